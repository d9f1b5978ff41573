"""Helpers shared by the GPU parity tests (inputs from synth, results via the C ABI)."""

import sys

import numpy as np
import torch

from synth.gen import bf16_bits_to_f32, f32_to_bf16_bits, normal_tensor


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def archer():
    from paper_2608_08086_amd import archer as a
    return a


def dev_i32(x):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, dtype=np.int32))).cuda()


def dev_bits(u16):
    """uint16 bf16 bit patterns -> CUDA bf16 tensor."""
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).cuda()


def dev_f32(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def rand_bf16(shape, seed, stream, scale=1.0):
    """(device tensor, float64 values) of an N(0, scale^2) bf16 tensor."""
    bits = normal_tensor(shape, seed, stream, scale, "bf16")
    return dev_bits(bits), bf16_bits_to_f32(bits).astype(np.float64)


def rand_f16(shape, seed, stream, scale=1.0):
    """(device tensor, float64 values) of an N(0, scale^2) tensor rounded to fp16."""
    v = normal_tensor(shape, seed, stream, scale, "fp32").astype(np.float16)
    return torch.from_numpy(np.ascontiguousarray(v)).cuda(), v.astype(np.float64)


def rand_f32(shape, seed, stream, scale=1.0):
    v = normal_tensor(shape, seed, stream, scale, "fp32")
    return dev_f32(v), v.astype(np.float64)


def make_ctx(shape, W, max_batch, max_prompt_len, max_prompt_total, resp_len, layout=None):
    """Context over host weights W.  layout None: the k-block weight layout for bf16 models
    (the one the bench runs), row-major for fp32."""
    a = archer()
    Wd = a.upload_weights(W, shape.dtype, getattr(shape, "gateup_fp16", False))
    if layout is None:
        layout = a.LAYOUT_KBLOCK if shape.dtype == "bf16" else a.LAYOUT_ROWMAJOR
    if layout == a.LAYOUT_KBLOCK:
        Wd = a.pack_weights(Wd, drop_source=True)
    return a.Context(shape, Wd, max_batch, max_prompt_len, max_prompt_total, resp_len)


def with_gains(W, seed):
    """Non-unit RMSNorm gains so that a dropped gain shows up."""
    rng = np.random.default_rng(seed)
    d = W["final_norm"].shape[0]
    W["final_norm"] = (1.0 + 0.2 * rng.standard_normal(d)).astype(np.float32)
    for L in W["layers"]:
        L["attn_norm"] = (1.0 + 0.2 * rng.standard_normal(d)).astype(np.float32)
        L["mlp_norm"] = (1.0 + 0.2 * rng.standard_normal(d)).astype(np.float32)
    return W


def rel_err(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-30))
