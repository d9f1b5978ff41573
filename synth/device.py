"""Seeded random-init weights generated directly on the GPU (timing runs only).

Host generation of an 8B-parameter model takes minutes, so throughput runs
draw their N(0, init_std^2) weights with torch's seeded device generator
(one generator per tensor, keyed by the stream ids of :mod:`synth.gen`).  The
values differ from :func:`synth.gen.model_weights`; nothing is compared
against the oracle on them.  Parity tests use :mod:`synth.gen`.
"""

from __future__ import annotations

import torch

from .workloads import ModelShape


def _normal(shape, seed, stream, std, dtype):
    g = torch.Generator(device="cuda")
    g.manual_seed((seed << 32) + stream)
    out = torch.empty(shape, dtype=dtype, device="cuda")
    rows = shape[0]
    step = max(1, (1 << 27) // max(1, int(torch.tensor(shape[1:]).prod().item()) if len(shape) > 1 else 1))
    for r0 in range(0, rows, step):
        r1 = min(rows, r0 + step)
        t = torch.randn((r1 - r0,) + tuple(shape[1:]), generator=g, device="cuda", dtype=torch.float32)
        out[r0:r1] = (t * std).to(dtype)
    return out


def _gateup(m: ModelShape, w):
    """A bf16 gate or up matrix as the model stores it: fp16 under gateup_fp16."""
    return w.to(torch.float16) if m.dtype == "bf16" and m.gateup_fp16 else w


def model_weights_cuda(m: ModelShape, seed: int = 0) -> dict:
    dt = torch.bfloat16 if m.dtype == "bf16" else torch.float32
    d, hd, s = m.d_model, m.head_dim, m.init_std
    ones = lambda: torch.ones(d, dtype=torch.float32, device="cuda")  # noqa: E731
    W = {"tok_emb": _normal((m.vocab, d), seed, 0, s, dt), "lm_head": _normal((m.vocab, d), seed, 1, s, dt),
         "final_norm": ones(), "layers": []}
    for l in range(m.n_layers):
        b = 16 + 8 * l
        W["layers"].append({
            "attn_norm": ones(),
            "w_qkv": _normal((m.qkv_dim, d), seed, b + 0, s, dt),
            "w_o": _normal((d, m.n_heads * hd), seed, b + 1, s, dt),
            "mlp_norm": ones(),
            "w_gate": _gateup(m, _normal((m.d_ff, d), seed, b + 2, s, dt)),
            "w_up": _gateup(m, _normal((m.d_ff, d), seed, b + 3, s, dt)),
            "w_down": _normal((d, m.d_ff), seed, b + 4, s, dt),
        })
    return W
