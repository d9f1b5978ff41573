"""Seeded generators for weights, prompts and ragged prompt lengths.

Every random tensor is drawn from NumPy's Philox-4x64 counter-based bit
generator keyed by ``(seed, stream id, chunk index)``, so each chunk of each
tensor can be produced independently (in parallel threads) and the result
does not depend on the thread count.  Weights are ``N(0, init_std^2)`` drawn in
float32; bf16 workloads store them as bf16 bit patterns (uint16) obtained by
round-to-nearest-even from the float32 draw.

Stream ids: token embedding 0, LM head 1, and for layer ``l`` the matrices
``16 + 8*l + j`` with ``j`` = 0 (W_qkv), 1 (W_o), 2 (W_gate), 3 (W_up),
4 (W_down).  RMSNorm gains are ones.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .workloads import ModelShape, Workload

_CHUNK = 1 << 22


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exactly equal float32 values."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _chunk_draw(seed: int, stream: int, chunk: int, n: int, scale: float) -> np.ndarray:
    key = np.array([seed & 0xFFFFFFFFFFFFFFFF, ((stream << 24) | chunk) & 0xFFFFFFFFFFFFFFFF],
                   dtype=np.uint64)
    g = np.random.Generator(np.random.Philox(key=key))
    v = g.standard_normal(n, dtype=np.float32)
    v *= np.float32(scale)
    return v


def normal_tensor(shape, seed: int, stream: int, scale: float, dtype: str = "bf16",
                  pool: ThreadPoolExecutor | None = None) -> np.ndarray:
    """N(0, scale^2) tensor; returns float32 (dtype="fp32") or uint16 bf16 bits."""
    numel = int(np.prod(shape))
    out = np.empty(numel, dtype=np.uint16 if dtype == "bf16" else np.float32)
    nchunks = (numel + _CHUNK - 1) // _CHUNK

    def work(c):
        lo = c * _CHUNK
        hi = min(numel, lo + _CHUNK)
        v = _chunk_draw(seed, stream, c, hi - lo, scale)
        out[lo:hi] = f32_to_bf16_bits(v) if dtype == "bf16" else v

    if nchunks == 1:
        work(0)
    elif pool is not None:
        list(pool.map(work, range(nchunks)))
    else:
        with ThreadPoolExecutor(_workers()) as ex:
            list(ex.map(work, range(nchunks)))
    return out.reshape(shape)


def model_weights(m: ModelShape, seed: int = 0, layers: int | None = None) -> dict:
    """Random-init weights in the row-major ``[out][in]`` layout.

    Returns ``{"tok_emb": [V][d], "lm_head": [V][d], "final_norm": [d],
    "layers": [{"attn_norm": [d], "w_qkv": [(Hq+2Hkv)hd][d], "w_o": [d][Hq hd],
    "mlp_norm": [d], "w_gate": [F][d], "w_up": [F][d], "w_down": [d][F]}]}``.
    Matrices are uint16 bf16 bits (bf16 models) or float32 (fp32 models); norm
    gains are float32 ones.  ``layers`` may cap the number of layers generated.
    """
    nl = m.n_layers if layers is None else layers
    d, hd = m.d_model, m.head_dim
    s, dt = m.init_std, m.dtype
    with ThreadPoolExecutor(_workers()) as pool:
        W = {
            "tok_emb": normal_tensor((m.vocab, d), seed, 0, s, dt, pool),
            "lm_head": normal_tensor((m.vocab, d), seed, 1, s, dt, pool),
            "final_norm": np.ones(d, np.float32),
            "layers": [],
        }
        for l in range(nl):
            b = 16 + 8 * l
            W["layers"].append({
                "attn_norm": np.ones(d, np.float32),
                "w_qkv": normal_tensor((m.qkv_dim, d), seed, b + 0, s, dt, pool),
                "w_o": normal_tensor((d, m.n_heads * hd), seed, b + 1, s, dt, pool),
                "mlp_norm": np.ones(d, np.float32),
                "w_gate": normal_tensor((m.d_ff, d), seed, b + 2, s, dt, pool),
                "w_up": normal_tensor((m.d_ff, d), seed, b + 3, s, dt, pool),
                "w_down": normal_tensor((d, m.d_ff), seed, b + 4, s, dt, pool),
            })
    return W


def prompt_lengths(w: Workload) -> list[int]:
    """Per-sequence prompt lengths: fixed, or uniform in the ragged range."""
    dec = w.decode
    if dec.ragged is None:
        return [dec.prompt_len] * dec.batch
    lo, hi = dec.ragged
    g = np.random.Generator(np.random.Philox(key=np.array([w.length_seed, 7], dtype=np.uint64)))
    return [int(v) for v in g.integers(lo, hi + 1, size=dec.batch)]


def prompts(w: Workload, lengths: list[int] | None = None) -> list[np.ndarray]:
    """Uniform-random prompt tokens over the non-MASK ids, one array per sequence."""
    lengths = prompt_lengths(w) if lengths is None else lengths
    out = []
    for b, n in enumerate(lengths):
        g = np.random.Generator(np.random.Philox(
            key=np.array([w.prompt_seed, (1 << 40) | b], dtype=np.uint64)))
        out.append(g.integers(0, w.model.vocab - 1, size=n, dtype=np.int64).astype(np.int32))
    return out
