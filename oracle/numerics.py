"""Elementary operations of the oracle (float64).

The paper treats the backbone Phi_theta abstractly (Sec. 4.1); the operations
below are those of the named backbones' architecture family (pre-norm
bidirectional transformer with RMSNorm, rotate-half RoPE, SwiGLU MLP).  The
paper fixes no precision, so the oracle computes in float64 and emulates the
storage points of the bf16 path with :func:`round_bf16` and
:func:`round_fp16`.
"""

from __future__ import annotations

import numpy as np


def weights_f64(w: np.ndarray) -> np.ndarray:
    """Weight array -> float64.  uint16 arrays hold bf16 bit patterns."""
    if w.dtype == np.uint16:
        return (w.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return np.asarray(w, dtype=np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even).

    bf16 keeps 8 significant bits (1 implicit + 7 stored) and float32's
    exponent range.  For normal numbers this rounds the 53-bit float64
    significand to 8 bits directly on the bit pattern.  Magnitudes below
    2^-126 (bf16 subnormals; they do not occur in the workloads) are rounded
    via float32.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    tiny = np.abs(x) < 2.0 ** -126
    u = x.view(np.uint64)
    # 52 - 7 = 45 low significand bits are dropped.
    lsb = (u >> np.uint64(45)) & np.uint64(1)
    r = (u + np.uint64((1 << 44) - 1) + lsb) & ~np.uint64((1 << 45) - 1)
    out[...] = r.view(np.float64)
    if np.any(tiny):
        f = x[tiny].astype(np.float32).view(np.uint32)
        f = (f + np.uint32(0x7FFF) + ((f >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
        out[tiny] = f.view(np.float32).astype(np.float64)
    return out


def round_fp16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest IEEE half-precision value (ties to
    even; 11 significant bits, subnormals below 2^-14, overflow to inf), by
    NumPy's float64 -> float16 conversion, which rounds once."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * gain."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, dtype=np.float64)


def rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary position embedding.

    ``x`` is ``[n][heads][hd]``; dimension pair (j, j + hd/2) of the row at
    absolute position ``pos`` is rotated by the angle ``pos * theta^(-2j/hd)``.
    """
    n, h, hd = x.shape
    half = hd // 2
    j = np.arange(half, dtype=np.float64)
    inv_freq = theta ** (-2.0 * j / hd)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def linear(a: np.ndarray, w: np.ndarray) -> np.ndarray:
    """A projection of the transformer: a W^T with W stored row-major [out][in]."""
    return np.asarray(a, dtype=np.float64) @ weights_f64(w).T


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Non-causal scaled dot-product attention of one head.

    ``q`` is ``[nq][hd]``, ``k`` and ``v`` are ``[nk][hd]``; every query
    attends to every key (no mask): softmax(q k^T / sqrt(hd)) v.
    """
    hd = q.shape[-1]
    s = (q @ k.T) / np.sqrt(hd)
    s = s - np.max(s, axis=-1, keepdims=True)
    p = np.exp(s)
    p /= np.sum(p, axis=-1, keepdims=True)
    return p @ v
