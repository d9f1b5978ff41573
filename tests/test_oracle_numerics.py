"""Pins of the oracle's elementary operations against library routines,
closed forms and brute force (no GPU)."""

import math
from itertools import product

import numpy as np
import pytest
import torch

from oracle import numerics as on


# --- bf16 rounding -----------------------------------------------------------

def test_round_bf16_matches_torch_on_float32_inputs(rng):
    x = (rng.standard_normal(200000) * np.exp(rng.uniform(-20, 20, 200000))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(on.round_bf16(x.astype(np.float64)), ref)


def test_round_bf16_ties_and_direct_rounding():
    u = 2.0 ** -7                         # bf16 spacing in [1, 2)
    cases = {
        1.0 + u / 2: 1.0,                 # tie -> even (1.0)
        1.0 + 3 * u / 2: 1.0 + 2 * u,     # tie -> even (1 + 2u)
        -(1.0 + u / 2): -1.0,
        1.0 + u / 2 + 2.0 ** -40: 1.0 + u,  # above the tie: a float32 detour would give 1.0
        3.0: 3.0,
        0.0: 0.0,
    }
    for x, want in cases.items():
        assert on.round_bf16(np.array([x]))[0] == want, x


# --- fp16 rounding (queries, keys and values of bf16 models) ------------------

def _fp16_values():
    """Every finite non-negative fp16 value, ascending, built from its bit fields."""
    sub = np.arange(1024) * 2.0 ** -24                                   # exponent field 0
    norm = [(1 + np.arange(1024) / 1024) * 2.0 ** (e - 15) for e in range(1, 31)]
    return np.concatenate([sub] + norm)


def test_round_fp16_exact_values_midpoints_and_overflow():
    h = _fp16_values()
    assert len(h) == 31744 and h[-1] == 65504.0
    np.testing.assert_array_equal(on.round_fp16(h), h)
    np.testing.assert_array_equal(on.round_fp16(-h), -h)
    mid = (h[:-1] + h[1:]) / 2                          # exact in float64
    even = np.where(np.arange(len(h) - 1) % 2 == 0, h[:-1], h[1:])   # the neighbour with an even significand
    np.testing.assert_array_equal(on.round_fp16(mid), even)
    up = np.nextafter(mid, np.inf)
    down = np.nextafter(mid, -np.inf)
    np.testing.assert_array_equal(on.round_fp16(up), h[1:])
    np.testing.assert_array_equal(on.round_fp16(down), h[:-1])
    # beyond the largest finite value: ties to even at 65520 (the next, unrepresentable, step) go to inf
    assert on.round_fp16(np.array([65519.99]))[0] == 65504.0
    assert on.round_fp16(np.array([65520.0]))[0] == np.inf


# --- bf16 bit patterns -> float64 (every bf16 weight the oracle reads) -------

def test_weights_f64_matches_torch_bf16_view_on_every_bit_pattern():
    """All 65536 bf16 bit patterns: the oracle's decoding equals torch's bf16 -> float64 cast
    (a library routine that shares no code with it), NaNs in the same places."""
    u = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = on.weights_f64(u)
    ref = torch.from_numpy(u.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    np.testing.assert_array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def test_weights_f64_closed_forms():
    pats = np.array([0x3F80, 0xC000, 0x3F81, 0x4049, 0x8000, 0x0001, 0x7F7F, 0x7F80], dtype=np.uint16)
    want = [1.0, -2.0, 1.0 + 2.0 ** -7, 3.140625, -0.0, 2.0 ** -133, (2 - 2.0 ** -7) * 2.0 ** 127, math.inf]
    got = on.weights_f64(pats)
    assert got.tolist() == want
    assert math.copysign(1.0, got[4]) == -1.0
    # float32 weights pass through unchanged
    x = np.array([0.1, -3.5e-7, 1e30], dtype=np.float32)
    np.testing.assert_array_equal(on.weights_f64(x), x.astype(np.float64))


# --- RMSNorm / SiLU against torch --------------------------------------------

def test_rms_norm_matches_torch(rng):
    x = rng.standard_normal((7, 33)) * 3
    g = rng.standard_normal(33)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), eps=1e-5)
    np.testing.assert_allclose(on.rms_norm(x, g, 1e-5), ref.numpy(), rtol=1e-13, atol=1e-13)


def test_silu_matches_torch(rng):
    x = rng.standard_normal(1000) * 6
    ref = torch.nn.functional.silu(torch.from_numpy(x)).numpy()
    np.testing.assert_allclose(on.silu(x), ref, rtol=1e-13, atol=1e-15)


# --- RoPE ---------------------------------------------------------------------

def test_rope_identity_at_position_zero(rng):
    x = rng.standard_normal((1, 3, 8))
    np.testing.assert_allclose(on.rope(x, np.array([0]), 10000.0), x, atol=0)


def test_rope_matches_complex_rotation(rng):
    """Rotate-half RoPE == multiplying (x_j + i x_{j+hd/2}) by exp(i pos theta^(-2j/hd))."""
    hd, theta = 16, 500.0
    x = rng.standard_normal((5, 2, hd))
    pos = np.array([0, 1, 7, 100, 4097])
    y = on.rope(x, pos, theta)
    for r, p in enumerate(pos):
        for h in range(2):
            for j in range(hd // 2):
                w = complex(x[r, h, j], x[r, h, j + hd // 2]) * complex(
                    math.cos(p * theta ** (-2 * j / hd)), math.sin(p * theta ** (-2 * j / hd)))
                assert abs(y[r, h, j] - w.real) < 1e-12
                assert abs(y[r, h, j + hd // 2] - w.imag) < 1e-12


def test_rope_scores_depend_on_relative_position_only(rng):
    q = rng.standard_normal((1, 1, 8))
    k = rng.standard_normal((1, 1, 8))
    def score(m, n):
        return float(np.sum(on.rope(q, np.array([m]), 10000.0) * on.rope(k, np.array([n]), 10000.0)))
    for m, n, c in [(3, 1, 10), (0, 5, 77), (100, 100, 3)]:
        assert abs(score(m, n) - score(m + c, n + c)) < 1e-12


def test_rope_fixed_value():
    # hd = 4: pairs (0, 2) rotate by pos * 1, pairs (1, 3) by pos * theta^-0.5
    x = np.array([[[1.0, 0.0, 0.0, 2.0]]])
    y = on.rope(x, np.array([2]), 100.0)[0, 0]
    a, b = 2.0, 2.0 * 100.0 ** -0.5
    want = [math.cos(a), -2.0 * math.sin(b), math.sin(a), 2.0 * math.cos(b)]
    np.testing.assert_allclose(y, want, atol=1e-15)


# --- attention ----------------------------------------------------------------

def _attention_loops(q, k, v):
    nq, hd = q.shape
    out = np.zeros((nq, v.shape[1]))
    for i in range(nq):
        s = [sum(q[i, c] * k[j, c] for c in range(hd)) / math.sqrt(hd) for j in range(k.shape[0])]
        mx = max(s)
        w = [math.exp(t - mx) for t in s]
        tot = sum(w)
        for j in range(k.shape[0]):
            for c in range(v.shape[1]):
                out[i, c] += w[j] / tot * v[j, c]
    return out


def test_attention_matches_triple_loop(rng):
    q, k, v = rng.standard_normal((5, 4)), rng.standard_normal((7, 4)), rng.standard_normal((7, 4))
    np.testing.assert_allclose(on.attention(q, k, v), _attention_loops(q, k, v), atol=1e-13)


def test_attention_matches_torch_sdpa_noncausal(rng):
    q, k, v = (rng.standard_normal((2, 3, n, 16)) * 2 for n in (9, 13, 13))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), is_causal=False).numpy()
    for b, h in product(range(2), range(3)):
        np.testing.assert_allclose(on.attention(q[b, h], k[b, h], v[b, h]), ref[b, h], atol=1e-12)


def test_attention_closed_forms(rng):
    q = rng.standard_normal((3, 8))
    v = rng.standard_normal((5, 8))
    same = np.tile(rng.standard_normal(8), (5, 1))    # identical keys -> uniform weights
    np.testing.assert_allclose(on.attention(q, same, v), np.tile(v.mean(0), (3, 1)), atol=1e-14)
    np.testing.assert_allclose(on.attention(q, same[:1], v[:1]), np.tile(v[0], (3, 1)), atol=0)
