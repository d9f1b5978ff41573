"""Pins of the oracle model Phi_theta (no GPU).

* a scalar-loop float64 transformer written independently here (pure Python,
  its own fp16 and bf16 rounding via frexp) must match
  ``oracle.model.transformer``, with and without single-term operands and
  with the fp16 gate/up operands (weights below fp16's normal range planted);
* permutation consistency of bidirectional attention, by brute force over all
  orders of tiny inputs;
* CachedForward(g; C_p(g)) equals FullForward(p, g) (D_t = 0 case of
  Eq. app-radius-bound), layer-1 prompt K/V do not depend on g, and the dense
  rollback closure of Prop. app-closure.
"""

import math
from itertools import permutations

import numpy as np
import pytest

from conftest import random_weights, tiny_shape
from oracle import model as om
from oracle import numerics as on


# --- independent scalar-loop reference ---------------------------------------

def _bf16(x):
    if x == 0.0 or not math.isfinite(x):
        return x
    mant, e = math.frexp(x)              # x = mant * 2^e, 0.5 <= |mant| < 1
    return round(mant * 256.0) / 256.0 * 2.0 ** e   # round() ties to even on floats


def _fp16(x):
    """IEEE half rounding written from its definition: 11 significant bits,
    spacing 2^-24 below 2^-14, ties to even (Python's round on floats)."""
    if x == 0.0 or not math.isfinite(x):
        return x
    if abs(x) < 2.0 ** -14:
        return round(x * 2.0 ** 24) / 2.0 ** 24
    mant, e = math.frexp(x)
    r = round(mant * 2048.0) / 2048.0 * 2.0 ** e
    return r if abs(r) <= 65504.0 else math.copysign(math.inf, x)


def _w(a):
    return on.weights_f64(a).tolist()


def _loop_model(W, m, tokens, positions, out_rows, round_gateup_w=True):
    ident = lambda t: t   # noqa: E731
    rnd = _fp16 if m.dtype == "bf16" else ident
    gu16 = m.dtype == "bf16" and m.gateup_fp16

    def op(name, row):
        """Activation operand of a projection: single bf16 where the model says so,
        single fp16 for gate/up under gateup_fp16."""
        if name == "gateup" and gu16:
            return [_fp16(t) for t in row]
        single = m.dtype == "bf16" and name in m.single_term
        return [_bf16(t) for t in row] if single else row
    d, hq, hkv, hd, F = m.d_model, m.n_heads, m.n_kv_heads, m.head_dim, m.d_ff
    n = len(tokens)
    emb = _w(W["tok_emb"])
    x = [list(emb[t]) for t in tokens]

    def norm(row, gain):
        ms = sum(v * v for v in row) / d
        r = 1.0 / math.sqrt(ms + m.rms_eps)
        return [row[c] * r * float(gain[c]) for c in range(d)]

    def matvec(Wm, a):
        return [sum(Wm[o][c] * a[c] for c in range(len(a))) for o in range(len(Wm))]

    def rot(vec, pos):
        half = hd // 2
        out = [0.0] * hd
        for j in range(half):
            ang = pos * m.rope_theta ** (-2.0 * j / hd)
            out[j] = vec[j] * math.cos(ang) - vec[j + half] * math.sin(ang)
            out[j + half] = vec[j + half] * math.cos(ang) + vec[j] * math.sin(ang)
        return out

    for L in W["layers"]:
        wqkv, wo, wg, wu, wd = (_w(L[k]) for k in ("w_qkv", "w_o", "w_gate", "w_up", "w_down"))
        if gu16 and round_gateup_w:
            wg = [[_fp16(t) for t in r] for r in wg]
            wu = [[_fp16(t) for t in r] for r in wu]
        Q, K, V = [], [], []
        for i in range(n):
            a = op("qkv", norm(x[i], L["attn_norm"]))
            y = matvec(wqkv, a)
            Q.append([[rnd(t) for t in rot(y[h * hd:(h + 1) * hd], positions[i])] for h in range(hq)])
            K.append([[rnd(t) for t in rot(y[(hq + h) * hd:(hq + h + 1) * hd], positions[i])] for h in range(hkv)])
            V.append([[rnd(t) for t in y[(hq + hkv + h) * hd:(hq + hkv + h + 1) * hd]] for h in range(hkv)])
        newx = []
        for i in range(n):
            o = []
            for h in range(hq):
                kh = h * hkv // hq
                s = [sum(Q[i][h][c] * K[j][kh][c] for c in range(hd)) / math.sqrt(hd) for j in range(n)]
                mx = max(s)
                p = [math.exp(t - mx) for t in s]
                tot = sum(p)
                o += [sum(p[j] / tot * V[j][kh][c] for j in range(n)) for c in range(hd)]
            proj = matvec(wo, op("o", o))
            xi = [x[i][c] + proj[c] for c in range(d)]
            b = op("gateup", norm(xi, L["mlp_norm"]))
            gate, up = matvec(wg, b), matvec(wu, b)
            hmid = [gate[f] / (1.0 + math.exp(-gate[f])) * up[f] for f in range(F)]
            down = matvec(wd, op("down", hmid))
            newx.append([xi[c] + down[c] for c in range(d)])
        x = newx
    head = _w(W["lm_head"])
    z = []
    for i in out_rows:
        c = op("head", norm(x[i], W["final_norm"]))
        z.append(matvec(head, c))
    return np.array(z)


@pytest.mark.parametrize("dtype,single,gu16", [("fp32", (), False), ("bf16", (), False),
                                               ("bf16", ("qkv", "o", "gateup", "down", "head"), False),
                                               ("bf16", ("o", "head"), False),
                                               ("bf16", (), True), ("bf16", ("o", "head"), True)])
def test_transformer_matches_scalar_loops(dtype, single, gu16):
    m = tiny_shape(dtype, single_term=single, gateup_fp16=gu16)
    W = random_weights(m, seed=3)
    tokens = np.array([1, 4, 9, 2, 9, 0])
    positions = np.arange(6)
    z, _, _ = om.transformer(W, m, tokens, positions)
    ref = _loop_model(W, m, tokens.tolist(), positions.tolist(), range(6))
    np.testing.assert_allclose(z, ref, rtol=0, atol=1e-11 if dtype == "fp32" else 1e-9)


def _bf16_bits(v):
    """float64 values -> uint16 bf16 bit patterns (round to nearest even via float32)."""
    f = np.asarray(v, dtype=np.float32).view(np.uint32)
    return ((f + np.uint32(0x7FFF) + ((f >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def test_gateup_fp16_rounds_weights_below_the_fp16_normal_range():
    """bf16 gate weights of magnitude 2^-21..2^-19 are not fp16 values (fp16 spaces
    them 2^-24 apart): the oracle must multiply their fp16 roundings.  The plant is
    large enough that leaving the weights unrounded misses the scalar loops by far
    more than the tolerance."""
    m = tiny_shape("bf16", gateup_fp16=True)
    W = random_weights(m, seed=5)
    rng = np.random.default_rng(17)
    for L in W["layers"]:
        v = rng.uniform(2.0 ** -21, 2.0 ** -19, size=(3, m.d_model)) * rng.choice([-1.0, 1.0], size=(3, m.d_model))
        L["w_gate"][:3] = _bf16_bits(v)
        L["w_up"][:3] = _bf16_bits(64.0 * rng.standard_normal((3, m.d_model)))
    tokens = np.array([3, 1, 4, 1, 5])
    positions = np.arange(5)
    z, _, _ = om.transformer(W, m, tokens, positions)
    ref = _loop_model(W, m, tokens.tolist(), positions.tolist(), range(5))
    np.testing.assert_allclose(z, ref, rtol=0, atol=1e-9)
    unrounded = _loop_model(W, m, tokens.tolist(), positions.tolist(), range(5), round_gateup_w=False)
    assert np.max(np.abs(unrounded - ref)) > 1e-7


# --- permutation consistency (brute force over all orders) -------------------

def test_attention_permutation_consistency_all_orders(rng):
    n = 5
    q, k, v = rng.standard_normal((3, 4)), rng.standard_normal((n, 4)), rng.standard_normal((n, 4))
    base = on.attention(q, k, v)
    for perm in permutations(range(n)):
        p = list(perm)
        np.testing.assert_allclose(on.attention(q, k[p], v[p]), base, atol=1e-13)
    qq = rng.standard_normal((4, 4))
    base_q = on.attention(qq, k, v)
    for perm in permutations(range(4)):
        p = list(perm)
        np.testing.assert_allclose(on.attention(qq[p], k, v), base_q[p], atol=1e-13)


def test_model_permutation_equivariance_with_positions():
    """Permuting tokens together with their position ids permutes every output row."""
    m = tiny_shape("fp32")
    W = random_weights(m, seed=5)
    tokens = np.array([3, 1, 4, 1, 5])
    pos = np.arange(5)
    z, kv, _ = om.transformer(W, m, tokens, pos)
    for perm in permutations(range(5)):
        p = np.array(perm)
        zp, kvp, _ = om.transformer(W, m, tokens[p], pos[p])
        np.testing.assert_allclose(zp, z[p], atol=1e-11)
        np.testing.assert_allclose(kvp[1][0], kv[1][0][:, p, :], atol=1e-11)


def test_no_causal_mask_later_token_changes_first_row():
    m = tiny_shape("fp32")
    W = random_weights(m, seed=6)
    t1 = np.array([1, 2, 3, 4, 5])
    t2 = t1.copy()
    t2[-1] = 8
    z1, _, _ = om.transformer(W, m, t1, np.arange(5))
    z2, _, _ = om.transformer(W, m, t2, np.arange(5))
    assert np.max(np.abs(z1[0] - z2[0])) > 1e-6


# --- cache invariants ---------------------------------------------------------

@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_cached_forward_on_own_cache_equals_full_forward(dtype):
    m = tiny_shape(dtype, n_layers=3)
    W = random_weights(m, seed=7)
    rng = np.random.default_rng(0)
    p = rng.integers(0, m.vocab - 1, 7)
    g = np.array([m.mask_id, 2, m.mask_id, 5, m.mask_id])
    z_full, cache, _ = om.full_forward(W, m, p, g)
    z_cached, _ = om.cached_forward(W, m, g, cache, len(p))
    np.testing.assert_allclose(z_cached, z_full, rtol=0, atol=1e-12)


def test_layer1_prompt_kv_independent_of_response_and_closure():
    """Layer-1 prompt K/V see only the prompt; a one-token response edit changes
    every position at layer 1 and the prompt K/V of later layers (Prop. app-closure)."""
    m = tiny_shape("fp32", n_layers=3)
    W = random_weights(m, seed=8)
    p = np.array([1, 2, 3, 4])
    g1 = np.array([m.mask_id, 6, m.mask_id])
    g2 = g1.copy()
    g2[1] = 7
    _, c1, h1 = om.full_forward(W, m, p, g1, keep_hidden=True)
    _, c2, h2 = om.full_forward(W, m, p, g2, keep_hidden=True)
    np.testing.assert_array_equal(c1[0][0], c2[0][0])
    np.testing.assert_array_equal(c1[0][1], c2[0][1])
    res1, res2 = h1[0], h2[0]
    # after layer 1 every one of the P+G positions differs
    assert np.all(np.max(np.abs(res1[1] - res2[1]), axis=1) > 1e-9)
    for l in (1, 2):
        assert np.max(np.abs(c1[l][0] - c2[l][0])) > 1e-9
        assert np.max(np.abs(c1[l][1] - c2[l][1])) > 1e-9


def test_stale_cache_differs_and_distance_zero_is_exact():
    m = tiny_shape("fp32", n_layers=3)
    W = random_weights(m, seed=9)
    p = np.array([0, 5, 2, 8, 1])
    g_r = np.array([m.mask_id] * 4)
    g = g_r.copy()
    g[2] = 3
    _, c_r, _ = om.full_forward(W, m, p, g_r)
    z_star, _, _ = om.full_forward(W, m, p, g)
    z_hat, _ = om.cached_forward(W, m, g, c_r, len(p))
    assert np.max(np.abs(z_star - z_hat)) > 1e-9      # anchored cache is an approximation
    z_same, _ = om.cached_forward(W, m, g_r, c_r, len(p))
    z_ref, _, _ = om.full_forward(W, m, p, g_r)
    np.testing.assert_allclose(z_same, z_ref, atol=1e-12)
