"""Pins of the controller and of Algorithm 1 in the oracle (no GPU).

* D_t on hand-built states; the refresh rules on hand-built trajectories;
* refresh every step (K = 0, or the "always" policy) is eager decoding;
* K = 1 reproduces the eager trajectory (D_t = 0 => exact logits);
* K = infinity never refreshes after the initial forward;
* the age rule gives R = ceil(T / K) refreshes;
* prompt tokens never change, exactly T forwards run, no MASK remains;
* decision fidelity (Prop. app-decision): at every cached step where
  ||z* - zhat||_inf is below the margin of the eager logits, the cached
  decision equals the eager one.
"""

import math

import numpy as np
import pytest

from conftest import random_weights, tiny_shape
from oracle import controller as oc
from oracle import decode as odec
from oracle import decoder as od
from oracle import model as om


def test_hamming_counts_mask_and_token_changes():
    M = 9
    g_r = np.array([M, M, 3, 4, M])
    g = np.array([1, M, 3, 5, M])     # MASK->1 and 4->5 differ
    assert oc.hamming(g, g_r) == 2
    assert oc.hamming(g_r, g_r) == 0


def test_refresh_rules_on_hand_built_trajectory():
    # (D, A) pairs seen before forwards 1..6 and the expected refresh decisions
    seq = [(1, 1), (2, 2), (3, 3), (0, 1), (5, 2), (1, 1)]
    assert [oc.should_refresh(oc.HAMMING, 3, D, A) for D, A in seq] == [False, False, True, False, True, False]
    assert [oc.should_refresh(oc.AGE, 2, D, A) for D, A in seq] == [False, True, True, False, True, False]
    assert all(oc.should_refresh(oc.HAMMING, 0, D, A) for D, A in seq)
    assert not any(oc.should_refresh(oc.HAMMING, math.inf, D, A) for D, A in seq)


def _setup(seed=21, std=0.5, coupling=1.0, **kw):
    m = tiny_shape("fp32", n_layers=2, d_model=16, n_heads=2, n_kv_heads=2, head_dim=8,
                   d_ff=24, vocab=13, init_std=std, **kw)
    W = random_weights(m, seed=seed)
    for L in W["layers"]:       # scale of cross-position mixing (attention output)
        L["w_o"] = (L["w_o"] * coupling).astype(np.float32)
    rng = np.random.default_rng(seed)
    p = rng.integers(0, m.vocab - 1, 6)
    g0 = np.full(8, m.mask_id)
    return m, W, p, g0


KW = dict(steps=8, k=1, tau=0.1)


def test_refresh_every_step_is_eager():
    m, W, p, g0 = _setup()
    g_a, tr_a = odec.decode(W, m, p, g0, policy=oc.ALWAYS, K=0, keep_logits=True, **KW)
    g_b, tr_b = odec.decode(W, m, p, g0, policy=oc.HAMMING, K=0, keep_logits=True, **KW)
    assert g_a.tolist() == g_b.tolist()
    assert all(tr_b.refreshed)
    for za, zb in zip(tr_a.logits, tr_b.logits):
        np.testing.assert_array_equal(za, zb)


@pytest.mark.parametrize("seed", [21, 22, 23])
def test_radius_one_reproduces_eager_trajectory(seed):
    m, W, p, g0 = _setup(seed)
    g_e, tr_e = odec.decode(W, m, p, g0, policy=oc.ALWAYS, K=0, **KW)
    g_1, tr_1 = odec.decode(W, m, p, g0, policy=oc.HAMMING, K=1, **KW)
    assert g_1.tolist() == g_e.tolist()
    assert [s.tolist() for s in tr_1.states] == [s.tolist() for s in tr_e.states]
    # cached forwards happen exactly when nothing changed since the anchor
    for ref, D in zip(tr_1.refreshed[1:], tr_1.dist[1:]):
        assert ref == (D >= 1)


def test_infinite_radius_never_refreshes_and_age_period():
    m, W, p, g0 = _setup()
    _, tr = odec.decode(W, m, p, g0, policy=oc.HAMMING, K=math.inf, **KW)
    assert tr.refreshed == [True] + [False] * (KW["steps"] - 1)
    for K in (1, 2, 3, 5, 8, 100):
        _, tr = odec.decode(W, m, p, g0, policy=oc.AGE, K=K, **KW)
        assert sum(tr.refreshed) == math.ceil(KW["steps"] / K)
        assert [t for t, r in enumerate(tr.refreshed) if r] == list(range(0, KW["steps"], K))


def test_prompt_fixed_T_forwards_no_mask_left():
    m, W, p, g0 = _setup()
    p0 = p.copy()
    g, tr = odec.decode(W, m, p, g0, policy=oc.HAMMING, K=2, **KW)
    assert p.tolist() == p0.tolist()
    assert len(tr.refreshed) == KW["steps"]
    assert len(tr.unmask) == KW["steps"]
    assert m.mask_id not in g.tolist()


def test_remask_branch_is_exercised_with_peaked_logits():
    """With a large init scale the logits are peaked, so both remask outcomes occur."""
    m, W, p, g0 = _setup(seed=31, std=1.5)
    _, tr = odec.decode(W, m, p, g0, policy=oc.HAMMING, K=3, steps=8, k=2, tau=0.3)
    n_remask = sum(len(r) for r in tr.remask[:-1])
    assert 0 < n_remask < len(tr.remask) - 1


@pytest.mark.parametrize("K", [2, 4, 100])
def test_decision_fidelity_under_margin_condition(K):
    """At each cached step, compare D on the cached logits with D on eager logits
    at the same state (a shadow full forward).  A weakly coupled model (small
    attention output projection) keeps ||z* - zhat|| small enough that the
    margin condition holds at many steps."""
    checked = 0
    for seed in range(44, 52):
        m, W, p, g0 = _setup(seed=seed, coupling=0.05)
        g = g0.copy()
        z, cache, _ = om.full_forward(W, m, p, g)
        g_r = g.copy()
        steps = 8
        for t in range(steps):
            final = t == steps - 1
            g, _, _, _ = od.decide(z, g, m.mask_id, 1, 0.1, final=final)
            if final:
                break
            if oc.hamming(g, g_r) >= K:
                z, cache, _ = om.full_forward(W, m, p, g)
                g_r = g.copy()
                continue
            z_hat, _ = om.cached_forward(W, m, g, cache, len(p))
            z_star, _, _ = om.full_forward(W, m, p, g)
            err = np.max(np.abs(z_star - z_hat))
            last = t + 1 == steps - 1
            if err < od.decision_margin(z_star, g, m.mask_id, 1, 0.1, final=last):
                a = od.decide(z_hat, g, m.mask_id, 1, 0.1, final=last)[0]
                b = od.decide(z_star, g, m.mask_id, 1, 0.1, final=last)[0]
                assert a.tolist() == b.tolist()
                checked += 1
            z = z_hat
    assert checked >= 5
