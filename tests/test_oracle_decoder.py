"""Pins of the oracle decoder D and its margin bound (no GPU).

* hand-derived planted cases (tests/golden/decoder_planted.json);
* brute force over every candidate unmask set / remask row for tiny G, with
  the selection characterised differently from the oracle (every chosen row
  beats every unchosen one);
* the margin bound of Eq. theory-margin: random perturbations strictly inside
  it never change the decision, and a perturbation just beyond a tight planted
  margin does.
"""

import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import decoder as od

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "decoder_planted.json")


def _cases():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_planted_cases(case):
    z = np.array(case["z"], dtype=np.float64)
    g = np.array(case["g"])
    g_next, U, Rm, _ = od.decide(z, g, case["mask_id"], case["k"], case["tau"], final=case["final"])
    assert g_next.tolist() == case["expected_g_next"]
    assert U == case["expected_U"]
    assert Rm == case["expected_Rm"]


def _brute_force(z, g, mask_id, k, tau):
    V = z.shape[1]
    G = len(g)
    ids = [v for v in range(V) if v != mask_id]
    lse = [math.log(sum(math.exp(z[i, v]) for v in ids)) for i in range(G)]
    conf = [max(z[i, v] for v in ids) - lse[i] for i in range(G)]
    tok = [min(v for v in ids if z[i, v] == max(z[i, u] for u in ids)) for i in range(G)]
    masked = [i for i in range(G) if g[i] == mask_id]
    kt = min(k, len(masked))
    chosen = []
    for S in itertools.combinations(masked, kt):
        rest = [j for j in masked if j not in S]
        if all((conf[i] > conf[j]) or (conf[i] == conf[j] and i < j) for i in S for j in rest):
            chosen.append(list(S))
    assert len(chosen) == 1
    U = chosen[0]
    decided = [i for i in range(G) if g[i] != mask_id]
    qv = {i: z[i, g[i]] - lse[i] for i in decided}
    Rm = []
    for j in decided:
        if all((qv[j] < qv[i]) or (qv[j] == qv[i] and j < i) for i in decided if i != j):
            if qv[j] < math.log(tau):
                Rm = [j]
    out = g.copy()
    for i in U:
        out[i] = tok[i]
    for i in Rm:
        out[i] = mask_id
    return out, U, Rm


def test_brute_force_enumeration_small_G():
    rng = np.random.default_rng(11)
    V, mask_id = 6, 5
    for trial in range(400):
        G = int(rng.integers(1, 7))
        z = np.round(rng.standard_normal((G, V)) * 2, 1)   # coarse values -> frequent ties
        g = rng.integers(0, V, G)
        k = int(rng.integers(1, 4))
        tau = float(rng.choice([0.1, 0.3, 0.6]))
        got = od.decide(z, g, mask_id, k, tau)
        want = _brute_force(z, g, mask_id, k, tau)
        assert got[0].tolist() == want[0].tolist()
        assert got[1] == want[1] and got[2] == want[2]


def test_mask_column_never_predicted():
    z = np.zeros((4, 5))
    z[:, 4] = 100.0
    g = np.full(4, 4)
    g_next, U, _, _ = od.decide(z, g, 4, 4, 0.1)
    assert 4 not in g_next[U].tolist()


def test_margin_lower_bound_holds_under_random_perturbations():
    rng = np.random.default_rng(12)
    V, mask_id = 8, 7
    checked = 0
    for trial in range(300):
        G = int(rng.integers(2, 7))
        z = rng.standard_normal((G, V)) * 1.5
        g = rng.integers(0, V, G)
        k = int(rng.integers(1, 3))
        tau = 0.2
        final = bool(rng.random() < 0.2)
        mD = od.decision_margin(z, g, mask_id, k, tau, final)
        base = od.decide(z, g, mask_id, k, tau, final)[0]
        if not math.isfinite(mD) or mD <= 0:
            continue
        for _ in range(20):
            delta = rng.uniform(-1, 1, z.shape)
            delta *= 0.999 * mD / np.max(np.abs(delta))
            assert od.decide(z + delta, g, mask_id, k, tau, final)[0].tolist() == base.tolist()
            checked += 1
    assert checked > 3000


def test_margin_is_tight_for_a_planted_argmax_gap():
    """Single masked row, top-2 gap 0.2: the bound is 0.1 and a 0.1001 shift flips the token."""
    z = np.array([[1.0, 0.8, -5.0, 9.0]])
    g = np.array([3])
    assert abs(od.decision_margin(z, g, 3, 1, 0.1) - 0.1) < 1e-15
    delta = np.array([[-0.1001, 0.1001, 0.0, 0.0]])
    assert od.decide(z + delta, g, 3, 1, 0.1)[0].tolist() == [1]
    assert od.decide(z, g, 3, 1, 0.1)[0].tolist() == [0]


def test_margin_zero_on_exact_tie():
    z = np.array([[1.0, 1.0, 0.0]])
    assert od.decision_margin(z, np.array([2]), 2, 1, 0.1) == 0.0


# --- tightness of the top-k and remask terms of the margin ---------------------
# Each case makes one term of the bound the binding one and applies the
# perturbation that moves the two compared log-confidences towards each other
# as fast as a sup-norm budget allows: on a flat row of V logits, lowering one
# logit by eps and raising the others by eps moves its log-probability by
# 2 eps (1 - p), p its probability.  The decision must hold just inside the
# bound and flip just beyond it, so the term's constant is pinned from both
# sides (a constant half as large would leave the flip unreached).

V_FLAT = 1000


def _peak_for_logprob(logp, V=V_FLAT):
    """Peak height c over V - 2 zero logits (MASK excluded) giving log-probability logp."""
    p = math.exp(logp)
    return math.log(p * (V - 2) / (1.0 - p))


def _flat_row(peak_id, c, V=V_FLAT):
    z = np.zeros(V)
    z[peak_id] = c
    return z


def _push(z, row, tok, eps, mask_id, down):
    """Move row's log-probability of tok by about -2 eps (down) or +2 eps (up)."""
    d = np.full(z.shape[1], eps if down else -eps)
    d[tok] = -eps if down else eps
    d[mask_id] = 0.0
    z[row] += d


def _check_tight(z, g, mask_id, k, tau, want_term, push, slack):
    mD = od.decision_margin(z, g, mask_id, k, tau)
    assert abs(mD - want_term) < 1e-12, (mD, want_term)
    base = od.decide(z, g, mask_id, k, tau)[0].tolist()
    inside, beyond = z.copy(), z.copy()
    push(inside, 0.99 * mD)
    push(beyond, slack * mD)
    assert od.decide(inside, g, mask_id, k, tau)[0].tolist() == base
    assert od.decide(beyond, g, mask_id, k, tau)[0].tolist() != base


def test_margin_is_tight_for_the_unmask_set():
    """k = 1, two masked rows whose log-confidences differ by 0.02: the bound is 0.005."""
    mask_id, k, tau = V_FLAT - 1, 1, 0.1
    l0 = -6.0
    gap = 0.02
    z = np.stack([_flat_row(3, _peak_for_logprob(l0)), _flat_row(5, _peak_for_logprob(l0 - gap))])
    g = np.array([mask_id, mask_id])

    def push(zz, eps):
        _push(zz, 0, 3, eps, mask_id, down=True)
        _push(zz, 1, 5, eps, mask_id, down=False)

    _check_tight(z, g, mask_id, k, tau, gap / 4, push, 1.01)


def test_margin_is_tight_for_the_remask_threshold():
    """A decided row whose log-probability sits 0.02 above log(tau): the bound is 0.01
    (tau small, so the row's probability is small and the push moves it by ~2 eps)."""
    mask_id, k, tau = V_FLAT - 1, 1, 1e-3
    q = math.log(tau) + 0.02
    z = np.stack([_flat_row(3, 8.0), _flat_row(5, _peak_for_logprob(q)), _flat_row(6, 9.0)])
    g = np.array([mask_id, 5, 6])

    def push(zz, eps):
        _push(zz, 1, 5, eps, mask_id, down=True)

    _check_tight(z, g, mask_id, k, tau, 0.01, push, 1.01)
    # and from below: the remask fires and a push up by just over the bound stops it
    q2 = math.log(tau) - 0.02
    z2 = z.copy()
    z2[1] = _flat_row(5, _peak_for_logprob(q2))
    assert od.decide(z2, g, mask_id, k, tau)[2] == [1]

    def push_up(zz, eps):
        _push(zz, 1, 5, eps, mask_id, down=False)

    _check_tight(z2, g, mask_id, k, tau, 0.01, push_up, 1.01)


def test_margin_is_tight_for_the_remasked_row():
    """Two decided rows below log(tau) whose log-probabilities differ by 0.02: which one is
    remasked has the bound 0.005."""
    mask_id, k, tau = V_FLAT - 1, 1, 0.1
    q1 = -7.0
    gap = 0.02
    z = np.stack([_flat_row(3, 8.0), _flat_row(5, _peak_for_logprob(q1)), _flat_row(6, _peak_for_logprob(q1 + gap))])
    g = np.array([mask_id, 5, 6])
    assert od.decide(z, g, mask_id, k, tau)[2] == [1]

    def push(zz, eps):
        _push(zz, 1, 5, eps, mask_id, down=False)
        _push(zz, 2, 6, eps, mask_id, down=True)

    _check_tight(z, g, mask_id, k, tau, gap / 4, push, 1.01)
