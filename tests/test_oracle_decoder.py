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
