"""Host statistics of the cache-validity probe (no GPU).

The probe's partial Spearman correlation is pinned to a different definition
of the same quantity -- the Pearson correlation of the residuals of the ranks
of x and y after regressing each on the ranks of z -- and its ranking to
scipy's average-rank routine; the calibration table to a hand-counted case.
"""

import numpy as np
import pytest
from scipy.stats import rankdata

from paper_2608_08086_amd import probe


def _partial_by_residuals(x, y, z):
    rx, ry, rz = rankdata(x), rankdata(y), rankdata(z)
    Z = np.stack([np.ones_like(rz), rz], axis=1)
    ex = rx - Z @ np.linalg.lstsq(Z, rx, rcond=None)[0]
    ey = ry - Z @ np.linalg.lstsq(Z, ry, rcond=None)[0]
    return float(np.corrcoef(ex, ey)[0, 1])


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_ranks_match_average_ranks(seed):
    x = np.random.default_rng(seed).integers(0, 6, 50)   # many ties
    np.testing.assert_array_equal(probe._ranks(x), rankdata(x))


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_partial_spearman_matches_residual_definition(seed):
    rng = np.random.default_rng(seed)
    z = rng.integers(0, 20, 300)
    x = z + rng.integers(0, 8, 300)                        # correlated with z, with ties
    y = (rng.random(300) < 0.2 + 0.03 * x).astype(int)     # a 0/1 outcome, like action disagreement
    got = probe.partial_spearman(x, y, z)
    assert abs(got - _partial_by_residuals(x, y, z)) < 1e-12


def test_partial_spearman_removes_a_shared_cause():
    # x and y both follow z and are otherwise independent: partial rho ~ 0, plain rho clearly > 0
    rng = np.random.default_rng(7)
    z = rng.normal(size=4000)
    x = z + 0.3 * rng.normal(size=4000)
    y = z + 0.3 * rng.normal(size=4000)
    assert np.corrcoef(rankdata(x), rankdata(y))[0, 1] > 0.8
    assert abs(probe.partial_spearman(x, y, z)) < 0.05


def test_summarize_bins_by_distance():
    recs = [dict(b=0, t=1, D=0, A=1, disagree=0, dH=0), dict(b=0, t=2, D=2, A=2, disagree=1, dH=2),
            dict(b=0, t=3, D=5, A=3, disagree=1, dH=1), dict(b=0, t=4, D=6, A=4, disagree=0, dH=0),
            dict(b=0, t=5, D=20, A=5, disagree=1, dH=3)]
    s = probe.summarize(recs)
    bins = {b["D"]: b for b in s["bins"]}
    assert s["probes"] == 5
    assert bins["0-3"]["probes"] == 2 and bins["0-3"]["action_disagreement_pct"] == 50.0
    assert bins["0-3"]["next_state_dH"] == 1.0
    assert bins["4-7"]["probes"] == 2 and bins["4-7"]["next_state_dH"] == 0.5
    assert bins["8-11"]["probes"] == 0 and bins["8-11"]["action_disagreement_pct"] is None
    assert bins[">=15"]["probes"] == 1 and bins[">=15"]["action_disagreement_pct"] == 100.0
    # a constant signal leaves the partial correlation undefined: reported as None
    flat = [dict(r, D=1) for r in recs]
    assert probe.summarize(flat)["partial_spearman"]["distance_vs_disagreement"] is None
