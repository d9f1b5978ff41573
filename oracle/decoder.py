"""The rollback decoder D and its decision margin (oracle; test infrastructure only).

Algorithm 1 leaves token acceptance, replacement, re-masking and termination
to the decoder D (Sec. 4.2).  The paper's own decoder (Saber) is not defined
in the paper, so the decoder here is the workload's: unmask k tokens per step
by maximum softmax confidence, and remask the lowest-confidence decided token
when its confidence drops below tau.

Reading of that rule, for response row i with logits z_i (MASK column
excluded from the softmax and from the argmax):

* m_i = max_v z_iv, xhat_i = the smallest v attaining it,
  lse_i = log sum_v exp(z_iv);
* confidence of a masked row: ell_i = m_i - lse_i (log of its top
  probability);  confidence of a decided row: q_i = z_{i,g_i} - lse_i (log of
  the probability of its current token, re-evaluated at every step);
* unmask U: the min(k, #masked) masked rows with the largest ell, ties to the
  smaller position; each gets g_i <- xhat_i;
* remask: among rows decided in g_t take the one with the smallest q (ties to
  the smaller position); if q < log(tau) set it to MASK (at most one per step);
* both use the same z_t and apply together; U and the remasked row are
  disjoint (one is masked in g_t, the other decided);
* on the final step every masked row is unmasked and nothing is remasked, so
  the output holds no MASK.

Comparisons are exact ``<`` in log space.
"""

from __future__ import annotations

import math

import numpy as np


def row_stats(z: np.ndarray, g: np.ndarray, mask_id: int) -> dict:
    """Per-row statistics of the logits, in float64.

    Returns ``m``, ``xhat``, ``lse``, ``ell`` (= m - lse) and ``q``
    (= z[g_i] - lse; NaN where g_i is MASK), plus ``top2`` (second-largest
    non-MASK logit, used by the margin).
    """
    z = np.array(z, dtype=np.float64, copy=True)
    z[:, mask_id] = -np.inf
    m = np.max(z, axis=1)
    xhat = np.argmax(z, axis=1)                 # first occurrence = smallest id
    s = np.sum(np.exp(z - m[:, None]), axis=1)
    lse = m + np.log(s)
    ell = -np.log(s)
    g = np.asarray(g)
    decided = g != mask_id
    q = np.full(z.shape[0], np.nan)
    idx = np.nonzero(decided)[0]
    q[idx] = z[idx, g[idx]] - lse[idx]
    zt = z.copy()
    zt[np.arange(z.shape[0]), xhat] = -np.inf
    top2 = np.max(zt, axis=1)
    return {"m": m, "xhat": xhat, "lse": lse, "ell": ell, "q": q, "top2": top2}


def select_unmask(ell: np.ndarray, masked: np.ndarray, k: int) -> list[int]:
    """The min(k, #masked) masked positions with the largest ell (ties: smaller position)."""
    cand = [i for i in range(len(ell)) if masked[i]]
    cand.sort(key=lambda i: (-ell[i], i))
    return sorted(cand[: min(k, len(cand))])


def select_remask(q: np.ndarray, decided: np.ndarray, tau: float) -> list[int]:
    """The decided position with the smallest q, if that q < log(tau) (ties: smaller position)."""
    cand = [i for i in range(len(q)) if decided[i]]
    if not cand:
        return []
    j = min(cand, key=lambda i: (q[i], i))
    return [j] if q[j] < math.log(tau) else []


def decide(z: np.ndarray, g: np.ndarray, mask_id: int, k: int, tau: float,
           final: bool = False, remask: bool = True):
    """One decoder step g_{t+1} = D(g_t, z_t).

    Returns ``(g_next, U, Rm, stats)`` with U the unmasked positions and Rm the
    remasked positions (both sorted).
    """
    g = np.asarray(g)
    st = row_stats(z, g, mask_id)
    masked = g == mask_id
    decided = ~masked
    if final:
        U = [int(i) for i in np.nonzero(masked)[0]]
        Rm = []
    else:
        U = select_unmask(st["ell"], masked, k)
        Rm = select_remask(st["q"], decided, tau) if remask else []
    g_next = g.copy()
    for i in U:
        g_next[i] = st["xhat"][i]
    for i in Rm:
        g_next[i] = mask_id
    return g_next, U, Rm, st


def decision_margin(z: np.ndarray, g: np.ndarray, mask_id: int, k: int, tau: float,
                    final: bool = False, remask: bool = True) -> float:
    """A lower bound on the decision margin m_D(g, z) of Eq. theory-margin.

    Under a perturbation with ||delta||_inf <= eps every non-MASK logit moves
    by at most eps, so m_i and lse_i move by at most eps and ell_i, q_i by at
    most 2 eps.  The decision D(g, z + delta) equals D(g, z) whenever eps is
    below each of:

    * half the top-1 / top-2 logit gap of every unmasked row (its token);
    * a quarter of the gap between the k-th and (k+1)-th largest ell among
      masked rows (the unmask set);
    * half the distance of the smallest q to log(tau) (remask or not), and,
      when a remask happens, a quarter of the gap between the smallest and
      second-smallest q among decided rows (which row).

    The minimum of these is returned (``inf`` if nothing can change).
    """
    g = np.asarray(g)
    st = row_stats(z, g, mask_id)
    masked = g == mask_id
    decided = ~masked
    _, U, Rm, _ = decide(z, g, mask_id, k, tau, final, remask)
    bounds = [math.inf]
    for i in U:
        bounds.append(0.5 * (st["m"][i] - st["top2"][i]))
    if not final:
        ells = np.sort(st["ell"][masked])[::-1]
        kt = min(k, len(ells))
        if 0 < kt < len(ells):
            bounds.append(0.25 * (ells[kt - 1] - ells[kt]))
        if remask and np.any(decided):
            qs = np.sort(st["q"][decided])
            bounds.append(0.5 * abs(qs[0] - math.log(tau)))
            if Rm and len(qs) > 1:
                bounds.append(0.25 * (qs[1] - qs[0]))
    return float(min(bounds))
