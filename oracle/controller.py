"""Anchor distance and refresh rules (oracle; test infrastructure only).

* D_t = d_H(g_t, g_r) = sum_i 1[g_{t,i} != g_{r,i}] over V u {MASK}
  (Sec. 4.2 Eq. archer-distance): a MASK <-> token change and a
  token <-> other-token change both count.
* Archer refreshes when D_t >= K and reuses the cache while D_t < K
  (Eq. archer-controller; Algorithm 1; the integer bound of App. A.4
  Eq. app-k-bound relies on reuse only for D_t <= K - 1).
* The cache-age signal A_t = t - r (Sec. 6.4) gives the fixed-period rule
  "refresh every K steps": refresh when A_t >= K.
* "always" refreshes at every step (eager decoding, Eq. archer-fresh).
"""

from __future__ import annotations

import numpy as np

HAMMING = "hamming"
AGE = "age"
ALWAYS = "always"


def hamming(g: np.ndarray, g_r: np.ndarray) -> int:
    """d_H(g, g_r)."""
    return int(np.sum(np.asarray(g) != np.asarray(g_r)))


def should_refresh(policy: str, K: float, D: int, A: int) -> bool:
    if policy == HAMMING:
        return D >= K
    if policy == AGE:
        return A >= K
    if policy == ALWAYS:
        return True
    raise ValueError(policy)
