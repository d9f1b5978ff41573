"""Algorithm 1: state-anchored rollback decoding (oracle; test infrastructure only).

Algorithm 1 of the paper: start from g <- g_0 and g_r <- g_0, run a full
forward; then repeatedly apply the decoder D and, unless decoding has
terminated, either refresh (full forward, replace the cache, g_r <- g) when
d_H(g, g_r) >= K or run the cached forward on the anchored cache.

Termination is not defined in the paper (it belongs to D).  Reading: a fixed
budget of T decisions -- decisions are numbered t = 0..T-1, the forward that
precedes decision t is forward t (forward 0 is the initial full forward) and
decoding ends after decision T-1, which unmasks every remaining masked row.
So every run has exactly T forwards; the number R of them that are full
refreshes gives the refresh fraction q_K = R / T of Eq. theory-speedup.

Batches are decoded sequence by sequence: each sequence has its own anchor
g_r, anchor step r and distance D_t.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import controller
from .decoder import decide
from .model import cached_forward, full_forward


@dataclass
class Trace:
    refreshed: list = field(default_factory=list)   # forward t was a full refresh
    dist: list = field(default_factory=list)        # D_t before forward t (0 at t = 0)
    age: list = field(default_factory=list)         # A_t = t - r before forward t
    unmask: list = field(default_factory=list)      # U of decision t
    remask: list = field(default_factory=list)      # Rm of decision t
    states: list = field(default_factory=list)      # g_t entering forward t
    logits: list = field(default_factory=list)      # z_t (kept only on request)


def decode(W: dict, m, prompt: np.ndarray, g0: np.ndarray, *, steps: int, k: int,
           tau: float, policy: str, K: float, remask: bool = True,
           keep_logits: bool = False):
    """Decode one sequence.  Returns ``(g_final, Trace)``."""
    prompt = np.asarray(prompt).copy()
    P = len(prompt)
    g = np.asarray(g0).copy()
    tr = Trace()
    z, cache, _ = full_forward(W, m, prompt, g)
    g_r, r = g.copy(), 0
    tr.refreshed.append(True)
    tr.dist.append(0)
    tr.age.append(0)
    tr.states.append(g.copy())
    if keep_logits:
        tr.logits.append(z)
    for t in range(steps):
        final = t == steps - 1
        g, U, Rm, _ = decide(z, g, m.mask_id, k, tau, final=final, remask=remask)
        tr.unmask.append(U)
        tr.remask.append(Rm)
        if final:
            break
        s = t + 1
        D = controller.hamming(g, g_r)
        A = s - r
        tr.dist.append(D)
        tr.age.append(A)
        tr.states.append(g.copy())
        if controller.should_refresh(policy, K, D, A):
            z, cache, _ = full_forward(W, m, prompt, g)
            g_r, r = g.copy(), s
            tr.refreshed.append(True)
        else:
            z, _ = cached_forward(W, m, g, cache, P)
            tr.refreshed.append(False)
        if keep_logits:
            tr.logits.append(z)
    return g, tr


def decode_batch(W: dict, m, prompts: list, g0: list, **kw):
    """Decode each sequence independently (per-sequence anchors and refreshes)."""
    outs = [decode(W, m, p, g, **kw) for p, g in zip(prompts, g0)]
    return [o[0] for o in outs], [o[1] for o in outs]
