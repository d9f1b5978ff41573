"""Archer decoding of one sequence (oracle; test infrastructure only).

What feeds the decoder at step t is the controller's choice of logits,
Eq. archer-controller (Sec. 4.2; Algorithm 1 states the same procedure):

    z~_t = Phi(g_t; C_p(g_t))   if the refresh predicate holds at t  (and then g_r := g_t, r := t)
    z~_t = Phi(g_t; C_p(g_r))   otherwise
    g_{t+1} = D(g_t, z~_t)

with D_t = d_H(g_t, g_r) and A_t = t - r the signals of the predicate
(:mod:`oracle.controller`).  Step 0 always takes the full forward: it
creates the first anchor, g_r = g_0.

Termination belongs to the decoder and the paper does not define it.
Reading: a fixed budget of T decisions t = 0..T-1, each preceded by its
forward (so exactly T forwards), the last decision unmasking every remaining
masked row.  The number R of full forwards among the T gives the refresh
fraction q_K = R / T of Eq. theory-speedup.

Batches are decoded sequence by sequence: each sequence has its own anchor
g_r, anchor step r and distance D_t.

``force`` overrides the predicate at chosen forwards ({t: True} refreshes,
{t: False} reuses the anchored cache): the two branches of the matched-state
feedback intervention (the paper's mechanism appendix) continue one decoder
state with an immediate refresh and with the old cache.
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
    age: list = field(default_factory=list)         # A_t = t - r before forward t (0 at t = 0)
    unmask: list = field(default_factory=list)      # U of decision t
    remask: list = field(default_factory=list)      # Rm of decision t
    states: list = field(default_factory=list)      # g_t entering forward t
    logits: list = field(default_factory=list)      # z~_t (kept only on request)


def decode(W: dict, m, prompt: np.ndarray, g0: np.ndarray, *, steps: int, k: int,
           tau: float, policy: str, K: float, remask: bool = True,
           keep_logits: bool = False, force: dict | None = None):
    """Decode one sequence for ``steps`` decisions.  Returns ``(g_final, Trace)``."""
    prompt = np.asarray(prompt).copy()
    P = len(prompt)
    g = np.asarray(g0).copy()
    tr = Trace()
    g_r, r, cache = None, 0, None
    for t in range(steps):
        # the controller's signals before forward t, and its choice of logits
        if t == 0:
            D, A, refresh = 0, 0, True
        else:
            D, A = controller.hamming(g, g_r), t - r
            refresh = controller.should_refresh(policy, K, D, A)
            if force is not None and t in force:
                refresh = bool(force[t])
        if refresh:
            z, cache, _ = full_forward(W, m, prompt, g)
            g_r, r = g.copy(), t
        else:
            z, _ = cached_forward(W, m, g, cache, P)
        tr.refreshed.append(refresh)
        tr.dist.append(D)
        tr.age.append(A)
        tr.states.append(g.copy())
        if keep_logits:
            tr.logits.append(z)
        # the decoder's step on those logits
        g, U, Rm, _ = decide(z, g, m.mask_id, k, tau, final=t == steps - 1, remask=remask)
        tr.unmask.append(U)
        tr.remask.append(Rm)
    return g, tr


def decode_batch(W: dict, m, prompts: list, g0: list, **kw):
    """Decode each sequence independently (per-sequence anchors and refreshes)."""
    outs = [decode(W, m, p, g, **kw) for p, g in zip(prompts, g0)]
    return [o[0] for o in outs], [o[1] for o in outs]
