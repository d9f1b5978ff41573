"""Decision-level cache-validity probe: non-intervening shadow forwards.

Sec. "Why Refresh by State Distance?" and App. "Decision-Level Cache
Validity" of the paper: at sampled cached steps of an Archer decode, a full
forward is run from the identical response state on a scratch cache; the
decoder is applied to the cached logits (the main trajectory's action) and
to the fresh logits, and the two actions and next states are compared.
Disagreement is then binned by the anchor distance D_t and related to D_t
and the cache age A_t by partial Spearman correlations.

The main trajectory is archer_decode's own: the probe runs it as a decode
session (archer_session_begin / archer_session_advance, one decision at a
time), so the refresh decisions come from the library's controller.  Before
each decision that follows a cached forward, it reads that forward's logits
and the current state, runs a FullForward of the same state on a second
context over the same weights (whose prompt cache is the scratch cache) and
applies the decoder to both sets of logits there; nothing on the main
context changes.  All model and decoder arithmetic runs in the library's
kernels; this module only orders the calls and computes the statistics of
the recorded integers.
"""

from __future__ import annotations

import numpy as np

# D_t bins of the paper's calibration table, plus everything above
D_BINS = ((0, 3), (4, 7), (8, 11), (12, 14), (15, None))


def shadow_probe(ctx, shadow, prompt, prompt_len, g0, *, policy, K, steps, k=1, tau=0.1, max_remask=1,
                 every=1):
    """Decode with Algorithm 1 on ``ctx`` and probe every ``every``-th cached forward.

    ctx, shadow: two ``archer.Context`` over the same weights and limits.
    prompt: device int32, the prompts of all sequences concatenated; prompt_len: host list.
    g0: device int32 [B][G], the initial response.  policy: archer.HAMMING / AGE / ALWAYS.
    Returns (g_final, trace, probes): g_final device int32 [B][G]; trace a dict of host arrays
    ``refreshed``, ``dist``, ``age`` [T][B] as archer_decode records them; probes a list of
    dicts (b, t, D, A, disagree, dH) -- t the forward index, D and A the controller's
    signals before forward t, disagree 1 if the cached and fresh decisions differ in any
    position, dH the Hamming distance between the two next states.
    """
    B, G = g0.shape
    T = int(steps)
    tr = ctx.session_begin(prompt, prompt_len, g0, policy=policy, K=K, steps=T, k=k, tau=tau,
                           max_remask=max_remask, trace=True, keep_logits=True)
    probes = []
    n_cached = 0
    for t in range(T):
        # forward t has run; decision t (on its logits z_t and the state g_t) comes next
        if t > 0:
            cached = np.nonzero(tr["refreshed"][t].cpu().numpy() == 0)[0]
            if len(cached):
                if n_cached % every == 0:
                    g_t = ctx.session_response()
                    z_c = ctx.read_logits(B)
                    z_f = shadow.refresh_prompt(prompt, prompt_len, g_t)
                    final = t == T - 1
                    a_c = shadow.decide(z_c, g_t, k=k, tau=tau, max_remask=max_remask, final=final)[0]
                    a_f = shadow.decide(z_f, g_t, k=k, tau=tau, max_remask=max_remask, final=final)[0]
                    a_c, a_f = a_c.cpu().numpy(), a_f.cpu().numpy()
                    D = tr["dist"][t].cpu().numpy()
                    A = tr["age"][t].cpu().numpy()
                    for b in cached:
                        diff = int(np.sum(a_c[b] != a_f[b]))
                        probes.append(dict(b=int(b), t=int(t), D=int(D[b]), A=int(A[b]), disagree=int(diff > 0),
                                           dH=diff))
                n_cached += 1
        ctx.session_advance(1)
    g = ctx.session_response()
    trace = {name: tr[name].cpu().numpy() for name in ("refreshed", "dist", "age")}
    return g, trace, probes


def _ranks(x):
    """Ranks 1..n with ties given their average rank."""
    x = np.asarray(x, dtype=np.float64)
    order = np.argsort(x, kind="stable")
    ranks = np.empty(len(x), dtype=np.float64)
    xs = x[order]
    i = 0
    while i < len(x):
        j = i
        while j + 1 < len(x) and xs[j + 1] == xs[i]:
            j += 1
        ranks[order[i:j + 1]] = 0.5 * (i + j) + 1.0
        i = j + 1
    return ranks


def _corr(a, b):
    a = a - a.mean()
    b = b - b.mean()
    den = np.sqrt(np.sum(a * a) * np.sum(b * b))
    return float(np.sum(a * b) / den) if den > 0 else float("nan")


def partial_spearman(x, y, z):
    """Spearman correlation of x and y controlling for z: the partial correlation of the ranks."""
    rx, ry, rz = _ranks(x), _ranks(y), _ranks(z)
    rxy, rxz, ryz = _corr(rx, ry), _corr(rx, rz), _corr(ry, rz)
    den = np.sqrt((1.0 - rxz * rxz) * (1.0 - ryz * ryz))
    return float((rxy - rxz * ryz) / den) if den > 0 else float("nan")


def summarize(probes):
    """The paper's calibration table (by D_t bin) and refresh-signal comparison."""
    D = np.array([p["D"] for p in probes], dtype=np.float64)
    A = np.array([p["A"] for p in probes], dtype=np.float64)
    dis = np.array([p["disagree"] for p in probes], dtype=np.float64)
    dH = np.array([p["dH"] for p in probes], dtype=np.float64)
    bins = []
    for lo, hi in D_BINS:
        sel = (D >= lo) & (D <= (np.inf if hi is None else hi))
        n = int(sel.sum())
        bins.append(dict(D=f"{lo}-{hi}" if hi is not None else f">={lo}", probes=n,
                         action_disagreement_pct=round(100.0 * dis[sel].mean(), 2) if n else None,
                         next_state_dH=round(float(dH[sel].mean()), 3) if n else None))

    def rho(x, y, z):   # None where a signal is constant over the probes (undefined)
        v = partial_spearman(x, y, z) if len(probes) > 2 else float("nan")
        return None if np.isnan(v) else round(v, 4)

    return dict(probes=len(probes), bins=bins,
                partial_spearman=dict(
                    distance_vs_disagreement=rho(D, dis, A),
                    distance_vs_next_state_dH=rho(D, dH, A),
                    age_vs_disagreement=rho(A, dis, D),
                    age_vs_next_state_dH=rho(A, dH, D)))
