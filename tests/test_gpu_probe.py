"""GPU parity of the cache-validity probe (non-intervening shadow forwards).

* the main trajectory the probe drives (refresh schedule, D_t, A_t, final
  response) is bitwise the one archer_decode produces: the shadow forwards
  intervene in nothing;
* on the tiny fp32 workload every probe record (forward index, D_t, A_t,
  action disagreement, next-state Hamming distance) equals the one of the
  same probe run by the oracle (cached and fresh forwards in float64), up to
  decisions whose oracle margin is below the fp32 error of the kernels;
* archer_decode on a ragged bf16 batch (per-sequence refreshes mixed with
  cached forwards) equals the same algorithm driven call by call, bitwise.
"""

import numpy as np
import pytest

from gpu_util import archer, dev_i32, make_ctx, say
from oracle import controller as oc
from oracle import decoder as od
from oracle import model as om
from synth.gen import model_weights, prompts
from synth.workloads import get_workload

pytestmark = pytest.mark.gpu

MARGIN = 1e-4   # fp32 error bound of the kernels' log-confidences, far above what they reach


def _oracle_probe(W, m, p, g0, *, steps, k, tau, policy, K):
    P = len(p)
    g = g0.copy()
    z, cache, _ = om.full_forward(W, m, p, g)
    g_r, r = g.copy(), 0
    recs, pending = [], None
    for t in range(steps):
        final = t == steps - 1
        g_next = od.decide(z, g, m.mask_id, k, tau, final=final)[0]
        if pending is not None:
            s, g_fresh, D, A, zc, zf, gs = pending
            diff = int(np.sum(g_next != g_fresh))
            recs.append(dict(t=s, D=D, A=A, disagree=int(diff > 0), dH=diff, zc=zc, zf=zf, g=gs))
            pending = None
        if final:
            break
        s = t + 1
        D, A = oc.hamming(g_next, g_r), s - r
        if oc.should_refresh(policy, K, D, A):
            z, cache, _ = om.full_forward(W, m, p, g_next)
            g_r, r = g_next.copy(), s
        else:
            z, _ = om.cached_forward(W, m, g_next, cache, P)
            zf, _, _ = om.full_forward(W, m, p, g_next)
            g_fresh = od.decide(zf, g_next, m.mask_id, k, tau, final=s == steps - 1)[0]
            pending = (s, g_fresh, D, A, z, zf, g_next.copy())
        g = g_next
    return recs


@pytest.mark.parametrize("policy,K", [("age", 4), ("hamming", 3)])
def test_probe_is_non_intervening_and_matches_oracle(policy, K):
    from paper_2608_08086_amd import probe

    a = archer()
    w = get_workload("tiny")
    m, dec = w.model, w.decode
    say(f"shadow probe, tiny fp32 workload, policy={policy} K={K}")
    W = model_weights(m, seed=w.weight_seed)
    p = prompts(w)[0]
    G, T, k, tau = dec.resp_len, dec.steps, dec.unmask_per_step, dec.remask_threshold
    ctx = make_ctx(m, W, 1, len(p), len(p), G)
    shadow = make_ctx(m, W, 1, len(p), len(p), G)
    pol = {"age": a.AGE, "hamming": a.HAMMING}[policy]
    g0 = dev_i32(np.full((1, G), m.mask_id))
    g_fin, tr, recs = probe.shadow_probe(ctx, shadow, dev_i32(p), [len(p)], g0, policy=pol, K=K, steps=T, k=k,
                                         tau=tau)
    # non-intervention: the same trajectory as archer_decode
    ref_ctx = make_ctx(m, W, 1, len(p), len(p), G)
    out, tr_d = ref_ctx.decode(dev_i32(p), [len(p)], dev_i32(np.full((1, G), m.mask_id)), policy=pol, K=K,
                               steps=T, k=k, tau=tau)
    np.testing.assert_array_equal(g_fin.cpu().numpy(), out.cpu().numpy())
    for key in ("refreshed", "dist", "age"):
        np.testing.assert_array_equal(tr[key], tr_d[key].cpu().numpy(), err_msg=key)
    n_cached = int(T - tr["refreshed"].sum())
    assert len(recs) == n_cached > 0
    # every record against the oracle's probe
    want = _oracle_probe(W, m, p, np.full(G, m.mask_id), steps=T, k=k, tau=tau,
                         policy={"age": oc.AGE, "hamming": oc.HAMMING}[policy], K=K)
    assert len(want) == len(recs)
    for got, o in zip(recs, want):
        fields = ("t", "D", "A", "disagree", "dH")
        if any(got[f] != o[f] for f in fields):
            final = o["t"] == T - 1
            mc = od.decision_margin(o["zc"], o["g"], m.mask_id, k, tau, final=final)
            mf = od.decision_margin(o["zf"], o["g"], m.mask_id, k, tau, final=final)
            assert min(mc, mf) <= MARGIN, (got, {f: o[f] for f in fields}, mc, mf)
            say(f"  margin-exempt record at forward {o['t']} (margins {mc:.2e}, {mf:.2e})")
            return
    say(f"  {len(recs)} probes, disagreement {np.mean([r['disagree'] for r in recs]):.3f}")


@pytest.mark.parametrize("policy,K", [("age", 3), ("hamming", 4)])
def test_batched_bf16_decode_equals_call_driven_trajectory(policy, K):
    """archer_decode on a ragged bf16 batch (k-block weights, per-sequence refreshes mixed with
    cached steps in one forward) against the same Algorithm 1 driven through archer_refresh_prompt /
    archer_step / archer_decide: bitwise the same trajectories and responses."""
    from paper_2608_08086_amd import probe
    from synth.workloads import ModelShape

    a = archer()
    m = ModelShape(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                   dtype="bf16", init_std=0.05)
    say(f"batched bf16 decode vs call-driven trajectory, policy={policy} K={K}")
    W = model_weights(m, seed=21)
    lens, G, T, k = [37, 90], 32, 24, 2
    rng = np.random.default_rng(22)
    ps = [rng.integers(0, m.vocab - 1, n).astype(np.int32) for n in lens]
    prompt = dev_i32(np.concatenate(ps))
    pol = {"age": a.AGE, "hamming": a.HAMMING}[policy]
    ctx = make_ctx(m, W, 2, max(lens), sum(lens), G)
    shadow = make_ctx(m, W, 2, max(lens), sum(lens), G)
    g0 = dev_i32(np.full((2, G), m.mask_id))
    g_fin, tr, _ = probe.shadow_probe(ctx, shadow, prompt, lens, g0, policy=pol, K=K, steps=T, k=k, tau=0.1,
                                      every=5)
    ref_ctx = make_ctx(m, W, 2, max(lens), sum(lens), G)
    out, tr_d = ref_ctx.decode(prompt, lens, dev_i32(np.full((2, G), m.mask_id)), policy=pol, K=K, steps=T, k=k,
                               tau=0.1)
    np.testing.assert_array_equal(g_fin.cpu().numpy(), out.cpu().numpy())
    for key in ("refreshed", "dist", "age"):
        np.testing.assert_array_equal(tr[key], tr_d[key].cpu().numpy(), err_msg=key)
    # after the initial forward both refreshes and cached forwards happened
    assert 0 < tr["refreshed"][1:].sum() < (T - 1) * 2, tr["refreshed"].T
    assert (out.cpu().numpy() != m.mask_id).all()
