"""GPU parity of the decoder and of Algorithm 1 against the oracle.

* the decision kernels on identical fp32 logits: the planted golden cases
  bit-exact; random full-vocabulary logits bit-exact except rows whose oracle
  margin is below the fp32 error of the kernel's log-sum-exp;
* archer_decode of the tiny fp32 workload under the age, Hamming and always
  rules: the free-run trajectory (schedule, D_t, A_t, unmasked positions and
  tokens, remasked positions, final response) equals the oracle's until a
  margin-exempt step (there is none: every decision is asserted bit-exact),
  with the rollback decoder and the no-rollback one (max_remask 0);
* a teacher-forced bf16 decode: at every step the GPU receives the oracle's
  state; logits agree within 2e-2 and decisions are bit-exact wherever the
  decision margin exceeds the logit error (the condition of Prop. app-decision).
"""

import json
import math
import os

import numpy as np
import pytest
import torch

from gpu_util import archer, dev_f32, dev_i32, host, make_ctx, say, with_gains
from oracle import controller as oc
from oracle import decode as odec
from oracle import decoder as od
from oracle import model as om
from synth.gen import model_weights, prompts
from synth.workloads import ModelShape, get_workload

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "decoder_planted.json")
LSE_SLACK = 1e-4   # fp32 error bound of the kernel's ell / q, far above what it reaches


def _decide_ctx(V, G, B=1):
    m = ModelShape(n_layers=1, d_model=64, n_heads=1, n_kv_heads=1, head_dim=64, d_ff=64, vocab=V,
                   dtype="fp32", init_std=0.02)
    W = model_weights(m, seed=1)
    ctx = make_ctx(m, W, B, 8, 8 * B, G)
    # establish the batch and an anchor (all MASK)
    ctx.refresh_prompt(dev_i32(np.zeros(8 * B, np.int32)), [8] * B, dev_i32(np.full((B, G), m.mask_id)))
    return m, ctx


def test_decide_planted_cases():
    cases = json.load(open(GOLDEN))["cases"]
    V, G = 64, 8
    m, ctx = _decide_ctx(V, G)
    for c in cases:
        Vc, mc = len(c["z"][0]), c["mask_id"]
        n = len(c["g"])
        z = np.full((G, V), -1000.0, np.float32)
        g = np.zeros(G, np.int32)
        for i in range(n):
            z[i, : Vc - 1] = c["z"][i][: Vc - 1]
            z[i, m.mask_id] = c["z"][i][mc]
            g[i] = m.mask_id if c["g"][i] == mc else c["g"][i]
        for i in range(n, G):            # padding rows: decided, probability 1
            z[i, 5] = 50.0
            g[i] = 5
        g_out, dist, um, rm = ctx.decide(dev_f32(z[None]), dev_i32(g[None]), k=c["k"], tau=c["tau"],
                                         final=c["final"])
        want = [m.mask_id if t == mc else t for t in c["expected_g_next"]]
        got = g_out.cpu().numpy()[0]
        assert got[:n].tolist() == want, c["name"]
        assert got[n:].tolist() == [5] * (G - n)
        # the position list holds at most k entries (the final step may unmask more; g_out is complete)
        assert [p for p in um.cpu().numpy()[0] if p >= 0] == c["expected_U"][: c["k"]], c["name"]
        assert rm.cpu().numpy()[0] == (c["expected_Rm"][0] if c["expected_Rm"] else -1), c["name"]


@pytest.mark.parametrize("V,G,B,k", [(126464, 256, 1, 1), (152064, 64, 4, 2), (1024, 32, 2, 3)])
def test_decide_random_logits_full_vocab(V, G, B, k):
    say(f"decide on random logits V={V} G={G} B={B} k={k}")
    m, ctx = _decide_ctx(V, G, B)
    rng = np.random.default_rng(V + G)
    z = (rng.standard_normal((B, G, V)) * 1.3).astype(np.float32)
    g = np.full((B, G), m.mask_id, np.int32)
    for b in range(B):
        dec = rng.choice(G, G // 3, replace=False)
        g[b, dec] = rng.integers(0, V - 1, len(dec))
        z[b, dec[:2], g[b, dec[:2]]] += 9.0          # some decided rows above tau
    exempt = 0
    for final in (False, True):
        g_out, dist, um, rm = ctx.decide(dev_f32(z), dev_i32(g), k=k, tau=0.1, final=final)
        go = g_out.cpu().numpy()
        for b in range(B):
            want, U, Rm, st = od.decide(z[b], g[b], m.mask_id, k, 0.1, final=final)
            # the argmax token of every unmasked row is exact (max is order-free)
            if go[b].tolist() != want.tolist():
                mD = od.decision_margin(z[b], g[b], m.mask_id, k, 0.1, final=final)
                assert mD <= LSE_SLACK, (b, mD)
                exempt += 1
            assert int(dist.cpu().numpy()[b]) == oc.hamming(go[b], np.full(G, m.mask_id))
    assert exempt == 0


def _gpu_traj(tr, b, k):
    T = tr["refreshed"].shape[0]
    out = []
    for t in range(T):
        U = [int(x) for x in tr["unmask_pos"][t, b].cpu().numpy() if x >= 0]
        toks = [int(x) for x in tr["unmask_tok"][t, b].cpu().numpy()[: len(U)]]
        rm = int(tr["remask_pos"][t, b].cpu().numpy())
        out.append(dict(ref=int(tr["refreshed"][t, b]), dist=int(tr["dist"][t, b]), age=int(tr["age"][t, b]),
                        U=U, tok=toks, Rm=[rm] if rm >= 0 else []))
    return out


@pytest.mark.parametrize("policy,K,max_remask", [("age", 4, 1), ("hamming", 4, 1), ("hamming", 1, 1),
                                                ("always", 0, 1), ("age", 4, 0), ("hamming", 3, 0)])
def test_tiny_decode_matches_oracle(policy, K, max_remask):
    """Free run of the fp32 workload: every step's record and the final response equal the
    oracle's, with no margin-exempt step (max_remask 0 is the no-rollback decoder)."""
    w = get_workload("tiny")
    m, dec = w.model, w.decode
    say(f"tiny fp32 decode policy={policy} K={K} max_remask={max_remask}")
    a = archer()
    W = model_weights(m, seed=w.weight_seed)
    p = prompts(w)[0]
    G, T, k = dec.resp_len, dec.steps, dec.unmask_per_step
    ctx = make_ctx(m, W, 1, len(p), len(p), G)
    pol = {"age": a.AGE, "hamming": a.HAMMING, "always": a.ALWAYS}[policy]
    resp = dev_i32(np.full((1, G), m.mask_id))
    out, tr = ctx.decode(dev_i32(p), [len(p)], resp, policy=pol, K=K, steps=T, k=k, tau=dec.remask_threshold,
                         max_remask=max_remask)
    g_o, tr_o = odec.decode(W, m, p, np.full(G, m.mask_id), steps=T, k=k, tau=dec.remask_threshold,
                            policy={"age": oc.AGE, "hamming": oc.HAMMING, "always": oc.ALWAYS}[policy], K=K,
                            remask=max_remask == 1, keep_logits=True)
    gt = _gpu_traj(tr, 0, k)
    remasks = 0
    for t in range(T):
        g_next = tr_o.states[t + 1] if t + 1 < T else g_o
        U = list(tr_o.unmask[t])[:k]            # the trace lists at most k positions per step
        want = dict(ref=int(tr_o.refreshed[t]), dist=int(tr_o.dist[t]), age=int(tr_o.age[t]),
                    U=U, tok=[int(g_next[i]) for i in U], Rm=list(tr_o.remask[t]))
        mD = od.decision_margin(tr_o.logits[t], tr_o.states[t], m.mask_id, k, dec.remask_threshold,
                                final=t == T - 1, remask=max_remask == 1)
        # the fp32 workload has no margin-exempt step: every decision is bit-exact
        assert gt[t] == want, f"step {t}: gpu {gt[t]} oracle {want} margin {mD:.2e}"
        remasks += len(want["Rm"])
    if max_remask == 0:
        assert remasks == 0
    else:
        assert remasks > 0        # the rollback branch is exercised
    assert out.cpu().numpy()[0].tolist() == g_o.tolist()
    assert m.mask_id not in g_o.tolist()


def test_teacher_forced_bf16_decode():
    m = ModelShape(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=1024,
                   dtype="bf16", init_std=0.08)
    say("teacher-forced bf16 decode (GQA hd 64), age K=4")
    W = with_gains(model_weights(m, seed=12), 12)
    P, G, T, k, tau, K = 100, 32, 32, 1, 0.1, 4
    p = np.random.default_rng(13).integers(0, m.vocab - 1, P).astype(np.int32)
    ctx = make_ctx(m, W, 1, P, P, G)
    g = np.full(G, m.mask_id)
    r = 0
    z, cache, _ = om.full_forward(W, m, p, g)
    zg = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g[None])))[0]
    exempt = 0
    worst = 0.0
    for t in range(T):
        final = t == T - 1
        eps = float(np.max(np.abs(zg - z)))
        worst = max(worst, eps)
        assert eps < 2e-2, (t, eps)
        g_next, U, Rm, _ = od.decide(z, g, m.mask_id, k, tau, final=final)
        go, dist, um, rm = ctx.decide(dev_f32(zg[None]), dev_i32(g[None]), k=k, tau=tau, final=final)
        go = go.cpu().numpy()[0]
        if go.tolist() != g_next.tolist():
            mD = od.decision_margin(z, g, m.mask_id, k, tau, final=final)
            assert mD <= eps + LSE_SLACK, (t, mD, eps)
            exempt += 1
        g = g_next
        if final:
            break
        s = t + 1
        if s - r >= K:
            z, cache, _ = om.full_forward(W, m, p, g)
            zg = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g[None])))[0]
            r = s
        else:
            z, _ = om.cached_forward(W, m, g, cache, P)
            zg = host(ctx.step(dev_i32(g[None])))[0]
    say(f"  worst logit error {worst:.2e}, margin-exempt steps {exempt}")
    assert exempt <= 2
