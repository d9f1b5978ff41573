"""GPU parity at the workloads' real depth and width (through archer.h / archer_ops.h).

Every comparison is against the float64 oracle on host weights from synth.gen:

* LLaDA-8B shape with all 32 layers, P 512, G 256, in the bench's launch
  configuration: FullForward and CachedForward logits, final normalised hidden
  state and final residual stream of the response rows, and the prompt cache
  C_p (Eq. app-cached) of the first, a middle and the last layer; the same at
  depth 2 and 8 (contexts over the first layers of the same weights), which
  gives the error-versus-depth curve;
* the long-prompt workload at its real depth: P 4096, 32 layers;
* Dream-7B shape (GQA 28 / 4 heads, F 18944, V 152064): all 28 layers at
  batch 1, and two layers at batch 2, P 1024, G 512: both passes, hidden
  state and C_p;
* the ragged batch of the batched workload (16 sequences, the workload's
  seeded prompt lengths in [256, 2048]), two layers at full width, in the
  bench's launch configuration for that batch (one split per pass, folded
  split-K in the refresh pass): three sampled sequences (the shortest, the
  longest and one in between) against the oracle run on each alone;
* decisions at full width, teacher-forced: the GPU decoder on GPU logits
  against the oracle decoder on oracle logits, bit-exact wherever the
  decision margin exceeds the logit error (Prop. app-decision).

Bar: 2e-2 max abs for the logits, the final normalised hidden state and the
prompt cache (stored as fp16 by the precision contract; the share of its
elements that differ from the oracle's fp16 values is reported beside it).
The residual stream grows with depth (max |x| about 72 after 32 layers of
the random-init model, where 2e-2 is 3e-4 relative, finer than bf16's own
resolution there), so it is held to 2e-2 in units of each row's RMS -- the
quantity every RMSNorm passes on to the next projection -- with its plain
max abs error reported beside it.
"""

import dataclasses
import time

import numpy as np
import pytest
import torch

from gpu_util import archer, dev_f32, dev_i32, host, say
from oracle import decoder as od
from oracle import model as om
from synth.gen import model_weights, prompt_lengths, prompts
from synth.workloads import get_workload

pytestmark = pytest.mark.gpu

BAR = 2e-2


def _cmp_cache(name, got, want):
    """got: the GPU's cache (fp16); want: the oracle's fp16-rounded float64 values (same shape).
    Bar: 2e-2 max abs; the share of elements that differ (rounding-boundary flips of inputs
    that differ by float32 accumulation order) is reported beside it."""
    g = host(got)
    d = np.abs(g - want)
    frac = float(np.mean(d > 0))
    say(f"  {name}: max abs {d.max():.3e} (max |ref| {np.abs(want).max():.2f}), "
        f"elements differing {100 * frac:.2f} %")
    assert d.max() < BAR, f"{name}: {d.max():.3e}"
    return float(d.max()), frac


def _resid(name, got, want):
    """Residual stream rows: the bar in units of each row's RMS (what the next RMSNorm passes on);
    the plain max abs is reported beside it."""
    rms = np.sqrt(np.mean(want * want, axis=1, keepdims=True))
    e = float(np.max(np.abs(got - want) / rms))
    say(f"  {name}: max abs err {np.max(np.abs(got - want)):.3e} (max |ref| {np.max(np.abs(want)):.2f}), "
        f"in row-RMS units {e:.3e}")
    assert e < BAR, f"{name}: {e:.3e}"
    return e


def _err(name, got, want, bar=BAR):
    e = float(np.max(np.abs(got - want)))
    say(f"  {name}: max abs err {e:.3e} (max |ref| {np.max(np.abs(want)):.2f})")
    assert e < bar, f"{name}: {e:.3e}"
    return e


def _device_weights(W, m):
    a = archer()
    return a.pack_weights(a.upload_weights(W, "bf16", m.gateup_fp16), drop_source=True)


def _ctx(m, Wd, max_batch, max_prompt_len, max_prompt_total, G, layers=None):
    a = archer()
    if layers is not None:
        m = dataclasses.replace(m, n_layers=layers)
        Wd = dict(Wd, layers=Wd["layers"][:layers])
    return a.Context(m, Wd, max_batch, max_prompt_len, max_prompt_total, G)


# ----------------------------------------------------------------------------------------------
# LLaDA-8B shape, all 32 layers


@pytest.fixture(scope="module")
def llada32():
    w = get_workload("llada_p512")
    m = w.model
    P, G = w.decode.prompt_len, w.decode.resp_len
    t0 = time.time()
    say(f"LLaDA-8B shape, {m.n_layers} layers: generating host weights")
    W = model_weights(m, seed=w.weight_seed)
    say(f"  host weights in {time.time() - t0:.1f} s; uploading")
    Wd = _device_weights(W, m)
    p = prompts(w)[0]
    g0 = np.full(G, m.mask_id)
    g0[:48] = (np.arange(48) * 131) % (m.vocab - 1)
    g1 = g0.copy()
    g1[96:160] = (np.arange(64) * 17 + 5) % (m.vocab - 1)
    g1[10:14] = m.mask_id
    st = dict(w=w, m=m, P=P, G=G, W=W, Wd=Wd, p=p, g0=g0, g1=g1, oracle={})
    yield st
    st.clear()
    torch.cuda.empty_cache()


def _oracle_full(st, layers):
    key = ("full", layers)
    if key not in st["oracle"]:
        m = dataclasses.replace(st["m"], n_layers=layers)
        W = dict(st["W"], layers=st["W"]["layers"][:layers])
        t0 = time.time()
        z, cache, hidden = om.full_forward(W, m, st["p"], st["g0"], keep_hidden=True)
        say(f"  oracle FullForward at depth {layers}: {time.time() - t0:.1f} s")
        resid = hidden[0][-1][st["P"]:]
        st["oracle"][key] = (z, cache, resid, hidden[1])
    return st["oracle"][key]


def _check_depth(st, layers, cache_layers):
    a = archer()
    m, P, G = st["m"], st["P"], st["G"]
    ctx = _ctx(m, st["Wd"], 1, P, P, G, layers=layers)
    say(f"depth {layers}: GPU FullForward")
    z = host(ctx.refresh_prompt(dev_i32(st["p"]), [P], dev_i32(st["g0"][None])))[0]
    hid = host(ctx.read_rows(a.READ_HIDDEN, 1))
    res = host(ctx.read_rows(a.READ_RESIDUAL, 1))
    kv = {l: ctx.read_prompt_kv(l, 0, P) for l in cache_layers}
    z_ref, cache, res_ref, hid_ref = _oracle_full(st, layers)
    out = dict(logits=_err(f"depth {layers} full logits", z, z_ref),
               hidden=_err(f"depth {layers} full normalised hidden", hid, hid_ref),
               residual=_resid(f"depth {layers} full residual", res, res_ref))
    for l, (k, v) in kv.items():
        _cmp_cache(f"depth {layers} C_p layer {l} K", k, cache[l][0])
        _cmp_cache(f"depth {layers} C_p layer {l} V", v, cache[l][1])
    return ctx, cache, out


def test_llada_depth_32(llada32):
    st = llada32
    ctx, cache, full = _check_depth(st, 32, (0, 15, 31))
    a = archer()
    m, P, G = st["m"], st["P"], st["G"]
    say("depth 32: GPU CachedForward on the anchored cache")
    zc = host(ctx.step(dev_i32(st["g1"][None])))[0]
    hid = host(ctx.read_rows(a.READ_HIDDEN, 1))
    res = host(ctx.read_rows(a.READ_RESIDUAL, 1))
    t0 = time.time()
    zc_ref, (stack, hid_ref) = om.cached_forward(st["W"], m, st["g1"], cache, P, keep_hidden=True)
    say(f"  oracle CachedForward: {time.time() - t0:.1f} s")
    _err("depth 32 cached logits", zc, zc_ref)
    _err("depth 32 cached normalised hidden", hid, hid_ref)
    _resid("depth 32 cached residual", res, stack[-1])
    # decisions on the two sets of logits (teacher-forced on the same state g1)
    go, _, _, _ = ctx.decide(dev_f32(zc[None]), dev_i32(st["g1"][None]), k=1, tau=0.1)
    want = od.decide(zc_ref, st["g1"], m.mask_id, 1, 0.1)[0]
    eps = float(np.max(np.abs(zc - zc_ref)))
    if go.cpu().numpy()[0].tolist() != want.tolist():
        mD = od.decision_margin(zc_ref, st["g1"], m.mask_id, 1, 0.1)
        say(f"  decision differs; oracle margin {mD:.3e}, logit error {eps:.3e}")
        assert mD <= eps + 1e-4
    ctx.close()


def test_llada_depth_curve_2_and_8(llada32):
    """Logit / hidden / residual error against depth: 2 and 8 layers of the same weights (32 above)."""
    for layers in (2, 8):
        ctx, _, _ = _check_depth(llada32, layers, (layers - 1,))
        ctx.close()


def test_llada_depth_32_long_prompt(llada32):
    """The long-prompt workload at its real depth: P 4096, G 256, 32 layers -- the 4352-row
    refresh pass (one split, folded split-K) and the cached pass (split-KV over 4352 keys)."""
    a = archer()
    st = llada32
    w = get_workload("llada_p4096")
    m, G = st["m"], st["G"]
    P = w.decode.prompt_len
    p = prompts(w)[0]
    ctx = _ctx(m, st["Wd"], 1, P, P, G)
    g0 = np.full(G, m.mask_id)
    g0[:64] = (np.arange(64) * 37) % (m.vocab - 1)
    g1 = g0.copy()
    g1[128:192] = (np.arange(64) * 13 + 3) % (m.vocab - 1)
    say("depth 32, P 4096: GPU FullForward and CachedForward")
    z = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g0[None])))[0]
    kv = ctx.read_prompt_kv(31, 0, P)
    zc = host(ctx.step(dev_i32(g1[None])))[0]
    hid = host(ctx.read_rows(a.READ_HIDDEN, 1))
    res = host(ctx.read_rows(a.READ_RESIDUAL, 1))
    ctx.close()
    t0 = time.time()
    z_ref, cache, _ = om.full_forward(st["W"], m, p, g0)
    say(f"  oracle FullForward over 4352 rows: {time.time() - t0:.1f} s")
    _err("P 4096 depth 32 full logits", z, z_ref)
    _cmp_cache("P 4096 depth 32 C_p layer 31 K", kv[0], cache[31][0])
    _cmp_cache("P 4096 depth 32 C_p layer 31 V", kv[1], cache[31][1])
    zc_ref, (stack, hid_ref) = om.cached_forward(st["W"], m, g1, cache, P, keep_hidden=True)
    _err("P 4096 depth 32 cached logits", zc, zc_ref)
    _err("P 4096 depth 32 cached normalised hidden", hid, hid_ref)
    _resid("P 4096 depth 32 cached residual", res, stack[-1])


# ----------------------------------------------------------------------------------------------
# Dream-7B shape (GQA): all 28 layers at batch 1, two layers at batch 2


def test_dream_all_28_layers():
    a = archer()
    w = get_workload("dream_gqa")
    m = w.model
    P, G = w.decode.prompt_len, w.decode.resp_len
    t0 = time.time()
    say(f"Dream shape, {m.n_layers} layers, B 1, P {P}, G {G}: generating host weights")
    W = model_weights(m, seed=w.weight_seed)
    say(f"  host weights in {time.time() - t0:.1f} s")
    Wd = _device_weights(W, m)
    p = prompts(w)[0]
    ctx = _ctx(m, Wd, 1, P, P, G)
    rng = np.random.default_rng(73)
    g0 = np.full(G, m.mask_id)
    idx = rng.choice(G, G // 4, replace=False)
    g0[idx] = rng.integers(0, m.vocab - 1, len(idx))
    g1 = g0.copy()
    idx = rng.choice(G, G // 8, replace=False)
    g1[idx] = rng.integers(0, m.vocab - 1, len(idx))
    z = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g0[None])))[0]
    hid = host(ctx.read_rows(a.READ_HIDDEN, 1))
    res = host(ctx.read_rows(a.READ_RESIDUAL, 1))
    kv = ctx.read_prompt_kv(m.n_layers - 1, 0, P)
    zc = host(ctx.step(dev_i32(g1[None])))[0]
    ctx.close()
    del Wd
    t0 = time.time()
    z_ref, cache, (stack, h_ref) = om.full_forward(W, m, p, g0, keep_hidden=True)
    say(f"  oracle FullForward: {time.time() - t0:.1f} s")
    _err("Dream depth 28 full logits", z, z_ref)
    _err("Dream depth 28 full normalised hidden", hid, h_ref)
    _resid("Dream depth 28 full residual", res, stack[-1][P:])
    _cmp_cache("Dream depth 28 C_p layer 27 K", kv[0], cache[-1][0])
    _cmp_cache("Dream depth 28 C_p layer 27 V", kv[1], cache[-1][1])
    zc_ref, _ = om.cached_forward(W, m, g1, cache, P)
    _err("Dream depth 28 cached logits", zc, zc_ref)


def test_dream_two_layers_full_width_batch2():
    a = archer()
    w = get_workload("dream_gqa")
    m = dataclasses.replace(w.model, n_layers=2)
    P, G, B = w.decode.prompt_len, w.decode.resp_len, 2
    say(f"Dream shape, 2 layers, B {B}, P {P}, G {G}: generating host weights")
    W = model_weights(m, seed=w.weight_seed)
    Wd = _device_weights(W, m)
    ps = prompts(w)[:B]
    ctx = _ctx(m, Wd, w.decode.batch, P, P * w.decode.batch, G)
    rng = np.random.default_rng(71)
    g0 = np.full((B, G), m.mask_id)
    for b in range(B):
        idx = rng.choice(G, G // 4, replace=False)
        g0[b, idx] = rng.integers(0, m.vocab - 1, len(idx))
    g1 = g0.copy()
    for b in range(B):
        idx = rng.choice(G, G // 8, replace=False)
        g1[b, idx] = rng.integers(0, m.vocab - 1, len(idx))
    z = host(ctx.refresh_prompt(dev_i32(np.concatenate(ps)), [P] * B, dev_i32(g0)))
    hid = host(ctx.read_rows(a.READ_HIDDEN, B))
    kv = [ctx.read_prompt_kv(1, b, P) for b in range(B)]
    zc = host(ctx.step(dev_i32(g1)))
    hidc = host(ctx.read_rows(a.READ_HIDDEN, B))
    for b in range(B):
        t0 = time.time()
        z_ref, cache, (_, h_ref) = om.full_forward(W, m, ps[b], g0[b], keep_hidden=True)
        say(f"  sequence {b}: oracle FullForward {time.time() - t0:.1f} s")
        _err(f"Dream seq {b} full logits", z[b], z_ref)
        _err(f"Dream seq {b} full normalised hidden", hid[b * G:(b + 1) * G], h_ref)
        _cmp_cache(f"Dream seq {b} C_p layer 1 K", kv[b][0], cache[1][0])
        _cmp_cache(f"Dream seq {b} C_p layer 1 V", kv[b][1], cache[1][1])
        zc_ref, (_, hc_ref) = om.cached_forward(W, m, g1[b], cache, P, keep_hidden=True)
        _err(f"Dream seq {b} cached logits", zc[b], zc_ref)
        _err(f"Dream seq {b} cached normalised hidden", hidc[b * G:(b + 1) * G], hc_ref)
    ctx.close()


# ----------------------------------------------------------------------------------------------
# the batched ragged workload, two layers at full width


def test_ragged16_two_layers_full_width_sampled():
    a = archer()
    w = get_workload("llada_ragged16")
    m = dataclasses.replace(w.model, n_layers=2)
    G, B = w.decode.resp_len, w.decode.batch
    lens = prompt_lengths(w)
    ps = prompts(w, lens)
    say(f"ragged batch, 2 layers, B {B}, P {lens}: generating host weights")
    W = model_weights(m, seed=w.weight_seed)
    Wd = _device_weights(W, m)
    ctx = _ctx(m, Wd, B, max(lens), sum(lens), G)
    rng = np.random.default_rng(72)
    g0 = np.full((B, G), m.mask_id)
    g1 = g0.copy()
    for b in range(B):
        idx = rng.choice(G, 40, replace=False)
        g0[b, idx] = rng.integers(0, m.vocab - 1, 40)
        g1[b] = g0[b]
        idx = rng.choice(G, 24, replace=False)
        g1[b, idx] = rng.integers(0, m.vocab - 1, 24)
    z = host(ctx.refresh_prompt(dev_i32(np.concatenate(ps)), lens, dev_i32(g0)))
    sample = [int(np.argmin(lens)), int(np.argmax(lens)), int(np.argsort(lens)[B // 2])]
    kv = {b: ctx.read_prompt_kv(1, b, lens[b]) for b in sample}
    zc = host(ctx.step(dev_i32(g1)))
    hidc = host(ctx.read_rows(a.READ_HIDDEN, B))
    for b in sample:
        t0 = time.time()
        z_ref, cache, _ = om.full_forward(W, m, ps[b], g0[b])
        say(f"  sequence {b} (P {lens[b]}): oracle FullForward {time.time() - t0:.1f} s")
        _err(f"ragged seq {b} full logits", z[b], z_ref)
        _cmp_cache(f"ragged seq {b} C_p layer 1 K", kv[b][0], cache[1][0])
        _cmp_cache(f"ragged seq {b} C_p layer 1 V", kv[b][1], cache[1][1])
        zc_ref, (_, hc_ref) = om.cached_forward(W, m, g1[b], cache, lens[b], keep_hidden=True)
        _err(f"ragged seq {b} cached logits", zc[b], zc_ref)
        _err(f"ragged seq {b} cached normalised hidden", hidc[b * G:(b + 1) * G], hc_ref)
    ctx.close()


# ----------------------------------------------------------------------------------------------
# teacher-forced decisions at full width (two LLaDA-shaped layers, P 512)


def test_teacher_forced_decisions_full_width():
    w = get_workload("llada_p512")
    m = dataclasses.replace(w.model, n_layers=2)
    P, G, k, tau, K = w.decode.prompt_len, w.decode.resp_len, 1, 0.1, 3
    say("teacher-forced decisions, 2 full-width LLaDA layers, age rule K 3, 6 steps")
    W = model_weights(m, seed=w.weight_seed)
    Wd = _device_weights(W, m)
    p = prompts(w)[0]
    ctx = _ctx(m, Wd, 1, P, P, G)
    g = np.full(G, m.mask_id)
    z, cache, _ = om.full_forward(W, m, p, g)
    zg = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g[None])))[0]
    r, exempt, worst = 0, 0, 0.0
    T = 6
    for t in range(T):
        eps = float(np.max(np.abs(zg - z)))
        worst = max(worst, eps)
        assert eps < BAR, (t, eps)
        g_next, U, Rm, _ = od.decide(z, g, m.mask_id, k, tau)
        go, _, _, _ = ctx.decide(dev_f32(zg[None]), dev_i32(g[None]), k=k, tau=tau)
        if go.cpu().numpy()[0].tolist() != g_next.tolist():
            mD = od.decision_margin(z, g, m.mask_id, k, tau)
            assert mD <= eps + 1e-4, (t, mD, eps)
            exempt += 1
        say(f"  step {t}: logit error {eps:.2e}, unmask {U}, remask {Rm}")
        g = g_next
        s = t + 1
        if s - r >= K:
            z, cache, _ = om.full_forward(W, m, p, g)
            zg = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g[None])))[0]
            r = s
        else:
            z, _ = om.cached_forward(W, m, g, cache, P)
            zg = host(ctx.step(dev_i32(g[None])))[0]
    say(f"  worst logit error {worst:.2e}, margin-exempt steps {exempt} of {T}")
    ctx.close()
