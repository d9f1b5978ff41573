"""GPU parity of the two forward modes against the oracle (through archer.h).

* tiny fp32 workload: FullForward and CachedForward logits within 1e-5
  (norm-relative);
* small bf16 models (GQA hd 64, MHA hd 128, ragged prompt lengths): logits
  within 2e-2 max abs;
* on the GPU, CachedForward on the cache of the same response equals
  FullForward bitwise, and a sequence's logits do not depend on the batch;
* a ragged batch with per-sequence refresh (seq_sel);
* the largest batch (64 sequences) with a one-token prompt;
* the k-block weight layout: the pack kernel is the stated permutation, and a
  model gives the same bits in either layout (bf16 contexts use the k-block
  layout unless a test says otherwise, as the bench does);
* full-width 2-layer LLaDA-8B-shaped models (d 4096, vocab 126464, G 256)
  at P 512 and P 4096 in the bench's launch configurations (at P 4096: the
  cached pass with 8-way split-KV, the 4352-row refresh with one split and
  split-K projections).
"""

import dataclasses

import numpy as np
import pytest
import torch

from gpu_util import archer, dev_i32, host, make_ctx, rand_bf16, rel_err, say, with_gains
from oracle import model as om
from synth.gen import model_weights, prompts
from synth.workloads import ModelShape, get_workload

pytestmark = pytest.mark.gpu

SMALL_BF16 = {
    "gqa_hd64": ModelShape(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512,
                           vocab=1024, dtype="bf16", init_std=0.05),
    "mha_hd128": ModelShape(n_layers=2, d_model=256, n_heads=2, n_kv_heads=2, head_dim=128, d_ff=768,
                            vocab=1024, dtype="bf16", init_std=0.05),
}
# the same models with fp16 gate/up operands (split-K gate/up partials, the fp16 RMSNorm
# fused into the O projection's split-K reduction)
SMALL_BF16.update({k + "_gateup_fp16": dataclasses.replace(v, gateup_fp16=True) for k, v in list(SMALL_BF16.items())})


def _resp(m, G, seed, frac=0.3):
    rng = np.random.default_rng(seed)
    g = np.full(G, m.mask_id)
    idx = rng.choice(G, int(frac * G), replace=False)
    g[idx] = rng.integers(0, m.vocab - 1, len(idx))
    return g


def _prompt(m, P, seed):
    return np.random.default_rng(seed).integers(0, m.vocab - 1, P).astype(np.int32)


def test_tiny_fp32_workload_full_and_cached():
    w = get_workload("tiny")
    m, G = w.model, w.decode.resp_len
    say("tiny fp32 workload: full + cached forward")
    W = model_weights(m, seed=w.weight_seed)
    p = prompts(w)[0]
    ctx = make_ctx(m, W, 1, len(p), len(p), G)
    g0 = np.full(G, m.mask_id)
    z = host(ctx.refresh_prompt(dev_i32(p), [len(p)], dev_i32(g0[None])))[0]
    z_ref, cache, _ = om.full_forward(W, m, p, g0)
    assert rel_err(z, z_ref) < 1e-5
    g1 = _resp(m, G, 3)
    zc = host(ctx.step(dev_i32(g1[None])))[0]
    zc_ref, _ = om.cached_forward(W, m, g1, cache, len(p))
    assert rel_err(zc, zc_ref) < 1e-5
    # the GPU follows the anchored cache, not the fresh one
    z1_ref, _, _ = om.full_forward(W, m, p, g1)
    assert np.max(np.abs(z1_ref - zc_ref)) > 10 * np.max(np.abs(zc - zc_ref))
    z1 = host(ctx.refresh_prompt(dev_i32(p), [len(p)], dev_i32(g1[None])))[0]
    assert rel_err(z1, z1_ref) < 1e-5


@pytest.mark.parametrize("name", list(SMALL_BF16))
def test_small_bf16_full_and_cached(name):
    m = SMALL_BF16[name]
    say(f"small bf16 model {name}")
    W = with_gains(model_weights(m, seed=4), 4)
    P, G = 100, 64
    p = _prompt(m, P, 5)
    ctx = make_ctx(m, W, 1, P, P, G)
    g0 = _resp(m, G, 6)
    z = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g0[None])))[0]
    z_ref, cache, _ = om.full_forward(W, m, p, g0)
    assert np.max(np.abs(z - z_ref)) < 2e-2
    # CachedForward on its own anchor equals FullForward bitwise on the GPU
    zc0 = host(ctx.step(dev_i32(g0[None])))[0]
    np.testing.assert_array_equal(zc0, z)
    g1 = _resp(m, G, 7, frac=0.6)
    zc = host(ctx.step(dev_i32(g1[None])))[0]
    zc_ref, _ = om.cached_forward(W, m, g1, cache, P)
    assert np.max(np.abs(zc - zc_ref)) < 2e-2


@pytest.mark.parametrize("rows,cols,half", [(1, 32, False), (100, 96, False), (257, 4096, False),
                                            (100, 96, True)])
def test_pack_weight_is_the_k_block_permutation(rows, cols, half):
    a = archer()
    say(f"pack weight {rows}x{cols}{' fp16' if half else ''}")
    w, _ = rand_bf16((rows, cols), 61, rows * 7 + cols)
    if half:
        w = w.to(torch.float16)
    got = a.pack_weight(w)
    # element (r, c) at ((c / 32) * rows + r) * 32 + c % 32
    want = w.view(rows, cols // 32, 32).permute(1, 0, 2).contiguous().view(rows, cols)
    assert torch.equal(got.view(torch.int16), want.view(torch.int16))


@pytest.mark.parametrize("name", ["gqa_hd64", "gqa_hd64_gateup_fp16"])
def test_weight_layouts_give_the_same_bits(name):
    """The k-block and row-major weight layouts feed the same tiles in the same order."""
    a = archer()
    m = SMALL_BF16[name]
    say(f"bf16 model {name}, row-major vs k-block weights")
    W = with_gains(model_weights(m, seed=12), 12)
    P, G = 77, 32
    p = _prompt(m, P, 13)
    g0, g1 = _resp(m, G, 14), _resp(m, G, 15, frac=0.5)
    out = []
    for layout in (a.LAYOUT_ROWMAJOR, a.LAYOUT_KBLOCK):
        ctx = make_ctx(m, W, 1, P, P, G, layout=layout)
        z = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g0[None])))[0]
        zc = host(ctx.step(dev_i32(g1[None])))[0]
        out.append((z, zc))
        ctx.close()
    np.testing.assert_array_equal(out[0][0], out[1][0])
    np.testing.assert_array_equal(out[0][1], out[1][1])


def test_gateup_fp16_full_pass_with_folded_slices():
    """A full pass above the partial-plane row capacity (4608 rows) runs the split-K
    projections with their slices folded in one workgroup, fp16 gate/up included, and
    the stand-alone fp16 RMSNorm before it."""
    m = SMALL_BF16["gqa_hd64_gateup_fp16"]
    say("small bf16 model, fp16 gate/up, P 4700: folded split-K slices in the full pass")
    W = with_gains(model_weights(m, seed=21), 21)
    P, G = 4700, 32
    p = _prompt(m, P, 22)
    ctx = make_ctx(m, W, 1, P, P, G)
    g0 = _resp(m, G, 23)
    z = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g0[None])))[0]
    z_ref, cache, _ = om.full_forward(W, m, p, g0)
    e = np.max(np.abs(z - z_ref))
    say(f"  full pass logits max abs err {e:.3e}")
    assert e < 2e-2
    g1 = _resp(m, G, 24, frac=0.6)
    zc = host(ctx.step(dev_i32(g1[None])))[0]
    zc_ref, _ = om.cached_forward(W, m, g1, cache, P)
    e = np.max(np.abs(zc - zc_ref))
    say(f"  cached pass logits max abs err {e:.3e}")
    assert e < 2e-2


def test_ragged_batch_per_sequence_refresh_and_batch_invariance():
    m = SMALL_BF16["gqa_hd64"]
    say("ragged batch bf16: lengths 37/100/64, per-sequence refresh")
    W = with_gains(model_weights(m, seed=8), 8)
    lens, G = [37, 100, 64], 32
    ps = [_prompt(m, n, 20 + i) for i, n in enumerate(lens)]
    packed = dev_i32(np.concatenate(ps))
    ctx = make_ctx(m, W, 4, 128, 256, G)
    g = [_resp(m, G, 30 + i) for i in range(3)]
    z = host(ctx.refresh_prompt(packed, lens, dev_i32(np.stack(g))))
    caches = []
    for b in range(3):
        zr, cb, _ = om.full_forward(W, m, ps[b], g[b])
        caches.append(cb)
        assert np.max(np.abs(z[b] - zr)) < 2e-2, b
    # batch invariance: sequence 1 alone gives the same bits
    solo = make_ctx(m, W, 1, 128, 128, G)
    z1 = host(solo.refresh_prompt(dev_i32(ps[1]), [lens[1]], dev_i32(g[1][None])))[0]
    np.testing.assert_array_equal(z1, z[1])
    # refresh sequence 1 only; the other rows of the logits stay untouched
    g1n = _resp(m, G, 41, frac=0.7)
    gs = np.stack([g[0], g1n, g[2]])
    logits = torch.full((3, G, m.vocab), 7.0, device="cuda")
    ctx.refresh_prompt(packed, lens, dev_i32(gs), seq_sel=[0, 1, 0], logits=logits)
    lz = host(logits)
    assert np.all(lz[0] == 7.0) and np.all(lz[2] == 7.0)
    zr1, caches[1], _ = om.full_forward(W, m, ps[1], g1n)
    assert np.max(np.abs(lz[1] - zr1)) < 2e-2
    # cached step of everyone: sequences 0 and 2 use their old anchors, 1 its new one
    g2 = [_resp(m, G, 50 + i, frac=0.5) for i in range(3)]
    zc = host(ctx.step(dev_i32(np.stack(g2))))
    for b in range(3):
        zr, _ = om.cached_forward(W, m, g2[b], caches[b], lens[b])
        assert np.max(np.abs(zc[b] - zr)) < 2e-2, b
    # cached step of a subset
    logits.fill_(3.0)
    ctx.step(dev_i32(np.stack(g2)), seq_sel=[1, 0, 1], logits=logits)
    lz = host(logits)
    assert np.all(lz[1] == 3.0)
    np.testing.assert_array_equal(lz[0], zc[0])
    np.testing.assert_array_equal(lz[2], zc[2])


def test_maximum_batch_of_64_with_one_token_prompt():
    """The largest batch the library takes (64 sequences), prompts of 1 to 90 tokens (the
    first sequence's prompt is a single token, whose 64-key cache tile holds one real key):
    FullForward and CachedForward against the oracle for the shortest, a middle and the longest
    sequence, and the one-token sequence alone in a context of the same limits gives the
    same bits."""
    m = SMALL_BF16["gqa_hd64"]
    B, G = 64, 16
    lens = [1 + (b * 37) % 90 for b in range(B)]
    say(f"maximum batch bf16: B {B}, prompts {min(lens)}..{max(lens)} (total {sum(lens)}), G {G}")
    W = with_gains(model_weights(m, seed=9), 9)
    ps = [_prompt(m, n, 300 + b) for b, n in enumerate(lens)]
    ctx = make_ctx(m, W, B, max(lens), sum(lens), G)
    g = [_resp(m, G, 400 + b) for b in range(B)]
    z = host(ctx.refresh_prompt(dev_i32(np.concatenate(ps)), lens, dev_i32(np.stack(g))))
    g2 = [_resp(m, G, 500 + b, frac=0.5) for b in range(B)]
    zc = host(ctx.step(dev_i32(np.stack(g2))))
    for b in (0, B // 2, int(np.argmax(lens))):
        zr, cache, _ = om.full_forward(W, m, ps[b], g[b])
        zcr, _ = om.cached_forward(W, m, g2[b], cache, lens[b])
        e_full, e_cached = np.max(np.abs(z[b] - zr)), np.max(np.abs(zc[b] - zcr))
        say(f"  sequence {b} (P {lens[b]}): full {e_full:.3e}, cached {e_cached:.3e}")
        assert e_full < 2e-2 and e_cached < 2e-2, b
    solo = make_ctx(m, W, B, max(lens), sum(lens), G)
    z0 = host(solo.refresh_prompt(dev_i32(ps[0]), [lens[0]], dev_i32(g[0][None])))[0]
    np.testing.assert_array_equal(z0, z[0])
    z0c = host(solo.step(dev_i32(g2[0][None])))[0]
    np.testing.assert_array_equal(z0c, zc[0])


@pytest.mark.parametrize("gateup_fp16", [True, False])
def test_full_width_two_layer_llada_shape(gateup_fp16):
    """d 4096, 32 heads x 128, F 12288, vocab 126464, P 512, G 256 (two layers); gate/up
    with fp16 operands (the workload's model) and with two-term bf16 ones."""
    w = get_workload("llada_p512")
    m = dataclasses.replace(w.model, n_layers=2, gateup_fp16=gateup_fp16)
    P, G = w.decode.prompt_len, w.decode.resp_len
    say("full-width 2-layer LLaDA shape: generating weights")
    W = model_weights(m, seed=w.weight_seed)
    p = prompts(w)[0]
    ctx = make_ctx(m, W, 1, P, P, G)
    g0 = np.full(G, m.mask_id)
    g0[:40] = np.arange(40) * 7
    z = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g0[None])))[0]
    say("  oracle full forward")
    z_ref, cache, _ = om.full_forward(W, m, p, g0)
    err = float(np.max(np.abs(z - z_ref)))
    say(f"  full forward max abs err {err:.3e} (max |z| {np.max(np.abs(z_ref)):.2f})")
    assert err < 2e-2
    g1 = g0.copy()
    g1[100:140] = np.arange(40) * 11
    zc = host(ctx.step(dev_i32(g1[None])))[0]
    say("  oracle cached forward")
    zc_ref, _ = om.cached_forward(W, m, g1, cache, P)
    err = float(np.max(np.abs(zc - zc_ref)))
    say(f"  cached forward max abs err {err:.3e}")
    assert err < 2e-2


@pytest.mark.parametrize("gateup_fp16", [True, False])
def test_full_width_two_layer_llada_long_prompt(gateup_fp16):
    """d 4096, 32 heads x 128, F 12288, vocab 126464, P 4096, G 256 (two layers); the
    4352-row refresh runs 128 x 256 gate/up tiles, fp16 or two-term."""
    import time
    w = get_workload("llada_p4096")
    m = dataclasses.replace(w.model, n_layers=2, gateup_fp16=gateup_fp16)
    P, G = w.decode.prompt_len, w.decode.resp_len
    say("full-width 2-layer LLaDA shape, P 4096: generating weights")
    W = model_weights(m, seed=w.weight_seed)
    p = prompts(w)[0]
    ctx = make_ctx(m, W, 1, P, P, G)
    g0 = np.full(G, m.mask_id)
    g0[:64] = np.arange(64) * 5
    z = host(ctx.refresh_prompt(dev_i32(p), [P], dev_i32(g0[None])))[0]
    g1 = g0.copy()
    g1[128:192] = np.arange(64) * 13
    zc = host(ctx.step(dev_i32(g1[None])))[0]
    t0 = time.time()
    say("  oracle full forward (4352 rows)")
    z_ref, cache, _ = om.full_forward(W, m, p, g0)
    err = float(np.max(np.abs(z - z_ref)))
    say(f"  full forward max abs err {err:.3e} (max |z| {np.max(np.abs(z_ref)):.2f}, oracle {time.time() - t0:.1f} s)")
    assert err < 2e-2
    zc_ref, _ = om.cached_forward(W, m, g1, cache, P)
    err = float(np.max(np.abs(zc - zc_ref)))
    say(f"  cached forward max abs err {err:.3e}")
    assert err < 2e-2
