"""GPU tests of the resumable decode session, its snapshots and the state reads.

* archer_decode equals the same schedule advanced in pieces (begin, then
  advance 3, 5 and the rest), bitwise: final response and every trace row;
* a snapshot taken mid-decode and restored replays the rest bitwise;
* the matched-state fork (the paper's feedback intervention: one decoder
  state continued with an immediate refresh and with the old cache) on the
  tiny fp32 workload: both branches equal the oracle's decode with the same
  forced forward, step by step;
* ARCHER_READ_LOGITS returns the logits the session decides on (equal to a
  FullForward of the same state on a second context), and the session calls
  refuse wrong states and foreign snapshots;
* the fused decision statistics: archer_decode, whose LM head writes only the
  statistics partials, equals the same schedule driven call by call
  (archer_refresh_prompt / archer_step with logits, archer_decide computing
  the partials from them) bitwise, for 128- and 192-column head tiles.
"""

import numpy as np
import pytest
import torch

from gpu_util import archer, dev_i32, host, make_ctx, say
from oracle import controller as oc
from oracle import decode as odec
from synth.gen import model_weights, prompts
from synth.workloads import ModelShape, get_workload

pytestmark = pytest.mark.gpu

TRACE_KEYS = ("refreshed", "dist", "age", "unmask_pos", "unmask_tok", "remask_pos")


def _tiny():
    w = get_workload("tiny")
    m, dec = w.model, w.decode
    W = model_weights(m, seed=w.weight_seed)
    p = prompts(w)[0]
    return w, m, dec, W, p


def _bf16_batch():
    # vocab 16384: the LM head runs one slice, so sessions use the fused decision statistics
    m = ModelShape(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=16384,
                   dtype="bf16", init_std=0.05)
    W = model_weights(m, seed=31)
    lens = [70, 129, 33]
    rng = np.random.default_rng(32)
    ps = [rng.integers(0, m.vocab - 1, n).astype(np.int32) for n in lens]
    return m, W, lens, ps


def _same_trace(a, b, rows=None):
    for k in TRACE_KEYS:
        x, y = a[k].cpu().numpy(), b[k].cpu().numpy()
        if rows is not None:
            x, y = x[rows], y[rows]
        np.testing.assert_array_equal(x, y, err_msg=k)


@pytest.mark.parametrize("kind", ["tiny_fp32_hamming", "bf16_ragged_age"])
def test_decode_equals_session_advanced_in_pieces(kind):
    a = archer()
    if kind.startswith("tiny"):
        w, m, dec, W, p = _tiny()
        lens, ps, G, T, B = [len(p)], [p], dec.resp_len, dec.steps, 1
        pol, K = a.HAMMING, 3
    else:
        m, W, lens, ps = _bf16_batch()
        G, T, B = 32, 24, 3
        pol, K = a.AGE, 4
    say(f"session in pieces vs archer_decode: {kind}")
    ctx = make_ctx(m, W, B, max(lens), sum(lens), G)
    prompt = dev_i32(np.concatenate(ps))
    g0 = np.full((B, G), m.mask_id, np.int32)
    out, tr = ctx.decode(prompt, lens, dev_i32(g0), policy=pol, K=K, steps=T, k=1, tau=0.1)
    tr2 = ctx.session_begin(prompt, lens, dev_i32(g0), policy=pol, K=K, steps=T, k=1, tau=0.1)
    assert ctx.session_advance(3) == 3
    assert ctx.session_advance(5) == 8
    assert ctx.session_advance(10 * T) == T
    assert ctx.session_advance(1) == T        # the schedule is complete
    out2 = ctx.session_response()
    np.testing.assert_array_equal(out.cpu().numpy(), out2.cpu().numpy())
    _same_trace(tr, tr2)
    ctx.sync()


def test_snapshot_restore_replays_bitwise():
    a = archer()
    m, W, lens, ps = _bf16_batch()
    G, T, B, s = 32, 24, 3, 9
    say("snapshot at decision 9 of 24, restore, replay")
    ctx = make_ctx(m, W, B, max(lens), sum(lens), G)
    prompt = dev_i32(np.concatenate(ps))
    g0 = dev_i32(np.full((B, G), m.mask_id, np.int32))
    tr = ctx.session_begin(prompt, lens, g0, policy=a.AGE, K=4, steps=T, k=2, tau=0.1, keep_logits=True)
    ctx.session_advance(s)
    snap = ctx.session_save()
    z_at_s = ctx.read_logits(B).clone()
    ctx.session_advance(T)
    out1 = ctx.session_response().clone()
    tr1 = {k: v.clone() for k, v in tr.items()}
    for v in tr.values():
        v.fill_(-7)
    ctx.session_restore(snap)
    assert torch.equal(ctx.read_logits(B), z_at_s)
    assert ctx.session_advance(T) == T
    out2 = ctx.session_response()
    assert torch.equal(out1, out2)
    # rows from the snapshot on are rewritten identically (dist row s + 1 onwards, the rest from s)
    _same_trace(tr1, tr, rows=slice(s + 1, None))
    ctx.sync()


def test_matched_state_fork_against_oracle():
    """Branch F refreshes at the forward after the fork, branch C reuses the old cache there."""
    a = archer()
    w, m, dec, W, p = _tiny()
    G, T, k, tau, K, s = dec.resp_len, dec.steps, 1, dec.remask_threshold, 8, 5
    say("matched-state fork on the tiny fp32 workload (age rule K 8, fork after decision 5)")
    ctx = make_ctx(m, W, 1, len(p), len(p), G)
    prompt = dev_i32(p)
    g0 = np.full(G, m.mask_id, np.int32)
    tr = ctx.session_begin(prompt, [len(p)], dev_i32(g0[None]), policy=a.AGE, K=K, steps=T, k=k, tau=tau)
    ctx.session_advance(s)
    snap = ctx.session_save()
    for mode, forced in ((a.FORWARD_REFRESH, True), (a.FORWARD_CACHED, False)):
        ctx.session_restore(snap)
        ctx.session_advance(1, first_forward=mode)
        ctx.session_advance(T)
        out = ctx.session_response().cpu().numpy()[0]
        g_o, tr_o = odec.decode(W, m, p, g0, steps=T, k=k, tau=tau, policy=oc.AGE, K=K, force={s + 1: forced})
        ref = tr["refreshed"].cpu().numpy()[:, 0]
        assert ref.tolist() == [int(x) for x in tr_o.refreshed], mode
        assert tr["age"].cpu().numpy()[:, 0].tolist() == tr_o.age, mode
        assert tr["dist"].cpu().numpy()[:, 0].tolist() == tr_o.dist, mode
        assert out.tolist() == g_o.tolist(), mode
        say(f"  branch {'fresh' if forced else 'cached'}: refreshes at {np.nonzero(ref)[0].tolist()}")


def test_read_logits_and_session_errors():
    a = archer()
    m, W, lens, ps = _bf16_batch()
    G, B = 32, 3
    ctx = make_ctx(m, W, B, max(lens), sum(lens), G)
    other = make_ctx(m, W, B, max(lens), sum(lens), G)
    prompt = dev_i32(np.concatenate(ps))
    g0 = np.full((B, G), m.mask_id, np.int32)
    g0[:, 3] = 17
    with pytest.raises(a.ArcherError) as e:
        ctx.session_advance(1)
    assert e.value.status == a.E_STATE
    ctx.session_begin(prompt, lens, dev_i32(g0), policy=a.AGE, K=4, steps=8)
    with pytest.raises(a.ArcherError) as e:          # this session keeps no logits
        ctx.read_logits(B)
    assert e.value.status == a.E_STATE
    ctx.session_begin(prompt, lens, dev_i32(g0), policy=a.AGE, K=4, steps=8, keep_logits=True)
    z = other.refresh_prompt(prompt, lens, dev_i32(g0))
    assert torch.equal(ctx.read_logits(B), z)
    # hidden / residual rows of the last pass: one FullForward of all three sequences
    assert ctx.read_rows(a.READ_HIDDEN, B).shape == (B * G, m.d_model)
    # a snapshot of a context with other limits is refused
    small = make_ctx(m, W, 1, max(lens), max(lens), G)
    small.session_begin(dev_i32(ps[0]), [lens[0]], dev_i32(g0[:1]), policy=a.AGE, K=4, steps=8)
    snap = small.session_save()
    with pytest.raises(a.ArcherError) as e:
        ctx.session_restore(snap)
    assert e.value.status in (a.E_ARG, a.E_WORKSPACE)
    # a refresh outside the session ends it
    ctx.refresh_prompt(prompt, lens, dev_i32(g0))
    with pytest.raises(a.ArcherError) as e:
        ctx.session_save()
    assert e.value.status == a.E_STATE
    ctx.sync()


@pytest.mark.parametrize("vocab,policy", [(16384, "age"), (18432, "age"), (18432, "hamming"), (65536, "age")])
def test_fused_statistics_decode_equals_call_driven(vocab, policy):
    """The LM head runs one slice (enough column tiles), so its epilogue produces the statistics:
    vocab 16384 in 128-column tiles, 18432 (a multiple of 192) in 192-column tiles, 65536 (256
    tiles of 256 columns) in 256-column tiles."""
    a = archer()
    m = ModelShape(n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512, vocab=vocab,
                   dtype="bf16", init_std=0.05)
    say(f"fused statistics vs call-driven decisions, vocab {vocab}, {policy}")
    W = model_weights(m, seed=33)
    lens, G, T, k, tau, K = [45, 101], 32, 20, 2, 0.1, 3
    rng = np.random.default_rng(34)
    ps = [rng.integers(0, m.vocab - 1, n).astype(np.int32) for n in lens]
    prompt = dev_i32(np.concatenate(ps))
    B = len(lens)
    pol = {"age": a.AGE, "hamming": a.HAMMING}[policy]
    ctx = make_ctx(m, W, B, max(lens), sum(lens), G)
    out, tr = ctx.decode(prompt, lens, dev_i32(np.full((B, G), m.mask_id)), policy=pol, K=K, steps=T, k=k,
                         tau=tau)
    # the fused path ran: the session kept no logits (only contexts with fused statistics may)
    with pytest.raises(a.ArcherError) as e:
        ctx.read_logits(B)
    assert e.value.status == a.E_STATE
    # the same algorithm through the call-level API (stand-alone statistics from stored logits)
    drv = make_ctx(m, W, B, max(lens), sum(lens), G)
    g = dev_i32(np.full((B, G), m.mask_id))
    z = drv.refresh_prompt(prompt, lens, g)
    r = np.zeros(B, dtype=np.int64)
    refreshed = [np.ones(B, dtype=np.int32)]
    for t in range(T):
        final = t == T - 1
        g_next, dist, _, _ = drv.decide(z, g, k=k, tau=tau, final=final)
        if final:
            g = g_next
            break
        s = t + 1
        D = dist.cpu().numpy()
        ref = (D >= K) if policy == "hamming" else (s - r >= K)
        r[ref] = s
        refreshed.append(ref.astype(np.int32))
        if ref.any():
            drv.refresh_prompt(prompt, lens, g_next, seq_sel=ref.tolist(), logits=z)
        if (~ref).any():
            drv.step(g_next, seq_sel=(~ref).tolist(), logits=z)
        g = g_next
    np.testing.assert_array_equal(out.cpu().numpy(), g.cpu().numpy())
    np.testing.assert_array_equal(tr["refreshed"].cpu().numpy(), np.stack(refreshed))
    assert 0 < np.stack(refreshed)[1:].sum() < (T - 1) * B
    ctx.sync()
