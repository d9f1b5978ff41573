"""Status codes of the C ABI on the GPU (all checked on the host before any
launch, except token ids, which the device flags and archer_sync reports)."""

import numpy as np
import pytest
import torch

from gpu_util import archer, dev_i32, make_ctx
from synth.gen import model_weights
from synth.workloads import ModelShape

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    m = ModelShape(n_layers=1, d_model=64, n_heads=1, n_kv_heads=1, head_dim=64, d_ff=64, vocab=128,
                   dtype="bf16")
    return m, make_ctx(m, model_weights(m, seed=2), 2, 16, 32, 8)


def test_step_before_refresh_is_a_state_error(ctx):
    m, c = ctx
    a = archer()
    with pytest.raises(a.ArcherError) as e:
        c.step(dev_i32(np.full((1, 8), m.mask_id)))
    assert e.value.status == a.E_STATE


def test_limits_and_arguments(ctx):
    m, c = ctx
    a = archer()
    g = dev_i32(np.full((1, 8), m.mask_id))
    with pytest.raises(a.ArcherError) as e:
        c.refresh_prompt(dev_i32(np.zeros(17, np.int32)), [17], g)          # P > max_prompt_len
    assert e.value.status == a.E_SHAPE
    with pytest.raises(a.ArcherError) as e:
        c.refresh_prompt(dev_i32(np.zeros(48, np.int32)), [16, 16, 16], dev_i32(np.full((3, 8), 0)))
    assert e.value.status == a.E_SHAPE                                       # batch > max_batch
    c.refresh_prompt(dev_i32(np.zeros(16, np.int32)), [8, 8], dev_i32(np.full((2, 8), m.mask_id)))
    with pytest.raises(a.ArcherError) as e:                                   # seq_sel with another batch
        c.refresh_prompt(dev_i32(np.zeros(8, np.int32)), [8], g, seq_sel=[1])
    assert e.value.status == a.E_STATE
    logits = torch.zeros(2, 8, m.vocab, device="cuda")
    gi = dev_i32(np.full((2, 8), m.mask_id))
    with pytest.raises(a.ArcherError) as e:
        a._check(a.lib.archer_decide(c.h, a._ptr(logits), a._ptr(gi), a._ptr(gi),
                                     a.C.byref(a.DecideCfg(1, 0.1, 1, 0)), None, None, None))
    assert e.value.status == a.E_ARG                                          # g_out aliases g_in
    with pytest.raises(a.ArcherError) as e:
        c.decide(logits, gi, k=1, tau=1.5)
    assert e.value.status == a.E_ARG


def test_bad_token_ids_are_flagged(ctx):
    m, c = ctx
    a = archer()
    p = np.zeros(8, np.int32)
    p[3] = m.mask_id                                                          # MASK inside the prompt
    c.refresh_prompt(dev_i32(p), [8], dev_i32(np.full((1, 8), m.mask_id)))
    with pytest.raises(a.ArcherError) as e:
        c.sync()
    assert e.value.status == a.E_ARG
    c.sync()                                                                  # flag cleared
    g = np.full((1, 8), m.mask_id)
    g[0, 2] = 10 ** 6                                                         # out of the vocabulary
    c.refresh_prompt(dev_i32(np.zeros(8, np.int32)), [8], dev_i32(g))
    with pytest.raises(a.ArcherError) as e:
        c.sync()
    assert e.value.status == a.E_ARG


def test_timing_stride(ctx):
    """archer_timing_begin records the 1st, (every+1)-th, ... launch of each class."""
    m, c = ctx
    a = archer()
    with pytest.raises(a.ArcherError) as e:
        c.timing_begin([a.K_GEMM_QKV], every=0)
    assert e.value.status == a.E_ARG
    p = dev_i32(np.arange(10) % (m.vocab - 1))
    g = dev_i32(np.full((1, 8), m.mask_id))
    c.refresh_prompt(p, [10], g)
    for every, want in ((1, 7), (3, 3), (7, 1)):
        # 7 forwards of a 1-layer model: 7 QKV GEMMs and 7 LM heads
        c.timing_begin([a.K_GEMM_QKV, a.K_GEMM_HEAD], every=every)
        for _ in range(7):
            c.step(g)
        t = c.timing_end()
        for k in ("gemm_qkv", "gemm_head"):
            assert t[k]["launches"] == want, (every, k, t[k])
            assert t[k]["ms"] > 0 and t[k]["flops"] > 0
        assert t["attn"]["launches"] == 0


def test_gateup_fp16_option_errors():
    """A model with fp16 gate/up operands takes fp16 w_gate / w_up (the binding refuses
    bf16 ones) and refuses a single-term request for gate/up (its operands are single
    fp16 values already); other classes still switch."""
    import dataclasses
    a = archer()
    m = ModelShape(n_layers=1, d_model=64, n_heads=1, n_kv_heads=1, head_dim=64, d_ff=64, vocab=128,
                   dtype="bf16", gateup_fp16=True)
    W = model_weights(m, seed=3)
    with pytest.raises(a.ArcherError) as e:
        a.Context(m, a.upload_weights(W, "bf16"), 1, 16, 16, 8)   # bf16 gate/up weights
    assert e.value.status == a.E_ARG
    c = make_ctx(m, W, 1, 16, 16, 8)
    with pytest.raises(a.ArcherError) as e:
        c.set_single_term(["gateup"])
    assert e.value.status == a.E_UNSUPPORTED
    c.set_single_term(["o"])
    c.set_single_term([])
    # the same shape without the option accepts a single-term gate/up
    m2 = dataclasses.replace(m, gateup_fp16=False)
    c2 = make_ctx(m2, W, 1, 16, 16, 8)
    c2.set_single_term(["gateup"])
