"""archer_op_attention_noalloc (split-KV partials in the library's fixed scratch
array) against archer_op_attention (partials in a caller workspace): the same
kernels and launch configuration, so the outputs must be bitwise equal.  Two
calls in a row, the second with a smaller input, so that the second reads
nothing the first left in the shared array; and a shape whose partials exceed
the array is refused on the host before any launch."""

import numpy as np
import pytest
import torch

from gpu_util import archer, rand_f16, say

pytestmark = pytest.mark.gpu

CASES = [
    (256, 32, 32, 128, 4096, 256),   # the LLaDA-8B-shaped long-prompt cached pass: 4 splits, 17 MB of partials
    (64, 8, 2, 64, 700, 40),         # smaller: GQA 4:1, 2 splits
]


def _inputs(Mq, Hq, Hkv, hd, nk1, nk2, seed):
    ld1 = (nk1 + 63) // 64 * 64
    ld2 = (nk2 + 63) // 64 * 64
    Q, _ = rand_f16((Hq, Mq, hd), seed, 1)
    K1, _ = rand_f16((Hkv, ld1, hd), seed, 2)
    V1, _ = rand_f16((Hkv, hd, ld1), seed, 3)
    K2, _ = rand_f16((Hkv, ld2, hd), seed, 4)
    V2, _ = rand_f16((Hkv, hd, ld2), seed, 5)
    return Q, K1, V1, nk1, K2, V2, nk2


def test_noalloc_attention_equals_the_workspace_call():
    a = archer()
    for i, (Mq, Hq, Hkv, hd, nk1, nk2) in enumerate(CASES):
        say(f"noalloc attention Mq={Mq} Hq={Hq} Hkv={Hkv} hd={hd} nk1={nk1} nk2={nk2}")
        args = _inputs(Mq, Hq, Hkv, hd, nk1, nk2, 40 + i)
        ref = a.op_attention(*args)
        got = a.op_attention_noalloc(*args)
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), (Mq, Hq, nk1)
        assert torch.isfinite(got.float()).all()


def test_noalloc_attention_refuses_shapes_beyond_the_scratch():
    a = archer()
    # 5 query tiles x 32 heads still split: 4 x 32 x 1280 x 128 fp32 partials = 84 MB > 64 MiB
    args = _inputs(1280, 32, 32, 128, 4096, 256, 50)
    with pytest.raises(a.ArcherError) as e:
        a.op_attention_noalloc(*args)
    assert e.value.status == a.E_SHAPE
    assert "scratch" in str(e.value)
