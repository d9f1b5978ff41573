"""GPU parity of single kernels (through archer_ops.h) against the oracle.

Small shapes span several tiles with ragged tails; full-size shapes are those
of the LLaDA-8B-shaped cached step and of the long-prompt / GQA attention, in
the same launch configuration the model path uses, checked on sampled rows
the oracle computes one by one.
"""

import numpy as np
import pytest

from gpu_util import archer, host, rand_bf16, rand_f16, rand_f32, say
from oracle import numerics as on

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,N,K", [(1, 64, 64), (37, 192, 320), (128, 128, 256), (300, 64, 1024),
                                   (513, 320, 128)])
def test_gemm_bf16_matches_oracle(M, N, K):
    say(f"gemm bf16 M={M} N={N} K={K}")
    a = archer()
    A, A64 = rand_bf16((M, K), 5, 1)
    W, W64 = rand_bf16((N, K), 5, 2)
    Y = host(a.op_gemm(A, W, a.BF16))
    ref = on.linear(A64, W64)
    # fp32 accumulation of exact bf16 products: error ~ sqrt(K) * 2^-24 * |a||w|
    np.testing.assert_allclose(Y, ref, rtol=0, atol=2e-5 * np.sqrt(K) * 4)


@pytest.mark.parametrize("M,N,K", [(1, 64, 64), (70, 128, 320), (200, 192, 64)])
def test_gemm_f32_matches_oracle(M, N, K):
    say(f"gemm fp32 M={M} N={N} K={K}")
    a = archer()
    A, A64 = rand_f32((M, K), 6, 1)
    W, W64 = rand_f32((N, K), 6, 2)
    Y = host(a.op_gemm(A, W, a.FP32))
    np.testing.assert_allclose(Y, on.linear(A64, W64), rtol=0, atol=1e-4)


@pytest.mark.parametrize("M,N,K", [(37, 192, 320), (256, 512, 4096), (300, 65536, 256), (3900, 4096, 256),
                                   (2600, 4608, 192)])
def test_gemm_two_term_activation_matches_oracle(M, N, K):
    """A = hi + lo (bf16 pair of an fp32 activation) against the unrounded activation; N 65536
    runs the 128 x 256 tiles (enough column tiles), with a ragged last row tile.  3900 x 4096
    (16 column tiles of 256, 31 row tiles) and 2600 x 4608 (24 column tiles of 192, 21 row
    tiles) have few column tiles and many row tiles, so their row tiles are split over 4 and 2
    XCDs per column-tile set, in shares of unequal size."""
    say(f"gemm two-term bf16 M={M} N={N} K={K}")
    a = archer()
    import torch
    from synth.gen import bf16_bits_to_f32, f32_to_bf16_bits, normal_tensor
    A32 = normal_tensor((M, K), 9, 1, 1.0, "fp32")
    hi = f32_to_bf16_bits(A32)
    lo = f32_to_bf16_bits(A32 - bf16_bits_to_f32(hi))
    W, W64 = rand_bf16((N, K), 9, 2)
    dev = lambda u: torch.from_numpy(u.view(np.int16)).view(torch.bfloat16).cuda()  # noqa: E731
    Y = host(a.op_gemm(dev(hi), W, a.BF16, A_lo=dev(lo)))
    ref = on.linear(A32.astype(np.float64), W64)
    # two-term residual ~2^-17 relative per element plus fp32 accumulation
    np.testing.assert_allclose(Y, ref, rtol=0, atol=4e-5 * np.sqrt(K) * 4)


@pytest.mark.parametrize("M,N,K", [(100, 256, 512), (37, 192, 4096)])
def test_gemm_misaligned_output_equals_aligned(M, N, K):
    """Y only 4-byte aligned (a view one float into a buffer): the epilogue's
    element-store fallback gives the same bits as the vector stores, and
    nothing outside Y is written."""
    import ctypes as C

    import torch
    say(f"gemm bf16 misaligned Y M={M} N={N} K={K}")
    a = archer()
    A, _ = rand_bf16((M, K), 11, 1)
    W, _ = rand_bf16((N, K), 11, 2)
    Y = host(a.op_gemm(A, W, a.BF16))
    buf = torch.full((M * N + 2,), 7.0, dtype=torch.float32, device="cuda")
    rc = a.lib.archer_op_gemm(a.BF16, M, N, K, C.c_void_p(A.data_ptr()), None, C.c_void_p(W.data_ptr()),
                              C.c_void_p(buf.data_ptr() + 4), C.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == a.OK
    got = host(buf)
    np.testing.assert_array_equal(got[1:-1].reshape(M, N), Y)
    assert got[0] == 7.0 and got[-1] == 7.0


def test_gemm_deterministic():
    a = archer()
    A, _ = rand_bf16((256, 4096), 7, 1)
    W, _ = rand_bf16((512, 4096), 7, 2)
    Y1 = a.op_gemm(A, W)
    Y2 = a.op_gemm(A, W)
    assert bool((Y1 == Y2).all())


@pytest.mark.parametrize("N,K", [(12288, 4096), (4096, 12288), (126464, 4096)])
def test_gemm_full_size_sampled(N, K):
    """LLaDA-8B-shaped cached-step projections (M = 256 response rows)."""
    say(f"gemm full size M=256 N={N} K={K}")
    a = archer()
    M = 256
    A, A64 = rand_bf16((M, K), 8, 1)
    W, W64 = rand_bf16((N, K), 8, 2, scale=0.02)
    Y = a.op_gemm(A, W)
    rng = np.random.default_rng(0)
    rows = np.sort(rng.choice(M, 12, replace=False))
    cols = np.sort(rng.choice(N, 1024, replace=False))
    got = host(Y[rows][:, cols])
    ref = on.linear(A64[rows], W64[cols])
    np.testing.assert_allclose(got, ref, rtol=0, atol=2e-5 * np.sqrt(K) * 4 * 0.02)


def _attn_case(dtype, Mq, Hq, Hkv, hd, nk1, nk2, seed, rows=None, heads=None, q_scale=1.0):
    a = archer()
    # the bf16 model path stores queries, keys and values as fp16
    rand = rand_f16 if dtype == a.BF16 else rand_f32
    ld1 = (nk1 + 63) // 64 * 64
    ld2 = (nk2 + 63) // 64 * 64
    Q, Q64 = rand((Hq, Mq, hd), seed, 1, q_scale)
    K1, K164 = rand((Hkv, ld1, hd), seed, 2)
    V1, V164 = rand((Hkv, hd, ld1), seed, 3)
    K2, K264 = rand((Hkv, ld2, hd), seed, 4)
    V2, V264 = rand((Hkv, hd, ld2), seed, 5)
    O = host(a.op_attention(Q, K1, V1, nk1, K2, V2, nk2, dtype))
    rows = np.arange(Mq) if rows is None else rows
    heads = range(Hq) if heads is None else heads
    worst = 0.0
    for h in heads:
        kh = h // (Hq // Hkv)
        k = np.concatenate([K164[kh, :nk1], K264[kh, :nk2]])
        v = np.concatenate([V164[kh, :, :nk1].T, V264[kh, :, :nk2].T])
        ref = on.attention(Q64[h, rows], k, v)
        worst = max(worst, float(np.max(np.abs(O[rows, h * hd:(h + 1) * hd] - ref))))
    return worst


@pytest.mark.parametrize("Mq,Hq,Hkv,hd,nk1,nk2", [
    (70, 4, 2, 64, 100, 40),       # GQA, ragged prompt keys, one split
    (256, 2, 2, 128, 513, 256),    # several splits, ragged prompt
    (16, 7, 1, 128, 1024, 512),    # GQA 7:1, many splits, few queries
    (130, 3, 3, 64, 1, 8),         # a single prompt key
])
def test_attention_bf16_matches_oracle(Mq, Hq, Hkv, hd, nk1, nk2):
    say(f"attention bf16 Mq={Mq} Hq={Hq} Hkv={Hkv} hd={hd} nk1={nk1} nk2={nk2}")
    a = archer()
    # fp16 inputs and fp16 probabilities in P V; the op returns the output's bf16 hi term
    # only (the model path also keeps the lo term), so |err| <~ 2^-9 max|o|
    err = _attn_case(a.BF16, Mq, Hq, Hkv, hd, nk1, nk2, 11)
    say(f"  max abs err {err:.3e}")
    assert err < 2e-2


@pytest.mark.parametrize("Mq,Hq,Hkv,nk1,nk2", [(256, 4, 4, 512, 256), (256, 4, 4, 4096, 256)])
def test_attention_bf16_peaked_softmax_accuracy(Mq, Hq, Hkv, nk1, nk2):
    """Scores with standard deviation 4 (a few keys dominate each query)."""
    say(f"attention bf16 peaked softmax Mq={Mq} Hq={Hq} nk1={nk1} nk2={nk2}")
    a = archer()
    err = _attn_case(a.BF16, Mq, Hq, Hkv, 128, nk1, nk2, 14, q_scale=4.0)
    say(f"  max abs err {err:.3e}")
    assert err < 2e-2


@pytest.mark.parametrize("Mq,Hq,Hkv,hd,nk1,nk2", [(33, 4, 2, 64, 100, 40), (8, 2, 1, 128, 300, 64)])
def test_attention_f32_matches_oracle(Mq, Hq, Hkv, hd, nk1, nk2):
    say(f"attention fp32 Mq={Mq} Hq={Hq} Hkv={Hkv} hd={hd} nk1={nk1} nk2={nk2}")
    a = archer()
    assert _attn_case(a.FP32, Mq, Hq, Hkv, hd, nk1, nk2, 12) < 1e-5


@pytest.mark.parametrize("Mq,Hq,Hkv,nk1,nk2", [
    (256, 32, 32, 4096, 256),   # LLaDA-8B-shaped long-prompt cached step
    (256, 32, 32, 512, 256),    # LLaDA-8B-shaped cached step
    (512, 28, 4, 1024, 512),    # Dream-7B-shaped GQA cached step
    (4352, 32, 32, 4096, 256),  # LLaDA-8B-shaped refresh pass at P 4096: enough query tiles, one split
])
def test_attention_full_size_sampled(Mq, Hq, Hkv, nk1, nk2):
    say(f"attention full size Mq={Mq} Hq={Hq} Hkv={Hkv} nk1={nk1} nk2={nk2}")
    a = archer()
    rng = np.random.default_rng(1)
    rows = np.sort(rng.choice(Mq, 24, replace=False))
    heads = sorted(rng.choice(Hq, 4, replace=False).tolist())
    err = _attn_case(a.BF16, Mq, Hq, Hkv, 128, nk1, nk2, 13, rows=rows, heads=heads)
    say(f"  max abs err {err:.3e}")
    assert err < 2e-2
