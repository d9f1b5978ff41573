// Projection GEMMs Y = A W^T of the Archer path with fused epilogues.
//
// bf16: LDS-tiled MFMA kernel (v_mfma_f32_16x16x32_bf16, fp32 accumulate),
//       256 threads = 4 wave64s stacked along M, BK = 64, double-buffered LDS.
// fp32: FMA kernel with a 64x64 tile (tiny fp32 model and fp32 checks).
//
// Column pairing.  Two epilogues need two output columns of the same row in
// one thread: RoPE rotates dimension j with j + hd/2 of a head, and SwiGLU
// multiplies gate feature f with up feature f.  The B tile rows (weight rows)
// are gathered so that tile column r and r + BN/2 form such a pair:
//   QKV (q and k heads): columns {h*hd + j0 + c} and {h*hd + hd/2 + j0 + c},
//                        c < BN/2, j0 = (tile offset within the head) * BN/2;
//   SWIGLU:              gate rows f0 + c and up rows f0 + c, f0 = tile * BN/2.
#include "launch.h"

template <int EPI, int BN>
__device__ __forceinline__ int64_t brow_index(const GemmArgs& a, int tile_n, int r, bool* second) {
  *second = false;
  if constexpr (EPI == EPI_SWIGLU) {
    const int f0 = tile_n * (BN / 2);
    if (r < BN / 2) return f0 + r;
    *second = true;
    return f0 + r - BN / 2;
  } else if constexpr (EPI == EPI_QKV) {
    const int col0 = tile_n * BN;
    if (col0 < (a.hq + a.hkv) * a.hd) {
      const int base = (col0 / a.hd) * a.hd;
      const int j0 = ((col0 % a.hd) / BN) * (BN / 2);
      return r < BN / 2 ? base + j0 + r : base + a.hd / 2 + j0 + (r - BN / 2);
    }
    return col0 + r;
  } else {
    return (int64_t)tile_n * BN + r;
  }
}

template <int EPI, class T, int BN>
__device__ __forceinline__ void epi_pair(const GemmArgs& a, int tile_n, int r, int row, float v1, float v2) {
  if constexpr (EPI == EPI_SWIGLU) {
    const int f = tile_n * (BN / 2) + r;
    const float s = v1 / (1.0f + expf(-v1));
    store_act<T>((T*)a.H, (T*)a.H2, (size_t)row * a.ldh + f, s * v2);
  } else if constexpr (EPI == EPI_QKV) {
    const int col0 = tile_n * BN;
    const int hd = a.hd;
    const int qk_end = (a.hq + a.hkv) * hd;
    const int dst = a.row_dst[row];
    if (col0 < qk_end) {
      const int head = col0 / hd;
      const int j = ((col0 % hd) / BN) * (BN / 2) + r;
      const float2 cs = a.rope[(size_t)a.row_pos[row] * (hd / 2) + j];
      const float o1 = v1 * cs.x - v2 * cs.y;
      const float o2 = v2 * cs.x + v1 * cs.y;
      T* p;
      if (head < a.hq) {
        p = (T*)a.Qb + ((size_t)head * a.ldq + row) * hd;
      } else if (dst_is_fresh(dst)) {
        p = (T*)a.Kf + ((size_t)(head - a.hq) * a.ldfresh + dst) * hd;
      } else {
        p = (T*)a.Kc + ((size_t)(head - a.hq) * a.ldcache + dst_cache_row(dst)) * hd;
      }
      p[j] = from_f32<T>(o1);
      p[j + hd / 2] = from_f32<T>(o2);
    } else {
      const int c1 = col0 - qk_end + r, c2 = c1 + BN / 2;
      T* vt;
      int ld, col;
      if (dst_is_fresh(dst)) { vt = (T*)a.Vtf; ld = a.ldfresh; col = dst; }
      else { vt = (T*)a.Vtc; ld = a.ldcache; col = dst_cache_row(dst); }
      vt[(size_t)c1 * ld + col] = from_f32<T>(v1);   // (vh*hd + d) == c
      vt[(size_t)c2 * ld + col] = from_f32<T>(v2);
    }
  }
}

template <int EPI>
__device__ __forceinline__ void epi_single(const GemmArgs& a, int row, int col, float v) {
  if constexpr (EPI == EPI_STORE) {
    const int orow = a.out_row ? a.out_row[row] : row;
    a.C[(size_t)orow * a.ldc + col] = v;
  } else if constexpr (EPI == EPI_RESID) {
    a.X[(size_t)row * a.ldx + col] += v;
  }
}

constexpr bool epi_paired(int epi) { return epi == EPI_SWIGLU || epi == EPI_QKV; }

// ---------------------------------------------------------------------------
// SPLIT: A is the two-term activation (A = hi, A2 = lo); every fragment
// product is issued twice, hi x W and lo x W, into the same fp32 accumulator.
template <int BM, int BN, int EPI, bool SPLIT>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int BK = 64, LDK = BK + 8;
  constexpr int WM = BM / 4;
  constexpr int RB = WM / 16, CB = BN / 16;
  constexpr int A_CH = BM * BK / 8 / 256;
  constexpr int B_CH = BN * BK / 8 / 256;
  constexpr int NA = SPLIT ? 2 : 1;
  static_assert(A_CH >= 1 && B_CH >= 1, "tile too small for 256 threads");
  __shared__ __attribute__((aligned(16))) bf16 As[2][NA][BM * LDK];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * LDK];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int tile_n = blockIdx.x, m0 = blockIdx.y * BM;
  const bf16* Ap[2] = {(const bf16*)a.A, (const bf16*)(SPLIT ? a.A2 : a.A)};

  size_t aoffg[A_CH];
  bool aval[A_CH];
  int aoff[A_CH];
#pragma unroll
  for (int j = 0; j < A_CH; ++j) {
    const int c = tid + 256 * j, r = c >> 3, kc = (c & 7) * 8;
    const int row = m0 + r;
    aval[j] = row < a.M;
    aoffg[j] = (size_t)(aval[j] ? row : 0) * a.lda + kc;
    aoff[j] = r * LDK + kc;
  }
  const bf16* bsrc[B_CH];
  int boff[B_CH];
#pragma unroll
  for (int j = 0; j < B_CH; ++j) {
    const int c = tid + 256 * j, r = c >> 3, kc = (c & 7) * 8;
    bool second;
    const int64_t wr = brow_index<EPI, BN>(a, tile_n, r, &second);
    const bf16* base = (const bf16*)(second ? a.W2 : a.W);
    bsrc[j] = base + wr * a.ldw + kc;
    boff[j] = r * LDK + kc;
  }

  uint4 ra[NA][A_CH], rbv[B_CH];
  f32x4 acc[RB][CB];
#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int j = 0; j < CB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto gload = [&](int k0) {
#pragma unroll
    for (int t = 0; t < NA; ++t)
#pragma unroll
      for (int j = 0; j < A_CH; ++j)
        ra[t][j] = aval[j] ? *(const uint4*)(Ap[t] + aoffg[j] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int j = 0; j < B_CH; ++j) rbv[j] = *(const uint4*)(bsrc[j] + k0);
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int t = 0; t < NA; ++t)
#pragma unroll
      for (int j = 0; j < A_CH; ++j) *(uint4*)&As[buf][t][aoff[j]] = ra[t][j];
#pragma unroll
    for (int j = 0; j < B_CH; ++j) *(uint4*)&Bs[buf][boff[j]] = rbv[j];
  };

  const int nk = a.K / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 bfr[CB];
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        bfr[cb] = *(const bf16x8*)&Bs[cur][(cb * 16 + (lane & 15)) * LDK + ks * 32 + (lane >> 4) * 8];
#pragma unroll
      for (int t = 0; t < NA; ++t) {
        bf16x8 af[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          af[rb] = *(const bf16x8*)&As[cur][t][(w * WM + rb * 16 + (lane & 15)) * LDK + ks * 32 + (lane >> 4) * 8];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int cb = 0; cb < CB; ++cb)
            acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[rb], bfr[cb], acc[rb][cb], 0, 0, 0);
      }
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // accumulator (rb, cb)[i] holds row 16*rb + 4*(lane/16) + i, column 16*cb + lane%16
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = m0 + w * WM + rb * 16 + (lane >> 4) * 4 + i;
      if (row >= a.M) continue;
      if constexpr (epi_paired(EPI)) {
#pragma unroll
        for (int cb = 0; cb < CB / 2; ++cb)
          epi_pair<EPI, bf16, BN>(a, tile_n, cb * 16 + (lane & 15), row, acc[rb][cb][i], acc[rb][cb + CB / 2][i]);
      } else {
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
          epi_single<EPI>(a, row, tile_n * BN + cb * 16 + (lane & 15), acc[rb][cb][i]);
      }
    }
  }
}

template <int BM, int BN, int EPI>
static void run_bf16(const GemmArgs& a, hipStream_t st) {
  dim3 grid(a.N / BN, (a.M + BM - 1) / BM);
  if (a.A2) gemm_bf16_kernel<BM, BN, EPI, true><<<grid, 256, 0, st>>>(a);
  else gemm_bf16_kernel<BM, BN, EPI, false><<<grid, 256, 0, st>>>(a);
}

int launch_gemm_bf16(int epi, const GemmArgs& a, hipStream_t st) {
  constexpr int BM = 128, BN = 64;
  if (a.M <= 0 || a.N % BN || a.K % 64) return 1;
  if (epi == EPI_QKV && (a.hd % BN)) return 1;
  switch (epi) {
    case EPI_STORE: run_bf16<BM, BN, EPI_STORE>(a, st); break;
    case EPI_RESID: run_bf16<BM, BN, EPI_RESID>(a, st); break;
    case EPI_SWIGLU: run_bf16<BM, BN, EPI_SWIGLU>(a, st); break;
    case EPI_QKV: run_bf16<BM, BN, EPI_QKV>(a, st); break;
    default: return 1;
  }
  return 0;
}

// ---------------------------------------------------------------------------
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BM][BK + 1];
  __shared__ float Bs[BN][BK + 1];
  const int tid = threadIdx.x, tx = tid & 31, ty = tid >> 5;
  const int tile_n = blockIdx.x, m0 = blockIdx.y * BM;
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  const float* A = (const float*)a.A;
  const int arow = m0 + lr;
  const bool aval = arow < a.M;
  const float* asrc = A + (size_t)(aval ? arow : 0) * a.lda + lk;
  bool second;
  const int64_t wr = brow_index<EPI, BN>(a, tile_n, lr, &second);
  const float* bsrc = (const float*)(second ? a.W2 : a.W) + wr * a.ldw + lk;
  float acc0[8], acc1[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) { acc0[i] = 0.f; acc1[i] = 0.f; }
  for (int k0 = 0; k0 < a.K; k0 += BK) {
    const float4 av = aval ? *(const float4*)(asrc + k0) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 bv = *(const float4*)(bsrc + k0);
    As[lr][lk + 0] = av.x; As[lr][lk + 1] = av.y; As[lr][lk + 2] = av.z; As[lr][lk + 3] = av.w;
    Bs[lr][lk + 0] = bv.x; Bs[lr][lk + 1] = bv.y; Bs[lr][lk + 2] = bv.z; Bs[lr][lk + 3] = bv.w;
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      const float b0 = Bs[tx][kk], b1 = Bs[tx + 32][kk];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float av2 = As[ty + 8 * i][kk];
        acc0[i] = fmaf(av2, b0, acc0[i]);
        acc1[i] = fmaf(av2, b1, acc1[i]);
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = m0 + ty + 8 * i;
    if (row >= a.M) continue;
    if constexpr (epi_paired(EPI)) {
      epi_pair<EPI, float, BN>(a, tile_n, tx, row, acc0[i], acc1[i]);
    } else {
      epi_single<EPI>(a, row, tile_n * BN + tx, acc0[i]);
      epi_single<EPI>(a, row, tile_n * BN + tx + 32, acc1[i]);
    }
  }
}

int launch_gemm_f32(int epi, const GemmArgs& a, hipStream_t st) {
  constexpr int BM = 64, BN = 64;
  if (a.M <= 0 || a.N % BN || a.K % 16) return 1;
  if (epi == EPI_QKV && (a.hd % BN)) return 1;
  dim3 grid(a.N / BN, (a.M + BM - 1) / BM);
  switch (epi) {
    case EPI_STORE: gemm_f32_kernel<EPI_STORE><<<grid, 256, 0, st>>>(a); break;
    case EPI_RESID: gemm_f32_kernel<EPI_RESID><<<grid, 256, 0, st>>>(a); break;
    case EPI_SWIGLU: gemm_f32_kernel<EPI_SWIGLU><<<grid, 256, 0, st>>>(a); break;
    case EPI_QKV: gemm_f32_kernel<EPI_QKV><<<grid, 256, 0, st>>>(a); break;
    default: return 1;
  }
  return 0;
}
