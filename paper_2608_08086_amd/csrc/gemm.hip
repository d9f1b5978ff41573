// Projection GEMMs Y = A W^T of the Archer path with fused epilogues.
//
// bf16 kernel: LDS-tiled MFMA (v_mfma_f32_16x16x32_bf16, fp32 accumulate),
// 256 threads = 4 wave64s in a WGM x WGN grid, double-buffered LDS tiles in
// an XOR-swizzled layout (16-byte chunk c of row r is stored at chunk
// c ^ (r mod chunks-per-row): conflict-free fragment reads, no padding), and a
// one-tile-ahead register prefetch of the global loads.
//
// Split-K.  The K range of a GEMM is cut into S slices, S chosen from (N, K)
// only.  A launch either gives each slice its own workgroup, which writes an
// fp32 partial, and a second kernel sums the partials in slice order and
// applies the epilogue; or runs all slices in one workgroup, accumulating each
// slice from zero and adding the slice sums in the same order.  Both give the
// same bits, so a row's result never depends on how many rows are in the
// launch (CachedForward on its own cache equals FullForward bitwise).
//
// Column pairing (gemm_common.h): tile column r and r + BN/2 are an RoPE or
// SwiGLU pair, and each wave's columns are taken from both halves of the tile
// so that a pair sits in one lane.
//
// Tile order (tile_of in gemm_common.h).  Workgroups are dispatched
// round-robin over the 8 XCDs; each XCD owns every eighth (N tile, slice)
// group (or, for passes with few groups and many M tiles, every second or
// fourth group and a share of the M tiles) and walks blocks of its groups
// times its M tiles, so that the tiles it runs at once share both operands
// through its L2 (with 8 slices each XCD owns one K slice, whose part of A
// stays in its L2).
#include <algorithm>

#include "launch.h"

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

#include "gemm_common.h"


int gemm_grid_size(int n_tiles, int m_tiles, int S) {
  // 8 XCDs times the most workgroups tile_of gives one XCD
  const int groups = n_tiles * S, py = tile_py(groups, m_tiles), px = 8 / py;
  return 8 * ((groups + px - 1) / px) * ((m_tiles + py - 1) / py);
}

#define GEMM_GLOAD(slot, k0)                                                             \
  do {                                                                                   \
    _Pragma("unroll") for (int t = 0; t < NA; ++t)                                       \
      _Pragma("unroll") for (int j = 0; j < A_CH; ++j)                                   \
        RA##slot[t][j] = *(const u32x4*)(Ap[t] + aoffg[j] + (size_t)(k0) * akmul);      \
    _Pragma("unroll") for (int j = 0; j < B_CH; ++j) RB##slot[j] = *(const u32x4*)(bsrc[j] + (size_t)(k0) * wkmul); \
  } while (0)
#define GEMM_SSTORE(slot, buf)                                                           \
  do {                                                                                   \
    _Pragma("unroll") for (int t = 0; t < NA; ++t)                                       \
      _Pragma("unroll") for (int j = 0; j < A_CH; ++j) *(u32x4*)&As[buf][t][aoff[j]] = RA##slot[t][j]; \
    _Pragma("unroll") for (int j = 0; j < B_CH; ++j) *(u32x4*)&Bs[buf][boff[j]] = RB##slot[j]; \
  } while (0)
#define GEMM_COMPUTE(cur)                                                                \
  do {                                                                                   \
    _Pragma("unroll") for (int ks = 0; ks < BK / 32; ++ks) {                             \
      const int ch = ks * 4 + lg;                                                        \
      bf16x8 bfr[CB];                                                                    \
      _Pragma("unroll") for (int cb = 0; cb < CB; ++cb)                                  \
        bfr[cb] = *(const bf16x8*)&Bs[cur][tc[cb] * BK + ((ch ^ (tc[cb] % CPR)) * 8)];  \
      _Pragma("unroll") for (int t = 0; t < NA; ++t) {                                   \
        bf16x8 af[RB];                                                                   \
        _Pragma("unroll") for (int rb = 0; rb < RB; ++rb) {                              \
          const int r_ = wm * WM + rb * 16 + lc;                                         \
          af[rb] = *(const bf16x8*)&As[cur][t][r_ * BK + ((ch ^ (r_ % CPR)) * 8)];       \
        }                                                                                \
        _Pragma("unroll") for (int rb = 0; rb < RB; ++rb)                                \
          _Pragma("unroll") for (int cb = 0; cb < CB; ++cb)                              \
            acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[rb], bfr[cb], acc[rb][cb], 0, 0, 0); \
      }                                                                                  \
    }                                                                                    \
  } while (0)

// ---------------------------------------------------------------------------
// SPLIT: A is the two-term activation (A = hi, A2 = lo); every fragment
// product is issued twice, hi x W and lo x W, into the same accumulator.
// MODE 0: one workgroup covers all of K in one accumulation (ksplit == 1).
// MODE 1: one workgroup covers all ksplit slices, each accumulated from zero
//         and added to the running total in slice order.
// MODE 2: one workgroup per slice, writing an fp32 partial.
template <int BM, int BN, int BK, int WGM, int WGN, int EPI, bool SPLIT, int MODE>
__global__ __launch_bounds__(256, 1) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int RB = WM / 16, CB = WN / 16;
  constexpr int CPR = BK / 8;                       // 16-byte chunks per tile row
  constexpr int A_CH = BM * CPR / 256, B_CH = BN * CPR / 256;
  constexpr int NA = SPLIT ? 2 : 1;
  constexpr bool PARTIAL = MODE == 2, FOLD = MODE == 1;
  static_assert(WGM * WGN == 4 && A_CH >= 1 && B_CH >= 1 && CB % 2 == 0 && RB >= 1, "bad tile");
  static_assert(BN % (32 * WGN) == 0, "each wave takes 16-column blocks from both tile halves");
  __shared__ __attribute__((aligned(16))) bf16 As[2][NA][BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * BK];

  const int n_tiles = a.N / BN, m_tiles = (a.M + BM - 1) / BM;
  int tile_n, tile_m, z;
  if (!tile_of(blockIdx.x, n_tiles, m_tiles, PARTIAL ? a.ksplit : 1, &tile_n, &tile_m, &z)) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int wm = w / WGN, wn = w % WGN;
  const int m0 = tile_m * BM;
  const int kslice = a.K / a.ksplit;
  const int kbeg = PARTIAL ? z * kslice : 0;
  const int nslices = FOLD ? a.ksplit : 1;
  const int kt_slice = (PARTIAL || FOLD ? kslice : a.K) / BK;   // k tiles per accumulation
  const bf16* Ap[2] = {(const bf16*)a.A, (const bf16*)(SPLIT ? a.A2 : a.A)};
  const int akmul = a.a_tiled ? a.lda : 1, wkmul = a.w_tiled ? a.ldw : 1;

  // rows past M load row M-1 (finite data; those output rows are never stored)
  uint32_t aoffg[A_CH], aoff[A_CH];
#pragma unroll
  for (int j = 0; j < A_CH; ++j) {
    const int c = tid + 256 * j, r = c / CPR, kc = c % CPR;
    const int row = min(m0 + r, a.M - 1);
    // k0 (a multiple of 32) contributes k0 * akmul elements
    aoffg[j] = a.a_tiled ? (uint32_t)((kc / 4) * a.lda * 32 + row * 32 + (kc % 4) * 8) : (uint32_t)row * a.lda + kc * 8;
    aoff[j] = r * BK + ((kc ^ (r % CPR)) * 8);
  }
  const bf16* bsrc[B_CH];
  uint32_t boff[B_CH];
#pragma unroll
  for (int j = 0; j < B_CH; ++j) {
    const int c = tid + 256 * j, r = c / CPR, kc = c % CPR;
    bool second;
    const int wr = brow_index<EPI, BN>(a, tile_n, r, &second);
    bsrc[j] = (const bf16*)(second ? a.W2 : a.W) +
              (a.w_tiled ? (size_t)(kc / 4) * a.ldw * 32 + (size_t)wr * 32 + (kc % 4) * 8 : (size_t)wr * a.ldw + kc * 8);
    boff[j] = r * BK + ((kc ^ (r % CPR)) * 8);
  }
  // tile column of accumulator block cb: blocks 0..CB/2-1 from the first tile
  // half, CB/2..CB-1 the partner columns from the second half
  int tc[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) tc[cb] = (cb / (CB / 2)) * (BN / 2) + wn * (WN / 2) + (cb % (CB / 2)) * 16 + lc;

  u32x4 RA0[NA][A_CH], RB0[B_CH], RA1[NA][A_CH], RB1[B_CH];   // two tiles of prefetch in flight
  f32x4 acc[RB][CB];
  f32x4 tot[FOLD ? RB : 1][FOLD ? CB : 1];
  if constexpr (FOLD) {
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int j = 0; j < CB; ++j) tot[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Pipeline: LDS buffer b holds tile g (b = g & 1), register slot (g + 1) & 1
  // holds tile g + 1 in flight; iteration g issues tile g + 2 into slot g & 1,
  // computes tile g, then moves tile g + 1 from its slot into LDS buffer b ^ 1.
  // Tile indices past the last tile are clamped (a redundant load whose LDS
  // copy is never read).  Tiles per accumulation are even (host-checked), so
  // the parity of g is static in the two unrolled halves.
  const int ntot = nslices * kt_slice;
#define kof(g) (kbeg + min((g), ntot - 1) * BK)
  GEMM_GLOAD(0, kof(0));
  GEMM_GLOAD(1, kof(1));
  GEMM_SSTORE(0, 0);
  __syncthreads();
  for (int sl = 0; sl < nslices; ++sl) {
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int j = 0; j < CB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int kt = 0; kt < kt_slice; kt += 2) {
      const int g = sl * kt_slice + kt;             // even
      GEMM_GLOAD(0, kof(g + 2));
      GEMM_COMPUTE(0);
      GEMM_SSTORE(1, 1);
      __syncthreads();
      GEMM_GLOAD(1, kof(g + 3));
      GEMM_COMPUTE(1);
      GEMM_SSTORE(0, 0);
      __syncthreads();
    }
    if constexpr (FOLD) {
#pragma unroll
      for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < CB; ++j) tot[i][j] += acc[i][j];
    }
  }

  // accumulator (rb, cb)[i]: row wm*WM + 16*rb + 4*lg + i, tile column tc[cb]
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = m0 + wm * WM + rb * 16 + lg * 4 + i;
      if (row >= a.M) continue;
      if constexpr (PARTIAL) {
        float* pr = a.part + ((size_t)z * a.M + row) * a.N;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) pr[logical_col<EPI, BN>(a, tile_n, tc[cb])] = acc[rb][cb][i];
      } else if constexpr (epi_paired(EPI)) {
#pragma unroll
        for (int cb = 0; cb < CB / 2; ++cb) epi_tile_pair<EPI, bf16, BN>(a, tile_n, tc[cb], row, FOLD ? tot[rb % (FOLD ? RB : 1)][cb % (FOLD ? CB : 1)][i] : acc[rb][cb][i],
                                         FOLD ? tot[rb % (FOLD ? RB : 1)][(cb + CB / 2) % (FOLD ? CB : 1)][i] : acc[rb][cb + CB / 2][i]);
      } else {
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
          const int col = tile_n * BN + tc[cb];
          const float v = FOLD ? tot[rb % (FOLD ? RB : 1)][cb % (FOLD ? CB : 1)][i] : acc[rb][cb][i];
          if constexpr (EPI == EPI_STORE) epi_store(a, row, col, v);
          else epi_resid(a, row, col, v);
        }
      }
    }
  }
}

// Sum of the S partials in slice order, then the epilogue.  One thread per
// (row, logical pair) for SWIGLU, per (row, column) otherwise.
template <int EPI, class T>
__global__ __launch_bounds__(256) void gemm_reduce_kernel(GemmArgs a) {
  static_assert(EPI != EPI_QKV, "QKV partials are reduced by gemm_reduce_qkv_kernel");
  const int npair = epi_paired(EPI) ? a.N / 2 : a.N;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)a.M * npair) return;
  const int row = (int)(idx / npair), p = (int)(idx % npair);
  const size_t plane = (size_t)a.M * a.N;
  const float* pr = a.part + (size_t)row * a.N;
  if constexpr (EPI == EPI_SWIGLU) {
    const int F = a.N / 2;
    float g = pr[p], u = pr[F + p];
    for (int s = 1; s < a.ksplit; ++s) { g += pr[s * plane + p]; u += pr[s * plane + F + p]; }
    epi_swiglu<T>(a, row, p, g, u);
  } else {
    float v = pr[p];
    for (int s = 1; s < a.ksplit; ++s) v += pr[s * plane + p];
    if constexpr (EPI == EPI_STORE) epi_store(a, row, p, v);
    else epi_resid(a, row, p, v);
  }
}

// Split-K reduction of an EPI_RESID GEMM fused with the RMSNorm of the
// updated rows: one block of NORM_THREADS per row; thread t owns the float4
// chunks t, t + NORM_THREADS, ... (KC of them, N <= 4 * KC * NORM_THREADS) as
// in rms_normalize_row, adds the slices in slice order into X (as
// gemm_reduce_kernel does) and normalises the row from the values it keeps in
// registers, with the same expressions in the same order as
// rms_normalize_row (same bits as the stand-alone kernel).
template <class T, int KC>
__global__ __launch_bounds__(NORM_THREADS) void gemm_reduce_resid_norm_kernel(GemmArgs a) {
  constexpr int GRP = KC < 4 ? KC : 4;   // chunks whose slices are requested together
  __shared__ float red[16];
  const int row = blockIdx.x;
  const size_t plane = (size_t)a.M * a.N;
  const float* pr = a.part + (size_t)row * a.N;
  float* xr = a.X + (size_t)row * a.ldx;
  const int step = NORM_THREADS * 4;
  f32x4 xv[KC];
  float4 gv[KC];
#pragma unroll
  for (int k = 0; k < KC; ++k) {
    const int c = threadIdx.x * 4 + k * step;
    if (c < a.N) gv[k] = *(const float4*)(a.ngain + c);
  }
#pragma unroll
  for (int g = 0; g < KC; g += GRP) {
    f32x4 sl[GRP][8];
#pragma unroll
    for (int u = 0; u < GRP; ++u) {
      const int c = threadIdx.x * 4 + (g + u) * step;
      if (c < a.N) {
        xv[g + u] = *(const f32x4*)(xr + c);
#pragma unroll
        for (int s = 0; s < 8; ++s)
          if (s < a.ksplit) sl[u][s] = *(const f32x4*)(pr + s * plane + c);
      }
    }
#pragma unroll
    for (int u = 0; u < GRP; ++u) {
      const int c = threadIdx.x * 4 + (g + u) * step;
      if (c < a.N) {
        f32x4 v = sl[u][0];
#pragma unroll
        for (int s = 1; s < 8; ++s)
          if (s < a.ksplit) v += sl[u][s];
        xv[g + u] += v;
        *(f32x4*)(xr + c) = xv[g + u];
      }
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < KC; ++k) {
    const int c = threadIdx.x * 4 + k * step;
    if (c < a.N) {
      const f32x4 v = xv[k];
      ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)a.N + a.neps);
#pragma unroll
  for (int k = 0; k < KC; ++k) {
    const int c = threadIdx.x * 4 + k * step;
    if (c < a.N) {
      const f32x4 v = xv[k];
      const float4 g = gv[k];
      const size_t i = act_at(row, c, a.nld, a.ntiled);
      store_act4<T>((T*)a.nout, (T*)a.nout2, i, v.x * inv * g.x, v.y * inv * g.y, v.z * inv * g.z, v.w * inv * g.w);
    }
  }
}

// Split-K reduction of a QKV projection in one launch.  Blocks [0, nvb) sum
// the value heads: 32 rows x hd dimensions of one value head per block
// (float4 loads, slices summed in slice order as in gemm_reduce_kernel),
// staged transposed in LDS and written to V^T with the rows running fastest
// across the threads, so that the 2-byte stores of consecutive rows
// (consecutive K/V destinations within a sequence) coalesce.  The remaining
// blocks sum the q/k column pairs (four consecutive pairs of a head per
// thread, float4 loads) and apply RoPE.
template <class T, int HD>
__global__ __launch_bounds__(256) void gemm_reduce_qkv_kernel(GemmArgs a, int nvb) {
  static_assert(sizeof(T) == 2, "bf16 activations");
  using Q = qkv_t<T>;   // stored q, k, v
  const size_t plane = (size_t)a.M * a.N;
  if ((int)blockIdx.x >= nvb) {
    // four consecutive pairs (j .. j + 3) of one head per thread
    constexpr int Q4 = HD / 8;                    // quads of pairs per head
    const int nquad = (a.hq + a.hkv) * Q4;
    const long idx = (long)(blockIdx.x - nvb) * blockDim.x + threadIdx.x;
    if (idx >= (long)a.M * nquad) return;
    const int row = (int)(idx / nquad), q = (int)(idx % nquad);
    const float* pr = a.part + (size_t)row * a.N;
    const int head = q / Q4, j = (q % Q4) * 4;
    const int c1 = head * HD + j, c2 = c1 + HD / 2;
    f32x4 v1 = *(const f32x4*)(pr + c1), v2 = *(const f32x4*)(pr + c2);
    for (int s = 1; s < a.ksplit; ++s) {
      v1 += *(const f32x4*)(pr + s * plane + c1);
      v2 += *(const f32x4*)(pr + s * plane + c2);
    }
    // RoPE of the four pairs with epi_qkv's expressions, one 8-byte store per half
    const int dst = a.row_dst[row];
    const float2* cs = a.rope + (size_t)a.row_pos[row] * (HD / 2) + j;
    Q* p;
    if (head < a.hq) p = (Q*)a.Qb + ((size_t)head * a.ldq + row) * HD;
    else if (dst_is_fresh(dst)) p = (Q*)a.Kf + ((size_t)(head - a.hq) * a.ldfresh + dst) * HD;
    else p = (Q*)a.Kc + ((size_t)(head - a.hq) * a.ldcache + dst_cache_row(dst)) * HD;
    f16x4 o1, o2;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float2 o = rope_rotate(v1[e], v2[e], cs[e]);
      o1[e] = from_f32<Q>(o.x);
      o2[e] = from_f32<Q>(o.y);
    }
    *(f16x4*)(p + j) = o1;
    *(f16x4*)(p + j + HD / 2) = o2;
    return;
  }
  constexpr int RT = 32, TPR = HD / 4, RG = 256 / TPR, RPT = RT / RG;
  static_assert(RPT >= 1 && RT % RG == 0, "row tiling");
  __shared__ Q tile[HD][RT + 2];
  const int mb = (a.M + RT - 1) / RT;
  const int vh = blockIdx.x / mb, r0 = (blockIdx.x % mb) * RT;
  const int d4 = (threadIdx.x % TPR) * 4, rg = threadIdx.x / TPR;
  const float* pr = a.part + (size_t)(a.hq + a.hkv + vh) * HD + d4;
  // every slice of this thread's rows is requested before any is summed
  f32x4 v[RPT];
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int row = min(r0 + rg + k * RG, a.M - 1);
    v[k] = *(const f32x4*)(pr + (size_t)row * a.N);
  }
  for (int s = 1; s < a.ksplit; ++s) {
    f32x4 t[RPT];
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
      const int row = min(r0 + rg + k * RG, a.M - 1);
      t[k] = *(const f32x4*)(pr + s * plane + (size_t)row * a.N);
    }
#pragma unroll
    for (int k = 0; k < RPT; ++k) v[k] += t[k];
  }
#pragma unroll
  for (int k = 0; k < RPT; ++k)
#pragma unroll
    for (int e = 0; e < 4; ++e) tile[d4 + e][rg + k * RG] = from_f32<Q>(v[k][e]);
  __syncthreads();
  for (int i = threadIdx.x; i < RT * HD; i += blockDim.x) {
    const int dd = i / RT, rr = i % RT, row = r0 + rr;
    if (row < a.M) {
      const int dst = a.row_dst[row];
      Q* vt;
      int ld, col;
      if (dst_is_fresh(dst)) { vt = (Q*)a.Vtf; ld = a.ldfresh; col = dst; }
      else { vt = (Q*)a.Vtc; ld = a.ldcache; col = dst_cache_row(dst); }
      vt[((size_t)vh * HD + dd) * ld + col] = tile[dd][rr];
    }
  }
}

template <int EPI>
static void reduce_epi(const GemmArgs& a, hipStream_t st) {
  if constexpr (EPI == EPI_RESID) {
    if (a.ngain) {
      if (a.nf16) {
        if (a.N <= 8 * NORM_THREADS) gemm_reduce_resid_norm_kernel<f16, 2><<<a.M, NORM_THREADS, 0, st>>>(a);
        else gemm_reduce_resid_norm_kernel<f16, 4><<<a.M, NORM_THREADS, 0, st>>>(a);
      } else {
        if (a.N <= 8 * NORM_THREADS) gemm_reduce_resid_norm_kernel<bf16, 2><<<a.M, NORM_THREADS, 0, st>>>(a);
        else gemm_reduce_resid_norm_kernel<bf16, 4><<<a.M, NORM_THREADS, 0, st>>>(a);
      }
      return;
    }
  }
  if constexpr (EPI == EPI_QKV) {
    const int nvb = (a.M + 31) / 32 * a.hkv;
    const long nqk = (long)a.M * (a.hq + a.hkv) * a.hd / 8;
    const unsigned grid = (unsigned)(nvb + (nqk + 255) / 256);
    if (a.hd == 128) gemm_reduce_qkv_kernel<bf16, 128><<<grid, 256, 0, st>>>(a, nvb);
    else gemm_reduce_qkv_kernel<bf16, 64><<<grid, 256, 0, st>>>(a, nvb);
  } else {
    const int npair = epi_paired(EPI) ? a.N / 2 : a.N;
    const long total = (long)a.M * npair;
    gemm_reduce_kernel<EPI, bf16><<<(unsigned)((total + 255) / 256), 256, 0, st>>>(a);
  }
}

void launch_gemm_reduce(int epi, const GemmArgs& a, hipStream_t st) {
  switch (epi) {
    case EPI_STORE: reduce_epi<EPI_STORE>(a, st); break;
    case EPI_RESID: reduce_epi<EPI_RESID>(a, st); break;
    case EPI_SWIGLU: reduce_epi<EPI_SWIGLU>(a, st); break;
    default: reduce_epi<EPI_QKV>(a, st); break;
  }
}

// ---------------------------------------------------------------------------
namespace {

template <int BM, int BN, int BK, int WGM, int WGN, int EPI, int MODE>
void run_mode(const GemmArgs& a, int grid, hipStream_t st) {
  if (a.A2) gemm_bf16_kernel<BM, BN, BK, WGM, WGN, EPI, true, MODE><<<grid, 256, 0, st>>>(a);
  else gemm_bf16_kernel<BM, BN, BK, WGM, WGN, EPI, false, MODE><<<grid, 256, 0, st>>>(a);
}

template <int BM, int BN, int BK, int WGM, int WGN, int EPI>
void run_cfg(const GemmArgs& a, bool partial, hipStream_t st) {
  const int n_tiles = a.N / BN, m_tiles = (a.M + BM - 1) / BM;
  const int grid = gemm_grid_size(n_tiles, m_tiles, partial ? a.ksplit : 1);
  if (partial) {
    run_mode<BM, BN, BK, WGM, WGN, EPI, 2>(a, grid, st);
    launch_gemm_reduce(EPI, a, st);
  } else if (a.ksplit > 1) {
    run_mode<BM, BN, BK, WGM, WGN, EPI, 1>(a, grid, st);
  } else {
    run_mode<BM, BN, BK, WGM, WGN, EPI, 0>(a, grid, st);
  }
}

template <int EPI>
void run_epi(int cfg, const GemmArgs& a, bool partial, hipStream_t st) {
  switch (cfg) {
    case 0: run_cfg<128, 128, 64, 2, 2, EPI>(a, partial, st); break;
    case 1: run_cfg<256, 128, 32, 2, 2, EPI>(a, partial, st); break;
    case 2: run_cfg<128, 64, 64, 4, 1, EPI>(a, partial, st); break;
    case 3: run_cfg<256, 64, 64, 4, 1, EPI>(a, partial, st); break;
    case 4: run_cfg<64, 128, 64, 1, 4, EPI>(a, partial, st); break;
    case 5: run_cfg<64, 128, 32, 1, 4, EPI>(a, partial, st); break;
    default: run_cfg<128, 64, 32, 4, 1, EPI>(a, partial, st); break;
  }
}

const int kCfgBN[GEMM_NCFG] = {128, 128, 64, 64, 128, 128, 64};
const int kCfgBK[GEMM_NCFG] = {64, 32, 64, 64, 64, 32, 32};
const int kCfgBM[GEMM_NCFG] = {128, 256, 128, 256, 64, 64, 128};

}  // namespace

int gemm_ksplit(int N, int K, int rows) {
  // One slice when the smallest launch has enough 128-row tiles to fill the
  // GPU on its own (rows >= 2048: at least 16 row tiles); otherwise enough
  // slices that a 256-row launch of 128 x 128 tiles fills the 256 CUs,
  // within the K granularity.  The count is fixed per context (rows is the
  // context's response-row capacity), never per launch, so every pass of a
  // context sums every output in the same order.
  // A 256-row launch that already has three quarters of a round of 128 x 128
  // tiles (N >= 12288) also takes one slice: measured on the LLaDA-8B QKV
  // projection, one slice is as fast as two at 256 rows (128 x 128 tiles)
  // and 17 % faster in a 4352-row refresh pass (128 x 256 tiles, no partial
  // planes or reduction).
  if (rows >= 2048) return 1;
  const int tiles = 2 * std::max(N / 128, 1);
  if (tiles >= 192) return 1;
  int S = 1;
  while (S < 8 && tiles * S < 256 && K % (2 * S * 64) == 0) S *= 2;
  return S;
}

int gemm_pick_cfg(const GemmArgs& a, int epi) {
  // The warp-specialised direct-to-LDS kernel (gemm_lds.hip).  Two-term
  // launches of one K slice take the tile (128 x 256: 64 x 128 wave tiles,
  // fewer LDS bytes per MFMA; 128 x 192; 128 x 128) with the fewest rounds of
  // 256 workgroups (one per CU) times the time of a tile: measured on the
  // LLaDA-8B projections, a 128 x 192 tile takes 1.5x and a 128 x 256 tile
  // 1.77x the time of a 128 x 128 tile (so, for example, 256-row gate/up
  // passes take 128 x 192 tiles, one round, and 256-row QKV passes 128 x 128
  // tiles).  The LM head decides on N alone, so that the column tile of its
  // fused decision statistics does not depend on the row count of a pass.
  // Split-K launches take 128 x 192 tiles when N is a multiple of 192, else
  // 128 x 128; the 128 x 192 tile is not used for slices folded in one
  // workgroup (its second accumulator set does not fit the registers of two
  // waves per SIMD).
  // Single-term fp16 launches (gate/up) choose the same way with their own
  // tile times: 1.34x (128 x 192) and 1.66x (128 x 256) that of a 128 x 128
  // tile, measured on the LLaDA-8B gate/up shape at 24853 rows.
  const bool wide = (a.A2 || a.f16) && a.ksplit == 1;
  const double t192 = a.f16 ? 1.34 : 1.5, t256 = a.f16 ? 1.66 : 1.77;
  if (wide && epi == EPI_STORE) {
    if (a.N % 256 == 0 && a.N / 256 >= 256 && gemm_lds_cfg_ok(2, a)) return GEMM_NCFG + 2;
  } else if (wide) {
    // the tile with the fewest rounds times tile time; a narrower tile must
    // be 5 % cheaper than a wider one to be taken
    const long mt = (a.M + 127) / 128;
    const auto cost = [&](int bn, double t) { return (double)((a.N / bn * mt + 255) / 256) * t; };
    int best = -1;
    double bc = 0;
    if (a.N % 256 == 0 && gemm_lds_cfg_ok(2, a)) { best = 2; bc = cost(256, t256); }
    if (a.N % 192 == 0 && gemm_lds_cfg_ok(0, a) && (best < 0 || cost(192, t192) < 0.95 * bc)) {
      best = 0;
      bc = cost(192, t192);
    }
    if (a.N % 128 == 0 && gemm_lds_cfg_ok(1, a) && (best < 0 || cost(128, 1.0) < 0.95 * bc)) {
      best = 1;
      bc = cost(128, 1.0);
    }
    if (best >= 0) return GEMM_NCFG + best;
  }
  if (a.N % 192 == 0 && gemm_lds_cfg_ok(0, a)) {
    const bool fold = a.ksplit > 1 && !(a.part && gemm_partial_wanted(GEMM_NCFG + 0, a));
    if (!fold) return GEMM_NCFG + 0;
  }
  if (a.N % 128 == 0 && gemm_lds_cfg_ok(1, a)) return GEMM_NCFG + 1;
  // register-staged kernel for the remaining shapes
  const bool bn128 = a.N % 128 == 0 && (epi != EPI_QKV || a.hd % 128 == 0) &&
                     (epi != EPI_SWIGLU || (a.N / 2) % 64 == 0);
  const bool bk64 = a.K % (2 * a.ksplit * 64) == 0;   // even number of 64-wide k tiles per slice
  if (bn128) {
    if (!bk64) return 5;
    return a.M <= 1024 ? 4 : 0;
  }
  if (!bk64) return 6;
  return a.M <= 1024 ? 2 : 3;
}

bool gemm_cfg_ok(int cfg, const GemmArgs& a, int epi) {
  if (cfg < 0 || cfg >= GEMM_NCFG) return false;
  const int BN = kCfgBN[cfg];
  if (a.M <= 0 || a.N % BN || a.ksplit < 1 || a.K % (2 * a.ksplit * kCfgBK[cfg])) return false;
  if (epi == EPI_QKV && (a.hd % BN)) return false;
  if (epi == EPI_SWIGLU && ((a.N / 2) % (BN / 2))) return false;
  return true;
}

int gemm_partial_wanted(int cfg, const GemmArgs& a) {
  // Measured on MI355X (LLaDA-8B projections, M = 256 .. 4352): one workgroup
  // per slice with a separate reduction is at least as fast as folding the
  // slices into one workgroup whenever a partial buffer is available.
  (void)cfg;
  return a.ksplit > 1;
}

bool gemm_args_ok(int epi, const GemmArgs& a) {
  if (!a.A || !a.W || a.M <= 0 || a.N <= 0 || a.K <= 0 || a.ksplit < 1) return false;
  if (a.f16 && (epi != EPI_SWIGLU || a.A2)) return false;   // fp16 operands: single-term gate/up only
  switch (epi) {
    case EPI_STORE: return (a.C && a.ldc >= a.N) || (a.tstat && a.targ && a.zg && a.tg);
    case EPI_RESID: return a.X && a.ldx >= a.N;
    case EPI_SWIGLU: return a.H && a.W2 && a.N % 2 == 0;
    case EPI_QKV:
      // the column mapping divides by hd / 2 and the epilogue indexes every table
      return a.hd > 0 && a.hd % 2 == 0 && a.hq > 0 && a.hkv > 0 && a.N == (a.hq + 2 * a.hkv) * a.hd && a.Qb &&
             a.Kf && a.Vtf && a.Kc && a.Vtc && a.row_dst && a.row_pos && a.rope;
    default: return false;
  }
}

int launch_gemm_bf16_cfg(int epi, int cfg, bool partial, const GemmArgs& a, hipStream_t st) {
  if (!gemm_args_ok(epi, a)) return 1;
  if (cfg >= GEMM_NCFG) return launch_gemm_lds_cfg(epi, cfg - GEMM_NCFG, partial, a, st);
  if (a.f16 || !gemm_cfg_ok(cfg, a, epi)) return 1;   // the register-staged kernel is bf16 only
  if (partial && (!a.part || a.ksplit < 2)) return 1;
  switch (epi) {
    case EPI_STORE: run_epi<EPI_STORE>(cfg, a, partial, st); break;
    case EPI_RESID: run_epi<EPI_RESID>(cfg, a, partial, st); break;
    case EPI_SWIGLU: run_epi<EPI_SWIGLU>(cfg, a, partial, st); break;
    case EPI_QKV: run_epi<EPI_QKV>(cfg, a, partial, st); break;
    default: return 1;
  }
  return 0;
}

bool gemm_fuses_norm(const GemmArgs& a) {
  if (!a.ngain || !a.part || a.N % 4 || a.N > 16 * NORM_THREADS || a.ldx % 4 || a.ksplit > 8) return false;
  const int cfg = gemm_pick_cfg(a, EPI_RESID);
  return gemm_partial_wanted(cfg, a) != 0;
}

int launch_gemm_bf16(int epi, const GemmArgs& a, hipStream_t st) {
  const int cfg = gemm_pick_cfg(a, epi);
  const bool partial = a.part != nullptr && gemm_partial_wanted(cfg, a);
  return launch_gemm_bf16_cfg(epi, cfg, partial, a, st);
}

// ---------------------------------------------------------------------------
// fp32 kernel: 64 x 64 tile, BK 16; thread (tx, ty) owns columns tx and
// tx + 32 (a pair) of rows ty + 8 i.
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
  const int wr = brow_index<EPI, BN>(a, tile_n, lr, &second);
  const float* bsrc = (const float*)(second ? a.W2 : a.W) + (size_t)wr * a.ldw + lk;
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
      epi_tile_pair<EPI, float, BN>(a, tile_n, tx, row, acc0[i], acc1[i]);
    } else if constexpr (EPI == EPI_STORE) {
      epi_store(a, row, tile_n * BN + tx, acc0[i]);
      epi_store(a, row, tile_n * BN + tx + 32, acc1[i]);
    } else {
      epi_resid(a, row, tile_n * BN + tx, acc0[i]);
      epi_resid(a, row, tile_n * BN + tx + 32, acc1[i]);
    }
  }
}

int launch_gemm_f32(int epi, const GemmArgs& a, hipStream_t st) {
  constexpr int BM = 64, BN = 64;
  if (!gemm_args_ok(epi, a)) return 1;
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
