// Projection GEMMs, multistage warp-specialised version.
//
// A workgroup has 8 waves: waves 0-3 multiply (a 2 x 2 or 4 x 1 grid of
// wave tiles, MFMA v_mfma_f32_16x16x32_bf16 -- _f16 for the single-term fp16
// operands of the gate/up projection -- fp32 accumulate), waves 4-7 only
// load.  The loaders move the A (two-term: hi and lo) and W tiles of 32-wide k
// chunks straight from global memory into NST LDS stages
// (global_load_lds_dwordx4, no register staging).  With one wave per SIMD
// doing both jobs, a wave blocked issuing loads into a full memory queue also
// stops issuing MFMAs; separate loader waves keep the MFMA pipes fed.
//
// Addressing.  A direct load writes the 16 bytes of lane l at LDS address
// M0 + 16 l, so the LDS layout is fixed by the slot order and each lane
// fetches the global chunk that belongs in its slot.  Tiles are stored
// row-major with 16-byte chunks XOR-swizzled inside a row (physical chunk =
// logical chunk ^ swz(row)), which keeps the MFMA fragment reads free of bank
// conflicts.  The global address of a slot is a per-lane 32-bit offset that
// never changes plus a wave-uniform 64-bit base that advances by 32 elements
// per tile, so the loaders spend no vector instructions on addresses.
//
// Synchronisation (one barrier per tile, all 8 waves).  The multiply waves
// hold the fragments of tile g in registers (read during tile g - 1) and
// place barrier X_g between the hi-term and lo-term MFMAs of tile g (single
// term: between the MFMAs of the first and second half of its weight blocks);
// after X_g they read the fragments of tile g + 1, overlapping the MFMAs that
// follow X_g.
// A loader arrives at X_g once its loads of tile g + 1 have landed
// (s_waitcnt vmcnt; the loads are issued from inline assembly, outside the
// compiler's own wait tracking) and after X_g loads tile g + NST into the
// stage of tile g, which no wave reads any more.
//
// Results are bitwise identical to the register-staged kernel in gemm.hip:
// the same k order (32-wide chunks in order, hi then lo term per chunk), the
// same split-K slices and the same epilogues.  fp16 operands run only here.
#include <algorithm>

#include "gemm_common.h"

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

namespace {

// s_waitcnt immediates (gfx9 encoding)
#define GL_VMCNT(n) (((n) & 15) | (7 << 4) | (15 << 8) | ((((n) >> 4) & 3) << 14))
#define GL_LGKMCNT0 (15 | (7 << 4) | (0 << 8) | (3 << 14))

// M0 is listed as clobbered; no other code of this file keeps a value in it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void gl_dma16(const void* sbase, unsigned voff, unsigned lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ void gl_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Chunk swizzle of a 64-byte row (four 16-byte chunks), chosen by measurement
// (LDS bank-conflict counter of ds_read_b128 over 16 rows x one chunk): the
// chunk index is XORed with (row / 2) mod 4.
__device__ __forceinline__ int gl_swz(int row) { return (row >> 1) & 3; }

constexpr int BK = 32;      // k chunk per tile (one MFMA k step)
constexpr int CPR = BK / 8; // 16-byte chunks per tile row

// QKV projection, value heads.  A tile whose column pairs are all value pairs
// is staged in LDS as the transposed tile (one row of BM + 8 keys per value
// dimension) and written to V^T in 16-byte chunks along the key axis wherever
// eight consecutive pass rows go to eight consecutive, aligned key columns of
// one buffer; element stores otherwise.  Written one element per lane, the
// transposed layout gives every two-byte store its own cache line, which the
// L2 then reads whole to merge.  The stored values are those of
// epi_tile_pair4.
template <int BN>
__device__ __forceinline__ bool qkv_value_tile(const GemmArgs& a, int tile_n) {
  return tile_n * (BN / 2) >= (a.hq + a.hkv) * (a.hd / 2);
}
constexpr int VT_PAD = 8;
template <int BM, int BN, int NTHREADS>
__device__ __forceinline__ void store_value_tile(const GemmArgs& a, const f16* vs, int tile_n, int m0, int t) {
  constexpr int KS = BM + VT_PAD, KC = BM / 8;
  static_assert(NTHREADS % KC == 0, "a thread keeps one key chunk");
  // this thread's chunk of eight keys is the same for every dimension row it stores
  const int kc = t % KC, k0 = m0 + kc * 8;
  if (k0 >= a.M) return;
  const int nk = min(8, a.M - k0);
  const int dst0 = a.row_dst[k0];
  const bool fresh = dst_is_fresh(dst0);
  const int col0 = fresh ? dst0 : dst_cache_row(dst0);
  f16* vt = (f16*)(fresh ? a.Vtf : a.Vtc);
  const int ld = fresh ? a.ldfresh : a.ldcache;
  bool vec = nk == 8 && col0 % 8 == 0 && ld % 8 == 0 && ((uintptr_t)vt & 15) == 0;
  for (int i = 1; i < 8 && vec; ++i) {
    const int di = a.row_dst[k0 + i];
    vec = dst_is_fresh(di) == fresh && (fresh ? di : dst_cache_row(di)) == col0 + i;
  }
  const int half = a.hd / 2, p0 = tile_n * (BN / 2);
  for (int drow = t / KC; drow < BN; drow += NTHREADS / KC) {
    const int p = p0 + (drow >> 1);
    const int vh = p / half - a.hq - a.hkv, d = p % half + (drow & 1) * half;
    const f16* src = vs + drow * KS + kc * 8;
    if (vec) {
      *(u32x4*)(vt + (size_t)(vh * a.hd + d) * ld + col0) = *(const u32x4*)src;
    } else {
      for (int i = 0; i < nk; ++i) {
        const int di = a.row_dst[k0 + i];
        if (dst_is_fresh(di)) ((f16*)a.Vtf)[(size_t)(vh * a.hd + d) * a.ldfresh + di] = src[i];
        else ((f16*)a.Vtc)[(size_t)(vh * a.hd + d) * a.ldcache + dst_cache_row(di)] = src[i];
      }
    }
  }
}

// QKV projection, query and key heads.  A tile whose column pairs are whole
// query or key heads is staged in LDS as rotated rows (the values of
// epi_tile_pair4) and written with 16-byte stores along each head's
// dimensions, so every store covers whole 128-byte lines.  Written straight
// from the accumulators, a store covers 32 bytes of each of 16 rows, and the
// L2 reads every partly written line from memory first: the query and key
// stores of a 4096-row pass fetched 0.5 GB for 67 MB of output.
template <int BN>
__device__ __forceinline__ bool qkv_qk_tile(const GemmArgs& a, int tile_n) {
  const int half = a.hd / 2;
  return (BN / 2) % half == 0 && (tile_n + 1) * (BN / 2) <= (a.hq + a.hkv) * half &&
         (((uintptr_t)a.Qb | (uintptr_t)a.Kf | (uintptr_t)a.Kc) & 15) == 0;
}
constexpr int QK_PAD = 8;
template <int BM, int BN, int NTHREADS>
__device__ __forceinline__ void store_qk_tile(const GemmArgs& a, const f16* qs, int tile_n, int m0, int t) {
  constexpr int RS = BN + QK_PAD, CH = BN / 8;   // staged row stride, 16-byte chunks per row
  const int hd = a.hd, h0 = tile_n * (BN / hd);
  for (int i = t; i < BM * CH; i += NTHREADS) {
    const int r = i / CH, ch = i % CH, row = m0 + r;
    if (row >= a.M) break;                        // i only grows, and so does row
    const int head = h0 + ch * 8 / hd, d = ch * 8 % hd;
    f16* p;
    if (head < a.hq) {
      p = (f16*)a.Qb + ((size_t)head * a.ldq + row) * hd;
    } else {
      const int dst = a.row_dst[row];
      p = dst_is_fresh(dst) ? (f16*)a.Kf + ((size_t)(head - a.hq) * a.ldfresh + dst) * hd
                            : (f16*)a.Kc + ((size_t)(head - a.hq) * a.ldcache + dst_cache_row(dst)) * hd;
    }
    *(u32x4*)(p + d) = *(const u32x4*)(qs + r * RS + ch * 8);
  }
}

template <int BM, int BN, int WGM, int WGN, int NST, int EPI, bool SPLIT, int MODE, bool F16 = false>
__global__ __launch_bounds__(512, 1) void gemm_lds_kernel(GemmArgs a) {
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int RB = WM / 16, CB = WN / 16;
  constexpr int NA = SPLIT ? 2 : 1;
  constexpr int A_SL = BM * CPR, B_SL = BN * CPR;          // 16-byte slots per tile
  constexpr int AI = A_SL / 256, BI = B_SL / 256;          // load instructions per loader wave per tile
  constexpr int IPT = NA * AI + BI;
  constexpr int STAGE = (NA * A_SL + B_SL) * 16;           // bytes
  constexpr bool PARTIAL = MODE == 2, FOLD = MODE == 1;
  static_assert(WGM * WGN == 4 && CB % 2 == 0 && RB >= 1, "bad wave grid");
  static_assert(!F16 || !SPLIT, "fp16 operands are single-term");
  static_assert(A_SL % 256 == 0 && B_SL % 256 == 0, "each loader wave issues whole load instructions");
  static_assert(BN % (32 * WGN) == 0, "each wave takes 16-column blocks from both tile halves");
  static_assert((NST - 1) * IPT <= 63 && NST >= 2, "vmcnt range");
  // the W / W2 split of a SwiGLU tile falls on a wave-instruction boundary
  static_assert((BN / 2) % (64 / CPR) == 0, "pair halves must not share a load instruction");
  __shared__ __attribute__((aligned(1024))) char smem[NST * STAGE];

  const int n_tiles = a.N / BN, m_tiles = (a.M + BM - 1) / BM;
  int tile_n, tile_m, z;
  if (!tile_of(blockIdx.x, n_tiles, m_tiles, PARTIAL ? a.ksplit : 1, &tile_n, &tile_m, &z)) return;
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int m0 = tile_m * BM;
  const int kslice = a.K / a.ksplit;
  const int kbeg = PARTIAL ? z * kslice : 0;
  const int nslices = FOLD ? a.ksplit : 1;
  const int kt_slice = (PARTIAL || FOLD ? kslice : a.K) / BK;
  const int ntot = nslices * kt_slice;

  if (w >= 4) {
    // ---- loader waves -------------------------------------------------------
    const int wp = w - 4;
    const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) char*)smem;
    // per-lane global byte offsets of the slots this lane fills (rows past M
    // load row M - 1: finite data, and those output rows are never stored)
    unsigned a_go[AI], b_go[BI];
    bool b_hi[BI];
#pragma unroll
    for (int j = 0; j < AI; ++j) {
      const int q = j * 256 + wp * 64 + lane, r = q / CPR, pc = q % CPR;
      const int row = min(m0 + r, a.M - 1);
      a_go[j] = ((unsigned)row * (a.a_tiled ? BK : a.lda) + (pc ^ gl_swz(r)) * 8) * 2;
    }
#pragma unroll
    for (int j = 0; j < BI; ++j) {
      const int q = j * 256 + wp * 64 + lane, r = q / CPR, pc = q % CPR;
      bool second;
      const int wr = brow_index<EPI, BN>(a, tile_n, r, &second);
      b_go[j] = ((unsigned)wr * (a.w_tiled ? BK : a.ldw) + (pc ^ gl_swz(r)) * 8) * 2;
      // uniform over the wave's 64 slots (rows j*256/CPR + wp*64/CPR + [0, 64/CPR))
      b_hi[j] = __builtin_amdgcn_readfirstlane(second ? 1 : 0) != 0;
    }
    const bf16* Abase[2] = {(const bf16*)a.A, (const bf16*)(SPLIT ? a.A2 : a.A)};
    const bf16* Wlo = (const bf16*)a.W;
    const bf16* Whi = (const bf16*)(a.W2 ? a.W2 : a.W);
    // tiles past the last are clamped: redundant loads into stages no wave reads again
    // k-block-major A: the block of k step k0 starts k0 * row-capacity elements in
    const size_t akmul = a.a_tiled ? (size_t)a.lda : 1, wkmul = a.w_tiled ? (size_t)a.ldw : 1;
    auto issue = [&](int g) {
      const int k0 = kbeg + min(g, ntot - 1) * BK;
      const unsigned st = lds0 + (unsigned)((g % NST) * STAGE);
#pragma unroll
      for (int t = 0; t < NA; ++t)
#pragma unroll
        for (int j = 0; j < AI; ++j)
          gl_dma16(Abase[t] + (size_t)k0 * akmul, a_go[j], st + (unsigned)((t * A_SL + j * 256 + wp * 64) * 16));
#pragma unroll
      for (int j = 0; j < BI; ++j)
        gl_dma16((b_hi[j] ? Whi : Wlo) + (size_t)k0 * wkmul, b_go[j], st + (unsigned)((NA * A_SL + j * 256 + wp * 64) * 16));
    };
#pragma unroll
    for (int s = 0; s < NST; ++s) issue(s);
    __builtin_amdgcn_s_waitcnt(GL_VMCNT((NST - 1) * IPT));   // tile 0 landed
    gl_barrier();                                             // X_-1
    for (int g = 0; g + 1 < ntot; ++g) {
      __builtin_amdgcn_s_waitcnt(GL_VMCNT((NST - 2) * IPT)); // tile g + 1 landed
      gl_barrier();                                           // X_g
      issue(g + NST);
    }
    // the trailing loads must land before the workgroup's LDS is released
    __builtin_amdgcn_s_waitcnt(GL_VMCNT(0));
    if constexpr (EPI == EPI_QKV && MODE == 0 && SPLIT) {
      if (qkv_value_tile<BN>(a, tile_n)) {
        __syncthreads();   // X_v1: every load landed, every fragment read done
        __syncthreads();   // X_v2: the multiply waves staged the tile
        store_value_tile<BM, BN, 512>(a, (const f16*)smem, tile_n, m0, tid);
      } else if (qkv_qk_tile<BN>(a, tile_n)) {
        __syncthreads();   // X_q1
        __syncthreads();   // X_q2
        store_qk_tile<BM, BN, 512>(a, (const f16*)smem, tile_n, m0, tid);
      }
    }
    return;
  }

  // ---- multiply waves --------------------------------------------------------
  const int lg = lane >> 4, lc = lane & 15;
  const int wm = w / WGN, wn = w % WGN;
  // LDS byte offsets of this lane's fragment reads within a stage
  unsigned a_lo[RB], b_lo[CB];
  int tc[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) tc[cb] = (cb / (CB / 2)) * (BN / 2) + wn * (WN / 2) + (cb % (CB / 2)) * 16 + lc;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int r = wm * WM + rb * 16 + lc;
    a_lo[rb] = (unsigned)((r * CPR + (lg ^ gl_swz(r))) * 16);
  }
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) b_lo[cb] = (unsigned)((NA * A_SL + tc[cb] * CPR + (lg ^ gl_swz(tc[cb]))) * 16);

  f32x4 acc[RB][CB];
  f32x4 tot[FOLD ? RB : 1][FOLD ? CB : 1];
#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int j = 0; j < CB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  if constexpr (FOLD) {
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int j = 0; j < CB; ++j) tot[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  bf16x8 fa[2][NA][RB], fb[2][CB];
  auto read_frags = [&](int g, int buf) {
    const char* stg = smem + (g % NST) * STAGE;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) fb[buf][cb] = *(const bf16x8*)(stg + b_lo[cb]);
#pragma unroll
    for (int t = 0; t < NA; ++t)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) fa[buf][t][rb] = *(const bf16x8*)(stg + t * A_SL * 16 + a_lo[rb]);
  };
  // Except for split-K partials, the weight fragment is the MFMA's A operand
  // and the activation fragment its B operand (C^T = W A^T), so that a lane's
  // four accumulator entries are four consecutive output columns of one row,
  // which the epilogue writes with vector stores (gate/up -2 %, LM head -3 %
  // measured).  Partial tiles keep C = A W^T and one store per element: their
  // vector stores would touch 16 rows per instruction instead of 4 and were
  // measured no faster.  Either orientation gives the same bits (each output
  // is the same sum of the same products).
  constexpr bool CT = !PARTIAL;
  // one MFMA of weight fragment wf and activation fragment xf in the tile's
  // orientation (the fragments hold fp16 bits when F16)
  auto mm = [&](const bf16x8& wf, const bf16x8& xf, const f32x4& c) __attribute__((always_inline)) {
    if constexpr (F16) {
      const f16x8 w16 = __builtin_bit_cast(f16x8, wf), x16 = __builtin_bit_cast(f16x8, xf);
      return CT ? __builtin_amdgcn_mfma_f32_16x16x32_f16(w16, x16, c, 0, 0, 0)
                : __builtin_amdgcn_mfma_f32_16x16x32_f16(x16, w16, c, 0, 0, 0);
    } else {
      return CT ? __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, xf, c, 0, 0, 0)
                : __builtin_amdgcn_mfma_f32_16x16x32_bf16(xf, wf, c, 0, 0, 0);
    }
  };
  auto mfma_term = [&](int buf, int t) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) acc[rb][cb] = mm(fb[buf][cb], fa[buf][t][rb], acc[rb][cb]);
  };
  // Two-term tiles of 64, 96 or 128 columns per wave, except in the folded
  // mode (its second accumulator set leaves no room): one fragment set,
  // refilled in place.  The lo-term fragments of tile g are read during its
  // hi-term MFMAs; after X_g the lo-term MFMAs run weight block by weight
  // block, and each weight fragment of tile g + 1 is read as soon as the
  // MFMAs of its block have taken the old one (the hi-term fragments of tile
  // g + 1 go in among the first blocks), so reads never come in a burst.
  // Measured against two fragment sets (a burst of reads after X_g for 96
  // columns, reads spread one per lo-term MFMA for 64): 128 x 192 tiles 5-10 %
  // faster (LLaDA-8B gate/up and QKV shapes at 256 and 768 rows), 128 x 128
  // tiles 0-3 %, bitwise the same.
  constexpr bool ROLL = NA == 2 && (CB == 4 || CB == 6 || CB == 8) && !FOLD;
  // Two-term tiles of 32 columns per wave: two fragment sets, the reads of
  // tile g + 1 spread one per lo-term MFMA of tile g.
  constexpr bool PIPE = NA == 2 && CB <= 4 && !FOLD && !ROLL;
  // Single-term tiles (except folded): the MFMAs of the first half of the
  // weight blocks of tile g run before X_g, those of the second half after
  // it.  After X_g the weight fragments of the first half are refilled with
  // those of tile g + 1 at once, each of the second half as soon as its
  // block's MFMAs have taken it (one weight fragment set, so that 64 x 128
  // wave tiles fit the registers), and the activation fragments of tile
  // g + 1 go to the second set in among them.
  constexpr bool PIPE1 = NA == 1 && !FOLD;
  auto mfma_blocks = [&](int buf, int cb0, int cb1) {
#pragma unroll
    for (int cb = cb0; cb < cb1; ++cb)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) acc[rb][cb] = mm(fb[0][cb], fa[buf][0][rb], acc[rb][cb]);
  };
  auto tile_roll = [&](int g, bool more) {
    if constexpr (ROLL) {
      const char* stg = smem + (g % NST) * STAGE;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
          acc[rb][cb] = mm(fb[0][cb], fa[0][0][rb], acc[rb][cb]);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) fa[0][1][rb] = *(const bf16x8*)(stg + A_SL * 16 + a_lo[rb]);
#pragma unroll
      for (int i = 0; i < RB; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, RB * CB - RB, 0);
      __builtin_amdgcn_sched_barrier(0);
      if (more) {
        __builtin_amdgcn_s_waitcnt(GL_LGKMCNT0);   // this wave's reads of tile g are done
        gl_barrier();                               // X_g
        const char* stn = smem + ((g + 1) % NST) * STAGE;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            acc[rb][cb] = mm(fb[0][cb], fa[0][1][rb], acc[rb][cb]);
          fb[0][cb] = *(const bf16x8*)(stn + b_lo[cb]);
          if (cb < RB) fa[0][0][cb] = *(const bf16x8*)(stn + a_lo[cb]);
        }
        static_assert(RB <= CB, "the hi-term reads go in among the first RB blocks");
#pragma unroll
        for (int cb = 0; cb < RB; ++cb) {
          __builtin_amdgcn_sched_group_barrier(0x008, RB, 0);   // the MFMAs of block cb
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);    // its weight and one hi-term fragment
        }
#pragma unroll
        for (int cb = RB; cb < CB; ++cb) {
          __builtin_amdgcn_sched_group_barrier(0x008, RB, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      } else {
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            acc[rb][cb] = mm(fb[0][cb], fa[0][1][rb], acc[rb][cb]);
      }
    }
  };
  // 64 x 128 wave tiles (8 weight blocks) keep one activation fragment set
  // too: the last block's MFMAs take the activation fragments one by one and
  // each is refilled right after, and the next tile starts with the MFMAs of
  // the first activation fragment over its first half of blocks.
  constexpr bool FA1 = PIPE1 && CB == 8;
  auto tile_p1 = [&](int g, int cur, bool more) {
    if constexpr (FA1) {
      constexpr int H = CB / 2;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int cb = 0; cb < H; ++cb) acc[rb][cb] = mm(fb[0][cb], fa[0][0][rb], acc[rb][cb]);
      if (more) {
        __builtin_amdgcn_s_waitcnt(GL_LGKMCNT0);   // this wave's reads of tile g are done
        gl_barrier();                               // X_g
        const char* stn = smem + ((g + 1) % NST) * STAGE;
#pragma unroll
        for (int cb = 0; cb < H; ++cb) fb[0][cb] = *(const bf16x8*)(stn + b_lo[cb]);
#pragma unroll
        for (int cb = H; cb < CB - 1; ++cb) {
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) acc[rb][cb] = mm(fb[0][cb], fa[0][0][rb], acc[rb][cb]);
          fb[0][cb] = *(const bf16x8*)(stn + b_lo[cb]);
        }
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          acc[rb][CB - 1] = mm(fb[0][CB - 1], fa[0][0][rb], acc[rb][CB - 1]);
          fa[0][0][rb] = *(const bf16x8*)(stn + a_lo[rb]);
        }
        fb[0][CB - 1] = *(const bf16x8*)(stn + b_lo[CB - 1]);
        __builtin_amdgcn_sched_group_barrier(0x100, H, 0);   // the first half's weight fragments
#pragma unroll
        for (int cb = H; cb < CB - 1; ++cb) {
          __builtin_amdgcn_sched_group_barrier(0x008, RB, 0);   // the MFMAs of block cb
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);    // its weight fragment
        }
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // last block, activation fragment rb
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);    // its refill
        }
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // the last weight fragment
        __builtin_amdgcn_sched_barrier(0);
      } else {
        mfma_blocks(0, H, CB);
      }
    } else if constexpr (PIPE1) {
      constexpr int H = CB / 2, NB2 = CB - H;
      mfma_blocks(cur, 0, H);
      if (more) {
        __builtin_amdgcn_s_waitcnt(GL_LGKMCNT0);   // this wave's reads of tile g are done
        gl_barrier();                               // X_g
        const char* stn = smem + ((g + 1) % NST) * STAGE;
#pragma unroll
        for (int cb = 0; cb < H; ++cb) fb[0][cb] = *(const bf16x8*)(stn + b_lo[cb]);
#pragma unroll
        for (int i = 0; i < NB2; ++i) {
          const int cb = H + i;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) acc[rb][cb] = mm(fb[0][cb], fa[cur][0][rb], acc[rb][cb]);
          fb[0][cb] = *(const bf16x8*)(stn + b_lo[cb]);
#pragma unroll
          for (int rb = RB * i / NB2; rb < RB * (i + 1) / NB2; ++rb)
            fa[cur ^ 1][0][rb] = *(const bf16x8*)(stn + a_lo[rb]);
        }
        __builtin_amdgcn_sched_group_barrier(0x100, H, 0);   // the first half's weight fragments
#pragma unroll
        for (int i = 0; i < NB2; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, RB, 0);   // the MFMAs of block H + i
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);    // its weight fragment
#pragma unroll
          for (int rb = RB * i / NB2; rb < RB * (i + 1) / NB2; ++rb)
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // activation fragments
        }
        __builtin_amdgcn_sched_barrier(0);
      } else {
        mfma_blocks(cur, H, CB);
      }
    }
  };
  auto tile_body = [&](int g, int cur) {
    mfma_term(cur, 0);
    if constexpr (PIPE) {
      if (g + 1 < ntot) {
        __builtin_amdgcn_s_waitcnt(GL_LGKMCNT0);   // this wave's reads of tile g are done
        gl_barrier();                               // X_g
        read_frags(g + 1, cur ^ 1);
        mfma_term(cur, 1);
        constexpr int NRD = CB + NA * RB, NM = RB * CB;
#pragma unroll
        for (int i = 0; i < (NRD < NM ? NRD : NM); ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
        }
        if constexpr (NM > NRD) __builtin_amdgcn_sched_group_barrier(0x008, NM - NRD, 0);
        if constexpr (NRD > NM) __builtin_amdgcn_sched_group_barrier(0x100, NRD - NM, 0);
        __builtin_amdgcn_sched_barrier(0);
      } else {
        mfma_term(cur, 1);
      }
    } else {
      if (g + 1 < ntot) {
        __builtin_amdgcn_s_waitcnt(GL_LGKMCNT0);   // this wave's reads of tile g are done
        gl_barrier();                               // X_g
        read_frags(g + 1, cur ^ 1);
      }
      if constexpr (NA == 2) mfma_term(cur, 1);
    }
    if constexpr (FOLD) {
      if ((g + 1) % kt_slice == 0) {
#pragma unroll
        for (int i = 0; i < RB; ++i)
#pragma unroll
          for (int j = 0; j < CB; ++j) {
            tot[i][j] += acc[i][j];
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
          }
      }
    }
  };
  gl_barrier();                                   // X_-1: tile 0 landed
  if constexpr (ROLL) {
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) fb[0][cb] = *(const bf16x8*)(smem + b_lo[cb]);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) fa[0][0][rb] = *(const bf16x8*)(smem + a_lo[rb]);
  } else {
    read_frags(0, 0);
  }
  if constexpr (ROLL) {
    // the last tile peeled off: no branch in the loop body
    for (int g = 0; g + 1 < ntot; ++g) tile_roll(g, true);
    tile_roll(ntot - 1, false);
  } else if constexpr (PIPE1) {
    for (int g = 0; g < ntot; g += 2) {           // fragment buffer parity static in the two halves
      tile_p1(g, 0, g + 1 < ntot);
      if (g + 1 < ntot) tile_p1(g + 1, 1, g + 2 < ntot);
    }
  } else {
    for (int g = 0; g < ntot; g += 2) {           // fragment buffer parity static in the two halves
      tile_body(g, 0);
      if (g + 1 < ntot) tile_body(g + 1, 1);
    }
  }

  if constexpr (PARTIAL) {
    // accumulator (rb, cb)[i]: row wm*WM + 16*rb + 4*lg + i, tile column tc[cb]
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = m0 + wm * WM + rb * 16 + lg * 4 + i;
        if (row >= a.M) continue;
        float* pr = a.part + ((size_t)z * a.M + row) * a.N;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) pr[logical_col<EPI, BN>(a, tile_n, tc[cb])] = acc[rb][cb][i];
      }
    }
    return;
  }
  // accumulator (rb, cb)[e]: row wm*WM + 16*rb + lc, tile column tb[cb] + e,
  // tb[cb] = tc[cb] - lc + 4*lg (tc evaluated at lane lc = 4*lg)
  if constexpr (EPI == EPI_QKV && MODE == 0 && SPLIT) {
    if (qkv_value_tile<BN>(a, tile_n)) {
      constexpr int KS = BM + VT_PAD;
      static_assert(BN * KS * 2 <= NST * STAGE, "the staged value tile fits the LDS stages");
      f16* vs = (f16*)smem;
      __syncthreads();   // X_v1
      // tile column c < BN / 2 is pair c (first dimension half), c + BN / 2 its partner
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int kl = wm * WM + rb * 16 + lc;
#pragma unroll
        for (int cb = 0; cb < CB / 2; ++cb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int c = tc[cb] - lc + 4 * lg + e;
            vs[(2 * c) * KS + kl] = from_f32<f16>(acc[rb][cb][e]);
            vs[(2 * c + 1) * KS + kl] = from_f32<f16>(acc[rb][cb + CB / 2][e]);
          }
      }
      __syncthreads();   // X_v2
      store_value_tile<BM, BN, 512>(a, vs, tile_n, m0, tid);
      return;
    }
    if (qkv_qk_tile<BN>(a, tile_n)) {
      constexpr int RS = BN + QK_PAD;
      static_assert(BM * RS * 2 <= NST * STAGE, "the staged query / key tile fits the LDS stages");
      f16* qs = (f16*)smem;
      const int half = a.hd / 2;
      __syncthreads();   // X_q1: every load landed, every fragment read done
      // pair c < BN / 2 of the tile: head c / half of the tile, dimensions j and j + half
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int r = wm * WM + rb * 16 + lc, row = m0 + r;
        if (row >= a.M) continue;
        const float2* cs = a.rope + (size_t)a.row_pos[row] * half;
#pragma unroll
        for (int cb = 0; cb < CB / 2; ++cb) {
          const int c = tc[cb] - lc + 4 * lg, j = c % half;
          f16* q = qs + r * RS + (c / half) * a.hd + j;
          f16x4 o1, o2;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float2 o = rope_rotate(acc[rb][cb][e], acc[rb][cb + CB / 2][e], cs[j + e]);
            o1[e] = from_f32<f16>(o.x);
            o2[e] = from_f32<f16>(o.y);
          }
          *(f16x4*)q = o1;
          *(f16x4*)(q + half) = o2;
        }
      }
      __syncthreads();   // X_q2
      store_qk_tile<BM, BN, 512>(a, qs, tile_n, m0, tid);
      return;
    }
  }
  if constexpr (EPI == EPI_STORE && !FOLD && WGN == 2) {
    // decision statistics partial (tile tile_n, wave half wn) of each row, from
    // the fp32 results (the values the logits store would write); columns
    // tb[cb] + e are stat_col(BN, wn, lg, cb, e).  All lanes take part in the
    // shuffles; rows past M (clamped loads) are computed and not written.
    if (a.tstat) {
      const int np = 2 * (a.N / BN);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int row = m0 + wm * WM + rb * 16 + lc;
        const int rowc = min(row, a.M - 1);
        const int orow = a.out_row ? a.out_row[rowc] : rowc;
        const int cur = a.tg[orow];
        float mx = -INFINITY;
        int ix = 0x7fffffff;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int col = tile_n * BN + tc[cb] - lc + 4 * lg + e;
            const float v = acc[rb][cb][e];
            if (col != a.mask_id && (v > mx || (v == mx && col < ix))) { mx = v; ix = col; }
          }
#pragma unroll
        for (int o = 16; o <= 32; o <<= 1) {
          const float m2 = __shfl_xor(mx, o, 64);
          const int i2 = __shfl_xor(ix, o, 64);
          if (m2 > mx || (m2 == mx && i2 < ix)) { mx = m2; ix = i2; }
        }
        float sum = 0.f;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int col = tile_n * BN + tc[cb] - lc + 4 * lg + e;
            const float v = acc[rb][cb][e];
            if (col != a.mask_id) sum += stat_exp(v, mx);
            if (col == cur && row < a.M) a.zg[orow] = v;
          }
        sum += __shfl_xor(sum, 16, 64);   // (s0 + s1), (s2 + s3)
        sum += __shfl_xor(sum, 32, 64);   // (s0 + s1) + (s2 + s3)
        if (lg == 0 && row < a.M) {
          const size_t pi = (size_t)orow * np + 2 * tile_n + wn;
          a.tstat[pi] = make_float2(mx, sum);
          a.targ[pi] = ix;
        }
      }
      if (!a.C) return;
    }
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = m0 + wm * WM + rb * 16 + lc;
    if (row >= a.M) continue;
    int tb[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) tb[cb] = tc[cb] - lc + 4 * lg;
    if constexpr (epi_paired(EPI)) {
#pragma unroll
      for (int cb = 0; cb < CB / 2; ++cb) {
        const f32x4 v1 = FOLD ? tot[rb % (FOLD ? RB : 1)][cb % (FOLD ? CB : 1)] : acc[rb][cb];
        const f32x4 v2 = FOLD ? tot[rb % (FOLD ? RB : 1)][(cb + CB / 2) % (FOLD ? CB : 1)] : acc[rb][cb + CB / 2];
        epi_tile_pair4<EPI, bf16, BN>(a, tile_n, tb[cb], row, v1, v2);
      }
    } else {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        const int col = tile_n * BN + tb[cb];
        const f32x4 v = FOLD ? tot[rb % (FOLD ? RB : 1)][cb % (FOLD ? CB : 1)] : acc[rb][cb];
        if constexpr (EPI == EPI_STORE) epi_store4(a, row, col, v);
        else epi_resid4(a, row, col, v);
      }
    }
  }
}


template <int BM, int BN, int WGM, int WGN, int NST, int EPI, int MODE>
void lds_mode(const GemmArgs& a, int grid, hipStream_t st) {
  if (a.f16) {
    if constexpr (EPI == EPI_SWIGLU) gemm_lds_kernel<BM, BN, WGM, WGN, NST, EPI, false, MODE, true><<<grid, 512, 0, st>>>(a);
  } else if (a.A2) {
    gemm_lds_kernel<BM, BN, WGM, WGN, NST, EPI, true, MODE><<<grid, 512, 0, st>>>(a);
  } else {
    gemm_lds_kernel<BM, BN, WGM, WGN, NST, EPI, false, MODE><<<grid, 512, 0, st>>>(a);
  }
}

template <int BM, int BN, int WGM, int WGN, int NST, int EPI>
void lds_cfg(const GemmArgs& a, bool partial, hipStream_t st) {
  const int n_tiles = a.N / BN, m_tiles = (a.M + BM - 1) / BM;
  const int grid = gemm_grid_size(n_tiles, m_tiles, partial ? a.ksplit : 1);
  if (partial) {
    lds_mode<BM, BN, WGM, WGN, NST, EPI, 2>(a, grid, st);
    launch_gemm_reduce(EPI, a, st);
  } else if (a.ksplit > 1) {
    lds_mode<BM, BN, WGM, WGN, NST, EPI, 1>(a, grid, st);
  } else {
    lds_mode<BM, BN, WGM, WGN, NST, EPI, 0>(a, grid, st);
  }
}

struct LdsCfg { int BM, BN; };
const LdsCfg kLds[GEMM_NCFG_LDS] = {
    {128, 192},   // 0: 2 x 2 multiply waves of 64 x 96, 4 stages
    {128, 128},   // 1: 2 x 2 multiply waves of 64 x 64, 4 stages
    {128, 256},   // 2: 2 x 2 multiply waves of 64 x 128, 4 stages, one K slice, two-term or fp16
};

template <int EPI>
void lds_epi(int c, const GemmArgs& a, bool partial, hipStream_t st) {
  switch (c) {
    case 0: lds_cfg<128, 192, 2, 2, 4, EPI>(a, partial, st); break;
    case 1: lds_cfg<128, 128, 2, 2, 4, EPI>(a, partial, st); break;
    default: {
      // one K slice; two-term activations (the in-place refill needs both
      // terms) or single-term fp16 ones (one fragment set of each kind)
      const int grid = gemm_grid_size(a.N / 256, (a.M + 127) / 128, 1);
      if (a.f16) {
        if constexpr (EPI == EPI_SWIGLU) gemm_lds_kernel<128, 256, 2, 2, 4, EPI, false, 0, true><<<grid, 512, 0, st>>>(a);
      } else {
        gemm_lds_kernel<128, 256, 2, 2, 4, EPI, true, 0><<<grid, 512, 0, st>>>(a);
      }
      break;
    }
  }
}

}  // namespace

int gemm_stats_bn(const GemmArgs& a) {
  // the configurations whose kernel is gemm_lds_kernel with a 2 x 2 wave grid
  const int cfg = gemm_pick_cfg(a, EPI_STORE) - GEMM_NCFG;
  if (cfg < 0 || a.ksplit != 1 || !gemm_lds_cfg_ok(cfg, a)) return 0;
  return kLds[cfg].BN;
}

bool gemm_lds_cfg_ok(int c, const GemmArgs& a) {
  if (c < 0 || c >= GEMM_NCFG_LDS) return false;
  const LdsCfg& k = kLds[c];
  if (a.M <= 0 || a.N % k.BN || a.ksplit < 1 || a.K % (a.ksplit * BK)) return false;
  if (c == 2 && ((!a.A2 && !a.f16) || a.ksplit != 1)) return false;
  // 32-bit lane offsets
  if ((size_t)a.N * (a.w_tiled ? BK : a.ldw) * 2 >= (1ull << 32) || (size_t)a.M * (a.a_tiled ? BK : a.lda) * 2 >= (1ull << 32))
    return false;
  return true;
}

int gemm_lds_tiles(int c, const GemmArgs& a) {
  const LdsCfg& k = kLds[c];
  return (a.N / k.BN) * ((a.M + k.BM - 1) / k.BM);
}

int launch_gemm_lds_cfg(int epi, int c, bool partial, const GemmArgs& a, hipStream_t st) {
  if (!gemm_args_ok(epi, a) || !gemm_lds_cfg_ok(c, a)) return 1;
  if (partial && (!a.part || a.ksplit < 2)) return 1;
  switch (epi) {
    case EPI_STORE: lds_epi<EPI_STORE>(c, a, partial, st); break;
    case EPI_RESID: lds_epi<EPI_RESID>(c, a, partial, st); break;
    case EPI_SWIGLU: lds_epi<EPI_SWIGLU>(c, a, partial, st); break;
    case EPI_QKV: lds_epi<EPI_QKV>(c, a, partial, st); break;
    default: return 1;
  }
  return 0;
}
