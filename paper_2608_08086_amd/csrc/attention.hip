// Non-causal attention of the Archer path (Eq. archer-attention): each query
// row of a sequence attends to that sequence's cached prompt keys followed by
// its fresh response keys, with no mask other than key validity.
//
// bf16-model kernel: flash-style online softmax with MFMA.  Queries, keys and
// values are fp16 (the bf16 path stores them so; see qkv_t in common.h), the
// scores S = Q K^T are fp16 MFMAs with fp32 accumulation, and P V multiplies
// the probabilities rounded to fp16 (11 significant bits: an absolute error
// of at most 2^-12 |v| in the output, whatever the key count).  The
// output is the two-term bf16 activation of the O projection.  A workgroup owns
// 16 * QB * NW query rows (256, 128 or 64) of one (sequence, query head) and
// a contiguous range of 64-key tiles; with split-KV the splits' unnormalised
// partial results are combined by attn_merge_kernel.  With 8 waves, two waves
// share each SIMD and run a ping-pong schedule: while one multiplies (scores
// of tile i and P V of tile i - 1) the other does its softmax, separated by
// one barrier per half tile.  K [64][hd] and V^T [hd][64] tiles are loaded
// straight into one of four LDS stages, two tiles ahead of the one being
// computed.  Scores are formed transposed, S^T = K Q^T, so that a lane holds
// 4 keys x 1 query per 16x16 block; the K rows of each MFMA block are
// permuted (att_key_row) so that the probabilities a lane holds for two key
// blocks are 8 consecutive keys, which is exactly the B operand of
// O^T = V^T P^T and whose V^T partner is one 16-byte LDS read.  Row
// statistics need only two lane-swap steps across the four lane groups.
#include <algorithm>

#include "launch.h"

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt immediate (gfx9 encoding) waiting until at most n vector-memory
// operations of this wave are outstanding; LGKM and export counts untouched.
#define ATT_VMCNT(n) (((n) & 15) | (7 << 4) | (15 << 8) | ((((n) >> 4) & 3) << 14))
#define ATT_LGKMCNT0 (15 | (7 << 4) | (0 << 8) | (3 << 14))

// Rescale threshold of the online softmax, in log2 units: the running maximum
// is raised (and the accumulators rescaled) when a tile's maximum exceeds it
// by more than this.  Zero is the plain online softmax (probabilities <= 1).
// A lazy threshold of 8 (probabilities below 2^8, most tiles skipping the
// rescale) computes the same softmax and was 1-5 % faster, but, measured
// when the probabilities entered P V as single bf16 values, it raised the
// largest logit error of a two-layer LLaDA-8B-shaped model from 5.8e-3 to
// 9.5e-3 at P 512: with threshold 0 the key that sets the maximum gets
// probability 2^0 = 1, which needs no rounding, while with a lazy threshold
// the dominant probabilities are arbitrary values in (1, 2^8) and carry the
// full rounding.
constexpr float ATT_RESCALE_LOG2 = 0.0f;

// LDS layout of one 64-key stage.  K: row r (key) holds HD/8 16-byte chunks,
// V^T: row d (dimension) holds 8 chunks of 8 keys.  Chunks are stored
// XOR-swizzled inside a row, physical = logical ^ swz(row), with swz chosen so
// that the 16 rows a fragment read touches fall on distinct banks.  Tiles are
// filled by direct global->LDS loads: the 16-byte slot a lane writes is fixed
// (slot = instruction base + lane), so each lane loads the global chunk that
// belongs in its slot.
// One direct global->LDS load of 16 bytes per lane from sbase + voff (sbase
// wave-uniform, voff a per-lane byte offset): lane l's bytes land at LDS byte
// address lds_base + 16 * l (lds_base wave-uniform, held in M0).
// Written as inline assembly so that the compiler's own wait insertion, which
// cannot tell the stages apart, does not drain the loads in flight; the
// kernel waits for them itself (ATT_VMCNT) before the barrier that publishes
// a stage.
// M0 is listed as clobbered; no other code of this file keeps a value in it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void att_dma16(const void* sbase, unsigned voff, unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_base)
               : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ unsigned att_lds_addr(const void* p) { return (unsigned)(uintptr_t)(lds_void*)p; }

// A pointer that is the same in every lane, moved to scalar registers (the
// direct loads take their base address there).
__device__ __forceinline__ const void* att_uniform(const void* p) {
  const uintptr_t v = (uintptr_t)p;
  const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)v);
  const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(v >> 32));
  return (const void*)(((uintptr_t)hi << 32) | lo);
}

// Four consecutive outputs of one query row as two-term bf16 (hi = bf16(v),
// lo = bf16(v - hi)), one 8-byte store per term.
__device__ __forceinline__ void att_store4(const AttnArgs& a, int row, int col, f32x4 v) {
  const size_t i = act_at(row, col, a.ldo, a.o_tiled);   // col is a multiple of 4
  bf16x4 hi, lo;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    hi[e] = (bf16)v[e];
    lo[e] = (bf16)(v[e] - (float)hi[e]);
  }
  *(bf16x4*)((bf16*)a.O + i) = hi;
  if (a.O2) *(bf16x4*)((bf16*)a.O2 + i) = lo;
}

// K stage: row = key (CPR chunks of 8 dimensions).  The score MFMA reads the
// 16 rows {b..b+3, b+8..b+11, b+16..b+19, b+24..b+27} at once (see
// att_key_row), which the swizzle spreads over all banks.
template <int CPR>
__device__ __forceinline__ int att_kswz(int row) {
  return CPR == 16 ? ((row + 4 * (row >> 4)) & 15) : (((row >> 1) + 2 * (row >> 4)) & 7);
}
// V^T stage: row = dimension (8 chunks of 8 keys); 16 consecutive rows are
// read at once.
__device__ __forceinline__ int att_vswz(int d) { return (d >> 1) & 7; }

// Instruction order of one MFMA phase of NR fragment reads from LDS, each
// feeding MPR MFMAs: four reads ahead, then MPR MFMAs per further read, so
// that the read latency is hidden (left to itself the scheduler waits for
// each read right before its first MFMA).
template <int NR, int MPR>
__device__ __forceinline__ void att_mfma_pipeline() {
  constexpr int AHEAD = 6;
  __builtin_amdgcn_sched_group_barrier(0x100, AHEAD, 0);       // DS reads
#pragma unroll
  for (int i = 0; i < NR - AHEAD; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, MPR, 0);       // MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, MPR * AHEAD, 0);
}

// Reductions over the four 16-lane groups of a wave (lanes l, l ^ 16, l ^ 32,
// l ^ 48) with the lane-swap instructions (v_permlane16_swap_b32 exchanges
// the odd 16-lane rows of one operand with the even rows of the other,
// v_permlane32_swap_b32 the upper half with the lower half): with both
// operands x, the two results hold x and its partner in every lane, so one
// max / add finishes each level, on the VALU instead of an LDS permute.  The
// sums give every lane the same bits as x + partner (fp addition commutes).
__device__ __forceinline__ float att_max_groups(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float att_sum_groups(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Key (within a 64-key tile) of row r of the score MFMA's A operand for key
// block kb.  The order makes the four scores a lane receives from blocks
// 2 ks and 2 ks + 1 the keys 32 ks + 8 lg .. 32 ks + 8 lg + 7 in order, which
// is exactly the B operand of the PV MFMA with k-step ks, and that operand's
// partner (V^T row d, the same 8 keys) is one 16-byte chunk.
__device__ __forceinline__ int att_key_row(int kb, int r) {
  return 32 * (kb >> 1) + 4 * (kb & 1) + 8 * (r >> 2) + (r & 3);
}

template <int HD, int QB, int NW>
__global__ __launch_bounds__(64 * NW, 1) void attn_bf16_kernel(SeqPlan pl, AttnArgs a) {
  constexpr int KT = 64, NST = 4;
  constexpr int NT = 64 * NW;                      // threads
  constexpr int KCPR = HD / 8;                     // K chunks per row
  constexpr int KSL = KT * KCPR, VSL = HD * (KT / 8);   // 16-byte slots per stage
  constexpr int KI = KSL / NT, VI = VSL / NT;      // load instructions per wave per stage
  constexpr int DS = HD / 32, DB = HD / 16;
  constexpr int QT = 16 * QB * NW;
  static_assert(KSL % NT == 0 && VSL % NT == 0, "whole load instructions per wave");
  __shared__ __attribute__((aligned(1024))) u32x4 Ks[NST * KSL];
  __shared__ __attribute__((aligned(1024))) u32x4 Vs[NST * VSL];
  __shared__ int simd_of[NW];

  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lg = lane >> 4, lc = lane & 15;
  // heads vary fastest in the dispatch order: workgroups are dealt to the 8
  // XCDs round-robin, so every query tile and split of a head runs on one XCD
  // and reads the head's keys and values through one L2
  const int h = blockIdx.x, gq = blockIdx.y, split = blockIdx.z;
  const int s = plan_find(pl.qt_off, pl.n, gq);
  const int nsplit = pl.nsplit[s];
  if (split >= nsplit) return;
  const int qt = gq - pl.qt_off[s];
  const int rbeg = pl.row_off[s], rend = pl.row_off[s + 1];
  const int b = pl.seq[s], P = pl.p_len[s], G = pl.G;
  const int ppad = (P + 63) & ~63;
  const int ntiles = (ppad + G + KT - 1) / KT;
  const int t0 = split * ntiles / nsplit, t1 = (split + 1) * ntiles / nsplit, nt = t1 - t0;
  const int kvh = h / (a.hq / a.hkv);

  const f16* Kc = (const f16*)a.Kc + (size_t)kvh * a.ldcache * HD;
  const f16* Vtc = (const f16*)a.Vtc + (size_t)kvh * HD * a.ldcache;
  const f16* Kf = (const f16*)a.Kf + (size_t)kvh * a.ldfresh * HD;
  const f16* Vtf = (const f16*)a.Vtf + (size_t)kvh * HD * a.ldfresh;
  const int coff = pl.cache_off[s], foff = b * G;
  const unsigned k_lds = att_lds_addr(Ks), v_lds = att_lds_addr(Vs);

  // Issue the direct loads of local tile i into stage i % NST.  Keys past the
  // segment read a clamped valid key (in bounds; K rows then give scores that
  // are masked, V chunks are zeroed after arrival).
  auto issue = [&](int i, int st) __attribute__((always_inline)) {
    const int k0 = (t0 + i) * KT;
    const bool ct = k0 < ppad;
    const int kb0 = ct ? k0 : k0 - ppad;
    const int kvalid = ct ? P : G;
    const bool part = kb0 + KT > kvalid;
    const f16* Kbase = (ct ? Kc + (size_t)coff * HD : Kf + (size_t)foff * HD) + (size_t)kb0 * HD;
    const f16* Vbase = (ct ? Vtc + coff : Vtf + foff) + kb0;
    const int vld = ct ? a.ldcache : a.ldfresh;
    const unsigned kofs = k_lds + (unsigned)(st * KSL * 16), vofs = v_lds + (unsigned)(st * VSL * 16);
#pragma unroll
    for (int j = 0; j < KI; ++j) {
      const int q = j * NT + w * 64 + lane;
      const int r = q / KCPR, pc = q % KCPR;
      const int rr = part ? min(r, kvalid - 1 - kb0) : r;
      att_dma16(att_uniform(Kbase), (unsigned)(rr * HD + (pc ^ att_kswz<KCPR>(r)) * 8) * 2, kofs + (j * NT + w * 64) * 16);
    }
#pragma unroll
    for (int j = 0; j < VI; ++j) {
      const int q = j * NT + w * 64 + lane;
      const int d = q / 8, pc = q % 8;
      const int c = pc ^ att_vswz(d);
      const int cc = part ? min(c * 8, ((kvalid - 1) & ~7) - kb0) : c * 8;
      att_dma16(att_uniform(Vbase), (unsigned)(d * vld + cc) * 2, vofs + (j * NT + w * 64) * 16);
    }
  };
  // After local tile i has landed: zero the V entries of keys past the
  // segment in the slots this lane loaded (only partial tiles have any).
  auto fix_tail = [&](int i, int st) __attribute__((always_inline)) {
    const int k0 = (t0 + i) * KT;
    const bool ct = k0 < ppad;
    const int kb0 = ct ? k0 : k0 - ppad;
    const int kvalid = ct ? P : G;
    if (kb0 + KT <= kvalid) return;
    u32x4* Vd = Vs + st * VSL;
#pragma unroll
    for (int j = 0; j < VI; ++j) {
      const int q = j * NT + w * 64 + lane;
      const int d = q / 8, pc = q % 8;
      const int c = pc ^ att_vswz(d);
      const int nv = kvalid - (kb0 + c * 8);
      if (nv < 8) {
        u32x4 v = Vd[q];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] &= (2 * e < nv ? 0xffffu : 0u) | (2 * e + 1 < nv ? 0xffff0000u : 0u);
        Vd[q] = v;
      }
    }
  };

  if (nt > 0) issue(0, 0);
  if (nt > 1) issue(1, 1);

  // Which of the two waves on this wave's SIMD it is: the first one (by wave
  // index) runs group 0, the other group 1.  Only the schedule depends on it.
  // s_getreg returns the 2-bit field SIMD_ID (bits 5:4 of HW_ID) already shifted down
  if (lane == 0) simd_of[w] = __builtin_amdgcn_s_getreg((1 << 11) | (4 << 6) | 4) & 3;

  f16x8 qf[QB][DS];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    // rows past the sequence read its last row; their outputs are never stored
    const int qrow = min(rbeg + qt * QT + w * 16 * QB + qb * 16 + lc, rend - 1);
    const f16* Qp = (const f16*)a.Q + ((size_t)h * a.ldq + qrow) * HD;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[qb][ds] = __builtin_bit_cast(f16x8, *(const u32x4*)(Qp + ds * 32 + lg * 8));
  }
  // wait for the Q fragments and the first two stages together, so that no
  // wait the compiler places for Q inside the loop drains later stages
  __builtin_amdgcn_s_waitcnt(ATT_VMCNT(0));
  __syncthreads();
  int grp = 0;
  for (int v = 0; v < w; ++v) grp += simd_of[v] == simd_of[w];
  grp = __builtin_amdgcn_readfirstlane(grp & 1);

  f32x4 o[QB][DB];
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_run[qb] = -INFINITY;
    l_run[qb] = 0.f;
#pragma unroll
    for (int i = 0; i < DB; ++i) o[qb][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  f32x4 sc[QB][4];
  // probabilities as fp16 (p <= 1; below fp16's normal range at most 2^-25
  // absolute), the B operands of O^T = V^T P^T
  f16x8 pb[2][QB];

  // S^T = K Q^T of local tile i: sc[qb][kb][e] = raw score of key kb*16 + 4*lg + e, query lc of block qb
  auto scores = [&](int st) __attribute__((always_inline)) {
    const u32x4* Kcur = Ks + st * KSL;
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kp = 0; kp < 4; kp += 2) {
      // the fragments of two key blocks are requested before the first is
      // used; the MFMAs go dimension step by dimension step over both key
      // blocks, so four independent accumulation chains are in flight
      f16x8 kf[2][DS];
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const int r = att_key_row(kp + k2, lc);
#pragma unroll
        for (int ds = 0; ds < DS; ++ds)
          kf[k2][ds] = __builtin_bit_cast(f16x8, Kcur[r * KCPR + ((ds * 4 + lg) ^ att_kswz<KCPR>(r))]);
      }
#pragma unroll
      for (int ds = 0; ds < DS; ++ds)
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            sc[qb][kp + k2] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf[k2][ds], qf[qb][ds],
                                                                      ds == 0 ? zero : sc[qb][kp + k2], 0, 0, 0);
    }
    att_mfma_pipeline<4 * DS, QB>();
  };
  // online softmax of local tile i (running maxima in log2 units); leaves the
  // fp16 probabilities in pb as the B operands of O^T = V^T P^T
  auto softmax = [&](int i) __attribute__((always_inline)) {
    const int k0 = (t0 + i) * KT;
    const bool ct = k0 < ppad;
    const int kb0 = ct ? k0 : k0 - ppad;
    const int kvalid = ct ? P : G;
    // keys past the segment (partial tiles only) get -inf, hence probability 0
    if (kb0 + KT > kvalid) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (kb0 + att_key_row(kb, 4 * lg + e) >= kvalid) sc[qb][kb][e] = -INFINITY;
    }
    bool grow = false;
    float mt[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float m = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) m = fmaxf(m, sc[qb][kb][e]);
      m = att_max_groups(m);
      mt[qb] = m * a.scale_log2;
      grow |= mt[qb] > m_run[qb] + ATT_RESCALE_LOG2;   // the query's own rule
    }
    // the branch is taken by the whole wave, but each query decides for
    // itself (alpha = 1 leaves it unchanged), so a row's result does not
    // depend on the rows sharing its wave
    if (__ballot(grow)) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const bool g = mt[qb] > m_run[qb] + ATT_RESCALE_LOG2;
        const float m_new = g ? mt[qb] : m_run[qb];
        const float alpha = g ? __builtin_amdgcn_exp2f(m_run[qb] - m_new) : 1.0f;
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[qb][db] *= alpha;
      }
    }
    // p = 2^(s * scale_log2 - m): at most 1 by the rescale rule; v_exp_f32
    // flushes results below the normal range to 0, which the sum tolerates
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float ls = 0.f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pv = __builtin_amdgcn_exp2f(fmaf(sc[qb][kb][e], a.scale_log2, -m_run[qb]));
          sc[qb][kb][e] = pv;
          ls += pv;
        }
      l_run[qb] += ls;
    }
    // scores of blocks 2 ks and 2 ks + 1 are the keys 32 ks + 8 lg + (0..7):
    // the k-slice 8 lg .. 8 lg + 7 of the PV MFMA with k-step ks
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pb[ks][qb][e] = (f16)sc[qb][2 * ks][e];
          pb[ks][qb][4 + e] = (f16)sc[qb][2 * ks + 1][e];
        }
  };
  // O^T += V^T P^T for local tile i (probabilities in pb)
  auto pv_update = [&](int st) __attribute__((always_inline)) {
    const u32x4* Vcur = Vs + st * VSL;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      // keys 32 ks + 8 lg .. + 7 of row d: logical chunk 4 ks + lg.  The
      // eight fragments of a k-step are requested before the first is used.
      f16x8 vf[DB];
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int d = db * 16 + lc;
        vf[db] = __builtin_bit_cast(f16x8, Vcur[d * 8 + ((4 * ks + lg) ^ att_vswz(d))]);
      }
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          o[qb][db] = __builtin_amdgcn_mfma_f32_16x16x32_f16(vf[db], pb[ks][qb], o[qb][db], 0, 0, 0);
        }
    }
    att_mfma_pipeline<2 * DB, QB>();
  };

  // Ping-pong schedule.  A wave's tile i is an MFMA half M(i) = [PV(i - 1);
  // S(i)] and a VALU half V(i) = softmax(i).  Iteration i has two half-steps,
  // each after a barrier: group 0 runs M(i) then V(i), group 1 runs V(i - 1)
  // then M(i), so on every SIMD one wave multiplies while the other one does
  // its softmax.  Tile j is loaded into stage j % 4 at the first half-step of
  // iteration j - 2 and must have landed before iteration j; its stage is last
  // read in the second half-step of iteration j + 1 (group 1's PV(j)).
  auto sync = [&]() __attribute__((always_inline)) {
    // a plain barrier: this wave's LDS traffic done (the fence of
    // __syncthreads would also drain the loads still in flight)
    __builtin_amdgcn_s_waitcnt(ATT_LGKMCNT0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
  };
  // iteration i uses stage st = i % NST, passed as a constant so that stage
  // offsets fold into the LDS instructions
  auto head = [&](int i, int st) __attribute__((always_inline)) {
    if (i < nt) {
      if (i + 1 < nt) __builtin_amdgcn_s_waitcnt(ATT_VMCNT(KI + VI));
      else __builtin_amdgcn_s_waitcnt(ATT_VMCNT(0));
      asm volatile("" ::: "memory");    // no LDS access moves above the wait
      fix_tail(i, st);
    }
    sync();
    if (i + 2 < nt) issue(i + 2, (st + 2) % NST);
  };
  auto mfma_half = [&](int i, int st) __attribute__((always_inline)) {
    if (i >= 1) pv_update((st + NST - 1) % NST);
    if (i < nt) scores(st);
  };
  auto iter0 = [&](int i, int st) __attribute__((always_inline)) {
    head(i, st);
    mfma_half(i, st);
    sync();
    if (i < nt) softmax(i);
  };
  auto iter1 = [&](int i, int st) __attribute__((always_inline)) {
    head(i, st);
    if (i >= 1) softmax(i - 1);
    sync();
    mfma_half(i, st);
  };
  // one loop per group (same barrier count), so that each loop carries only
  // its own registers from one iteration to the next
  static_assert(NST == 4, "the loops below are unrolled by the stage count");
  if (grp == 0) {
    for (int i = 0; i <= nt; i += 4) {
      iter0(i, 0);
      if (i + 1 <= nt) iter0(i + 1, 1);
      if (i + 2 <= nt) iter0(i + 2, 2);
      if (i + 3 <= nt) iter0(i + 3, 3);
    }
  } else {
    for (int i = 0; i <= nt; i += 4) {
      iter1(i, 0);
      if (i + 1 <= nt) iter1(i + 1, 1);
      if (i + 2 <= nt) iter1(i + 2, 2);
      if (i + 3 <= nt) iter1(i + 3, 3);
    }
  }

  // o[qb][db][e]: dimension db*16 + 4*lg + e of query lc of block qb
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    l_run[qb] = att_sum_groups(l_run[qb]);
  }
  if (nsplit == 1) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int qrow = rbeg + qt * QT + w * 16 * QB + qb * 16 + lc;
      if (qrow >= rend) continue;
      const float inv = 1.0f / l_run[qb];
#pragma unroll
      for (int db = 0; db < DB; ++db) att_store4(a, qrow, h * HD + db * 16 + lg * 4, o[qb][db] * inv);
    }
    return;
  }

  // Split-KV: publish this split's unnormalised (O, m, l); attn_merge_kernel
  // combines the splits.
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qrow = rbeg + qt * QT + w * 16 * QB + qb * 16 + lc;
    if (qrow >= rend) continue;
    const size_t base = ((size_t)split * a.hq + h) * pl.rows + qrow;
    float* op = a.Opart + base * HD;
#pragma unroll
    for (int db = 0; db < DB; ++db) *(f32x4v*)(op + db * 16 + lg * 4) = o[qb][db];
    if (lg == 0) *(float2*)(a.ML + base * 2) = make_float2(m_run[qb], l_run[qb]);
  }
}

// Merge of the split-KV partial results of the bf16 kernel, spread over the
// whole GPU: thread t of a workgroup owns 4 consecutive dimensions of one
// (query row, head); every split's partial is requested before any is used.
// Splits are combined in split order, so the result is a function of the
// row's own partials only.  Rows of sequences with one split were stored by
// the attention kernel itself.
constexpr int MERGE_ROWS = 8;
template <int HD>
__global__ __launch_bounds__(MERGE_ROWS * HD / 4) void attn_merge_kernel(SeqPlan pl, AttnArgs a) {
  constexpr int TPR = HD / 4;                       // threads per row
  const int row = blockIdx.x * MERGE_ROWS + threadIdx.x / TPR, h = blockIdx.y, d0 = (threadIdx.x % TPR) * 4;
  if (row >= pl.rows) return;
  const int s = plan_find(pl.row_off, pl.n, row);
  const int nsplit = pl.nsplit[s];
  if (nsplit == 1) return;
  float2 ml[ATTN_MAX_SPLIT];
  f32x4v part[ATTN_MAX_SPLIT];
#pragma unroll
  for (int sp = 0; sp < ATTN_MAX_SPLIT; ++sp) {
    if (sp < nsplit) {
      const size_t base = ((size_t)sp * a.hq + h) * pl.rows + row;
      ml[sp] = *(const float2*)(a.ML + base * 2);
      part[sp] = *(const f32x4v*)(a.Opart + base * HD + d0);
    }
  }
  float M = -INFINITY;
#pragma unroll
  for (int sp = 0; sp < ATTN_MAX_SPLIT; ++sp)
    if (sp < nsplit) M = fmaxf(M, ml[sp].x);
  float den = 0.f;
  f32x4v num = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int sp = 0; sp < ATTN_MAX_SPLIT; ++sp) {
    if (sp < nsplit) {
      const float wgt = exp2f(ml[sp].x - M);
      den += wgt * ml[sp].y;
      num += wgt * part[sp];
    }
  }
  att_store4(a, row, h * HD + d0, num * (1.0f / den));
}

int attn_nsplit_for_keys(int nkeys) {
  const int tiles = (nkeys + 63) / 64;
  return std::max(1, std::min(ATTN_MAX_SPLIT, (tiles + ATTN_TILES_PER_SPLIT - 1) / ATTN_TILES_PER_SPLIT));
}

bool attn_split_wanted(const int* rows, int n, int hq) {
  long wgs = 0;
  for (int s = 0; s < n; ++s) wgs += (long)((rows[s] + 255) / 256) * hq;
  return 4 * wgs < 3 * ATTN_MIN_WGS;
}

int attn_split_rows_max(int hq) { return 256 * ((ATTN_MIN_WGS + hq - 1) / hq); }

int attn_qt_bf16(const int* rows, const int* nsplit, int n, int hq) {
  for (int qt : {256, 128}) {
    long wgs = 0;
    for (int s = 0; s < n; ++s) wgs += (long)((rows[s] + qt - 1) / qt) * nsplit[s] * hq;
    if (wgs >= ATTN_MIN_WGS) return qt;
  }
  return 64;
}

template <int HD>
void attn_launch_hd(const SeqPlan& pl, const AttnArgs& a, dim3 grid, hipStream_t st) {
  if (pl.qt == 256) attn_bf16_kernel<HD, 2, 8><<<grid, 512, 0, st>>>(pl, a);
  else if (pl.qt == 128) attn_bf16_kernel<HD, 1, 8><<<grid, 512, 0, st>>>(pl, a);
  else attn_bf16_kernel<HD, 1, 4><<<grid, 256, 0, st>>>(pl, a);
  if (pl.max_split > 1)
    attn_merge_kernel<HD><<<dim3((pl.rows + MERGE_ROWS - 1) / MERGE_ROWS, a.hq), MERGE_ROWS * HD / 4, 0, st>>>(pl, a);
}

int launch_attn_bf16(const SeqPlan& pl, const AttnArgs& a, hipStream_t st) {
  const dim3 grid(a.hq, pl.qt_off[pl.n], pl.max_split);
  if (grid.y == 0) return 0;
  if (grid.y > 65535 || (pl.max_split > 1 && (!a.Opart || !a.ML))) return 1;
  if ((pl.qt != 256 && pl.qt != 128 && pl.qt != 64) || (a.hd != 128 && a.hd != 64)) return 1;
  if (a.hd == 128) attn_launch_hd<128>(pl, a, grid, st);
  else attn_launch_hd<64>(pl, a, grid, st);
  return 0;
}

// ---------------------------------------------------------------------------
// fp32 kernel: one workgroup per (query row, head); scores staged in LDS.
__global__ __launch_bounds__(128) void attn_f32_kernel(SeqPlan pl, AttnArgs a) {
  extern __shared__ float sh[];
  __shared__ float red[16];
  const int row = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, hd = a.hd;
  const int s = plan_find(pl.row_off, pl.n, row);
  const int b = pl.seq[s], P = pl.p_len[s], G = pl.G;
  const int ppad = (P + 63) & ~63, nkv = ppad + G;
  const int kvh = h / (a.hq / a.hkv);
  float* q = sh;
  float* sc = sh + hd;
  const float* Qp = (const float*)a.Q + ((size_t)h * a.ldq + row) * hd;
  for (int d = tid; d < hd; d += blockDim.x) q[d] = Qp[d];
  __syncthreads();
  const float* Kc = (const float*)a.Kc + ((size_t)kvh * a.ldcache + pl.cache_off[s]) * hd;
  const float* Kf = (const float*)a.Kf + ((size_t)kvh * a.ldfresh + b * G) * hd;
  const float scale = 1.0f / sqrtf((float)hd);
  float mloc = -INFINITY;
  for (int kv = tid; kv < nkv; kv += blockDim.x) {
    const float* kr = nullptr;
    if (kv < P) kr = Kc + (size_t)kv * hd;
    else if (kv >= ppad) kr = Kf + (size_t)(kv - ppad) * hd;
    float v = -INFINITY;
    if (kr) {
      float acc = 0.f;
      for (int d = 0; d < hd; ++d) acc = fmaf(q[d], kr[d], acc);
      v = acc * scale;
    }
    sc[kv] = v;
    mloc = fmaxf(mloc, v);
  }
  mloc = wave_max(mloc);
  __syncthreads();
  if ((tid & 63) == 0) red[tid >> 6] = mloc;
  __syncthreads();
  float M = -INFINITY;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) M = fmaxf(M, red[i]);
  float ssum = 0.f;
  for (int kv = tid; kv < nkv; kv += blockDim.x) {
    const float p = expf(sc[kv] - M);
    sc[kv] = p;
    ssum += p;
  }
  __syncthreads();
  ssum = block_sum(ssum, red + 8);
  const float* Vtc = (const float*)a.Vtc + (size_t)kvh * hd * a.ldcache + pl.cache_off[s];
  const float* Vtf = (const float*)a.Vtf + (size_t)kvh * hd * a.ldfresh + b * G;
  for (int d = tid; d < hd; d += blockDim.x) {
    float acc = 0.f;
    for (int kv = 0; kv < P; ++kv) acc = fmaf(sc[kv], Vtc[(size_t)d * a.ldcache + kv], acc);
    for (int kv = 0; kv < G; ++kv) acc = fmaf(sc[ppad + kv], Vtf[(size_t)d * a.ldfresh + kv], acc);
    ((float*)a.O)[(size_t)row * a.ldo + h * hd + d] = acc / ssum;
  }
}

int launch_attn_f32(const SeqPlan& pl, const AttnArgs& a, int max_keys, hipStream_t st) {
  const size_t shm = (size_t)(a.hd + max_keys) * sizeof(float);
  if (shm > 64 * 1024 || a.hd > 128) return 1;
  attn_f32_kernel<<<dim3(pl.rows, a.hq), 128, shm, st>>>(pl, a);
  return 0;
}
