// Non-causal attention of the Archer path (Eq. archer-attention): each query
// row of a sequence attends to that sequence's cached prompt keys followed by
// its fresh response keys, with no mask other than key validity.
//
// bf16 kernel: flash-style online softmax with MFMA.  A workgroup (4 wave64s)
// owns 64 * QB query rows of one (sequence, query head) and a contiguous
// range of 64-key tiles (split-KV over blockIdx.z; the last split to finish
// merges the partial results).  Per tile, K [64][hd] and V^T [hd][64] are
// loaded straight into one of three LDS stages, two tiles ahead of the one
// being computed.  Scores are formed transposed, S^T = K Q^T, so
// that a lane holds 4 keys x 1 query per 16x16 block; the probabilities of two
// key blocks then form exactly the B operand of O^T = V^T P^T with the key
// order permuted identically on both operands (the contraction is order-free),
// which removes any register shuffle between the two MFMA stages.  Row
// statistics need only two xor-shuffles across the four lane groups.
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
// is raised (and the accumulators rescaled) only when a tile's maximum exceeds
// it by more than this, so probabilities stay below 2^8 and most tiles skip
// the rescale.  The result is the same softmax (the final division uses the
// same reference maximum); only rounding differs.
constexpr float ATT_RESCALE_LOG2 = 8.0f;

// LDS layout of one 64-key stage.  K: row r (key) holds HD/8 16-byte chunks,
// V^T: row d (dimension) holds 8 chunks of 8 keys.  Chunks are stored
// XOR-swizzled inside a row, physical = logical ^ swz(row), with swz chosen so
// that the 16 rows a fragment read touches fall on distinct banks.  Tiles are
// filled by direct global->LDS loads: the 16-byte slot a lane writes is fixed
// (slot = instruction base + lane), so each lane loads the global chunk that
// belongs in its slot.
// One direct global->LDS load of 16 bytes per lane: lane l's bytes land at
// LDS byte address lds_base + 16 * l (lds_base wave-uniform, held in M0).
// Written as inline assembly so that the compiler's own wait insertion, which
// cannot tell the stages apart, does not drain the loads in flight; the
// kernel waits for them itself (ATT_VMCNT) before the barrier that publishes
// a stage.
// M0 is listed as clobbered; no other code of this file keeps a value in it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void att_dma16(const void* src, unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(lds_base)
               : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ unsigned att_lds_addr(const void* p) { return (unsigned)(uintptr_t)(lds_void*)p; }

// Four consecutive outputs of one query row as two-term bf16 (hi = bf16(v),
// lo = bf16(v - hi)), one 8-byte store per term.
__device__ __forceinline__ void att_store4(const AttnArgs& a, size_t i, f32x4 v) {
  bf16x4 hi, lo;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    hi[e] = (bf16)v[e];
    lo[e] = (bf16)(v[e] - (float)hi[e]);
  }
  *(bf16x4*)((bf16*)a.O + i) = hi;
  if (a.O2) *(bf16x4*)((bf16*)a.O2 + i) = lo;
}

template <int CPR>
__device__ __forceinline__ int att_swz(int row) {
  return CPR == 16 ? (row & 15) : ((row >> 1) & 7);
}

template <int HD, int QB>
__global__ __launch_bounds__(256, 1) void attn_bf16_kernel(SeqPlan pl, AttnArgs a) {
  constexpr int KT = 64, NST = 3;
  constexpr int KCPR = HD / 8;                     // K chunks per row
  constexpr int KSL = KT * KCPR, VSL = HD * (KT / 8);   // 16-byte slots per stage
  constexpr int KI = KSL / 256, VI = VSL / 256;    // load instructions per wave per stage
  constexpr int DS = HD / 32, DB = HD / 16;
  constexpr int QT = 64 * QB;
  // one LDS object per stage: the compiler can then tell a stage being read
  // from the stages still being filled and does not wait for their loads
  __shared__ __attribute__((aligned(1024))) u32x4 Ks0[KSL], Ks1[KSL], Ks2[KSL];
  __shared__ __attribute__((aligned(1024))) u32x4 Vs0[VSL], Vs1[VSL], Vs2[VSL];
  __shared__ int last_flag;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, lg = lane >> 4, lc = lane & 15;
  const int gq = blockIdx.x, h = blockIdx.y, split = blockIdx.z;
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

  const bf16* Kc = (const bf16*)a.Kc + (size_t)kvh * a.ldcache * HD;
  const bf16* Vtc = (const bf16*)a.Vtc + (size_t)kvh * HD * a.ldcache;
  const bf16* Kf = (const bf16*)a.Kf + (size_t)kvh * a.ldfresh * HD;
  const bf16* Vtf = (const bf16*)a.Vtf + (size_t)kvh * HD * a.ldfresh;
  const int coff = pl.cache_off[s], foff = b * G;

  // Issue the direct loads of local tile i into stage i % NST.  Keys past the
  // segment read a clamped valid key (in bounds; K rows then give scores that
  // are masked, V chunks are zeroed after arrival).
  const int wu = __builtin_amdgcn_readfirstlane(w);
  auto issue = [&](int i, unsigned kofs, unsigned vofs) {
    const int k0 = (t0 + i) * KT;
    const bool ct = k0 < ppad;
    const int kb0 = ct ? k0 : k0 - ppad;
    const int kvalid = ct ? P : G;
    const bf16* Kseg = ct ? Kc + (size_t)coff * HD : Kf + (size_t)foff * HD;
    const bf16* Vseg = ct ? Vtc + coff : Vtf + foff;
    const int vld = ct ? a.ldcache : a.ldfresh;
#pragma unroll
    for (int j = 0; j < KI; ++j) {
      const int q = j * 256 + w * 64 + lane;
      const int r = q / KCPR, pc = q % KCPR;
      const int key = min(kb0 + r, kvalid - 1);
      const bf16* src = Kseg + (size_t)key * HD + (pc ^ att_swz<KCPR>(r)) * 8;
      att_dma16(src, kofs + (j * 256 + wu * 64) * 16);
    }
#pragma unroll
    for (int j = 0; j < VI; ++j) {
      const int q = j * 256 + w * 64 + lane;
      const int d = q / 8, pc = q % 8;
      const int c = pc ^ att_swz<8>(d);
      const int keyc = min(kb0 + c * 8, (kvalid - 1) & ~7);
      const bf16* src = Vseg + (size_t)d * vld + keyc;
      att_dma16(src, vofs + (j * 256 + wu * 64) * 16);
    }
  };
  // After local tile i has landed: zero the V entries of keys past the
  // segment in the slots this lane loaded (only partial tiles have any).
  auto fix_tail = [&](int i, u32x4* Vd) {
    const int k0 = (t0 + i) * KT;
    const bool ct = k0 < ppad;
    const int kb0 = ct ? k0 : k0 - ppad;
    const int kvalid = ct ? P : G;
    if (kb0 + KT <= kvalid) return;
#pragma unroll
    for (int j = 0; j < VI; ++j) {
      const int q = j * 256 + w * 64 + lane;
      const int d = q / 8, pc = q % 8;
      const int c = pc ^ att_swz<8>(d);
      const int nv = kvalid - (kb0 + c * 8);
      if (nv < 8) {
        u32x4 v = Vd[q];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] &= (2 * e < nv ? 0xffffu : 0u) | (2 * e + 1 < nv ? 0xffff0000u : 0u);
        Vd[q] = v;
      }
    }
  };

  const unsigned k_ofs[NST] = {att_lds_addr(Ks0), att_lds_addr(Ks1), att_lds_addr(Ks2)};
  const unsigned v_ofs[NST] = {att_lds_addr(Vs0), att_lds_addr(Vs1), att_lds_addr(Vs2)};
  if (nt > 0) issue(0, k_ofs[0], v_ofs[0]);
  if (nt > 1) issue(1, k_ofs[1], v_ofs[1]);

  bf16x8 qf[QB][DS];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    // rows past the sequence read its last row; their outputs are never stored
    const int qrow = min(rbeg + qt * QT + w * 16 * QB + qb * 16 + lc, rend - 1);
    const bf16* Qp = (const bf16*)a.Q + ((size_t)h * a.ldq + qrow) * HD;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) qf[qb][ds] = __builtin_bit_cast(bf16x8, *(const u32x4*)(Qp + ds * 32 + lg * 8));
  }
  // the Q fragments were loaded after the first two stages were issued: wait
  // for all of them here (the stages arrive about together), so that no wait
  // the compiler places for Q inside the loop drains later stages
  __builtin_amdgcn_s_waitcnt(ATT_VMCNT(0));
  asm volatile("" ::: "memory");
  f32x4 o[QB][DB];
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_run[qb] = -INFINITY;
    l_run[qb] = 0.f;
#pragma unroll
    for (int i = 0; i < DB; ++i) o[qb][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // local tile i from stage (Kcur, Vcur); tile i + 2 goes into stage nxt,
  // the one computed at i - 1, which every wave has left at the barrier
  auto tile = [&](int i, const u32x4* Kcur, u32x4* Vcur, int nxt) {
    if (i + 1 < nt) __builtin_amdgcn_s_waitcnt(ATT_VMCNT(KI + VI));
    else __builtin_amdgcn_s_waitcnt(ATT_VMCNT(0));
    asm volatile("" ::: "memory");    // no LDS access moves above the wait
    fix_tail(i, Vcur);
    // a plain barrier: LDS traffic of this wave done (the fence of
    // __syncthreads would also drain the loads still in flight)
    __builtin_amdgcn_s_waitcnt(ATT_LGKMCNT0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (i + 2 < nt) issue(i + 2, k_ofs[nxt], v_ofs[nxt]);
    const int k0 = (t0 + i) * KT;
    const bool ct = k0 < ppad;
    const int kb0 = ct ? k0 : k0 - ppad;
    const int kvalid = ct ? P : G;

    f32x4 sc[QB][4];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) sc[qb][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const int r = kb * 16 + lc;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        const bf16x8 kf = __builtin_bit_cast(bf16x8, Kcur[r * KCPR + ((ds * 4 + lg) ^ att_swz<KCPR>(r))]);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          sc[qb][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[qb][ds], sc[qb][kb], 0, 0, 0);
      }
    }
    // sc[qb][kb][i]: raw score of key kb*16 + 4*lg + i and query lc of block qb.
    // Keys past the segment (partial tiles only) get -inf, hence probability 0.
    if (kb0 + KT > kvalid) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (kb0 + kb * 16 + lg * 4 + e >= kvalid) sc[qb][kb][e] = -INFINITY;
    }
    // running maxima are kept in log2 units (score * scale_log2)
    bool grow = false;
    float mt[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float m = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) m = fmaxf(m, sc[qb][kb][e]);
      m = fmaxf(m, __shfl_xor(m, 16, 64));
      m = fmaxf(m, __shfl_xor(m, 32, 64));
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
    // p = 2^(s * scale_log2 - m): below 2^8 by the rescale rule; v_exp_f32
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
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 pb[QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pb[qb][e] = (bf16)sc[qb][2 * ks][e];
          pb[qb][4 + e] = (bf16)sc[qb][2 * ks + 1][e];
        }
      // keys ks*32 + 4*lg + (0..3) and ks*32 + 16 + 4*lg + (0..3): half lg & 1
      // of logical chunks 4*ks + lg/2 and 4*ks + 2 + lg/2 of row d
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int d = db * 16 + lc;
        const int sw = att_swz<8>(d);
        const unsigned* rowp = (const unsigned*)&Vcur[d * 8];
        const int c0 = (4 * ks + (lg >> 1)) ^ sw, c1 = (4 * ks + 2 + (lg >> 1)) ^ sw;
        const uint2 lo = *(const uint2*)(rowp + c0 * 4 + (lg & 1) * 2);
        const uint2 hi = *(const uint2*)(rowp + c1 * 4 + (lg & 1) * 2);
        const u32x4 vv = {lo.x, lo.y, hi.x, hi.y};
        const bf16x8 vf = __builtin_bit_cast(bf16x8, vv);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          o[qb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb[qb], o[qb][db], 0, 0, 0);
      }
    }
  };
  for (int i = 0; i < nt; i += NST) {
    tile(i, Ks0, Vs0, 2);
    if (i + 1 < nt) tile(i + 1, Ks1, Vs1, 0);
    if (i + 2 < nt) tile(i + 2, Ks2, Vs2, 1);
  }

  // o[qb][db][e]: dimension db*16 + 4*lg + e of query lc of block qb
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    l_run[qb] += __shfl_xor(l_run[qb], 16, 64);
    l_run[qb] += __shfl_xor(l_run[qb], 32, 64);
  }
  if (nsplit == 1) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int qrow = rbeg + qt * QT + w * 16 * QB + qb * 16 + lc;
      if (qrow >= rend) continue;
      const size_t ob = (size_t)qrow * a.ldo + h * HD;
      const float inv = 1.0f / l_run[qb];
#pragma unroll
      for (int db = 0; db < DB; ++db) att_store4(a, ob + db * 16 + lg * 4, o[qb][db] * inv);
    }
    return;
  }

  // Split-KV: publish this split's (O, m, l); the last split of the
  // (query tile, head) to arrive merges all of them and resets the counter.
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
  __syncthreads();
  int* cnt = a.cnt + (size_t)gq * a.hq + h;
  if (tid == 0) {
    const int prev = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    last_flag = prev == nsplit - 1;
    if (last_flag) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!last_flag) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qrow = rbeg + qt * QT + w * 16 * QB + qb * 16 + lc;
    if (qrow >= rend) continue;
    float M = -INFINITY;
    for (int sp = 0; sp < nsplit; ++sp) M = fmaxf(M, a.ML[(((size_t)sp * a.hq + h) * pl.rows + qrow) * 2]);
    float den = 0.f;
    f32x4 num[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) num[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < nsplit; ++sp) {
      const size_t base = ((size_t)sp * a.hq + h) * pl.rows + qrow;
      const float2 ml = *(const float2*)(a.ML + base * 2);
      const float wgt = exp2f(ml.x - M);
      den += wgt * ml.y;
      const float* op = a.Opart + base * HD;
#pragma unroll
      for (int db = 0; db < DB; ++db) num[db] += wgt * *(const f32x4v*)(op + db * 16 + lg * 4);
    }
    const float inv = 1.0f / den;
    const size_t ob = (size_t)qrow * a.ldo + h * HD;
#pragma unroll
    for (int db = 0; db < DB; ++db) att_store4(a, ob + db * 16 + lg * 4, num[db] * inv);
  }
}

int attn_nsplit_for_keys(int nkeys) {
  const int tiles = (nkeys + 63) / 64;
  return std::max(1, std::min(ATTN_MAX_SPLIT, (tiles + ATTN_TILES_PER_SPLIT - 1) / ATTN_TILES_PER_SPLIT));
}

int launch_attn_bf16(const SeqPlan& pl, const AttnArgs& a, hipStream_t st) {
  dim3 grid(pl.qt_off[pl.n], a.hq, pl.max_split);
  if (grid.x == 0) return 0;
  if (pl.max_split > 1 && (!a.Opart || !a.ML || !a.cnt)) return 1;
  if (pl.qt != 64 && pl.qt != 128) return 1;
  const bool wide = pl.qt == 128;
  if (a.hd == 128) {
    if (wide) attn_bf16_kernel<128, 2><<<grid, 256, 0, st>>>(pl, a);
    else attn_bf16_kernel<128, 1><<<grid, 256, 0, st>>>(pl, a);
  } else if (a.hd == 64) {
    if (wide) attn_bf16_kernel<64, 2><<<grid, 256, 0, st>>>(pl, a);
    else attn_bf16_kernel<64, 1><<<grid, 256, 0, st>>>(pl, a);
  } else {
    return 1;
  }
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
