// Non-causal attention of the Archer path (Eq. archer-attention): each query
// row of a sequence attends to that sequence's cached prompt keys followed by
// its fresh response keys, with no mask other than key validity.
//
// bf16 kernel: flash-style online softmax with MFMA.  A workgroup (4 wave64s)
// owns 64 query rows of one (sequence, query head) and a contiguous range of
// 64-key tiles (split-KV over blockIdx.z).  Per tile, K [64][hd] and V^T
// [hd][64] are staged in LDS.  Scores are formed transposed, S^T = K Q^T, so
// that a lane holds 4 keys x 1 query per 16x16 block; the probabilities of two
// key blocks then form exactly the B operand of O^T = V^T P^T with the key
// order permuted identically on both operands (the contraction is order-free),
// which removes any register shuffle between the two MFMA stages.  Row
// statistics need only two xor-shuffles across the four lane groups.
#include <algorithm>

#include "launch.h"

template <int HD>
__global__ __launch_bounds__(256) void attn_bf16_kernel(SeqPlan pl, AttnArgs a) {
  constexpr int KT = 64, LDK = HD + 8, LDV = KT + 8;
  constexpr int DS = HD / 32, DB = HD / 16;
  constexpr int KCH = KT * HD / 8 / 256, VCH = HD * KT / 8 / 256;
  __shared__ __attribute__((aligned(16))) bf16 Ks[KT * LDK];
  __shared__ __attribute__((aligned(16))) bf16 Vs[HD * LDV];

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
  const int t0 = split * ntiles / nsplit, t1 = (split + 1) * ntiles / nsplit;
  const int kvh = h / (a.hq / a.hkv);
  const int qrow = rbeg + qt * ATTN_QT_BF16 + w * 16 + lc;
  const bool qval = qrow < rend;

  bf16x8 qf[DS];
  {
    const bf16* Qp = (const bf16*)a.Q + ((size_t)h * a.ldq + (qval ? qrow : rbeg)) * HD;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      const uint4 v = qval ? *(const uint4*)(Qp + ds * 32 + lg * 8) : make_uint4(0, 0, 0, 0);
      qf[ds] = *(const bf16x8*)&v;
    }
  }
  f32x4 o[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const bf16* Kc = (const bf16*)a.Kc + (size_t)kvh * a.ldcache * HD;
  const bf16* Vtc = (const bf16*)a.Vtc + (size_t)kvh * HD * a.ldcache;
  const bf16* Kf = (const bf16*)a.Kf + (size_t)kvh * a.ldfresh * HD;
  const bf16* Vtf = (const bf16*)a.Vtf + (size_t)kvh * HD * a.ldfresh;
  const int coff = pl.cache_off[s], foff = b * G;

  for (int t = t0; t < t1; ++t) {
    const int k0 = t * KT;
    const bool ct = k0 < ppad;
    const int kb0 = ct ? k0 : k0 - ppad;     // first key of the tile within its segment
    const int kvalid = ct ? P : G;           // keys of the segment that exist
    const bf16* Kseg = ct ? Kc + (size_t)coff * HD : Kf + (size_t)foff * HD;
    const bf16* Vseg = ct ? Vtc + coff : Vtf + foff;
    const int vld = ct ? a.ldcache : a.ldfresh;
#pragma unroll
    for (int j = 0; j < KCH; ++j) {
      const int c = tid + 256 * j, r = c / (HD / 8), dc = (c % (HD / 8)) * 8;
      const int key = kb0 + r;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (key < kvalid) v = *(const uint4*)(Kseg + (size_t)key * HD + dc);
      *(uint4*)&Ks[r * LDK + dc] = v;
    }
#pragma unroll
    for (int j = 0; j < VCH; ++j) {
      const int c = tid + 256 * j, d = c / (KT / 8), kc = (c % (KT / 8)) * 8;
      const int key = kb0 + kc;
      const int nv = min(max(kvalid - key, 0), 8);
      const bf16* src = Vseg + (size_t)d * vld + key;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (nv == 8) {
        v = *(const uint4*)src;
      } else if (nv > 0) {
        bf16 tmp[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) tmp[e] = e < nv ? src[e] : (bf16)0.f;
        v = *(const uint4*)tmp;
      }
      *(uint4*)&Vs[d * LDV + kc] = v;
    }
    __syncthreads();

    f32x4 sc[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      sc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        const bf16x8 kf = *(const bf16x8*)&Ks[(kb * 16 + lc) * LDK + ds * 32 + lg * 8];
        sc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ds], sc[kb], 0, 0, 0);
      }
    }
    // sc[kb][i]: key kb*16 + 4*lg + i of the tile, query lc of this wave
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ok = kb0 + kb * 16 + lg * 4 + i < kvalid;
        const float v = ok ? sc[kb][i] * a.scale_log2 : -INFINITY;
        sc[kb][i] = v;
        mt = fmaxf(mt, v);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = exp2f(m_run - m_new);
    float ls = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = exp2f(sc[kb][i] - m_new);
        sc[kb][i] = p;
        ls += p;
      }
    l_run = l_run * alpha + ls;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] *= alpha;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 pb;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pb[i] = (bf16)sc[2 * ks][i];
        pb[4 + i] = (bf16)sc[2 * ks + 1][i];
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const bf16* vr = &Vs[(db * 16 + lc) * LDV + ks * 32 + lg * 4];
        const bf16x4 lo = *(const bf16x4*)vr;
        const bf16x4 hi = *(const bf16x4*)(vr + 16);
        const bf16x8 vf = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb, o[db], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  float l = l_run;
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (!qval) return;
  // o[db][i]: dimension db*16 + 4*lg + i of query lc
  if (nsplit == 1) {
    const size_t ob = (size_t)qrow * a.ldo + h * HD;
    const float inv = 1.0f / l;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        store_act<bf16>((bf16*)a.O, (bf16*)a.O2, ob + db * 16 + lg * 4 + i, o[db][i] * inv);
  } else {
    const size_t base = ((size_t)split * a.hq + h) * pl.rows + qrow;
    float* op = a.Opart + base * HD;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) op[db * 16 + lg * 4 + i] = o[db][i];
    if (lg == 0) {
      a.ML[base * 2] = m_run;
      a.ML[base * 2 + 1] = l;
    }
  }
}

int attn_nsplit_for_keys(int nkeys) {
  const int tiles = (nkeys + 63) / 64;
  return std::max(1, std::min(8, (tiles + 3) / 4));
}

int launch_attn_bf16(const SeqPlan& pl, const AttnArgs& a, hipStream_t st) {
  dim3 grid(pl.qt_off[pl.n], a.hq, pl.max_split);
  if (grid.x == 0) return 0;
  if (a.hd == 128) attn_bf16_kernel<128><<<grid, 256, 0, st>>>(pl, a);
  else if (a.hd == 64) attn_bf16_kernel<64><<<grid, 256, 0, st>>>(pl, a);
  else return 1;
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
