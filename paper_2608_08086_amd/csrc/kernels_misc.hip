// Row-wise kernels of the Archer path: RoPE table, embedding gather, RMSNorm,
// decision row statistics and selection, and the split-KV attention merge.
#include <algorithm>

#include "launch.h"

// ---------------------------------------------------------------------------
// RoPE table: tab[pos][j] = (cos, sin)(pos * theta^(-2j/hd)), computed in fp64.
__global__ void rope_table_kernel(float2* tab, int max_pos, int half, int hd, double theta) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)max_pos * half) return;
  const int pos = (int)(i / half), j = (int)(i % half);
  const double ang = (double)pos * pow(theta, -2.0 * (double)j / (double)hd);
  tab[i] = make_float2((float)cos(ang), (float)sin(ang));
}

void launch_rope_table(float2* tab, int max_pos, int hd, double theta, hipStream_t st) {
  const long n = (long)max_pos * (hd / 2);
  rope_table_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(tab, max_pos, hd / 2, hd, theta);
}

// ---------------------------------------------------------------------------
// Weight packing: row-major [rows][cols] -> k-block-major (32-column blocks of
// all rows one after another).  One thread per 16-byte chunk, enumerated in
// destination order so the stores are contiguous; each source row segment of
// one block is 64 contiguous bytes.
__global__ void pack_kblock_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, size_t rows,
                                   size_t cols, size_t nchunk) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nchunk; i += (size_t)gridDim.x * blockDim.x) {
    const size_t cb = i / (rows * 4), rem = i - cb * rows * 4, r = rem >> 2, q = rem & 3;
    dst[i] = src[(r * cols + cb * 32 + q * 8) / 8];
  }
}

void launch_pack_kblock(const void* src, void* dst, int rows, int cols, hipStream_t st) {
  const size_t nchunk = (size_t)rows * cols / 8;
  const size_t blocks = std::min<size_t>((nchunk + 255) / 256, 65536);
  pack_kblock_kernel<<<(unsigned)blocks, 256, 0, st>>>((const uint4*)src, (uint4*)dst, rows, cols, nchunk);
}

// ---------------------------------------------------------------------------
// Embedding gather.  One block per pass row: resolve (sequence, token,
// position, K/V destination) from the plan, copy E[token] into the fp32
// residual stream, and in a full pass record the response token as anchor g_r.
template <class T>
__global__ __launch_bounds__(256) void embed_kernel(SeqPlan pl, const T* __restrict__ emb, int d,
                                                    int V, int mask_id, const int* __restrict__ prompt,
                                                    const int* __restrict__ resp, float* __restrict__ x,
                                                    int* __restrict__ row_pos, int* __restrict__ row_dst,
                                                    int* __restrict__ g_anchor, int* __restrict__ err) {
  const int i = blockIdx.x;
  const int s = plan_find(pl.row_off, pl.n, i);
  const int j = i - pl.row_off[s];
  const int b = pl.seq[s], P = pl.p_len[s], G = pl.G;
  int tok, pos, dst;
  bool is_prompt = pl.full && j < P;
  if (is_prompt) {
    tok = prompt[pl.tok_off[s] + j];
    pos = j;
    dst = -1 - (pl.cache_off[s] + j);
  } else {
    const int r = pl.full ? j - P : j;
    tok = resp[b * G + r];
    pos = P + r;
    dst = b * G + r;
    if (pl.full && threadIdx.x == 0) g_anchor[b * G + r] = tok;
  }
  const bool bad = tok < 0 || tok >= V || (is_prompt && tok == mask_id);
  if (bad) {
    if (threadIdx.x == 0) atomicOr(err, 1);
    tok = 0;
  }
  if (threadIdx.x == 0) {
    row_pos[i] = pos;
    row_dst[i] = dst;
  }
  const T* e = emb + (size_t)tok * d;
  float* xr = x + (size_t)i * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) xr[c] = to_f32(e[c]);
}

template <class T>
void launch_embed(const SeqPlan& pl, const void* emb, int d, int V, int mask_id, const int* prompt,
                  const int* resp, float* x, int* row_pos, int* row_dst, int* g_anchor, int* err,
                  hipStream_t st) {
  embed_kernel<T><<<pl.rows, 256, 0, st>>>(pl, (const T*)emb, d, V, mask_id, prompt, resp, x, row_pos,
                                           row_dst, g_anchor, err);
}
template void launch_embed<float>(const SeqPlan&, const void*, int, int, int, const int*, const int*,
                                  float*, int*, int*, int*, int*, hipStream_t);
template void launch_embed<bf16>(const SeqPlan&, const void*, int, int, int, const int*, const int*,
                                 float*, int*, int*, int*, int*, hipStream_t);

// ---------------------------------------------------------------------------
// RMSNorm: out[r] = round_T(x[r] / sqrt(mean(x[r]^2) + eps) * gain), fp32 math.
// gather = 1 (final norm): output row ri in [0, n*G) is response row ri % G of
// pass sequence ri / G; its logits row b*G + (ri % G) is written to out_row.
template <class T>
__global__ __launch_bounds__(NORM_THREADS) void rmsnorm_kernel(SeqPlan pl, int gather, const float* __restrict__ x,
                                                      const float* __restrict__ gain, T* __restrict__ out,
                                                      T* __restrict__ out2, int ld, int tiled, int d, float eps,
                                                      int* __restrict__ out_row) {
  __shared__ float red[16];
  const int ro = blockIdx.x;
  int ri = ro;
  if (gather) {
    const int s = ro / pl.G, r = ro % pl.G;
    ri = pl.row_off[s] + (pl.full ? pl.p_len[s] : 0) + r;
    if (threadIdx.x == 0) out_row[ro] = pl.seq[s] * pl.G + r;
  }
  rms_normalize_row<T>(x + (size_t)ri * d, gain, out, out2, ro, ld, tiled, d, eps, red);
}

template <class T>
void launch_rmsnorm(const SeqPlan& pl, int gather, int nrows, const float* x, const float* gain, void* out,
                    void* out2, int ld, int tiled, int d, float eps, int* out_row, hipStream_t st) {
  rmsnorm_kernel<T><<<nrows, NORM_THREADS, 0, st>>>(pl, gather, x, gain, (T*)out, (T*)out2, ld, tiled, d, eps, out_row);
}
template void launch_rmsnorm<float>(const SeqPlan&, int, int, const float*, const float*, void*, void*, int, int,
                                    int, float, int*, hipStream_t);
template void launch_rmsnorm<bf16>(const SeqPlan&, int, int, const float*, const float*, void*, void*, int, int,
                                   int, float, int*, hipStream_t);
template void launch_rmsnorm<f16>(const SeqPlan&, int, int, const float*, const float*, void*, void*, int, int,
                                  int, float, int*, hipStream_t);

// ---------------------------------------------------------------------------
// Decision pass 1: per response row, over the non-MASK vocabulary:
//   m = max z, xhat = smallest id attaining m, s = sum exp(z - m),
//   ell = -log s (= m - lse, log top probability),
//   q = z[g] - m - log s (log probability of the current token; decided rows).
// Built from partials (stat_col in common.h).  The LM head produces them in
// its epilogue; tile_stats_kernel produces the same bits from stored logits.
// Thread (row, partial p): tile p / 2, wave half p % 2; its four lane groups'
// sums are formed one after the other and combined as the epilogue's
// xor-shuffles combine them.  Columns past V (a last partial tile) are skipped.
__global__ __launch_bounds__(256) void tile_stats_kernel(const float* __restrict__ logits, int V, int BN, int np,
                                                         int mask_id, const int* __restrict__ g, int rows,
                                                         float2* __restrict__ tstat, int* __restrict__ targ,
                                                         float* __restrict__ zg) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)rows * np) return;
  const int row = (int)(idx / np), p = (int)(idx % np);
  const int c0 = (p >> 1) * BN, h = p & 1, CB = BN / 32;
  const float* z = logits + (size_t)row * V;
  const int cur = g[row];
  float mx = -INFINITY;
  int ix = 0x7fffffff;
  for (int lg = 0; lg < 4; ++lg)
    for (int cb = 0; cb < CB; ++cb)
      for (int e = 0; e < 4; ++e) {
        const int col = c0 + stat_col(BN, h, lg, cb, e);
        if (col >= V || col == mask_id) continue;
        const float v = z[col];
        if (v > mx || (v == mx && col < ix)) { mx = v; ix = col; }
      }
  float sl[4];
  for (int lg = 0; lg < 4; ++lg) {
    float sum = 0.f;
    for (int cb = 0; cb < CB; ++cb)
      for (int e = 0; e < 4; ++e) {
        const int col = c0 + stat_col(BN, h, lg, cb, e);
        if (col >= V) continue;
        const float v = z[col];
        if (col != mask_id) sum += stat_exp(v, mx);
        if (col == cur) zg[row] = v;
      }
    sl[lg] = sum;
  }
  tstat[(size_t)row * np + p] = make_float2(mx, (sl[0] + sl[1]) + (sl[2] + sl[3]));
  targ[(size_t)row * np + p] = ix;
}

void launch_tile_stats(int rows, const float* logits, int V, int BN, int np, int mask_id, const int* g,
                       float2* tstat, int* targ, float* zg, hipStream_t st) {
  const long n = (long)rows * np;
  tile_stats_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(logits, V, BN, np, mask_id, g, rows, tstat, targ,
                                                                 zg);
}

// Merge of a row's partials, one wave per row: lane l takes partials
// l, l + 64, ... in order; M and xhat are order-free (max; smallest column at
// the max), the sum s = sum_p s_p exp(m_p - M) runs per lane in partial
// order and then over a fixed xor tree, read from lane 0.
constexpr int FS_ROWS = 4;   // rows (waves) per block
__global__ __launch_bounds__(64 * FS_ROWS) void finalize_stats_kernel(const float2* __restrict__ tstat,
                                                                      const int* __restrict__ targ,
                                                                      const float* __restrict__ zg,
                                                                      const int* __restrict__ g, int np, int V,
                                                                      int mask_id, int rows, int* __restrict__ xhat,
                                                                      float* __restrict__ ell,
                                                                      float* __restrict__ qv) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * FS_ROWS + (threadIdx.x >> 6);
  if (row >= rows) return;
  const float2* ts = tstat + (size_t)row * np;
  const int* ta = targ + (size_t)row * np;
  float m = -INFINITY;
  for (int p = lane; p < np; p += 64) m = fmaxf(m, ts[p].x);
  const float M = wave_max(m);
  int id = 0x7fffffff;
  float s = 0.f;
  for (int p = lane; p < np; p += 64) {
    const float2 t = ts[p];
    if (t.x == M) id = min(id, ta[p]);
    if (t.y > 0.f) s += t.y * stat_exp(t.x, M);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    id = min(id, __shfl_xor(id, o, 64));
    s += __shfl_xor(s, o, 64);
  }
  if (lane == 0) {
    const float logs = logf(s);
    xhat[row] = id;
    ell[row] = -logs;
    const int cur = g[row];
    qv[row] = (cur != mask_id && cur >= 0 && cur < V) ? (zg[row] - M) - logs : 0.f;
  }
}

void launch_finalize_stats(int rows, int np, const float2* tstat, const int* targ, const float* zg, const int* g,
                           int V, int mask_id, int* xhat, float* ell, float* qv, hipStream_t st) {
  finalize_stats_kernel<<<(unsigned)((rows + FS_ROWS - 1) / FS_ROWS), 64 * FS_ROWS, 0, st>>>(
      tstat, targ, zg, g, np, V, mask_id, rows, xhat, ell, qv);
}

// ---------------------------------------------------------------------------
// Decision pass 2 (one block per sequence): unmask the top-k masked rows by
// ell (ties: smaller position) to xhat, remask the decided row of smallest q
// (ties: smaller position) when q < log(tau), then D = d_H(g_out, g_anchor).
__global__ __launch_bounds__(512) void select_kernel(const int* __restrict__ g_in, int* __restrict__ g_out,
                                                     const int* __restrict__ g_anchor,
                                                     const int* __restrict__ xhat, const float* __restrict__ ell,
                                                     const float* __restrict__ qv, int G, int mask_id, int k,
                                                     float log_tau, int max_remask, int final_step,
                                                     int* __restrict__ dist, int* __restrict__ unmask_pos,
                                                     int* __restrict__ remask_pos, int* __restrict__ tr_dist,
                                                     int* __restrict__ tr_unmask, int* __restrict__ tr_utok,
                                                     int* __restrict__ tr_remask) {
  extern __shared__ float4 smem_raw4[];
  // key[i] = ell[i] for masked rows, -inf for decided rows (which then never
  // outrank a masked row: ell = -log sum exp(z - max) is finite)
  float* skey = (float*)smem_raw4;              // [G], G % 4 == 0
  int* ssel = (int*)(skey + G);                 // [G]
  __shared__ float rq[512];
  __shared__ int ri[512];
  __shared__ int rcnt[512];
  __shared__ int wcnt[8];
  const int b = blockIdx.x;
  const int* gi = g_in + (size_t)b * G;
  for (int i = threadIdx.x; i < G; i += blockDim.x)
    skey[i] = gi[i] == mask_id ? ell[(size_t)b * G + i] : -INFINITY;
  __syncthreads();
  // unmask selection by rank among the masked rows (ties: smaller position)
  for (int i = threadIdx.x; i < G; i += blockDim.x) {
    int sel = 0;
    const float ei = skey[i];
    if (gi[i] == mask_id) {
      if (final_step) {
        sel = 1;
      } else {
        int rank = 0;
        const float4* k4 = (const float4*)skey;
#pragma unroll 4
        for (int j4 = 0; j4 < G / 4; ++j4) {
          const float4 kk = k4[j4];
          const int j = 4 * j4;
          rank += (kk.x > ei || (kk.x == ei && j + 0 < i)) + (kk.y > ei || (kk.y == ei && j + 1 < i)) +
                  (kk.z > ei || (kk.z == ei && j + 2 < i)) + (kk.w > ei || (kk.w == ei && j + 3 < i));
        }
        sel = rank < k;
      }
    }
    ssel[i] = sel;
  }
  // remask candidate: argmin (q, position) over decided rows
  float bq = INFINITY;
  int bi = 0x7fffffff;
  for (int i = threadIdx.x; i < G; i += blockDim.x) {
    if (gi[i] != mask_id) {
      const float q = qv[(size_t)b * G + i];
      if (q < bq || (q == bq && i < bi)) { bq = q; bi = i; }
    }
  }
  rq[threadIdx.x] = bq;
  ri[threadIdx.x] = bi;
  __syncthreads();
  for (int w = blockDim.x / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) {
      const float q2 = rq[threadIdx.x + w];
      const int i2 = ri[threadIdx.x + w];
      if (q2 < rq[threadIdx.x] || (q2 == rq[threadIdx.x] && i2 < ri[threadIdx.x])) {
        rq[threadIdx.x] = q2;
        ri[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  const int rm = (!final_step && max_remask > 0 && ri[0] < G && rq[0] < log_tau) ? ri[0] : -1;
  // write g_out, count the distance to the anchor, list the unmasked
  // positions in ascending order (position among the selected rows by a
  // ballot scan over blocks of blockDim rows)
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
  const bool list = unmask_pos || tr_unmask || tr_utok;
  int cnt = 0, nsel = 0;
  for (int i0 = 0; i0 < G; i0 += blockDim.x) {
    const int i = i0 + threadIdx.x;
    const int f = i < G ? ssel[i] : 0;
    const unsigned long long bal = __ballot(f);
    if (lane == 0) wcnt[wv] = __popcll(bal);
    __syncthreads();
    int before = nsel, total = nsel;
    for (int w = 0; w < nw; ++w) {
      if (w < wv) before += wcnt[w];
      total += wcnt[w];
    }
    if (i < G) {
      int v = gi[i];
      if (f) v = xhat[(size_t)b * G + i];
      if (i == rm) v = mask_id;
      g_out[(size_t)b * G + i] = v;
      cnt += v != g_anchor[(size_t)b * G + i];
      const int order = before + __popcll(bal & ((1ull << lane) - 1));
      if (f && list && order < k) {
        if (unmask_pos) unmask_pos[(size_t)b * k + order] = i;
        if (tr_unmask) tr_unmask[(size_t)b * k + order] = i;
        if (tr_utok) tr_utok[(size_t)b * k + order] = v;
      }
    }
    nsel = total;
    __syncthreads();
  }
  rcnt[threadIdx.x] = cnt;
  __syncthreads();
  for (int w = blockDim.x / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) rcnt[threadIdx.x] += rcnt[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    for (int o = nsel; o < k; ++o) {
      if (unmask_pos) unmask_pos[(size_t)b * k + o] = -1;
      if (tr_unmask) tr_unmask[(size_t)b * k + o] = -1;
      if (tr_utok) tr_utok[(size_t)b * k + o] = -1;
    }
    if (dist) dist[b] = rcnt[0];
    if (tr_dist) tr_dist[b] = rcnt[0];
    if (remask_pos) remask_pos[b] = rm;
    if (tr_remask) tr_remask[b] = rm;
  }
}

void launch_select(int B, const int* g_in, int* g_out, const int* g_anchor, const int* xhat, const float* ell,
                   const float* qv, int G, int mask_id, int k, float log_tau, int max_remask, int final_step,
                   int* dist, int* unmask_pos, int* remask_pos, int* tr_dist, int* tr_unmask, int* tr_utok,
                   int* tr_remask, hipStream_t st) {
  const size_t shm = (size_t)G * 8;
  select_kernel<<<B, 512, shm, st>>>(g_in, g_out, g_anchor, xhat, ell, qv, G, mask_id, k, log_tau, max_remask,
                                     final_step, dist, unmask_pos, remask_pos, tr_dist, tr_unmask, tr_utok,
                                     tr_remask);
}

// ---------------------------------------------------------------------------
// Split-KV merge: O[row][h*hd + d] = sum_s w_s O_s / sum_s w_s l_s with
// w_s = 2^(m_s - max_s m_s); partials are unnormalised, m in log2 units.
// Rows of sequences attended in one split were written directly and are skipped.
__global__ void fill_i32_kernel(int* p, int v, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

void launch_fill_i32(int* p, int v, size_t n, hipStream_t st) {
  if (n == 0) return;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 1024);
  fill_i32_kernel<<<blocks, 256, 0, st>>>(p, v, n);
}

// ---------------------------------------------------------------------------
// Small copies of the session and state-read calls.
//
// Two rows of n <= ARCHER_MAXB ints passed by value (per-sequence trace rows of
// a session step); a null destination is skipped.
// Response rows of a FullForward pass moved into the row layout of a
// CachedForward pass (row s G + i of selected sequence s): the residual row
// (d floats) and the query row of every head (Q [hq][ldq][hd], qbytes bytes
// per row).  The last layer of a full pass needs nothing else of its prompt
// rows once their keys and values are in the cache, so it continues on the
// response rows only.
__global__ __launch_bounds__(256) void gather_resp_rows_kernel(SeqPlan pl, const float* __restrict__ x,
                                                               float* __restrict__ xc, int d,
                                                               const char* __restrict__ Q, char* __restrict__ Qc,
                                                               int ldq, int ldqc, int hq, int qbytes) {
  const int r = blockIdx.x, s = r / pl.G, i = r % pl.G;
  const int src = pl.row_off[s] + pl.p_len[s] + i;
  const float4* xs = (const float4*)(x + (size_t)src * d);
  float4* xd = (float4*)(xc + (size_t)r * d);
  for (int k = threadIdx.x; k < d / 4; k += blockDim.x) xd[k] = xs[k];
  const int nq = qbytes / 16;
  for (int k = threadIdx.x; k < hq * nq; k += blockDim.x) {
    const int h = k / nq, c = k % nq;
    ((uint4*)(Qc + ((size_t)h * ldqc + r) * qbytes))[c] = ((const uint4*)(Q + ((size_t)h * ldq + src) * qbytes))[c];
  }
}

void launch_gather_resp_rows(const SeqPlan& pl, const float* x, float* xc, int d, const void* Q, void* Qc, int ldq,
                             int ldqc, int hq, int qbytes, hipStream_t st) {
  const int n = pl.n * pl.G;
  if (n > 0)
    gather_resp_rows_kernel<<<n, 256, 0, st>>>(pl, x, xc, d, (const char*)Q, (char*)Qc, ldq, ldqc, hq, qbytes);
}

__global__ void store_rows_kernel(int* a, int* b, I32Row va, I32Row vb, int n) {
  const int i = threadIdx.x;
  if (i < n) {
    if (a) a[i] = va.v[i];
    if (b) b[i] = vb.v[i];
  }
}

void launch_store_rows(int* a, int* b, const I32Row& va, const I32Row& vb, int n, hipStream_t st) {
  if (n < 1 || (!a && !b)) return;
  store_rows_kernel<<<1, ARCHER_MAXB, 0, st>>>(a, b, va, vb, n);
}

// Prompt K / V of one sequence out of one layer of the cache: K rows
// [off, off + P) of every head plane [Hkv][ld][hd] and the same key columns of
// V^T [Hkv][hd][ld], both written as [Hkv][P][hd].
template <class T>
__global__ void read_cache_kernel(const T* __restrict__ K, const T* __restrict__ Vt, int ld, int off, int P,
                                  int hkv, int hd, T* __restrict__ Kd, T* __restrict__ Vd) {
  const size_t n = (size_t)hkv * P * hd;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int e = (int)(i % hd);
    const size_t r = i / hd;
    const int p = (int)(r % P), h = (int)(r / P);
    if (Kd) Kd[i] = K[((size_t)h * ld + off + p) * hd + e];
    if (Vd) Vd[i] = Vt[((size_t)h * hd + e) * ld + off + p];
  }
}

template <class T>
void launch_read_cache(const void* K, const void* Vt, int ld, int off, int P, int hkv, int hd, void* Kd, void* Vd,
                       hipStream_t st) {
  const size_t n = (size_t)hkv * P * hd;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 4096);
  read_cache_kernel<T><<<blocks, 256, 0, st>>>((const T*)K, (const T*)Vt, ld, off, P, hkv, hd, (T*)Kd, (T*)Vd);
}
template void launch_read_cache<float>(const void*, const void*, int, int, int, int, int, void*, void*, hipStream_t);
template void launch_read_cache<f16>(const void*, const void*, int, int, int, int, int, void*, void*, hipStream_t);

// Activation rows (hi and optional lo term, layout act_at(row, k, ld, tiled))
// -> fp32 row-major [n][d] holding hi + lo.  The sum is exact in fp32: lo is
// the bf16 rounding of v - hi, at most 16 significant bits below hi's leading one.
template <class T>
__global__ void read_act_kernel(const T* __restrict__ hi, const T* __restrict__ lo, int n, int d, int ld, int tiled,
                                float* __restrict__ out) {
  const size_t tot = (size_t)n * d;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < tot; i += (size_t)gridDim.x * blockDim.x) {
    const int r = (int)(i / d), k = (int)(i % d);
    const size_t j = act_at(r, k, ld, tiled);
    out[i] = to_f32(hi[j]) + (lo ? to_f32(lo[j]) : 0.f);
  }
}

template <class T>
void launch_read_act(const void* hi, const void* lo, int n, int d, int ld, int tiled, float* out, hipStream_t st) {
  const size_t tot = (size_t)n * d;
  if (tot == 0) return;
  const int blocks = (int)std::min<size_t>((tot + 255) / 256, 4096);
  read_act_kernel<T><<<blocks, 256, 0, st>>>((const T*)hi, (const T*)lo, n, d, ld, tiled, out);
}
template void launch_read_act<float>(const void*, const void*, int, int, int, int, float*, hipStream_t);
template void launch_read_act<bf16>(const void*, const void*, int, int, int, int, float*, hipStream_t);
