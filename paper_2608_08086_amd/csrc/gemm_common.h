// Shared pieces of the bf16 / fp32 projection GEMMs: weight-row gathering for
// paired epilogues, the fused epilogues, and the XCD-aware tile order.
//
// Column pairing.  RoPE rotates dimension j with j + hd/2 of a head, SwiGLU
// multiplies gate feature f with up feature f.  The B tile rows (weight rows)
// are gathered so that tile column r and r + BN/2 form such a pair:
//   QKV:    pair p = tile * BN/2 + c (c < BN/2) is (head p / (hd/2), dim
//           j = p mod (hd/2)); its columns are head*hd + j and head*hd + hd/2 + j
//           (q, k and v heads alike);
//   SWIGLU: gate row f and up row f, f = tile * BN/2 + c.
#pragma once

#include "launch.h"

namespace {

// weight row of tile column r; *second = the row is in W2 (SWIGLU up rows)
template <int EPI, int BN>
__device__ __forceinline__ int brow_index(const GemmArgs& a, int tile_n, int r, bool* second) {
  *second = false;
  if constexpr (EPI == EPI_SWIGLU) {
    const int f0 = tile_n * (BN / 2);
    if (r < BN / 2) return f0 + r;
    *second = true;
    return f0 + r - BN / 2;
  } else if constexpr (EPI == EPI_QKV) {
    // rotation pairs are numbered across heads: pair p = (head, j), j < hd/2
    const int half = a.hd / 2;
    const int p = tile_n * (BN / 2) + (r < BN / 2 ? r : r - BN / 2);
    return (p / half) * a.hd + (r < BN / 2 ? 0 : half) + p % half;
  } else {
    return tile_n * BN + r;
  }
}

// ---- epilogues on logical (global) columns ----------------------------------
__device__ __forceinline__ void epi_store(const GemmArgs& a, int row, int col, float v) {
  const int orow = a.out_row ? a.out_row[row] : row;
  a.C[(size_t)orow * a.ldc + col] = v;
}

__device__ __forceinline__ void epi_resid(const GemmArgs& a, int row, int col, float v) {
  a.X[(size_t)row * a.ldx + col] += v;
}

// SiLU(g) * u with the hardware exponential and reciprocal (v_exp_f32,
// v_rcp_f32): a few ulp in fp32, far below the two-term bf16 rounding of the
// stored product, for a fraction of the instructions of the IEEE-exact forms;
// the denominator is >= 1 (and rcp(inf) = 0 gives the limit for large -g)
__device__ __forceinline__ float silu_times(float g, float u) {
  const float s = g * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
  return s * u;
}

template <class T>
__device__ __forceinline__ void epi_swiglu(const GemmArgs& a, int row, int f, float g, float u) {
  store_act<T>((T*)a.H, (T*)a.H2, act_at(row, f, a.ldh, a.h_tiled), silu_times(g, u));
}

// RoPE of one (first-half, second-half) dimension pair by (cos, sin); the
// single definition used by every epilogue that rotates q/k.
__device__ __forceinline__ float2 rope_rotate(float v1, float v2, float2 cs) {
  return make_float2(v1 * cs.x - v2 * cs.y, v2 * cs.x + v1 * cs.y);
}

// head in [0, hq + 2 hkv): q heads, k heads, v heads; v1 / v2 = dims j, j + hd/2
// (q, k and v are stored as qkv_t<T>)
template <class T>
__device__ __forceinline__ void epi_qkv(const GemmArgs& a, int row, int head, int j, float v1, float v2) {
  using Q = qkv_t<T>;
  const int hd = a.hd;
  const int dst = a.row_dst[row];
  if (head < a.hq + a.hkv) {
    const float2 o = rope_rotate(v1, v2, a.rope[(size_t)a.row_pos[row] * (hd / 2) + j]);
    const float o1 = o.x, o2 = o.y;
    Q* p;
    if (head < a.hq) p = (Q*)a.Qb + ((size_t)head * a.ldq + row) * hd;
    else if (dst_is_fresh(dst)) p = (Q*)a.Kf + ((size_t)(head - a.hq) * a.ldfresh + dst) * hd;
    else p = (Q*)a.Kc + ((size_t)(head - a.hq) * a.ldcache + dst_cache_row(dst)) * hd;
    p[j] = from_f32<Q>(o1);
    p[j + hd / 2] = from_f32<Q>(o2);
  } else {
    const int vh = head - a.hq - a.hkv;
    Q* vt;
    int ld, col;
    if (dst_is_fresh(dst)) { vt = (Q*)a.Vtf; ld = a.ldfresh; col = dst; }
    else { vt = (Q*)a.Vtc; ld = a.ldcache; col = dst_cache_row(dst); }
    vt[((size_t)vh * hd + j) * ld + col] = from_f32<Q>(v1);
    vt[((size_t)vh * hd + j + hd / 2) * ld + col] = from_f32<Q>(v2);
  }
}

constexpr bool epi_paired(int epi) { return epi == EPI_SWIGLU || epi == EPI_QKV; }

// Fused epilogue of one pair of tile columns (r, r + BN/2) or single column r.
template <int EPI, class T, int BN>
__device__ __forceinline__ void epi_tile_pair(const GemmArgs& a, int tile_n, int r, int row, float v1, float v2) {
  if constexpr (EPI == EPI_SWIGLU) {
    epi_swiglu<T>(a, row, tile_n * (BN / 2) + r, v1, v2);
  } else if constexpr (EPI == EPI_QKV) {
    const int half = a.hd / 2, p = tile_n * (BN / 2) + r;
    epi_qkv<T>(a, row, p / half, p % half, v1, v2);
  }
}

// Epilogues of four consecutive tile columns r .. r + 3 of one row (r a
// multiple of 4, so the four outputs are consecutive columns in every map
// below): the same values as four single-column calls, written with vector
// stores where the destination is aligned for them.
__device__ __forceinline__ void epi_store4(const GemmArgs& a, int row, int col, f32x4 v) {
  const int orow = a.out_row ? a.out_row[row] : row;
  float* p = a.C + (size_t)orow * a.ldc + col;
  if (((a.ldc & 3) | ((uintptr_t)a.C & 15)) == 0) {
    *(f32x4*)p = v;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) p[e] = v[e];
  }
}

__device__ __forceinline__ void epi_resid4(const GemmArgs& a, int row, int col, f32x4 v) {
  float* p = a.X + (size_t)row * a.ldx + col;
  if (((a.ldx & 3) | ((uintptr_t)a.X & 15)) == 0) {
    *(f32x4*)p += v;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) p[e] += v[e];
  }
}

template <int EPI, class T, int BN>
__device__ __forceinline__ void epi_tile_pair4(const GemmArgs& a, int tile_n, int r, int row, f32x4 v1, f32x4 v2) {
  if constexpr (EPI == EPI_SWIGLU) {
    const int f = tile_n * (BN / 2) + r;
    const bool vec = sizeof(T) == 2 && ((a.h_tiled ? 0 : (a.ldh & 3)) | ((uintptr_t)a.H & 7) |
                                        ((uintptr_t)a.H2 & 7)) == 0;
    if (vec) {
      float s[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) s[e] = silu_times(v1[e], v2[e]);
      store_act4<T>((T*)a.H, (T*)a.H2, act_at(row, f, a.ldh, a.h_tiled), s[0], s[1], s[2], s[3]);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) epi_swiglu<T>(a, row, f + e, v1[e], v2[e]);
    }
  } else if constexpr (EPI == EPI_QKV && sizeof(T) == 2) {
    // four consecutive rotation pairs j .. j + 3 of one head (r and hd / 2 are
    // multiples of 4): q / k halves as one 8-byte store each, v as four
    // transposed element stores per half; the values of epi_qkv
    using Q = qkv_t<T>;
    const int half = a.hd / 2, p0 = tile_n * (BN / 2) + r;
    const int head = p0 / half, j = p0 % half;
    const int dst = a.row_dst[row];
    if (head < a.hq + a.hkv) {
      const float2* cs = a.rope + (size_t)a.row_pos[row] * half + j;
      Q* p;
      if (head < a.hq) p = (Q*)a.Qb + ((size_t)head * a.ldq + row) * a.hd;
      else if (dst_is_fresh(dst)) p = (Q*)a.Kf + ((size_t)(head - a.hq) * a.ldfresh + dst) * a.hd;
      else p = (Q*)a.Kc + ((size_t)(head - a.hq) * a.ldcache + dst_cache_row(dst)) * a.hd;
      f16x4 o1, o2;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float2 o = rope_rotate(v1[e], v2[e], cs[e]);
        o1[e] = from_f32<Q>(o.x);
        o2[e] = from_f32<Q>(o.y);
      }
      *(f16x4*)(p + j) = o1;
      *(f16x4*)(p + j + half) = o2;
    } else {
      const int vh = head - a.hq - a.hkv;
      Q* vt;
      int ld, col;
      if (dst_is_fresh(dst)) { vt = (Q*)a.Vtf; ld = a.ldfresh; col = dst; }
      else { vt = (Q*)a.Vtc; ld = a.ldcache; col = dst_cache_row(dst); }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vt[((size_t)vh * a.hd + j + e) * ld + col] = from_f32<Q>(v1[e]);
        vt[((size_t)vh * a.hd + j + e + half) * ld + col] = from_f32<Q>(v2[e]);
      }
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) epi_tile_pair<EPI, T, BN>(a, tile_n, r + e, row, v1[e], v2[e]);
  }
}

// logical column of tile column r in the [S][M][N] partial buffer
template <int EPI, int BN>
__device__ __forceinline__ int logical_col(const GemmArgs& a, int tile_n, int r) {
  bool second;
  const int w = brow_index<EPI, BN>(a, tile_n, r, &second);
  return second ? w + a.N / 2 : w;
}

// XCD-aware decomposition of the linear workgroup id.  Workgroups are
// dispatched round-robin over the 8 XCDs, so XCD x runs ids x, x + 8, ....
// With few M tiles (M up to 1024 rows) XCD x owns the (N tile, slice) groups
// g with g mod 8 = x and runs all M tiles of one group back to back, so a
// weight tile is read from memory once and then hits the XCD's L2.  With many
// M tiles, an XCD's workgroups walk blocks of 8 of its groups and inside a
// block its M tiles, the groups varying fastest: the workgroups an XCD runs
// at once cover a few M tiles times 8 weight tiles, so that activation rows
// are not re-read from memory for every weight tile.  An XCD needs 6 or more
// groups for that; when 8 XCDs would leave it fewer (N = 4096 at 256-column
// tiles: 2 each, and every XCD would read all of A), py = 2 or 4 XCDs share
// one set of groups (g mod px with px = 8 / py) and split its M tiles
// (m mod py), which cuts the L2-miss reads of such a pass by about a third.
__host__ __device__ inline int tile_py(int groups, int m_tiles) {
  return m_tiles > 8 && groups < 48 ? (groups < 24 ? 4 : 2) : 1;
}
__device__ __forceinline__ bool tile_of(int id, int n_tiles, int m_tiles, int S, int* tn, int* tm, int* z) {
  const int groups = n_tiles * S;
  const int py = tile_py(groups, m_tiles), px = 8 / py;
  const int x = id % 8, rest = id / 8, xn = x % px, xm = x / px;
  const int gx = (groups - xn + px - 1) / px;          // groups of XCD x
  const int mx = (m_tiles - xm + py - 1) / py;         // M tiles of XCD x
  if (rest >= gx * mx) return false;
  const int gb = m_tiles > 8 ? 8 : 1;                  // groups per block
  const int blk = rest / (gb * mx);
  const int nb = min(gb, gx - blk * gb);               // groups in this block
  const int within = rest - blk * gb * mx;
  const int group = (blk * gb + within % nb) * px + xn;
  *tn = group / S;
  *z = group % S;
  *tm = (within / nb) * py + xm;
  return true;
}

}  // namespace
