// Shared device types and helpers of the Archer HIP library (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <type_traits>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16;
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

#define ARCHER_MAXB 64

// Per-pass description of the rows a forward recomputes, passed to kernels
// by value.  A full pass (FullForward) recomputes, for each selected
// sequence, its prompt rows followed by its G response rows; a cached pass
// (CachedForward) recomputes only the G response rows.  Key index space of
// sequence s, shared by both passes: [0, ppad) are the cached prompt keys
// (valid below p_len), [ppad, ppad + G) the fresh response keys, with
// ppad = p_len rounded up to 64 so that every 64-key tile lies in one segment.
struct SeqPlan {
  int n;                          // sequences in this pass
  int full;                       // 1 = rows are [prompt; response], 0 = response only
  int G;                          // response length
  int rows;                       // total rows of the pass
  int seq[ARCHER_MAXB];           // batch index b of pass sequence s
  int row_off[ARCHER_MAXB + 1];   // first pass row of sequence s (row_off[n] = rows)
  int p_len[ARCHER_MAXB];         // prompt length P_b
  int cache_off[ARCHER_MAXB];     // 64-aligned offset of b's prompt keys in a cache head plane
  int tok_off[ARCHER_MAXB];       // offset of b's prompt tokens in the packed prompt array
  int qt_off[ARCHER_MAXB + 1];    // prefix sum of attention query tiles per sequence
  int nsplit[ARCHER_MAXB];        // split-KV count of sequence s (a function of its key count only)
  int max_split;                  // max over s of nsplit
  int qt;                         // attention query rows per workgroup (qt_off counts tiles of qt rows)
};

__device__ __forceinline__ int plan_find(const int* off, int n, int v) {
  // largest s in [0, n) with off[s] <= v (off ascending, off[0] = 0)
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (off[mid] <= v) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(f16 x) { return (float)x; }

template <class T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }
template <> __device__ __forceinline__ f16 from_f32<f16>(float x) { return (f16)x; }

// Element type of the stored queries, keys and values -- and so of the prompt
// cache -- for activation type T: fp16 on the bf16 path (three more significant
// bits than bf16 in the same two bytes; a single rounding of each of them
// feeds every later layer, so its precision sets the error growth with
// depth), fp32 on the fp32 path.
template <class T> struct QkvOf { using type = T; };
template <> struct QkvOf<bf16> { using type = f16; };
template <class T> using qkv_t = typename QkvOf<T>::type;

// Two-term bf16 representation of an fp32 activation: v ~= hi + lo with
// hi = bf16(v) and lo = bf16(v - hi), about 16 significant bits.  The bf16
// GEMMs multiply both terms by the weights (two MFMAs), so activations keep
// near-fp32 precision while every MFMA operand is bf16.
template <class T>
__device__ __forceinline__ void store_act(T* hi, T* lo, size_t i, float v) {
  const T h = from_f32<T>(v);
  hi[i] = h;
  if (lo) lo[i] = from_f32<T>(v - to_f32(h));
}

// Four consecutive activations (i a multiple of 4, so the 4 elements are
// contiguous and 8-byte aligned in either activation layout): the same values
// as four store_act calls, written with one vector store per term.
template <class T>
__device__ __forceinline__ void store_act4(T* hi, T* lo, size_t i, float v0, float v1, float v2, float v3) {
  if constexpr (sizeof(T) == 2) {
    using V4 = std::conditional_t<std::is_same_v<T, f16>, f16x4, bf16x4>;
    const float v[4] = {v0, v1, v2, v3};
    V4 h, l;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      h[e] = from_f32<T>(v[e]);
      l[e] = from_f32<T>(v[e] - to_f32((T)h[e]));
    }
    *(V4*)(hi + i) = h;
    if (lo) *(V4*)(lo + i) = l;
  } else {
    store_act<T>(hi, lo, i + 0, v0);
    store_act<T>(hi, lo, i + 1, v1);
    store_act<T>(hi, lo, i + 2, v2);
    store_act<T>(hi, lo, i + 3, v3);
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide sum for blockDim.x a multiple of 64 (<= 1024).  Uses 16 floats of LDS.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

// Activations feeding the bf16 projection GEMMs are stored k-block-major:
// 32-column blocks of all rows one after the other, element (row, k) at
// ((k / 32) * ld + row) * 32 + k % 32 with ld the row capacity, so that the
// rows a GEMM tile reads for one 32-wide k step are one contiguous block.
// Row-major (element (row, k) at row * ld + k) otherwise.
__device__ __forceinline__ size_t act_at(int row, int k, int ld, int tiled) {
  return tiled ? ((size_t)(k >> 5) * ld + row) * 32 + (k & 31) : (size_t)row * ld + k;
}

// Threads per row of the RMSNorm kernels (stand-alone and fused into the
// split-K reduction; both must use the same count to give the same bits).
constexpr int NORM_THREADS = 512;

// RMSNorm of one row of x (d columns) into a two-term activation row (with T
// = f16 and out2 null: one fp16 rounding per element), by a block of
// NORM_THREADS threads: thread t owns the float4 chunks at
// t * 4 + k * 4 * NORM_THREADS.
// Shared by the stand-alone RMSNorm kernel and the split-K reduction that
// fuses it, so that both give the same bits.
template <class T>
__device__ __forceinline__ void rms_normalize_row(const float* xr, const float* gain, T* out, T* out2, int orow,
                                                  int ld, int tiled, int d, float eps, float* red) {
  float ss = 0.f;
  for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
    const float4 v = *(const float4*)(xr + c);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
    const float4 v = *(const float4*)(xr + c);
    const float4 g = *(const float4*)(gain + c);
    const size_t i = act_at(orow, c, ld, tiled);   // 4 consecutive elements in either layout
    store_act4<T>(out, out2, i, v.x * inv * g.x, v.y * inv * g.y, v.z * inv * g.z, v.w * inv * g.w);
  }
}

// Decision statistics of the logits (the decoder's m = max, xhat = argmax,
// log-sum-exp and log p(current token)) are built from partials.  One partial
// covers the columns of a row that one LM-head multiply wave holds in one
// column tile of BN columns: wave half h (0 or 1) holds, in lane group lg
// (0..3), the columns
//   stat_col(BN, h, lg, cb, e) = (cb / (CB/2)) * (BN/2) + h * (BN/4) + (cb % (CB/2)) * 16 + 4 lg + e
// of the tile, cb < CB = BN / 32, e < 4.  A partial is (m, s, argmax) with m
// the largest non-MASK logit, argmax the smallest column attaining it and
// s = sum over lg of its lane sums, combined as (s0 + s1) + (s2 + s3), each lane
// sum adding stat_exp(z, m) over cb then e in increasing order.  The LM-head
// epilogue and the stand-alone kernel that reads stored logits produce the
// same bits, and one kernel merges the partials of a row, so a decision does
// not depend on which of the two produced them.
__host__ __device__ __forceinline__ int stat_col(int BN, int h, int lg, int cb, int e) {
  const int hcb = BN / 64;   // CB / 2
  return (cb / hcb) * (BN / 2) + h * (BN / 4) + (cb % hcb) * 16 + 4 * lg + e;
}
__device__ __forceinline__ float stat_exp(float z, float m) {
  return __builtin_amdgcn_exp2f((z - m) * 1.4426950408889634f);
}

// dst-row encoding of the K/V destination of a pass row: >= 0 is a row of the
// fresh (response) K/V buffers, < 0 encodes prompt-cache row (-1 - v).
__device__ __forceinline__ bool dst_is_fresh(int v) { return v >= 0; }
__device__ __forceinline__ int dst_cache_row(int v) { return -1 - v; }
