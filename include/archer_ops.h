/*
 * archer_ops.h -- single-kernel entry points and timing of the Archer library.
 *
 * These calls run one kernel of the decoding path exactly as the model path
 * launches it (same kernels, same tile and split choices for the same
 * shapes), on caller-provided device buffers.  They exist so that the
 * kernels can be checked element by element at full model sizes and timed in
 * isolation.  Conventions as in archer.h: device pointers, caller-owned
 * memory, asynchronous on the given stream, host-side argument checks.
 */
#ifndef ARCHER_OPS_H
#define ARCHER_OPS_H

#include "archer.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Y = A W^T (a projection of the transformer layer; the alpha_l work of
 * Eq. theory-cost).  A: [M][K], W: [N][K], both of element type dtype,
 * row-major; Y: fp32 [M][N].  M >= 1; N and K multiples of 64.
 * A_lo (bf16 only, may be NULL): low part of a two-term activation, so that
 * A + A_lo carries about 16 significant bits; the product is then
 * (A + A_lo) W^T, as in every projection of the bf16 model path. */
archer_status archer_op_gemm(int32_t dtype, int32_t M, int32_t N, int32_t K, const void *A,
                             const void *A_lo, const void *W, float *Y, void *hip_stream);

/* Non-causal attention of one sequence over two key segments, the anchored
 * attention of Eq. archer-attention: every query of head h attends to the nk1
 * keys of segment 1 followed by the nk2 keys of segment 2 of key/value head
 * h / (Hq / Hkv), scale 1 / sqrt(hd).  Q, K and V are fp16 for ARCHER_BF16
 * (as the bf16 model path stores them) and fp32 for ARCHER_FP32; O has the
 * element type dtype (bf16 / fp32).
 *   Q   [Hq][Mq][hd]                    O  [Mq][Hq hd]
 *   K1  [Hkv][ld1][hd]   Vt1 [Hkv][hd][ld1]   (segment 1, keys 0..nk1-1)
 *   K2  [Hkv][ld2][hd]   Vt2 [Hkv][hd][ld2]   (segment 2, keys 0..nk2-1)
 * V is stored transposed (Vt[h][d][key]).  ld1, ld2 multiples of 64,
 * nk1 <= ld1, nk2 <= ld2, head_dim 64 or 128.  Keys are read in tiles of
 * 64, so segment 1 must be readable up to nk1 rounded up to 64 (the values
 * there are ignored).
 * workspace: device scratch of archer_op_attention_ws_bytes(...) bytes,
 * 256-byte aligned (split-KV partial results; none is needed, and NULL is
 * accepted, when the key count gives one split).  Calls sharing a workspace
 * must not overlap. */
size_t archer_op_attention_ws_bytes(int32_t dtype, int32_t Mq, int32_t Hq, int32_t hd, int32_t nk);
archer_status archer_op_attention(int32_t dtype, int32_t Mq, int32_t Hq, int32_t Hkv, int32_t hd,
                                  const void *Q, const void *K1, const void *Vt1, int32_t nk1,
                                  int32_t ld1, const void *K2, const void *Vt2, int32_t nk2,
                                  int32_t ld2, void *O, void *workspace, size_t ws_bytes,
                                  void *hip_stream);

/* archer_op_attention for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels, launch configuration and results, with the
 * split-KV partials in a fixed scratch array that the library holds in each
 * device's memory (64 MiB per device, for the life of the process) instead
 * of a caller workspace.  Arguments as archer_op_attention without the
 * workspace; hip_stream must belong to the calling thread's current device.
 * Allocates nothing: ARCHER_E_SHAPE (before any launch) when the shape's
 * split-KV partials, archer_op_attention_ws_bytes, exceed 64 MiB.  All calls
 * on one device share its array: calls that overlap in time on one device
 * (other streams, other threads) race, and must be serialised by the caller.
 * The array is fully rewritten before it is read in every call, so nothing
 * carries over from the previous call. */
archer_status archer_op_attention_noalloc(int32_t dtype, int32_t Mq, int32_t Hq, int32_t Hkv, int32_t hd,
                                          const void *Q, const void *K1, const void *Vt1, int32_t nk1,
                                          int32_t ld1, const void *K2, const void *Vt2, int32_t nk2,
                                          int32_t ld2, void *O, void *hip_stream);

/* Kernel classes for timing.  The projection classes _QKV, _O, _GATEUP and
 * _DOWN are the launches of CachedForward passes (M = G per sequence); their
 * _FULL twins are the same projections in FullForward (refresh) passes
 * (M = P_b + G per sequence).  The LM head runs on the response rows in both
 * passes and has one class. */
enum {
  ARCHER_K_EMBED = 0, ARCHER_K_NORM = 1, ARCHER_K_GEMM_QKV = 2,
  ARCHER_K_ATTN = 3 /* attention of CachedForward passes (with its split-KV merge) */,
  ARCHER_K_ATTN_FULL = 4 /* attention of FullForward (refresh) passes */,
  ARCHER_K_GEMM_O = 5, ARCHER_K_GEMM_GATEUP = 6,
  ARCHER_K_GEMM_DOWN = 7, ARCHER_K_GEMM_HEAD = 8, ARCHER_K_DECIDE = 9,
  ARCHER_K_GEMM_QKV_FULL = 10, ARCHER_K_GEMM_O_FULL = 11, ARCHER_K_GEMM_GATEUP_FULL = 12,
  ARCHER_K_GEMM_DOWN_FULL = 13,
  ARCHER_K_COUNT = 14
};

/* Start recording HIP events around launches of the classes in class_mask
 * (bit c = class c) made by this context: the 1st, (every+1)-th, (2 every+1)-th
 * ... launch of each class (every >= 1; 1 = every launch).  Each event pair
 * idles the GPU for a few microseconds, so a stride keeps the measurement from
 * slowing what it measures.  Stops and clears any earlier recording;
 * ARCHER_E_ARG if every < 1. */
archer_status archer_timing_begin(archer_ctx *ctx, uint32_t class_mask, int32_t every);

/* Synchronise, stop recording and return, per class c < ARCHER_K_COUNT:
 * launches[c] (recorded launches), total_ms[c] (sum of their event-bracketed
 * durations) and the algorithmic bytes[c] and flops[c] of those launches
 * (minimum HBM traffic: operands read once and results written once).  Any
 * output may be NULL. */
archer_status archer_timing_end(archer_ctx *ctx, int64_t *launches, double *total_ms,
                                double *bytes, double *flops);

/* Read-only copies of context state, for checking it against a reference
 * (none of these changes the state).  dst: device, caller-owned, >= the
 * stated size in bytes; copies are enqueued on the context's stream.
 *   ARCHER_READ_LOGITS    fp32 [B][G][V]: the logits the session's decoder reads
 *                         (those of the last forward of archer_decode or a session).
 *   ARCHER_READ_HIDDEN    fp32 [n][d]: the final normalised hidden state (the LM
 *                         head's input) of the response rows of the most recent
 *                         forward pass, n = G x (sequences in that pass), in
 *                         ascending sequence order.  bf16 models hold it as a
 *                         two-term pair; the copy is hi + lo (exact in fp32).
 *   ARCHER_READ_RESIDUAL  fp32 [n][d]: the residual stream after the last layer
 *                         for the same rows.
 *   ARCHER_READ_PROMPT_K  [Hkv][P_b][hd] of the cache's element type (fp16 for
 *                         ARCHER_BF16 models, fp32 for ARCHER_FP32): the cached
 *   ARCHER_READ_PROMPT_V  post-RoPE prompt K / prompt V of layer `layer`,
 *                         sequence `seq` -- C_p of Eq. app-cached (App. "Formal
 *                         Analysis"), one layer of it.
 * layer and seq are ignored where they do not apply.  ARCHER_E_STATE before
 * the first forward (or for a sequence without a cache), ARCHER_E_ARG for a
 * short dst or an unknown `what`. */
enum {
  ARCHER_READ_LOGITS = 0, ARCHER_READ_HIDDEN = 1, ARCHER_READ_RESIDUAL = 2,
  ARCHER_READ_PROMPT_K = 3, ARCHER_READ_PROMPT_V = 4
};
archer_status archer_read_state(archer_ctx *ctx, int32_t what, int32_t layer, int32_t seq, void *dst,
                                size_t bytes);

/* Precision of the activation operand of each projection class (bf16 models).
 * By default every projection multiplies a two-term bf16 activation
 * (hi + lo, about 16 significant bits; two MFMAs per fragment), except the
 * gate/up projection of a model with gateup_fp16 (single fp16).  A set bit
 * ARCHER_K_GEMM_QKV, _O, _GATEUP, _DOWN or _HEAD in class_mask makes that
 * class's producer store and its GEMM read the single bf16 rounding hi = bf16(v)
 * instead (half the MFMA work of that projection).  Applies to forwards
 * enqueued after the call.  ARCHER_E_ARG for other bits, ARCHER_E_UNSUPPORTED
 * for a nonzero mask on an fp32 model and for _GATEUP on a model with
 * gateup_fp16 (whose gate/up operands are single fp16 values already). */
archer_status archer_set_single_term(archer_ctx *ctx, uint32_t class_mask);

#ifdef __cplusplus
}
#endif
#endif /* ARCHER_OPS_H */
