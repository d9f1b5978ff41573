/*
 * archer.h -- C ABI of the Archer cached-prompt decoding library (gfx950 / MI355X).
 *
 * The library implements the per-step hot path of Archer (arXiv 2608.08086):
 * a bidirectional diffusion-LM forward that either recomputes every position
 * (FullForward, the refresh pass) or only the G mutable response positions
 * against an anchored prompt K/V cache (CachedForward); the confidence
 * unmask / threshold remask decoder on the logits; and Algorithm 1, which
 * refreshes the cache under the bounded-reuse rule.
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every function returns archer_status (0 = ARCHER_OK, negative = error);
 *   no C++ exception crosses this boundary.  archer_last_error() returns a
 *   thread-local description of the last failure.
 * - "device" pointers are HIP device memory on the context's device;
 *   "host" pointers are ordinary host memory.  The caller owns all memory:
 *   weights, token arrays, logits, traces and the one workspace.  The library
 *   never allocates device memory.
 * - All work is enqueued on the HIP stream given to archer_init, in order,
 *   asynchronously, except where a call says it synchronises.
 * - Argument checks (null pointers, shapes against the limits, call order)
 *   happen on the host before anything is enqueued; a failed check enqueues
 *   nothing.  Token ids read on the device are clamped into [0, V) and an
 *   out-of-range id raises a device error flag that archer_sync() and
 *   archer_decode() report as ARCHER_E_ARG.
 * - Response rows are response positions in order; sequence b of a batch
 *   owns rows b*G .. b*G + G - 1 of every [B][G] or [B][G][V] array.
 */
#ifndef ARCHER_H
#define ARCHER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ARCHER_OK = 0,
  ARCHER_E_ARG = -1,          /* null / misaligned pointer, bad value, bad token id  */
  ARCHER_E_SHAPE = -2,        /* a size exceeds the context limits or is unsupported  */
  ARCHER_E_STATE = -3,        /* wrong call order (e.g. archer_step before a refresh) */
  ARCHER_E_HIP = -4,          /* a HIP runtime call failed (text in last_error)       */
  ARCHER_E_WORKSPACE = -5,    /* workspace too small                                  */
  ARCHER_E_UNSUPPORTED = -6   /* model shape outside what the kernels implement       */
} archer_status;

/* ARCHER_FP16 is no model dtype: it is the element type of w_gate and w_up
 * in bf16 models with gateup_fp16 set (and an archer_pack_weight dtype). */
typedef enum { ARCHER_BF16 = 0, ARCHER_FP32 = 1, ARCHER_FP16 = 2 } archer_dtype;

/* Refresh rules of the cache controller.
 * HAMMING: refresh when D_t = d_H(g_t, g_r) >= K (Sec. 4.2 Eq. archer-distance and
 *          Eq. archer-controller; Algorithm 1).  K = 0 refreshes every step.
 * AGE:     refresh when A_t = t - r >= K, the cache-age signal of Sec. 6.4, i.e. a
 *          refresh every K steps.
 * ALWAYS:  refresh at every step: eager decoding (Eq. archer-fresh).          */
typedef enum { ARCHER_REFRESH_HAMMING = 0, ARCHER_REFRESH_AGE = 1, ARCHER_REFRESH_ALWAYS = 2 } archer_policy;

/* Model: pre-norm bidirectional transformer, RMSNorm, rotate-half RoPE,
 * SwiGLU MLP, untied LM head, grouped-query attention by contiguous groups.
 * Supported: head_dim 64 or 128, n_heads % n_kv_heads == 0, d_model, d_ff,
 * vocab and (n_heads + 2 n_kv_heads) head_dim multiples of 64. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab, mask_id;
  float rms_eps, rope_theta;
  int32_t dtype;              /* archer_dtype of weights and activations; ARCHER_BF16
                                 models store queries, keys and values (and so the
                                 prompt cache) as fp16, ARCHER_FP32 models as fp32 */
  int32_t gateup_fp16;        /* ARCHER_BF16 only (else ARCHER_E_UNSUPPORTED).  Nonzero:
                                 the gate/up projection multiplies single fp16 operands
                                 (one fp16 MFMA per fragment, half the matrix work of
                                 the two-term bf16 form): its input, the normalised MLP
                                 input, is stored as one fp16 rounding, and w_gate and
                                 w_up are fp16 matrices (the bf16 weights converted,
                                 exact for magnitudes in [2^-14, 65504]).  Zero: that
                                 input is two-term bf16 and w_gate, w_up are bf16. */
} archer_model_cfg;

/* Layouts of the projection matrices (lm_head, w_qkv, w_o, w_gate, w_up,
 * w_down).  ROWMAJOR: element (r, c) of a [rows][cols] matrix at r * cols + c.
 * KBLOCK (bf16 only): 32-column blocks of all rows one after another,
 * element (r, c) at ((c / 32) * rows + r) * 32 + c % 32, which lets every
 * projection GEMM tile read the weights of one 32-wide k step as one
 * contiguous block; archer_pack_weight converts a matrix.  tok_emb is always
 * row-major. */
typedef enum { ARCHER_LAYOUT_ROWMAJOR = 0, ARCHER_LAYOUT_KBLOCK = 1 } archer_weight_layout;

/* Weights [out][in] in `layout`, element type = cfg.dtype (w_gate and w_up:
 * fp16 when cfg.gateup_fp16 is set); norm gains fp32.
 * Every pointer is a device pointer; the per-layer fields are HOST arrays of
 * n_layers device pointers.  Weights must outlive the context.  A zeroed
 * `layout` is row-major.                                                   */
typedef struct {
  const void *tok_emb;                /* [V][d]                              */
  const void *lm_head;                /* [V][d]                              */
  const float *final_norm;            /* [d]                                 */
  const float *const *attn_norm;      /* L x [d]                             */
  const void *const *w_qkv;           /* L x [(Hq + 2 Hkv) hd][d]: q heads, k heads, v heads */
  const void *const *w_o;             /* L x [d][Hq hd]                      */
  const float *const *mlp_norm;       /* L x [d]                             */
  const void *const *w_gate;          /* L x [F][d]                          */
  const void *const *w_up;            /* L x [F][d]                          */
  const void *const *w_down;          /* L x [d][F]                          */
  int32_t layout;                     /* archer_weight_layout                */
} archer_weights;

/* Context limits: they size the workspace. */
typedef struct {
  int32_t max_batch;          /* B <= max_batch <= 64                          */
  int32_t max_prompt_len;     /* every P_b <= max_prompt_len                   */
  int32_t max_prompt_total;   /* sum_b P_b <= max_prompt_total                 */
  int32_t resp_len;           /* G: response length of every sequence, % 8 == 0 */
} archer_limits;

typedef struct archer_ctx archer_ctx;

/* Decoder D (workload reading): unmask the min(k, #masked) masked rows of
 * largest log-confidence m_i - lse_i (ties: smaller position) to their argmax
 * (MASK excluded; ties: smaller id); remask at most one decided row, the one
 * whose current token has the smallest log-probability, if that probability
 * is below tau (ties: smaller position).  final_step: unmask every masked row,
 * remask nothing. */
typedef struct {
  int32_t unmask_per_step;    /* k >= 1                                         */
  float remask_threshold;     /* tau in (0, 1)                                  */
  int32_t max_remask;         /* 0 (no rollback) or 1                           */
  int32_t final_step;         /* nonzero on the last decision                   */
} archer_decide_cfg;

typedef struct {
  int32_t policy;             /* archer_policy                                   */
  int32_t K;                  /* radius (HAMMING) or period (AGE), >= 0; INT32_MAX = never */
  int32_t steps;              /* T >= 1: number of decisions = number of forwards */
  int32_t unmask_per_step;    /* k >= 1                                          */
  float remask_threshold;     /* tau                                             */
  int32_t max_remask;         /* 0 or 1                                          */
  int32_t keep_logits;        /* nonzero: every forward also stores its fp32 logits in the
                                 workspace (archer_read_state ARCHER_READ_LOGITS).  Zero:
                                 bf16 models whose LM head runs the fused-statistics
                                 epilogue write only the decoder's row statistics, not the
                                 [B][G][V] logits (decisions are the same bits either way) */
} archer_decode_cfg;

/* Optional per-step record of archer_decode (device pointers; any may be NULL). */
typedef struct {
  int32_t *refreshed;         /* [T][B] 1 if forward t of sequence b was a full refresh */
  int32_t *dist;              /* [T][B] D_t evaluated before forward t (0 at t = 0)     */
  int32_t *age;               /* [T][B] A_t = t - r before forward t (0 at t = 0)       */
  int32_t *unmask_pos;        /* [T][B][k] positions unmasked by decision t, ascending, -1 padded */
  int32_t *unmask_tok;        /* [T][B][k] token given to each of those positions, -1 padded   */
  int32_t *remask_pos;        /* [T][B] position remasked by decision t, or -1          */
} archer_trace;

/* Bytes of workspace archer_init needs for this model and these limits
 * (0 if the arguments are invalid; see archer_last_error). */
size_t archer_workspace_bytes(const archer_model_cfg *cfg, const archer_limits *lim);

/* Layout helper (no operation of the method; the model is the same in
 * either layout and the results are bitwise the same): copy the row-major
 * bf16 (or fp16) matrix src [rows][cols] into dst in the KBLOCK layout.
 * Device pointers, 16-byte aligned, not overlapping; rows >= 1, cols a
 * positive multiple of 32; dtype must be ARCHER_BF16 or ARCHER_FP16 (else
 * ARCHER_E_UNSUPPORTED).
 * Enqueued on hip_stream (NULL = default stream); does not synchronise. */
archer_status archer_pack_weight(int32_t dtype, int32_t rows, int32_t cols, const void *src, void *dst,
                                 void *hip_stream);

/* Create a context.  workspace: device, >= archer_workspace_bytes bytes,
 * 256-byte aligned, owned by the caller and not touched by anything else
 * while the context lives.  hip_stream: a hipStream_t (NULL = default stream).
 * Synchronises once (device constant tables).  w->layout KBLOCK needs
 * cfg.dtype ARCHER_BF16 (else ARCHER_E_UNSUPPORTED). */
archer_status archer_init(const archer_model_cfg *cfg, const archer_weights *w,
                          const archer_limits *lim, void *workspace, size_t ws_bytes,
                          void *hip_stream, archer_ctx **out);

/* FullForward(p, g) of Algorithm 1 for the selected sequences: recompute all
 * P_b + G positions, write the post-RoPE prompt K and the prompt V of every
 * layer into the context's prompt cache C_p, set the anchor g_r := g, and
 * write the logits of the G response rows.
 *   batch       B (1..max_batch)
 *   prompt      device int32, prompts of all B sequences concatenated
 *   prompt_len  host int32 [B], 1 <= P_b <= max_prompt_len, sum <= max_prompt_total
 *   response    device int32 [B][G] (MASK allowed anywhere)
 *   seq_sel     host uint8 [B] (nonzero = recompute) or NULL = all.  With NULL
 *               the call starts a new batch (B and prompt_len are recorded);
 *               otherwise B and prompt_len must equal the recorded ones.
 *   logits      device fp32 [B][G][V]; rows of unselected sequences untouched. */
archer_status archer_refresh_prompt(archer_ctx *ctx, int32_t batch, const int32_t *prompt,
                                    const int32_t *prompt_len, const int32_t *response,
                                    const uint8_t *seq_sel, float *logits);

/* CachedForward(g; C_r) (Eq. archer-cached, archer-attention): recompute only
 * the G response rows of each selected sequence; at every layer their queries
 * attend, without a causal mask, to the anchored prompt K/V of that sequence
 * followed by the fresh response K/V.  No response state of an earlier call
 * is used.  response: device int32 [B][G]; seq_sel as above (NULL = all);
 * logits: device fp32 [B][G][V].  ARCHER_E_STATE if a selected sequence has
 * no cache yet. */
archer_status archer_step(archer_ctx *ctx, const int32_t *response, const uint8_t *seq_sel,
                          float *logits);

/* One decision g_out = D(g_in, logits) for all B sequences of the current
 * batch (device arrays, [B][G] and [B][G][V]; g_out must not alias g_in).
 * D is the rollback decoder of Sec. 4.2 ("State-Anchored Refresh") and
 * Algorithm 1, which owns token acceptance, replacement and re-masking; its
 * rule here is the one described at archer_decide_cfg.
 * dist_out   device int32 [B]: d_H(g_out_b, g_r_b) against the current anchor, or NULL.
 * unmask_pos device int32 [B][k]: unmasked positions ascending, -1 padded, or NULL.
 *            (With final_step the list holds at most k entries; g_out is complete.)
 * remask_pos device int32 [B]: remasked position or -1, or NULL. */
archer_status archer_decide(archer_ctx *ctx, const float *logits, const int32_t *g_in,
                            int32_t *g_out, const archer_decide_cfg *dc, int32_t *dist_out,
                            int32_t *unmask_pos, int32_t *remask_pos);

/* Algorithm 1 end to end for a batch of B sequences: an initial full forward,
 * then T decisions; before each later forward the controller picks, per
 * sequence, a refresh (full forward, new anchor) or a cached forward.
 * response_inout: device int32 [B][G], the initial response g_0 on entry
 * (normally all MASK) and the decoded response on return.  prompt and
 * prompt_len as in archer_refresh_prompt.  Synchronises: under HAMMING once
 * per step (4 bytes per sequence come back to the host), otherwise at the end. */
archer_status archer_decode(archer_ctx *ctx, int32_t batch, const int32_t *prompt,
                            const int32_t *prompt_len, int32_t *response_inout,
                            const archer_decode_cfg *cfg, archer_trace *trace);

/* Algorithm 1 as a resumable session.  archer_decode is exactly
 * archer_session_begin + archer_session_advance(T) + archer_session_response,
 * then a synchronisation; the split lets a caller advance the schedule a few
 * decisions at a time, read the state between decisions (archer_read_state),
 * and save / restore the decoder state, e.g. to branch two continuations from
 * one matched state as the matched-state feedback intervention of the
 * paper's mechanism appendix does ("Fresh" rebuilds the prompt cache at once,
 * "Cached" keeps the snapshot's cache).
 *
 * archer_session_begin: validate cfg as archer_decode does, start a new batch
 * (as archer_refresh_prompt with seq_sel NULL), copy response_init (device
 * int32 [B][G]) and run forward 0, a FullForward of every sequence.  Decision
 * count t = 0.  prompt (device) and the trace arrays (device, optional; same
 * meaning as for archer_decode) must stay valid while the session is used;
 * row 0 of the trace is written here.  Does not synchronise.  The session
 * ends when the context starts another batch (archer_refresh_prompt,
 * archer_decode or another archer_session_begin); archer_step and
 * archer_decide leave it intact. */
archer_status archer_session_begin(archer_ctx *ctx, int32_t batch, const int32_t *prompt,
                                   const int32_t *prompt_len, const int32_t *response_init,
                                   const archer_decode_cfg *cfg, const archer_trace *trace);

/* Which kind of pass the first forward of an archer_session_advance call is. */
typedef enum {
  ARCHER_FORWARD_CONTROLLER = 0,   /* the controller's rule, per sequence (normal decoding)  */
  ARCHER_FORWARD_REFRESH = 1,      /* every sequence refreshes (FullForward, new anchor)     */
  ARCHER_FORWARD_CACHED = 2        /* every sequence reuses its anchored cache (CachedForward) */
} archer_forward_mode;

/* Make up to n more decisions (stopping at the schedule's T), each followed,
 * unless it is the last of the schedule, by the next forward: per sequence a
 * refresh or a cached pass as the controller decides -- except the first
 * forward of this call, whose kind first_forward (archer_forward_mode) may
 * force.  *t_out (host, may be NULL) receives the number of decisions made so
 * far.  ARCHER_E_STATE without an active session.  Synchronises once per
 * decision under ARCHER_REFRESH_HAMMING (the controller reads D_t), never
 * otherwise. */
archer_status archer_session_advance(archer_ctx *ctx, int32_t n, int32_t first_forward, int32_t *t_out);

/* Copy the session's current response g_t (device int32 [B][G]) to dst
 * (device).  Asynchronous. */
archer_status archer_session_response(archer_ctx *ctx, int32_t *dst);

/* Bytes of a session snapshot of this context (0 and last_error if ctx is NULL). */
size_t archer_session_state_bytes(const archer_ctx *ctx);

/* Save the decoder state of the active session -- g_t, the anchor g_r, the
 * logits z_t of the last forward, the prompt cache of every layer, the anchor
 * steps r_b, t, the batch and the session's configuration -- into dst (device,
 * 256-byte aligned, >= archer_session_state_bytes bytes, caller-owned).
 * Synchronises.  archer_session_restore makes that state the context's active
 * session again (same model and limits; the snapshot's prompt and trace
 * pointers are used again), after which archer_session_advance continues
 * exactly as it would have from the saved point.  Restore is asynchronous
 * after it has read the snapshot's header (one synchronisation). */
archer_status archer_session_save(archer_ctx *ctx, void *dst, size_t bytes);
archer_status archer_session_restore(archer_ctx *ctx, const void *src, size_t bytes);

/* Wait for all work of the context and report device-side argument errors. */
archer_status archer_sync(archer_ctx *ctx);

void archer_destroy(archer_ctx *ctx);

/* Thread-local text of the last error ("" if none). */
const char *archer_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* ARCHER_H */
