// Kernel launchers of the Archer HIP library (internal interface between the
// host engine and the kernels).
#pragma once

#include "common.h"

// Epilogues of the projection GEMM Y = A W^T.
enum GemmEpi {
  EPI_STORE = 0,   // C[out_row ? out_row[r] : r][c] = y (fp32; LM-head logits, op hook)
  EPI_RESID = 1,   // X[r][c] += y (fp32 residual stream; O and down projections)
  EPI_SWIGLU = 2,  // H[r][f] = silu(y_gate) * y_up (W = gate rows, W2 = up rows)
  EPI_QKV = 3,     // RoPE on q/k, then scatter q -> Q, k/v -> prompt cache or fresh buffers
};

struct GemmArgs {
  const void* A; int lda;               // [M][K] row-major (lda = row stride), or k-block-major (a_tiled,
  int a_tiled;                          //   lda = row capacity; see act_at in common.h)
  const void* A2;                       // optional low part of a two-term A (same layout), or null
  int f16;                               // A, W and W2 are fp16 (A single-term, A2 null): one fp16
                                         //   MFMA per fragment (EPI_SWIGLU, direct-to-LDS kernel only)
  const void* W; const void* W2; int ldw; // [N][K] (SWIGLU: W = gate [F][K], W2 = up [F][K], N = 2F)
  int w_tiled;                           //   k-block-major W (ldw = rows of each matrix), see act_at
  int M, N, K;
  int ksplit;                            // K slices (bf16): fixed per (N, K, context), see gemm_ksplit
  float* part;                           // fp32 partials [ksplit][M][N] for the per-slice launch, or null
  float* C; int ldc; const int* out_row; // EPI_STORE (C may be null when tstat is set: statistics only)
  // EPI_STORE with decision statistics (LM head; see stat_col in common.h):
  // partials tstat / targ [logits row][2 N / BN], the current token's logit
  // zg [logits row]; tg = current tokens [logits row]
  float2* tstat; int* targ; float* zg; const int* tg; int mask_id;
  float* X; int ldx;                     // EPI_RESID
  // EPI_RESID with a split-K reduction: optionally RMSNorm the updated rows of
  // X (gain ngain, epsilon neps) into the two-term activation (nout, nout2)
  // laid out as act_at(row, k, nld, ntiled); nf16: into a single fp16 value
  // (nout2 null) instead
  const float* ngain; void* nout; void* nout2; float neps; int nld, ntiled, nf16;
  void* H; void* H2; int ldh, h_tiled;   // EPI_SWIGLU: H = hi part, H2 = lo part (or null), act_at layout
  // EPI_QKV
  void* Qb; int ldq;                     // Q [Hq][ldq][hd]
  void* Kc; void* Vtc; int ldcache;      // prompt cache of this layer: K [Hkv][ldcache][hd], Vt [Hkv][hd][ldcache]
  void* Kf; void* Vtf; int ldfresh;      // fresh response K/V: K [Hkv][ldfresh][hd], Vt [Hkv][hd][ldfresh]
  int hq, hkv, hd;
  const int* row_pos; const int* row_dst; const float2* rope;
};

struct AttnArgs {
  const void* Q; int ldq;                // [Hq][ldq][hd]
  const void* Kc; const void* Vtc; int ldcache;
  const void* Kf; const void* Vtf; int ldfresh;
  void* O; void* O2; int ldo, o_tiled;   // hi part, lo part (or null), layout act_at(row, col, ldo, o_tiled)
  float* Opart; float* ML;               // split partials [max_split][Hq][rows][hd], [max_split][Hq][rows][2]
  int hq, hkv, hd;
  float scale_log2;                      // log2(e) / sqrt(hd)
};

// Query tile (rows per attention workgroup) of the bf16 kernel: 256 rows (8
// waves of 32, two waves per SIMD), 128 rows (8 waves of 16) or 64 rows (4
// waves of 16).  The largest tile that still gives the pass enough
// workgroups is used; the result of a query row does not depend on the tiling
// (every softmax decision is per query).
// At most 4 splits: a long-prompt pass that would take 8 splits of 256-row
// tiles takes 4 of 128-row tiles instead (the same number of workgroups, half
// the partial bytes; measured at P 4096, 256 rows, 32 heads: 42.1 against
// 43.3 us with the merge).
constexpr int ATTN_MAX_SPLIT = 4;          // split-KV bound (workspace is sized for it)
constexpr int ATTN_TILES_PER_SPLIT = 8;    // 64-key tiles per split (target)
constexpr int ATTN_MIN_WGS = 256;          // workgroups wanted per pass (one per CU)
int attn_qt_bf16(const int* rows, const int* nsplit, int n, int hq);
// Split-KV only for passes short of workgroups: false when the pass's 256-row
// query tiles alone give three quarters of ATTN_MIN_WGS workgroups (a split
// would only add partial-result traffic and a merge; measured on the
// Dream-7B-shaped cached pass, 224 workgroups unsplit take 67 us against
// 101 us for three splits with the merge).  A split pass therefore has fewer
// than attn_split_rows_max(hq) rows (sizes the partial buffers).
bool attn_split_wanted(const int* rows, int n, int hq);
int attn_split_rows_max(int hq);
constexpr int ATTN_QT_F32 = 1;

void launch_rope_table(float2* tab, int max_pos, int hd, double theta, hipStream_t st);
// bf16 [rows][cols] row-major -> k-block-major (cols % 32 == 0)
void launch_pack_kblock(const void* src, void* dst, int rows, int cols, hipStream_t st);
template <class T>
void launch_embed(const SeqPlan& pl, const void* emb, int d, int V, int mask_id, const int* prompt,
                  const int* resp, float* x, int* row_pos, int* row_dst, int* g_anchor, int* err,
                  hipStream_t st);
template <class T>
void launch_rmsnorm(const SeqPlan& pl, int gather, int nrows, const float* x, const float* gain, void* out,
                    void* out2, int ld, int tiled, int d, float eps, int* out_row, hipStream_t st);
// Decision statistics: partials from stored logits (stat_col order, tiles of
// BN columns, np = 2 ceil(V / BN) per row), then the per-row merge into
// xhat (argmax), ell (log top probability) and qv (log p of the current token).
void launch_tile_stats(int rows, const float* logits, int V, int BN, int np, int mask_id, const int* g,
                       float2* tstat, int* targ, float* zg, hipStream_t st);
void launch_finalize_stats(int rows, int np, const float2* tstat, const int* targ, const float* zg, const int* g,
                           int V, int mask_id, int* xhat, float* ell, float* qv, hipStream_t st);
void launch_select(int B, const int* g_in, int* g_out, const int* g_anchor, const int* xhat, const float* ell,
                   const float* qv, int G, int mask_id, int k, float log_tau, int max_remask, int final_step,
                   int* dist, int* unmask_pos, int* remask_pos, int* tr_dist, int* tr_unmask, int* tr_utok,
                   int* tr_remask, hipStream_t st);
void launch_fill_i32(int* p, int v, size_t n, hipStream_t st);
// Session and state-read copies (kernels_misc.hip).
struct I32Row { int v[ARCHER_MAXB]; };
void launch_store_rows(int* a, int* b, const I32Row& va, const I32Row& vb, int n, hipStream_t st);
// FullForward response rows (residual, queries) into CachedForward row order
void launch_gather_resp_rows(const SeqPlan& pl, const float* x, float* xc, int d, const void* Q, void* Qc, int ldq,
                             int ldqc, int hq, int qbytes, hipStream_t st);
template <class T>
void launch_read_cache(const void* K, const void* Vt, int ld, int off, int P, int hkv, int hd, void* Kd, void* Vd,
                       hipStream_t st);
template <class T>
void launch_read_act(const void* hi, const void* lo, int n, int d, int ld, int tiled, float* out, hipStream_t st);

// GEMM: returns 0 on success, nonzero if the shape is unsupported.
// Configurations 0 .. GEMM_NCFG-1: register-staged kernel (gemm.hip);
// GEMM_NCFG .. GEMM_NCFG+GEMM_NCFG_LDS-1: direct-to-LDS multistage kernel
// (gemm_lds.hip).  All give the same bits for the same (N, K) split.
constexpr int GEMM_NCFG = 7;
constexpr int GEMM_NCFG_LDS = 3;
int gemm_ksplit(int N, int K, int rows);
bool gemm_lds_cfg_ok(int c, const GemmArgs& a);
int gemm_lds_tiles(int c, const GemmArgs& a);
int launch_gemm_lds_cfg(int epi, int c, bool partial, const GemmArgs& a, hipStream_t st);
void launch_gemm_reduce(int epi, const GemmArgs& a, hipStream_t st);
int gemm_grid_size(int n_tiles, int m_tiles, int S);
int gemm_pick_cfg(const GemmArgs& a, int epi);
int gemm_partial_wanted(int cfg, const GemmArgs& a);
int launch_gemm_bf16_cfg(int epi, int cfg, bool partial, const GemmArgs& a, hipStream_t st);
int launch_gemm_bf16(int epi, const GemmArgs& a, hipStream_t st);
// Column tile of the LM-head GEMM when it can also produce the decision
// statistics partials (bf16, one slice, a 2 x 2 wave grid), else 0.
int gemm_stats_bn(const GemmArgs& a);
// true if launch_gemm_bf16 runs this EPI_RESID GEMM with a separate split-K
// reduction, which then also applies the RMSNorm described by a.ngain
bool gemm_fuses_norm(const GemmArgs& a);
// Host-side check of the operands an epilogue uses (pointers, the QKV head
// shape); every launcher rejects arguments that fail it before any launch.
bool gemm_args_ok(int epi, const GemmArgs& a);
int launch_gemm_f32(int epi, const GemmArgs& a, hipStream_t st);

// Split-KV count for a sequence with nkeys keys (padded key space); the same
// function is used by every pass so results do not depend on the batch or pass.
int attn_nsplit_for_keys(int nkeys);
// Attention over the plan's sequences; split-KV partials are merged by a second kernel.
int launch_attn_bf16(const SeqPlan& pl, const AttnArgs& a, hipStream_t st);
int launch_attn_f32(const SeqPlan& pl, const AttnArgs& a, int max_keys, hipStream_t st);
