// Host engine of the Archer library: the C ABI of archer.h / archer_ops.h.
//
// A context holds the model description, the weight pointers, the carved-up
// caller workspace (prompt K/V cache of every layer, activations, logits and
// decision scratch) and the per-batch session state (prompt lengths, cache
// offsets, which sequences have a cache).  Each forward builds a SeqPlan on
// the host (passed to kernels by value) and enqueues, per layer:
//   RMSNorm -> QKV GEMM (+RoPE, K/V to cache or fresh buffers) -> attention
//   [-> split-KV merge] -> O GEMM (+residual) -> RMSNorm -> gate/up GEMM
//   (+SwiGLU) -> down GEMM (+residual),
// then the final RMSNorm of the response rows and the LM head.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "archer.h"
#include "archer_ops.h"
#include "launch.h"

namespace {

thread_local std::string g_err;

archer_status fail(archer_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

#define HIPCHK(x)                                                                           \
  do {                                                                                      \
    hipError_t e_ = (x);                                                                    \
    if (e_ != hipSuccess) return fail(ARCHER_E_HIP, std::string(#x) + ": " + hipGetErrorString(e_)); \
  } while (0)

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Layout {
  size_t rope, Kc, Vtc, Kf, Vtf, x, act, act2, Q, O, O2, H, H2, Cn, Cn2, logits, Opart, ML;
  size_t xc, Qc;   // residual and query rows of the response rows in CachedForward order (last full layer)
  size_t part, row_pos, row_dst, out_row, g_anchor, gbuf0, gbuf1, dist, xhat, ell, qv, err, total;
  size_t tstat, targ, zg;   // decision statistics partials [Rmax][npmax], current-token logits [Rmax]
  int npmax;
  int ldcache, ldfresh, Mmax, Rmax, max_pos, ldq;
  int part_rows;   // rows the split-K partial buffer holds
  size_t cache_layer_elems;
};

constexpr int kMaxSplit = ATTN_MAX_SPLIT;
constexpr int kPartRowsFull = 4608;

std::string check_cfg(const archer_model_cfg* c, const archer_limits* l) {
  if (!c || !l) return "null cfg or limits";
  if (c->n_layers < 1 || c->d_model < 64 || c->n_heads < 1 || c->n_kv_heads < 1 || c->d_ff < 64 || c->vocab < 64)
    return "model dimensions must be positive (d_model, d_ff, vocab >= 64)";
  if (c->head_dim != 64 && c->head_dim != 128) return "head_dim must be 64 or 128";
  if (c->n_heads % c->n_kv_heads) return "n_heads must be a multiple of n_kv_heads";
  if (c->d_model % 64 || c->d_ff % 64 || c->vocab % 64) return "d_model, d_ff and vocab must be multiples of 64";
  if (c->mask_id < 0 || c->mask_id >= c->vocab) return "mask_id outside the vocabulary";
  if (c->dtype != ARCHER_BF16 && c->dtype != ARCHER_FP32) return "dtype must be ARCHER_BF16 or ARCHER_FP32";
  if (c->gateup_fp16 && c->dtype != ARCHER_BF16) return "gateup_fp16 is a bf16-model option";
  if (!(c->rms_eps > 0.f) || !(c->rope_theta > 1.f)) return "rms_eps must be > 0 and rope_theta > 1";
  if (l->max_batch < 1 || l->max_batch > ARCHER_MAXB) return "max_batch must be in [1, 64]";
  if (l->max_prompt_len < 1 || l->max_prompt_total < l->max_prompt_len) return "bad prompt limits";
  if (l->resp_len < 8 || l->resp_len % 8 || l->resp_len > 4096) return "resp_len must be a multiple of 8 in [8, 4096]";
  if (c->dtype == ARCHER_FP32 && (size_t)c->head_dim + align_up(l->max_prompt_len, 64) + l->resp_len > 16000)
    return "fp32 path supports at most ~16k keys per sequence";
  return "";
}

Layout make_layout(const archer_model_cfg* c, const archer_limits* l) {
  Layout L{};
  const size_t esz = c->dtype == ARCHER_BF16 ? 2 : 4;
  const int d = c->d_model, hq = c->n_heads, hkv = c->n_kv_heads, hd = c->head_dim;
  L.Rmax = l->max_batch * l->resp_len;
  L.ldcache = (int)align_up((size_t)l->max_prompt_total + 64 * (size_t)l->max_batch, 64);
  L.ldfresh = (int)align_up((size_t)L.Rmax, 64);
  L.Mmax = l->max_prompt_total + L.Rmax;
  L.ldq = L.Mmax;
  L.max_pos = l->max_prompt_len + l->resp_len;
  L.cache_layer_elems = (size_t)hkv * L.ldcache * hd;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes, 256); return o; };
  L.rope = take((size_t)L.max_pos * (hd / 2) * sizeof(float2));
  L.Kc = take((size_t)c->n_layers * L.cache_layer_elems * esz);
  L.Vtc = take((size_t)c->n_layers * L.cache_layer_elems * esz);
  L.Kf = take((size_t)hkv * L.ldfresh * hd * esz);
  L.Vtf = take((size_t)hkv * L.ldfresh * hd * esz);
  L.x = take((size_t)L.Mmax * d * 4);
  // bf16 activations feeding a GEMM are two-term (hi, lo); fp32 ones are single
  const size_t lo = c->dtype == ARCHER_BF16 ? 1 : 0;
  L.act = take((size_t)L.Mmax * d * esz);
  L.act2 = take(lo * L.Mmax * d * esz);
  L.Q = take((size_t)hq * L.ldq * hd * esz);
  L.xc = take((size_t)L.Rmax * d * 4);
  L.Qc = take((size_t)hq * L.Rmax * hd * esz);
  L.O = take((size_t)L.Mmax * hq * hd * esz);
  L.O2 = take(lo * L.Mmax * hq * hd * esz);
  L.H = take((size_t)L.Mmax * c->d_ff * esz);
  L.H2 = take(lo * L.Mmax * c->d_ff * esz);
  L.Cn = take((size_t)L.Rmax * d * esz);
  L.Cn2 = take(lo * L.Rmax * d * esz);
  L.logits = take((size_t)L.Rmax * c->vocab * 4);
  // split-KV partials: only passes with fewer than attn_split_rows_max rows split
  const size_t part_rows =
      c->dtype == ARCHER_BF16 ? (size_t)std::min(L.Mmax, attn_split_rows_max(hq)) : 1;
  L.Opart = take((size_t)kMaxSplit * hq * part_rows * hd * 4);
  L.ML = take((size_t)kMaxSplit * hq * part_rows * 2 * 4);
  // split-K partials of response-row launches: max over the projections of ksplit * N
  size_t sn = 0;
  if (c->dtype == ARCHER_BF16) {
    const int F = c->d_ff, qkv = (hq + 2 * hkv) * hd;
    const int NK[5][2] = {{qkv, d}, {d, hq * hd}, {2 * F, d}, {d, F}, {c->vocab, d}};
    for (auto& nk : NK) {
      const int S = gemm_ksplit(nk[0], nk[1], L.Rmax);
      if (S > 1) sn = std::max(sn, (size_t)S * nk[0]);
    }
  }
  // split-K partials: every cached pass, and full passes of up to
  // kPartRowsFull rows (larger ones run the slices folded in one workgroup)
  L.part_rows = std::min(L.Mmax, std::max(L.Rmax, kPartRowsFull));
  L.part = take(sn * L.part_rows * 4);
  L.row_pos = take((size_t)L.Mmax * 4);
  L.row_dst = take((size_t)L.Mmax * 4);
  L.out_row = take((size_t)L.Rmax * 4);
  L.g_anchor = take((size_t)L.Rmax * 4);
  L.gbuf0 = take((size_t)L.Rmax * 4);
  L.gbuf1 = take((size_t)L.Rmax * 4);
  L.dist = take((size_t)ARCHER_MAXB * 4);
  L.xhat = take((size_t)L.Rmax * 4);
  L.ell = take((size_t)L.Rmax * 4);
  L.qv = take((size_t)L.Rmax * 4);
  // statistics partials: at most two per 128 columns (the smallest column tile)
  L.npmax = 2 * ((c->vocab + 127) / 128);
  L.tstat = take((size_t)L.Rmax * L.npmax * sizeof(float2));
  L.targ = take((size_t)L.Rmax * L.npmax * 4);
  L.zg = take((size_t)L.Rmax * 4);
  L.err = take(256);
  L.total = off;
  return L;
}

struct TimerRec {
  hipEvent_t a, b;
  int cls;
  double bytes, flops;
};

}  // namespace

struct archer_ctx {
  archer_model_cfg cfg;
  archer_limits lim;
  Layout L;
  hipStream_t stream;
  char* ws;
  size_t esz;
  // weights
  const void* tok_emb;
  const void* lm_head;
  const float* final_norm;
  std::vector<const float*> attn_norm, mlp_norm;
  std::vector<const void*> w_qkv, w_o, w_gate, w_up, w_down;
  int w_tiled = 0;   // projection matrices in the k-block-major layout
  // session
  int batch = 0;
  int plen[ARCHER_MAXB] = {0};
  int cache_off[ARCHER_MAXB] = {0};
  int tok_off[ARCHER_MAXB] = {0};
  bool has_cache[ARCHER_MAXB] = {false};
  // projection classes (bits ARCHER_K_GEMM_*) whose activation operand is a
  // single bf16 value instead of the two-term pair
  uint32_t single_mask = 0;
  // decision statistics: column tile of their partials (that of the LM-head
  // GEMM when its epilogue produces them, stat_fused) and partials per row
  int stat_tile = 128, np = 0;
  bool stat_fused = false;
  // the most recent forward pass (for archer_read_state)
  SeqPlan last{};
  size_t last_x = 0;   // workspace offset of the residual rows of the last forward (x, or xc after a full pass)
  bool have_last = false;
  uint32_t last_single = 0;
  // decode session: Algorithm 1 advanced a number of decisions at a time
  struct {
    bool active = false;
    archer_decode_cfg cfg{};
    archer_trace tr{};
    const int32_t* prompt = nullptr;
    int T = 0, t = 0;          // decisions in the schedule / made so far
    int cur = 0;               // g buffer (gbuf0 / gbuf1) holding the current response
    bool keep = true;          // forwards store their logits in the workspace
    int r[ARCHER_MAXB] = {0};  // step of each sequence's anchor
  } ses;
  // timing
  bool t_on = false;
  uint32_t t_mask = 0;
  int t_every = 1;                       // record every t_every-th launch of a class
  int64_t t_seen[ARCHER_K_COUNT] = {0};  // launches of each class since timing began
  std::vector<TimerRec> t_recs;
  size_t t_used = 0;

  template <class P> P* at(size_t off) { return (P*)(ws + off); }
};

namespace {

bool is_bf16(const archer_ctx* c) { return c->cfg.dtype == ARCHER_BF16; }

// low part of a two-term activation buffer (bf16 path only)
void* lo_part(archer_ctx* c, size_t off) { return is_bf16(c) ? (void*)(c->ws + off) : nullptr; }

template <class F>
archer_status timed(archer_ctx* c, int cls, double bytes, double flops, F&& launch) {
  const bool rec = c->t_on && ((c->t_mask >> cls) & 1u) && (c->t_seen[cls]++ % c->t_every) == 0;
  if (rec) {
    if (c->t_used == c->t_recs.size()) {
      TimerRec r{};
      // timing-only events: no system-scope fence (an L2 writeback and
      // invalidate per record, which idles the GPU ~5 us between kernels)
      HIPCHK(hipEventCreateWithFlags(&r.a, hipEventDisableSystemFence));
      HIPCHK(hipEventCreateWithFlags(&r.b, hipEventDisableSystemFence));
      c->t_recs.push_back(r);
    }
    HIPCHK(hipEventRecord(c->t_recs[c->t_used].a, c->stream));
  }
  const int rc = launch();
  if (rc) return fail(ARCHER_E_UNSUPPORTED, "kernel launch rejected the shape");
  if (rec) {
    TimerRec& r = c->t_recs[c->t_used++];
    HIPCHK(hipEventRecord(r.b, c->stream));
    r.cls = cls;
    r.bytes = bytes;
    r.flops = flops;
  }
  return ARCHER_OK;
}


SeqPlan build_plan(const archer_ctx* c, bool full, const std::vector<int>& sel) {
  SeqPlan p;
  memset(&p, 0, sizeof(p));
  p.n = (int)sel.size();
  p.full = full ? 1 : 0;
  p.G = c->lim.resp_len;
  int rows = 0, tiles = 0;
  int nrows[ARCHER_MAXB];
  for (int s = 0; s < p.n; ++s) nrows[s] = full ? c->plen[sel[s]] + p.G : p.G;
  const bool split = is_bf16(c) && attn_split_wanted(nrows, p.n, c->cfg.n_heads);
  for (int s = 0; s < p.n; ++s)
    p.nsplit[s] = split ? attn_nsplit_for_keys(((c->plen[sel[s]] + 63) & ~63) + p.G) : 1;
  const int qt = is_bf16(c) ? attn_qt_bf16(nrows, p.nsplit, p.n, c->cfg.n_heads) : ATTN_QT_F32;
  p.qt = qt;
  for (int s = 0; s < p.n; ++s) {
    const int b = sel[s];
    p.seq[s] = b;
    p.p_len[s] = c->plen[b];
    p.cache_off[s] = c->cache_off[b];
    p.tok_off[s] = c->tok_off[b];
    p.row_off[s] = rows;
    p.qt_off[s] = tiles;
    const int nr = full ? c->plen[b] + p.G : p.G;
    rows += nr;
    tiles += (nr + qt - 1) / qt;
    p.max_split = std::max(p.max_split, p.nsplit[s]);
  }
  p.row_off[p.n] = rows;
  p.qt_off[p.n] = tiles;
  p.rows = rows;
  return p;
}

// split-K slice count and partial buffer of a bf16 projection
void gemm_prepare(archer_ctx* c, GemmArgs& a) {
  if (!is_bf16(c)) return;
  a.ksplit = gemm_ksplit(a.N, a.K, c->L.Rmax);
  if (a.M <= c->L.part_rows) a.part = c->at<float>(c->L.part);
}

archer_status gemm(archer_ctx* c, int cls, int epi, GemmArgs& a) {
  gemm_prepare(c, a);
  const double es = (double)c->esz;
  double bytes = (double)a.M * a.K * es * (a.A2 ? 2 : 1) + (double)a.N * a.K * es;
  if (epi == EPI_STORE) bytes += (a.C ? (double)a.M * a.N * 4 : 0.0) + (a.tstat ? (double)a.M * c->np * 12 : 0.0);
  else if (epi == EPI_RESID)
    bytes += 2.0 * a.M * a.N * 4 + (gemm_fuses_norm(a) ? (double)a.M * a.N * es * (a.nout2 ? 2 : 1) : 0.0);
  else if (epi == EPI_SWIGLU) bytes += (double)a.M * (a.N / 2) * es * (a.H2 ? 2 : 1);
  else bytes += (double)a.M * a.N * es;
  const double flops = 2.0 * a.M * a.N * a.K;
  return timed(c, cls, bytes, flops, [&] {
    return is_bf16(c) ? launch_gemm_bf16(epi, a, c->stream) : launch_gemm_f32(epi, a, c->stream);
  });
}

GemmArgs gargs(const void* A, int lda, const void* W, int ldw, int M, int N, int K) {
  GemmArgs a;
  memset(&a, 0, sizeof(a));
  a.A = A; a.lda = lda; a.W = W; a.ldw = ldw; a.M = M; a.N = N; a.K = K;
  a.ksplit = 1;
  return a;
}

// One forward over the selected sequences (full = FullForward, else CachedForward).
// stats: the LM head also writes the decision statistics partials of the
// response rows (contexts with stat_fused); logits may then be null.
archer_status run_forward(archer_ctx* c, bool full, const std::vector<int>& sel, const int32_t* prompt,
                          const int32_t* resp, float* logits, bool stats = false) {
  if (sel.empty()) return ARCHER_OK;
  const archer_model_cfg& m = c->cfg;
  const Layout& L = c->L;
  const SeqPlan pl = build_plan(c, full, sel);
  const int d = m.d_model, hq = m.n_heads, hkv = m.n_kv_heads, hd = m.head_dim, F = m.d_ff;
  // The layers run on plan P over R rows with residual X; in a full pass the
  // last layer switches to the CachedForward plan of the same sequences after
  // its QKV projection: the prompt rows' keys and values are then in the cache
  // and nothing reads their attention, MLP or final residual.
  const SeqPlan plc = full ? build_plan(c, false, sel) : pl;
  const SeqPlan* P = &pl;
  int rows = pl.rows;
  const int qkv_n = (hq + 2 * hkv) * hd;
  const size_t es = c->esz;
  float* x = c->at<float>(L.x);
  void* qbuf = c->at<char>(L.Q);
  int ldq = L.ldq;
  void* act = c->at<char>(L.act);
  // low terms of the activations feeding each projection class (null where the
  // class takes a single bf16 operand)
  const uint32_t sm = c->single_mask;
  auto lo_for = [&](int cls, size_t off) -> void* { return ((sm >> cls) & 1u) ? nullptr : lo_part(c, off); };
  void* act2_qkv = lo_for(ARCHER_K_GEMM_QKV, L.act2);
  // gate/up with fp16 operands: its input is a single fp16 value
  const bool mlp16 = is_bf16(c) && m.gateup_fp16;
  void* act2_mlp = mlp16 ? nullptr : lo_for(ARCHER_K_GEMM_GATEUP, L.act2);
  void* o2 = lo_for(ARCHER_K_GEMM_O, L.O2);
  void* h2 = lo_for(ARCHER_K_GEMM_DOWN, L.H2);
  void* cn2 = lo_for(ARCHER_K_GEMM_HEAD, L.Cn2);
  int* row_pos = c->at<int>(L.row_pos);
  int* row_dst = c->at<int>(L.row_dst);
  archer_status st;

  st = timed(c, ARCHER_K_EMBED, (double)rows * d * (es + 4), 0.0, [&] {
    if (is_bf16(c))
      launch_embed<bf16>(pl, c->tok_emb, d, m.vocab, m.mask_id, prompt, resp, x, row_pos, row_dst,
                         c->at<int>(L.g_anchor), c->at<int>(L.err), c->stream);
    else
      launch_embed<float>(pl, c->tok_emb, d, m.vocab, m.mask_id, prompt, resp, x, row_pos, row_dst,
                          c->at<int>(L.g_anchor), c->at<int>(L.err), c->stream);
    return 0;
  });
  if (st) return st;

  // bf16 activations that feed a projection GEMM are stored k-block-major
  // with the buffer's row capacity as ld (act, O, H: Mmax rows; Cn: Rmax)
  const int tiled = is_bf16(c) ? 1 : 0;
  auto norm = [&](const float* gain, int gather, int nrows, void* out, void* out2, int cap, bool half = false) {
    return timed(c, ARCHER_K_NORM, (double)nrows * d * (4 + es * (out2 ? 2 : 1)), 0.0, [&] {
      if (half)
        launch_rmsnorm<f16>(*P, gather, nrows, x, gain, out, nullptr, cap, 1, d, m.rms_eps, c->at<int>(L.out_row),
                            c->stream);
      else if (is_bf16(c))
        launch_rmsnorm<bf16>(*P, gather, nrows, x, gain, out, out2, cap, 1, d, m.rms_eps, c->at<int>(L.out_row),
                             c->stream);
      else
        launch_rmsnorm<float>(*P, gather, nrows, x, gain, out, out2, d, 0, d, m.rms_eps, c->at<int>(L.out_row),
                              c->stream);
      return 0;
    });
  };

  double kv_keys = 0;
  for (int s = 0; s < pl.n; ++s) kv_keys += pl.p_len[s] + pl.G;
  auto q_keys = [&](const SeqPlan& p) {
    double v = 0;
    for (int s = 0; s < p.n; ++s) v += (double)(p.row_off[s + 1] - p.row_off[s]) * (p.p_len[s] + p.G);
    return v;
  };

  // RMSNorms whose input is the residual just updated by a split-K GEMM run
  // inside that GEMM's reduction (same arithmetic as the stand-alone kernel)
  auto fuse_norm = [&](GemmArgs& a, const float* gain, void* out2, bool half = false) {
    if (!is_bf16(c)) return;
    a.ngain = gain; a.nout = act; a.nout2 = out2; a.neps = m.rms_eps; a.nld = L.Mmax; a.ntiled = 1;
    a.nf16 = half ? 1 : 0;
  };
  bool normed = false;   // attn_norm of the current layer already applied
  for (int l = 0; l < m.n_layers; ++l) {
    if (!normed && (st = norm(c->attn_norm[l], 0, rows, act, act2_qkv, L.Mmax))) return st;
    normed = false;
    {
      GemmArgs a = gargs(act, tiled ? L.Mmax : d, c->w_qkv[l], c->w_tiled ? qkv_n : d, rows, qkv_n, d);
      a.A2 = act2_qkv; a.a_tiled = tiled; a.w_tiled = c->w_tiled;
      a.Qb = c->at<char>(L.Q); a.ldq = L.ldq;
      a.Kc = c->at<char>(L.Kc) + (size_t)l * L.cache_layer_elems * es;
      a.Vtc = c->at<char>(L.Vtc) + (size_t)l * L.cache_layer_elems * es;
      a.ldcache = L.ldcache;
      a.Kf = c->at<char>(L.Kf); a.Vtf = c->at<char>(L.Vtf); a.ldfresh = L.ldfresh;
      a.hq = hq; a.hkv = hkv; a.hd = hd;
      a.row_pos = row_pos; a.row_dst = row_dst; a.rope = c->at<float2>(L.rope);
      if ((st = gemm(c, full ? ARCHER_K_GEMM_QKV_FULL : ARCHER_K_GEMM_QKV, EPI_QKV, a))) return st;
    }
    if (full && l + 1 == m.n_layers) {
      float* xc = c->at<float>(L.xc);
      void* qc = c->at<char>(L.Qc);
      launch_gather_resp_rows(pl, x, xc, d, qbuf, qc, L.ldq, L.Rmax, hq, hd * (int)es, c->stream);
      HIPCHK(hipGetLastError());
      P = &plc; rows = plc.rows; x = xc; qbuf = qc; ldq = L.Rmax;
    }
    {
      AttnArgs a;
      memset(&a, 0, sizeof(a));
      a.Q = qbuf; a.ldq = ldq;
      a.Kc = c->at<char>(L.Kc) + (size_t)l * L.cache_layer_elems * es;
      a.Vtc = c->at<char>(L.Vtc) + (size_t)l * L.cache_layer_elems * es;
      a.ldcache = L.ldcache;
      a.Kf = c->at<char>(L.Kf); a.Vtf = c->at<char>(L.Vtf); a.ldfresh = L.ldfresh;
      a.O = c->at<char>(L.O); a.O2 = o2; a.ldo = tiled ? L.Mmax : hq * hd; a.o_tiled = tiled;
      a.Opart = c->at<float>(L.Opart); a.ML = c->at<float>(L.ML);
      a.hq = hq; a.hkv = hkv; a.hd = hd;
      a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)hd));
      // Q read once, O written once (two terms for bf16), every real key's K
      // and V read once
      const double bytes = (double)rows * hq * hd * es * (a.O2 ? 3 : 2) + kv_keys * hkv * hd * es * 2;
      const double flops = 4.0 * q_keys(*P) * hq * hd;
      int max_keys = 0;
      for (int s = 0; s < P->n; ++s) max_keys = std::max(max_keys, ((P->p_len[s] + 63) & ~63) + P->G);
      st = timed(c, full ? ARCHER_K_ATTN_FULL : ARCHER_K_ATTN, bytes, flops, [&] {
        return is_bf16(c) ? launch_attn_bf16(*P, a, c->stream) : launch_attn_f32(*P, a, max_keys, c->stream);
      });
      if (st) return st;
    }
    {
      GemmArgs a = gargs(c->at<char>(L.O), tiled ? L.Mmax : hq * hd, c->w_o[l], c->w_tiled ? d : hq * hd, rows,
                         d, hq * hd);
      a.A2 = o2; a.a_tiled = tiled; a.w_tiled = c->w_tiled;
      a.X = x; a.ldx = d;
      fuse_norm(a, c->mlp_norm[l], act2_mlp, mlp16);
      if ((st = gemm(c, full ? ARCHER_K_GEMM_O_FULL : ARCHER_K_GEMM_O, EPI_RESID, a))) return st;
      normed = gemm_fuses_norm(a);
    }
    if (!normed && (st = norm(c->mlp_norm[l], 0, rows, act, act2_mlp, L.Mmax, mlp16))) return st;
    normed = false;
    {
      GemmArgs a = gargs(act, tiled ? L.Mmax : d, c->w_gate[l], c->w_tiled ? F : d, rows, 2 * F, d);
      a.A2 = act2_mlp; a.a_tiled = tiled; a.w_tiled = c->w_tiled; a.f16 = mlp16 ? 1 : 0;
      a.W2 = c->w_up[l];
      a.H = c->at<char>(L.H); a.H2 = h2; a.ldh = tiled ? L.Mmax : F; a.h_tiled = tiled;
      if ((st = gemm(c, full ? ARCHER_K_GEMM_GATEUP_FULL : ARCHER_K_GEMM_GATEUP, EPI_SWIGLU, a))) return st;
    }
    {
      GemmArgs a = gargs(c->at<char>(L.H), tiled ? L.Mmax : F, c->w_down[l], c->w_tiled ? d : F, rows, d, F);
      a.A2 = h2; a.a_tiled = tiled; a.w_tiled = c->w_tiled;
      a.X = x; a.ldx = d;
      if (l + 1 < m.n_layers) fuse_norm(a, c->attn_norm[l + 1], act2_qkv);
      if ((st = gemm(c, full ? ARCHER_K_GEMM_DOWN_FULL : ARCHER_K_GEMM_DOWN, EPI_RESID, a))) return st;
      normed = gemm_fuses_norm(a);
    }
  }
  const int nresp = pl.n * pl.G;
  if ((st = norm(c->final_norm, 1, nresp, c->at<char>(L.Cn), cn2, L.Rmax))) return st;
  {
    GemmArgs a = gargs(c->at<char>(L.Cn), tiled ? L.Rmax : d, c->lm_head, c->w_tiled ? m.vocab : d, nresp,
                       m.vocab, d);
    a.A2 = cn2; a.a_tiled = tiled; a.w_tiled = c->w_tiled;
    a.C = logits; a.ldc = m.vocab; a.out_row = c->at<int>(L.out_row);
    if (stats && c->stat_fused) {
      a.tstat = c->at<float2>(L.tstat); a.targ = c->at<int>(L.targ); a.zg = c->at<float>(L.zg);
      a.tg = resp; a.mask_id = m.mask_id;
    } else if (!logits) {
      return fail(ARCHER_E_STATE, "a forward without logits needs the fused decision statistics");
    }
    if ((st = gemm(c, ARCHER_K_GEMM_HEAD, EPI_STORE, a))) return st;
  }
  HIPCHK(hipGetLastError());
  c->last = *P;
  c->last_x = full ? L.xc : L.x;
  c->have_last = true;
  c->last_single = sm;
  return ARCHER_OK;
}

// fused: the partials of these logits were written by the LM head of the
// forward that produced them (same bits as the stand-alone kernel would give)
archer_status decide_impl(archer_ctx* c, const float* logits, const int32_t* g_in, int32_t* g_out, int k,
                          float tau, int max_remask, int final_step, int32_t* dist, int32_t* unmask_pos,
                          int32_t* remask_pos, int32_t* tr_dist, int32_t* tr_unmask, int32_t* tr_utok,
                          int32_t* tr_remask, bool fused = false) {
  const int B = c->batch, G = c->lim.resp_len, V = c->cfg.vocab;
  const int rows = B * G;
  const float log_tau = (float)std::log((double)tau);
  const Layout& L = c->L;
  float2* tstat = c->at<float2>(L.tstat);
  int* targ = c->at<int>(L.targ);
  float* zg = c->at<float>(L.zg);
  return timed(c, ARCHER_K_DECIDE, fused ? (double)rows * c->np * 12 : (double)rows * V * 4, 0.0, [&] {
    if (!fused) launch_tile_stats(rows, logits, V, c->stat_tile, c->np, c->cfg.mask_id, g_in, tstat, targ, zg,
                                  c->stream);
    launch_finalize_stats(rows, c->np, tstat, targ, zg, g_in, V, c->cfg.mask_id, c->at<int>(L.xhat),
                          c->at<float>(L.ell), c->at<float>(L.qv), c->stream);
    launch_select(B, g_in, g_out, c->at<int>(L.g_anchor), c->at<int>(L.xhat), c->at<float>(L.ell),
                  c->at<float>(L.qv), G, c->cfg.mask_id, k, log_tau, max_remask, final_step,
                  dist ? dist : c->at<int>(L.dist), unmask_pos, remask_pos, tr_dist, tr_unmask, tr_utok,
                  tr_remask, c->stream);
    return 0;
  });
}

archer_status set_batch(archer_ctx* c, int batch, const int32_t* prompt_len) {
  if (batch < 1 || batch > c->lim.max_batch) return fail(ARCHER_E_SHAPE, "batch outside [1, max_batch]");
  if (!prompt_len) return fail(ARCHER_E_ARG, "null prompt_len");
  long total = 0;
  for (int b = 0; b < batch; ++b) {
    if (prompt_len[b] < 1 || prompt_len[b] > c->lim.max_prompt_len)
      return fail(ARCHER_E_SHAPE, "prompt length outside [1, max_prompt_len]");
    total += prompt_len[b];
  }
  if (total > c->lim.max_prompt_total) return fail(ARCHER_E_SHAPE, "sum of prompt lengths exceeds max_prompt_total");
  c->batch = batch;
  int coff = 0, toff = 0;
  for (int b = 0; b < batch; ++b) {
    c->plen[b] = prompt_len[b];
    c->cache_off[b] = coff;
    c->tok_off[b] = toff;
    c->has_cache[b] = false;
    coff += (prompt_len[b] + 63) & ~63;
    toff += prompt_len[b];
  }
  return ARCHER_OK;
}

archer_status check_same_batch(const archer_ctx* c, int batch, const int32_t* prompt_len) {
  if (batch != c->batch) return fail(ARCHER_E_STATE, "batch differs from the current batch");
  if (!prompt_len) return fail(ARCHER_E_ARG, "null prompt_len");
  for (int b = 0; b < batch; ++b)
    if (prompt_len[b] != c->plen[b]) return fail(ARCHER_E_STATE, "prompt_len differs from the current batch");
  return ARCHER_OK;
}

archer_status read_err_flag(archer_ctx* c) {
  int flag = 0;
  HIPCHK(hipMemcpyAsync(&flag, c->at<int>(c->L.err), sizeof(int), hipMemcpyDeviceToHost, c->stream));
  HIPCHK(hipStreamSynchronize(c->stream));
  if (flag) {
    int zero = 0;
    HIPCHK(hipMemcpyAsync(c->at<int>(c->L.err), &zero, sizeof(int), hipMemcpyHostToDevice, c->stream));
    HIPCHK(hipStreamSynchronize(c->stream));
    return fail(ARCHER_E_ARG, "a token id was outside [0, vocab) or a prompt token was MASK");
  }
  return ARCHER_OK;
}

archer_status check_decode_cfg(const archer_ctx* c, const archer_decode_cfg* dc) {
  if (dc->policy < ARCHER_REFRESH_HAMMING || dc->policy > ARCHER_REFRESH_ALWAYS) return fail(ARCHER_E_ARG, "bad policy");
  if (dc->K < 0) return fail(ARCHER_E_ARG, "K must be >= 0");
  if (dc->steps < 1) return fail(ARCHER_E_ARG, "steps must be >= 1");
  if (dc->unmask_per_step < 1 || dc->unmask_per_step > c->lim.resp_len) return fail(ARCHER_E_ARG, "unmask_per_step outside [1, G]");
  if (!(dc->remask_threshold > 0.f && dc->remask_threshold < 1.f)) return fail(ARCHER_E_ARG, "remask_threshold outside (0, 1)");
  if (dc->max_remask != 0 && dc->max_remask != 1) return fail(ARCHER_E_ARG, "max_remask must be 0 or 1");
  return ARCHER_OK;
}

// The refresh rule of the controller (the one place it is decided):
// Eq. archer-controller refreshes when the anchor distance D_t >= K; the age
// rule refreshes when A_t = t - r >= K (the cache-age signal of Sec. 6.4);
// ALWAYS refreshes at every forward (eager decoding).
bool controller_refresh(int policy, int K, int D, int A) {
  if (policy == ARCHER_REFRESH_ALWAYS) return true;
  if (policy == ARCHER_REFRESH_AGE) return A >= K;
  return D >= K;
}

// Session snapshot: a header (host state) followed by the device state of the
// session -- the current response g_t, the anchor g_r, the logits z_t of the
// last forward and the prompt cache of every layer.
constexpr uint64_t kSnapMagic = 0x3170616e73726861ull;
constexpr size_t kSnapHdr = 4096;

struct SnapHeader {
  uint64_t magic, total, cache_bytes;
  int32_t n_layers, vocab, rmax, ldcache;
  int32_t batch, plen[ARCHER_MAXB], cache_off[ARCHER_MAXB], tok_off[ARCHER_MAXB];
  uint8_t has_cache[ARCHER_MAXB];
  archer_decode_cfg cfg;
  archer_trace tr;
  const int32_t* prompt;
  int32_t T, t, cur, keep, r[ARCHER_MAXB];
};
static_assert(sizeof(SnapHeader) <= kSnapHdr, "snapshot header");

struct SnapRegion {
  size_t ws_off, snap_off, bytes;
};

size_t cache_bytes(const archer_ctx* c) { return (size_t)c->cfg.n_layers * c->L.cache_layer_elems * c->esz; }

std::vector<SnapRegion> snapshot_regions(const archer_ctx* c) {
  const Layout& L = c->L;
  const size_t g = (size_t)L.Rmax * 4, z = (size_t)L.Rmax * c->cfg.vocab * 4, kv = cache_bytes(c);
  std::vector<SnapRegion> r;
  size_t off = kSnapHdr;
  auto add = [&](size_t ws_off, size_t n) { r.push_back({ws_off, off, n}); off = align_up(off + n, 256); };
  add(c->ses.cur ? L.gbuf1 : L.gbuf0, g);
  add(L.g_anchor, g);
  add(L.logits, z);
  add(L.tstat, (size_t)L.Rmax * L.npmax * sizeof(float2));
  add(L.targ, (size_t)L.Rmax * L.npmax * 4);
  add(L.zg, (size_t)L.Rmax * 4);
  add(L.Kc, kv);
  add(L.Vtc, kv);
  return r;
}

size_t snapshot_bytes(const archer_ctx* c) {
  const SnapRegion last = snapshot_regions(c).back();
  return align_up(last.snap_off + last.bytes, 256);
}

void fill_header(const archer_ctx* c, SnapHeader& h) {
  h.magic = kSnapMagic;
  h.total = snapshot_bytes(c);
  h.cache_bytes = cache_bytes(c);
  h.n_layers = c->cfg.n_layers;
  h.vocab = c->cfg.vocab;
  h.rmax = c->L.Rmax;
  h.ldcache = c->L.ldcache;
  h.batch = c->batch;
  for (int b = 0; b < ARCHER_MAXB; ++b) {
    h.plen[b] = c->plen[b];
    h.cache_off[b] = c->cache_off[b];
    h.tok_off[b] = c->tok_off[b];
    h.has_cache[b] = c->has_cache[b] ? 1 : 0;
    h.r[b] = c->ses.r[b];
  }
  h.cfg = c->ses.cfg;
  h.tr = c->ses.tr;
  h.prompt = c->ses.prompt;
  h.T = c->ses.T;
  h.t = c->ses.t;
  h.cur = c->ses.cur;
  h.keep = c->ses.keep ? 1 : 0;
}

}  // namespace

// ===========================================================================
extern "C" {

const char* archer_last_error(void) { return g_err.c_str(); }

size_t archer_workspace_bytes(const archer_model_cfg* cfg, const archer_limits* lim) {
  const std::string e = check_cfg(cfg, lim);
  if (!e.empty()) { g_err = e; return 0; }
  return make_layout(cfg, lim).total;
}

archer_status archer_init(const archer_model_cfg* cfg, const archer_weights* w, const archer_limits* lim,
                          void* workspace, size_t ws_bytes, void* hip_stream, archer_ctx** out) {
  if (!out) return fail(ARCHER_E_ARG, "null out");
  *out = nullptr;
  const std::string e = check_cfg(cfg, lim);
  if (!e.empty()) return fail(ARCHER_E_UNSUPPORTED, e);
  if (!w || !w->tok_emb || !w->lm_head || !w->final_norm || !w->attn_norm || !w->w_qkv || !w->w_o ||
      !w->mlp_norm || !w->w_gate || !w->w_up || !w->w_down)
    return fail(ARCHER_E_ARG, "null weight pointer");
  for (int l = 0; l < cfg->n_layers; ++l)
    if (!w->attn_norm[l] || !w->w_qkv[l] || !w->w_o[l] || !w->mlp_norm[l] || !w->w_gate[l] || !w->w_up[l] ||
        !w->w_down[l])
      return fail(ARCHER_E_ARG, "null per-layer weight pointer");
  if (w->layout != ARCHER_LAYOUT_ROWMAJOR && w->layout != ARCHER_LAYOUT_KBLOCK)
    return fail(ARCHER_E_ARG, "unknown weight layout");
  if (w->layout == ARCHER_LAYOUT_KBLOCK && cfg->dtype != ARCHER_BF16)
    return fail(ARCHER_E_UNSUPPORTED, "the k-block weight layout is bf16 only");
  if (!workspace || ((uintptr_t)workspace & 255)) return fail(ARCHER_E_ARG, "workspace null or not 256-byte aligned");
  const Layout L = make_layout(cfg, lim);
  if (ws_bytes < L.total) return fail(ARCHER_E_WORKSPACE, "workspace smaller than archer_workspace_bytes()");
  archer_ctx* c = new archer_ctx();
  c->cfg = *cfg;
  c->lim = *lim;
  c->L = L;
  c->stream = (hipStream_t)hip_stream;
  c->ws = (char*)workspace;
  c->esz = cfg->dtype == ARCHER_BF16 ? 2 : 4;
  c->tok_emb = w->tok_emb;
  c->w_tiled = w->layout == ARCHER_LAYOUT_KBLOCK;
  c->lm_head = w->lm_head;
  c->final_norm = w->final_norm;
  for (int l = 0; l < cfg->n_layers; ++l) {
    c->attn_norm.push_back(w->attn_norm[l]);
    c->mlp_norm.push_back(w->mlp_norm[l]);
    c->w_qkv.push_back(w->w_qkv[l]);
    c->w_o.push_back(w->w_o[l]);
    c->w_gate.push_back(w->w_gate[l]);
    c->w_up.push_back(w->w_up[l]);
    c->w_down.push_back(w->w_down[l]);
  }
  if (cfg->dtype == ARCHER_BF16) {
    // the LM head of a full batch of response rows, as run_forward launches it
    GemmArgs h = gargs(c->at<char>(L.Cn), L.Rmax, c->lm_head, c->w_tiled ? cfg->vocab : cfg->d_model, L.Rmax,
                       cfg->vocab, cfg->d_model);
    h.A2 = c->at<char>(L.Cn2); h.a_tiled = 1; h.w_tiled = c->w_tiled;
    h.ksplit = gemm_ksplit(cfg->vocab, cfg->d_model, L.Rmax);
    h.C = c->at<float>(L.logits); h.ldc = cfg->vocab;
    const int bn = gemm_stats_bn(h);
    c->stat_fused = bn > 0;
    if (bn > 0) c->stat_tile = bn;
  }
  c->np = 2 * ((cfg->vocab + c->stat_tile - 1) / c->stat_tile);
  launch_rope_table(c->at<float2>(L.rope), L.max_pos, cfg->head_dim, (double)cfg->rope_theta, c->stream);
  hipError_t he = hipMemsetAsync(c->at<int>(L.err), 0, 256, c->stream);
  if (he == hipSuccess) he = hipGetLastError();
  if (he == hipSuccess) he = hipStreamSynchronize(c->stream);
  if (he != hipSuccess) {
    delete c;
    return fail(ARCHER_E_HIP, std::string("archer_init: ") + hipGetErrorString(he));
  }
  *out = c;
  return ARCHER_OK;
}

archer_status archer_refresh_prompt(archer_ctx* c, int32_t batch, const int32_t* prompt, const int32_t* prompt_len,
                                    const int32_t* response, const uint8_t* seq_sel, float* logits) {
  if (!c) return fail(ARCHER_E_ARG, "null ctx");
  if (!prompt || !response || !logits) return fail(ARCHER_E_ARG, "null prompt, response or logits");
  archer_status st = seq_sel ? check_same_batch(c, batch, prompt_len) : set_batch(c, batch, prompt_len);
  if (st) return st;
  c->ses.active = false;   // the anchors change outside the session's controller
  std::vector<int> sel;
  for (int b = 0; b < batch; ++b)
    if (!seq_sel || seq_sel[b]) sel.push_back(b);
  st = run_forward(c, true, sel, prompt, response, logits);
  if (st) return st;
  for (int b : sel) c->has_cache[b] = true;
  return ARCHER_OK;
}

archer_status archer_step(archer_ctx* c, const int32_t* response, const uint8_t* seq_sel, float* logits) {
  if (!c) return fail(ARCHER_E_ARG, "null ctx");
  if (!response || !logits) return fail(ARCHER_E_ARG, "null response or logits");
  if (c->batch == 0) return fail(ARCHER_E_STATE, "archer_step before any archer_refresh_prompt");
  std::vector<int> sel;
  for (int b = 0; b < c->batch; ++b)
    if (!seq_sel || seq_sel[b]) {
      if (!c->has_cache[b]) return fail(ARCHER_E_STATE, "a selected sequence has no prompt cache");
      sel.push_back(b);
    }
  return run_forward(c, false, sel, nullptr, response, logits);
}

archer_status archer_decide(archer_ctx* c, const float* logits, const int32_t* g_in, int32_t* g_out,
                            const archer_decide_cfg* dc, int32_t* dist_out, int32_t* unmask_pos,
                            int32_t* remask_pos) {
  if (!c || !dc) return fail(ARCHER_E_ARG, "null ctx or cfg");
  if (!logits || !g_in || !g_out) return fail(ARCHER_E_ARG, "null logits or token arrays");
  if (g_in == g_out) return fail(ARCHER_E_ARG, "g_out must not alias g_in");
  if (c->batch == 0) return fail(ARCHER_E_STATE, "archer_decide before any archer_refresh_prompt");
  if (dc->unmask_per_step < 1 || dc->unmask_per_step > c->lim.resp_len) return fail(ARCHER_E_ARG, "unmask_per_step outside [1, G]");
  if (!(dc->remask_threshold > 0.f && dc->remask_threshold < 1.f)) return fail(ARCHER_E_ARG, "remask_threshold outside (0, 1)");
  if (dc->max_remask != 0 && dc->max_remask != 1) return fail(ARCHER_E_ARG, "max_remask must be 0 or 1");
  archer_status st = decide_impl(c, logits, g_in, g_out, dc->unmask_per_step, dc->remask_threshold, dc->max_remask,
                                 dc->final_step, dist_out, unmask_pos, remask_pos, nullptr, nullptr, nullptr,
                                 nullptr);
  if (st) return st;
  HIPCHK(hipGetLastError());
  return ARCHER_OK;
}

archer_status archer_session_begin(archer_ctx* c, int32_t batch, const int32_t* prompt,
                                   const int32_t* prompt_len, const int32_t* response_init,
                                   const archer_decode_cfg* dc, const archer_trace* tr) {
  if (!c || !dc) return fail(ARCHER_E_ARG, "null ctx or cfg");
  if (!prompt || !response_init) return fail(ARCHER_E_ARG, "null prompt or response");
  archer_status st = check_decode_cfg(c, dc);
  if (st) return st;
  c->ses.active = false;
  if ((st = set_batch(c, batch, prompt_len))) return st;
  const int B = batch, G = c->lim.resp_len;
  auto& S = c->ses;
  S.cfg = *dc;
  S.tr = tr ? *tr : archer_trace{};
  S.prompt = prompt;
  S.T = dc->steps;
  S.t = 0;
  S.cur = 0;
  S.keep = dc->keep_logits != 0 || !c->stat_fused;
  for (int b = 0; b < ARCHER_MAXB; ++b) S.r[b] = 0;
  int* g0 = c->at<int>(c->L.gbuf0);
  HIPCHK(hipMemcpyAsync(g0, response_init, (size_t)B * G * 4, hipMemcpyDeviceToDevice, c->stream));
  // trace row 0: forward 0 is a full refresh, D_0 = A_0 = 0
  I32Row ones{}, zeros{};
  for (int b = 0; b < B; ++b) ones.v[b] = 1;
  launch_store_rows(S.tr.refreshed, S.tr.age, ones, zeros, B, c->stream);
  launch_store_rows(S.tr.dist, nullptr, zeros, zeros, B, c->stream);
  std::vector<int> all(B);
  for (int b = 0; b < B; ++b) all[b] = b;
  float* logits = S.keep ? c->at<float>(c->L.logits) : nullptr;
  if ((st = run_forward(c, true, all, prompt, g0, logits, true))) return st;
  for (int b = 0; b < B; ++b) c->has_cache[b] = true;
  S.active = true;
  return ARCHER_OK;
}

archer_status archer_session_advance(archer_ctx* c, int32_t n, int32_t first_forward, int32_t* t_out) {
  if (!c) return fail(ARCHER_E_ARG, "null ctx");
  auto& S = c->ses;
  if (!S.active) return fail(ARCHER_E_STATE, "no active decode session");
  if (n < 0) return fail(ARCHER_E_ARG, "n must be >= 0");
  if (first_forward < ARCHER_FORWARD_CONTROLLER || first_forward > ARCHER_FORWARD_CACHED)
    return fail(ARCHER_E_ARG, "bad first_forward");
  const int B = c->batch, T = S.T, k = S.cfg.unmask_per_step;
  const archer_trace& tr = S.tr;
  int* g[2] = {c->at<int>(c->L.gbuf0), c->at<int>(c->L.gbuf1)};
  float* logits = S.keep ? c->at<float>(c->L.logits) : nullptr;
  archer_status st;
  for (int i = 0; i < n && S.t < T; ++i) {
    const int t = S.t;
    const bool final = t == T - 1;
    // decision t: g_{t+1} = D(g_t, z_t); its distance to the anchor is D_{t+1}
    int32_t* trd = (tr.dist && !final) ? tr.dist + (size_t)(t + 1) * B : nullptr;
    int32_t* tru = tr.unmask_pos ? tr.unmask_pos + (size_t)t * B * k : nullptr;
    int32_t* trt = tr.unmask_tok ? tr.unmask_tok + (size_t)t * B * k : nullptr;
    int32_t* trr = tr.remask_pos ? tr.remask_pos + (size_t)t * B : nullptr;
    st = decide_impl(c, logits, g[S.cur], g[S.cur ^ 1], k, S.cfg.remask_threshold, S.cfg.max_remask,
                     final ? 1 : 0, nullptr, nullptr, nullptr, trd, tru, trt, trr, c->stat_fused);
    if (st) return st;
    S.cur ^= 1;
    S.t = t + 1;
    if (final) break;
    // forward s = t + 1: the controller picks, per sequence, a refresh or a cached pass
    const int s = t + 1;
    const int mode = i == 0 ? first_forward : ARCHER_FORWARD_CONTROLLER;
    int D[ARCHER_MAXB] = {0};
    if (mode == ARCHER_FORWARD_CONTROLLER && S.cfg.policy == ARCHER_REFRESH_HAMMING) {
      HIPCHK(hipMemcpyAsync(D, c->at<int>(c->L.dist), (size_t)B * 4, hipMemcpyDeviceToHost, c->stream));
      HIPCHK(hipStreamSynchronize(c->stream));
    }
    std::vector<int> full, cached;
    I32Row ref_row{}, age_row{};
    for (int b = 0; b < B; ++b) {
      const int A = s - S.r[b];
      bool refresh;
      if (mode == ARCHER_FORWARD_REFRESH) refresh = true;
      else if (mode == ARCHER_FORWARD_CACHED) refresh = false;
      else refresh = controller_refresh(S.cfg.policy, S.cfg.K, D[b], A);
      (refresh ? full : cached).push_back(b);
      ref_row.v[b] = refresh ? 1 : 0;
      age_row.v[b] = A;
      if (refresh) S.r[b] = s;
    }
    launch_store_rows(tr.refreshed ? tr.refreshed + (size_t)s * B : nullptr,
                      tr.age ? tr.age + (size_t)s * B : nullptr, ref_row, age_row, B, c->stream);
    if ((st = run_forward(c, true, full, S.prompt, g[S.cur], logits, true))) return st;
    if ((st = run_forward(c, false, cached, nullptr, g[S.cur], logits, true))) return st;
  }
  HIPCHK(hipGetLastError());
  if (t_out) *t_out = S.t;
  return ARCHER_OK;
}

archer_status archer_session_response(archer_ctx* c, int32_t* dst) {
  if (!c || !dst) return fail(ARCHER_E_ARG, "null ctx or dst");
  if (!c->ses.active) return fail(ARCHER_E_STATE, "no active decode session");
  const int* g = c->at<int>(c->ses.cur ? c->L.gbuf1 : c->L.gbuf0);
  HIPCHK(hipMemcpyAsync(dst, g, (size_t)c->batch * c->lim.resp_len * 4, hipMemcpyDeviceToDevice, c->stream));
  return ARCHER_OK;
}

size_t archer_session_state_bytes(const archer_ctx* c) {
  if (!c) { g_err = "null ctx"; return 0; }
  return snapshot_bytes(c);
}

archer_status archer_session_save(archer_ctx* c, void* dst, size_t bytes) {
  if (!c || !dst) return fail(ARCHER_E_ARG, "null ctx or dst");
  if (!c->ses.active) return fail(ARCHER_E_STATE, "no active decode session");
  if (bytes < snapshot_bytes(c)) return fail(ARCHER_E_WORKSPACE, "snapshot buffer smaller than archer_session_state_bytes()");
  if ((uintptr_t)dst & 255) return fail(ARCHER_E_ARG, "snapshot buffer must be 256-byte aligned");
  SnapHeader h{};
  fill_header(c, h);
  char* d = (char*)dst;
  for (const SnapRegion& r : snapshot_regions(c))
    HIPCHK(hipMemcpyAsync(d + r.snap_off, c->ws + r.ws_off, r.bytes, hipMemcpyDeviceToDevice, c->stream));
  HIPCHK(hipMemcpyAsync(d, &h, sizeof(h), hipMemcpyHostToDevice, c->stream));
  HIPCHK(hipStreamSynchronize(c->stream));
  return ARCHER_OK;
}

archer_status archer_session_restore(archer_ctx* c, const void* src, size_t bytes) {
  if (!c || !src) return fail(ARCHER_E_ARG, "null ctx or src");
  if (bytes < snapshot_bytes(c)) return fail(ARCHER_E_WORKSPACE, "snapshot smaller than archer_session_state_bytes()");
  if ((uintptr_t)src & 255) return fail(ARCHER_E_ARG, "snapshot buffer must be 256-byte aligned");
  SnapHeader h{};
  HIPCHK(hipMemcpyAsync(&h, src, sizeof(h), hipMemcpyDeviceToHost, c->stream));
  HIPCHK(hipStreamSynchronize(c->stream));
  SnapHeader want{};
  fill_header(c, want);
  if (h.magic != kSnapMagic || h.total != want.total || h.n_layers != want.n_layers || h.vocab != want.vocab ||
      h.rmax != want.rmax || h.ldcache != want.ldcache || h.cache_bytes != want.cache_bytes)
    return fail(ARCHER_E_ARG, "not a snapshot of a context of this model and these limits");
  if (h.batch < 1 || h.batch > c->lim.max_batch || h.cur < 0 || h.cur > 1 || h.t < 0 || h.t > h.T)
    return fail(ARCHER_E_ARG, "corrupt snapshot header");
  c->batch = h.batch;
  for (int b = 0; b < ARCHER_MAXB; ++b) {
    c->plen[b] = h.plen[b];
    c->cache_off[b] = h.cache_off[b];
    c->tok_off[b] = h.tok_off[b];
    c->has_cache[b] = h.has_cache[b] != 0;
    c->ses.r[b] = h.r[b];
  }
  c->ses.cfg = h.cfg;
  c->ses.tr = h.tr;
  c->ses.prompt = h.prompt;
  c->ses.T = h.T;
  c->ses.t = h.t;
  c->ses.cur = h.cur;
  c->ses.keep = h.keep != 0;
  const char* s = (const char*)src;
  for (const SnapRegion& r : snapshot_regions(c))
    HIPCHK(hipMemcpyAsync(c->ws + r.ws_off, s + r.snap_off, r.bytes, hipMemcpyDeviceToDevice, c->stream));
  HIPCHK(hipGetLastError());
  c->ses.active = true;
  c->have_last = false;
  return ARCHER_OK;
}

archer_status archer_decode(archer_ctx* c, int32_t batch, const int32_t* prompt, const int32_t* prompt_len,
                            int32_t* response_inout, const archer_decode_cfg* dc, archer_trace* tr) {
  archer_status st = archer_session_begin(c, batch, prompt, prompt_len, response_inout, dc, tr);
  if (st) return st;
  if ((st = archer_session_advance(c, dc->steps, ARCHER_FORWARD_CONTROLLER, nullptr))) return st;
  if ((st = archer_session_response(c, response_inout))) return st;
  HIPCHK(hipStreamSynchronize(c->stream));
  return read_err_flag(c);
}

archer_status archer_read_state(archer_ctx* c, int32_t what, int32_t layer, int32_t seq, void* dst, size_t bytes) {
  if (!c || !dst) return fail(ARCHER_E_ARG, "null ctx or dst");
  const archer_model_cfg& m = c->cfg;
  const Layout& L = c->L;
  const int G = c->lim.resp_len, d = m.d_model;
  const size_t es = c->esz;
  if (what == ARCHER_READ_LOGITS) {
    if (!c->ses.active) return fail(ARCHER_E_STATE, "no active decode session");
    if (!c->ses.keep) return fail(ARCHER_E_STATE, "the session keeps no logits (archer_decode_cfg.keep_logits = 0)");
    const size_t need = (size_t)c->batch * G * m.vocab * 4;
    if (bytes < need) return fail(ARCHER_E_ARG, "dst too small");
    HIPCHK(hipMemcpyAsync(dst, c->at<float>(L.logits), need, hipMemcpyDeviceToDevice, c->stream));
    return ARCHER_OK;
  }
  if (what == ARCHER_READ_HIDDEN || what == ARCHER_READ_RESIDUAL) {
    if (!c->have_last) return fail(ARCHER_E_STATE, "no forward pass since the context was created or restored");
    const SeqPlan& pl = c->last;
    const int n = pl.n * G;
    if (bytes < (size_t)n * d * 4) return fail(ARCHER_E_ARG, "dst too small");
    if (what == ARCHER_READ_HIDDEN) {
      const bool two = is_bf16(c) && !((c->last_single >> ARCHER_K_GEMM_HEAD) & 1u);
      if (is_bf16(c))
        launch_read_act<bf16>(c->at<char>(L.Cn), two ? c->at<char>(L.Cn2) : nullptr, n, d, L.Rmax, 1, (float*)dst,
                              c->stream);
      else
        launch_read_act<float>(c->at<char>(L.Cn), nullptr, n, d, d, 0, (float*)dst, c->stream);
    } else {
      const float* x = c->at<float>(c->last_x);
      for (int s = 0; s < pl.n; ++s) {
        const size_t r0 = (size_t)pl.row_off[s] + (pl.full ? pl.p_len[s] : 0);
        HIPCHK(hipMemcpyAsync((float*)dst + (size_t)s * G * d, x + r0 * d, (size_t)G * d * 4,
                              hipMemcpyDeviceToDevice, c->stream));
      }
    }
    HIPCHK(hipGetLastError());
    return ARCHER_OK;
  }
  if (what == ARCHER_READ_PROMPT_K || what == ARCHER_READ_PROMPT_V) {
    if (layer < 0 || layer >= m.n_layers) return fail(ARCHER_E_ARG, "layer outside [0, n_layers)");
    if (seq < 0 || seq >= c->batch || !c->has_cache[seq]) return fail(ARCHER_E_STATE, "sequence has no prompt cache");
    const int P = c->plen[seq];
    if (bytes < (size_t)m.n_kv_heads * P * m.head_dim * es) return fail(ARCHER_E_ARG, "dst too small");
    const char* K = c->at<char>(L.Kc) + (size_t)layer * L.cache_layer_elems * es;
    const char* Vt = c->at<char>(L.Vtc) + (size_t)layer * L.cache_layer_elems * es;
    void* kd = what == ARCHER_READ_PROMPT_K ? dst : nullptr;
    void* vd = what == ARCHER_READ_PROMPT_V ? dst : nullptr;
    if (is_bf16(c))
      launch_read_cache<f16>(K, Vt, L.ldcache, c->cache_off[seq], P, m.n_kv_heads, m.head_dim, kd, vd, c->stream);
    else
      launch_read_cache<float>(K, Vt, L.ldcache, c->cache_off[seq], P, m.n_kv_heads, m.head_dim, kd, vd, c->stream);
    HIPCHK(hipGetLastError());
    return ARCHER_OK;
  }
  return fail(ARCHER_E_ARG, "unknown state");
}

archer_status archer_set_single_term(archer_ctx* c, uint32_t class_mask) {
  if (!c) return fail(ARCHER_E_ARG, "null ctx");
  const uint32_t allowed = (1u << ARCHER_K_GEMM_QKV) | (1u << ARCHER_K_GEMM_O) | (1u << ARCHER_K_GEMM_GATEUP) |
                           (1u << ARCHER_K_GEMM_DOWN) | (1u << ARCHER_K_GEMM_HEAD);
  if (class_mask & ~allowed) return fail(ARCHER_E_ARG, "class_mask names a class that is not a projection");
  if (class_mask && !is_bf16(c)) return fail(ARCHER_E_UNSUPPORTED, "single-term activations are a bf16 option");
  if (((class_mask >> ARCHER_K_GEMM_GATEUP) & 1u) && c->cfg.gateup_fp16)
    return fail(ARCHER_E_UNSUPPORTED, "gate/up of this model multiplies single fp16 operands already");
  c->single_mask = class_mask;
  return ARCHER_OK;
}

archer_status archer_sync(archer_ctx* c) {
  if (!c) return fail(ARCHER_E_ARG, "null ctx");
  HIPCHK(hipGetLastError());
  return read_err_flag(c);
}

void archer_destroy(archer_ctx* c) {
  if (!c) return;
  for (auto& r : c->t_recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  delete c;
}

archer_status archer_timing_begin(archer_ctx* c, uint32_t mask, int32_t every) {
  if (!c) return fail(ARCHER_E_ARG, "null ctx");
  if (every < 1) return fail(ARCHER_E_ARG, "every must be >= 1");
  c->t_on = mask != 0;
  c->t_mask = mask;
  c->t_every = every;
  for (int k = 0; k < ARCHER_K_COUNT; ++k) c->t_seen[k] = 0;
  c->t_used = 0;
  return ARCHER_OK;
}

archer_status archer_timing_end(archer_ctx* c, int64_t* launches, double* total_ms, double* bytes, double* flops) {
  if (!c) return fail(ARCHER_E_ARG, "null ctx");
  HIPCHK(hipStreamSynchronize(c->stream));
  int64_t nl[ARCHER_K_COUNT] = {0};
  double ms[ARCHER_K_COUNT] = {0}, by[ARCHER_K_COUNT] = {0}, fl[ARCHER_K_COUNT] = {0};
  for (size_t i = 0; i < c->t_used; ++i) {
    const TimerRec& r = c->t_recs[i];
    float e = 0.f;
    HIPCHK(hipEventElapsedTime(&e, r.a, r.b));
    nl[r.cls] += 1;
    ms[r.cls] += e;
    by[r.cls] += r.bytes;
    fl[r.cls] += r.flops;
  }
  for (int k = 0; k < ARCHER_K_COUNT; ++k) {
    if (launches) launches[k] = nl[k];
    if (total_ms) total_ms[k] = ms[k];
    if (bytes) bytes[k] = by[k];
    if (flops) flops[k] = fl[k];
  }
  c->t_on = false;
  c->t_used = 0;
  return ARCHER_OK;
}

// ---------------------------------------------------------------------------
archer_status archer_pack_weight(int32_t dtype, int32_t rows, int32_t cols, const void* src, void* dst,
                                 void* hip_stream) {
  if (dtype != ARCHER_BF16 && dtype != ARCHER_FP16)
    return fail(ARCHER_E_UNSUPPORTED, "the k-block weight layout holds bf16 or fp16 matrices");
  if (!src || !dst) return fail(ARCHER_E_ARG, "null src or dst");
  if (((uintptr_t)src & 15) || ((uintptr_t)dst & 15)) return fail(ARCHER_E_ARG, "src and dst must be 16-byte aligned");
  if (rows < 1 || cols < 32 || cols % 32) return fail(ARCHER_E_SHAPE, "need rows >= 1 and cols a multiple of 32");
  const size_t bytes = (size_t)rows * cols * 2;
  const uintptr_t s0 = (uintptr_t)src, d0 = (uintptr_t)dst;
  if (s0 < d0 + bytes && d0 < s0 + bytes) return fail(ARCHER_E_ARG, "src and dst overlap");
  launch_pack_kblock(src, dst, rows, cols, (hipStream_t)hip_stream);
  HIPCHK(hipGetLastError());
  return ARCHER_OK;
}

archer_status archer_op_gemm(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, const void* A_lo,
                             const void* W, float* Y, void* hip_stream) {
  if (!A || !W || !Y) return fail(ARCHER_E_ARG, "null operand");
  if (M < 1 || N < 64 || K < 64 || N % 64 || K % 64) return fail(ARCHER_E_SHAPE, "need M >= 1 and N, K multiples of 64");
  if (A_lo && dtype != ARCHER_BF16) return fail(ARCHER_E_ARG, "A_lo is only meaningful for bf16");
  GemmArgs a = gargs(A, K, W, K, M, N, K);
  a.A2 = A_lo;
  if (dtype == ARCHER_BF16) a.ksplit = gemm_ksplit(N, K, M);
  a.C = Y; a.ldc = N;
  int rc;
  if (dtype == ARCHER_BF16) rc = launch_gemm_bf16(EPI_STORE, a, (hipStream_t)hip_stream);
  else if (dtype == ARCHER_FP32) rc = launch_gemm_f32(EPI_STORE, a, (hipStream_t)hip_stream);
  else return fail(ARCHER_E_ARG, "bad dtype");
  if (rc) return fail(ARCHER_E_UNSUPPORTED, "gemm shape unsupported");
  HIPCHK(hipGetLastError());
  return ARCHER_OK;
}

static int op_attn_nsplit(int dtype, int Mq, int Hq, int nk) {
  return dtype == ARCHER_BF16 && attn_split_wanted(&Mq, 1, Hq) ? attn_nsplit_for_keys(nk) : 1;
}

size_t archer_op_attention_ws_bytes(int32_t dtype, int32_t Mq, int32_t Hq, int32_t hd, int32_t nk) {
  if (Mq < 1 || Hq < 1 || hd < 1 || nk < 1) return 0;
  const int ns = op_attn_nsplit(dtype, Mq, Hq, nk);
  return align_up((size_t)ns * Hq * Mq * hd * 4, 256) + align_up((size_t)ns * Hq * Mq * 2 * 4, 256);
}

}  // extern "C"

namespace {

archer_status op_attention_impl(int32_t dtype, int32_t Mq, int32_t Hq, int32_t Hkv, int32_t hd, const void* Q,
                                const void* K1, const void* Vt1, int32_t nk1, int32_t ld1, const void* K2,
                                const void* Vt2, int32_t nk2, int32_t ld2, void* O, void* workspace,
                                size_t ws_bytes, void* hip_stream) {
  if (!Q || !K1 || !Vt1 || !K2 || !Vt2 || !O) return fail(ARCHER_E_ARG, "null operand");
  if (Mq < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv || (hd != 64 && hd != 128)) return fail(ARCHER_E_SHAPE, "bad head shape");
  if (nk1 < 1 || nk2 < 1 || ld1 % 64 || ld2 % 64 || nk1 > ld1 || nk2 > ld2) return fail(ARCHER_E_SHAPE, "bad key segments");
  if (dtype != ARCHER_BF16 && dtype != ARCHER_FP32) return fail(ARCHER_E_ARG, "bad dtype");
  const int ns = op_attn_nsplit(dtype, Mq, Hq, ((nk1 + 63) & ~63) + nk2);
  const size_t need = archer_op_attention_ws_bytes(dtype, Mq, Hq, hd, ((nk1 + 63) & ~63) + nk2);
  if (ns > 1 && (!workspace || ws_bytes < need || ((uintptr_t)workspace & 255)))
    return fail(ARCHER_E_WORKSPACE, "attention workspace too small or misaligned");
  SeqPlan p;
  memset(&p, 0, sizeof(p));
  p.n = 1; p.full = 0; p.G = nk2; p.rows = Mq;
  p.row_off[1] = Mq; p.p_len[0] = nk1;
  const int qt = dtype == ARCHER_BF16 ? attn_qt_bf16(&Mq, &ns, 1, Hq) : ATTN_QT_F32;
  p.qt = qt;
  p.qt_off[1] = (Mq + qt - 1) / qt;
  p.nsplit[0] = ns;
  p.max_split = ns;
  AttnArgs a;
  memset(&a, 0, sizeof(a));
  a.Q = Q; a.ldq = Mq;
  a.Kc = K1; a.Vtc = Vt1; a.ldcache = ld1;
  a.Kf = K2; a.Vtf = Vt2; a.ldfresh = ld2;
  a.O = O; a.ldo = Hq * hd;
  a.hq = Hq; a.hkv = Hkv; a.hd = hd;
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)hd));
  hipStream_t st = (hipStream_t)hip_stream;
  if (ns > 1) {
    const size_t o1 = align_up((size_t)ns * Hq * Mq * hd * 4, 256);
    a.Opart = (float*)workspace;
    a.ML = (float*)((char*)workspace + o1);
  }
  int rc;
  if (dtype == ARCHER_BF16) {
    rc = launch_attn_bf16(p, a, st);
  } else {
    rc = launch_attn_f32(p, a, ((nk1 + 63) & ~63) + nk2, st);
  }
  if (rc) return fail(ARCHER_E_UNSUPPORTED, "attention shape unsupported");
  HIPCHK(hipGetLastError());
  return ARCHER_OK;
}

}  // namespace

extern "C" {

archer_status archer_op_attention(int32_t dtype, int32_t Mq, int32_t Hq, int32_t Hkv, int32_t hd, const void* Q,
                                  const void* K1, const void* Vt1, int32_t nk1, int32_t ld1, const void* K2,
                                  const void* Vt2, int32_t nk2, int32_t ld2, void* O, void* workspace,
                                  size_t ws_bytes, void* hip_stream) {
  return op_attention_impl(dtype, Mq, Hq, Hkv, hd, Q, K1, Vt1, nk1, ld1, K2, Vt2, nk2, ld2, O, workspace, ws_bytes,
                           hip_stream);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The attention op for callers that cannot allocate device memory.  Its
// split-KV partials live in `scratch`, a fixed array of this library in every
// device's memory, instead of a caller workspace.  Host code never passes the
// array's name to a kernel or a copy: it looks up each device's address once
// (with that device current) and passes that address.
namespace {
constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

static __device__ __align__(256) char scratch[kScratchBytes];

namespace {
// Device address of the current device's `scratch` (looked up on the first call per device).
archer_status scratch_address(void** out) {
  int dev = 0;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(ARCHER_E_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(ARCHER_E_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ARCHER_OK;
}
}  // namespace

extern "C" archer_status archer_op_attention_noalloc(int32_t dtype, int32_t Mq, int32_t Hq, int32_t Hkv, int32_t hd,
                                                     const void* Q, const void* K1, const void* Vt1, int32_t nk1,
                                                     int32_t ld1, const void* K2, const void* Vt2, int32_t nk2,
                                                     int32_t ld2, void* O, void* hip_stream) {
  if (Mq < 1 || Hq < 1 || hd < 1 || nk1 < 1 || nk2 < 1) return fail(ARCHER_E_SHAPE, "bad attention shape");
  const int nkeys = ((nk1 + 63) & ~63) + nk2;
  const int ns = op_attn_nsplit(dtype, Mq, Hq, nkeys);
  void* ws = nullptr;
  if (ns > 1) {
    const size_t need = archer_op_attention_ws_bytes(dtype, Mq, Hq, hd, nkeys);
    if (need > kScratchBytes)
      return fail(ARCHER_E_SHAPE, "archer_op_attention_noalloc: this shape needs " + std::to_string(need) +
                                      " bytes of split-KV scratch, more than the library's fixed " +
                                      std::to_string(kScratchBytes) + " bytes; use archer_op_attention");
    const archer_status st = scratch_address(&ws);
    if (st) return st;
  }
  return op_attention_impl(dtype, Mq, Hq, Hkv, hd, Q, K1, Vt1, nk1, ld1, K2, Vt2, nk2, ld2, O, ws, kScratchBytes,
                           hip_stream);
}
