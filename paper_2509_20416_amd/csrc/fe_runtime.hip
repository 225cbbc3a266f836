// fe_runtime.hip -- host side of libfe.so: the C ABI of include/fe.h,
// argument validation, workspace layout, the launch sequence of one drafting
// pass and HIP graph capture/replay.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <initializer_list>
#include <mutex>
#include <new>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "../../include/fe.h"
#include "fe_internal.h"

using namespace fe;

namespace {

thread_local char g_err[512];

fe_status fail(fe_status st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return st;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

#define FE_TRY(x)                                                           \
  do {                                                                      \
    hipError_t e_ = (x);                                                    \
    if (e_ != hipSuccess) return fail(FE_E_HIP, "%s: %s", #x, hipGetErrorString(e_)); \
  } while (0)

size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

// A roctx range over a host scope: the entry points, the pass and its layers
// show up by name on a rocprofv3 --marker-trace timeline (host time: when the
// work was enqueued, or captured).
struct Range {
  explicit Range(const char *name) { roctxRangePushA(name); }
  ~Range() { roctxRangePop(); }
  Range(const Range &) = delete;
  Range &operator=(const Range &) = delete;
};

struct Layout {
  size_t cat, X, Xp, ssqX, ssqP, AQ, AM, AF, an, bn, q, knew, vnew, part, rope, ao, s, pmax,
      psum, cval, cidx, cz, img, splitk, tagged, total;
  size_t splitk_floats;
  size_t acc_pre;
  int acc_pre_batch;
  // Layer-private buffers (x', its norms and sums of squares, Q/K/V, attention
  // partials and output, SwiGLU rows, split-K slices): one lane, or under
  // FE_CTX_PARALLEL one lane per layer, so that the independent layers can
  // run side by side; bytes per lane of each.
  int lanes;
  size_t Xp_l, ssqP_l, AM_l, an_l, bn_l, q_l, knew_l, vnew_l, part_l, ao_l, s_l, splitk_l;
  int nchmax, nwg, npos;
  // tagged words of the persistent batch-1 pass (offsets in words from `tagged`)
  size_t t_sync, t_g, t_ssq, t_ssqp, t_copy, t_xp, t_s, t_cand, t_words;
};

int es_of(const fe_config &c) { return c.dtype == FE_BF16 ? 2 : 4; }

Layout layout_of(const fe_config &c) {
  Layout L{};
  const size_t B = c.max_batch, N = c.n_layers, d = c.hidden, es = es_of(c);
  const size_t Hq = c.n_q_heads, Hkv = c.n_kv_heads, D = c.head_dim, I = c.intermediate;
  // partial slots per (sequence, head): one per prefix chunk, one for the
  // cascade keys when they run as a unit of their own
  L.nchmax = (c.max_prefix > 0 ? (c.max_prefix + kAttnChunk - 1) / kAttnChunk : 1) + 1;
  L.nwg = lmhead_tiles(c.draft_vocab);
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o += up256(bytes); return at; };
  L.lanes = c.cascade_ctx == FE_CTX_PARALLEL ? (int)N : 1;
  auto lane = [&](size_t bytes, size_t &lane_bytes) {
    lane_bytes = up256(bytes);
    return take(lane_bytes * L.lanes);
  };
  L.cat = take(B * 2 * d * es);
  L.X = take(B * (N + 1) * d * 4);
  L.Xp = lane(B * d * 4, L.Xp_l);
  L.ssqX = take(B * (N + 1) * (d / 16) * 4);  // sums of squares of x_j per 16-column tile
  L.ssqP = lane(B * (d / 16) * 4, L.ssqP_l);  // ... of x' (post-attention residual)
  // gamma * x operands of the fused-RMSNorm GEMMs: per layer l the QKV rows
  // (b, j) of x_j, the MLP rows of x', the final-norm rows (b, i-1) of x_i
  L.AQ = take(N * B * N * d * es);
  L.AM = lane(B * d * es, L.AM_l);
  L.AF = take(B * N * d * es);
  L.an = lane(B * N * d * es, L.an_l);
  L.bn = lane(B * d * es, L.bn_l);
  L.q = lane(B * Hq * D * 4, L.q_l);
  L.knew = lane(B * N * Hkv * D * 4, L.knew_l);
  L.vnew = lane(B * N * Hkv * D * 4, L.vnew_l);
  L.part = lane(B * Hq * ((size_t)L.nchmax * (D + 2) + 1) * 4, L.part_l);  // + partial counts
  L.npos = c.max_prefix + c.n_layers;  // positions P_b + j, j < N
  L.rope = take((size_t)L.npos * (D / 2) * 2 * 4);
  L.ao = lane(B * Hq * D * es, L.ao_l);
  L.s = lane(B * I * es, L.s_l);
  L.pmax = take(B * N * (size_t)L.nwg * 4);
  L.psum = take(B * N * (size_t)L.nwg * 4);
  L.cval = take(B * N * (size_t)L.nwg * kMaxTopk * 4);
  L.cidx = take(B * N * (size_t)L.nwg * kMaxTopk * 4);
  L.cz = take(B * N * (size_t)L.nwg * kMaxTopk * 4);  // z / T of sampled candidates
  L.img = take(((size_t)c.target_vocab + 31) / 32 * 4);  // target ids that d2t reaches
  // the sampling acceptance's row pre-pass for batches of a few sequences
  L.acc_pre_batch = (int)std::min<size_t>(B, kAccPreMaxBatch);
  L.acc_pre = take(acc_pre_bytes(L.acc_pre_batch, 1 + (int)N * c.max_topk, c.draft_vocab));
  // the persistent batch-1 pass: sync words, g_t, sums of squares of x_j and
  // x'_i per workgroup, normalised copies of x_j for every consumer (QKV of
  // layer l, or the LM head), of x'_i, the SwiGLU rows, LM-head candidates
  {
    size_t w = 0;
    auto words = [&](size_t n) { size_t at = w; w += (n + 31) / 32 * 32; return at; };
    L.t_sync = words(kSegSyncWords / 2 + 1);
    L.t_g = words(d / 2);
    L.t_ssq = words((N + 1) * (size_t)kSegMaxWg);
    L.t_ssqp = words(N * (size_t)kSegMaxWg);
    L.t_copy = words((N + 1) * (N + 1) * (d / 2));
    L.t_xp = words(N * (d / 2));
    L.t_s = words(N * (I / 2));
    L.t_cand = words(N * (size_t)kSegMaxWg * (2 + 2 * kMaxTopk));
    L.t_words = w;
    L.tagged = take(w * 8);
  }
  // split-K slices of the batched GEMMs with narrow outputs: up to 8 slices of
  // the QKV rows (B * N at most, 256 per launch) over 128-column tiles
  {
    const size_t rows = std::min<size_t>(256, B * N);
    const size_t cols = (std::max<size_t>((Hq + 2 * Hkv) * D, d) + 127) / 128 * 128;
    L.splitk_floats = rows > 16 ? 8 * rows * cols : 0;
    L.splitk = lane(L.splitk_floats * 4, L.splitk_l);
  }
  L.total = o;
  return L;
}

// Workspace of fe_kv_update for chunks of C rows: the fused inputs, x_0 in
// fp32, its per-layer RMSNorm (bf16: every layer's rows side by side, for the
// one K/V launch over all layers), the rows' sums of squares for the fused
// norm of chunks up to kFusedRows rows, and split-K slices for the 256-row
// launches.  Chunks of more rows than one such launch takes (bf16) run the
// fusion and input FCs as 2-D tiled GEMMs; below that the split-K launches
// are faster (measured on the 8B shapes: 192 rows 205 against 278 us, 256
// rows 219 against 287 us).
constexpr int kTiledRows = kGemmMaxRows + 1, kFusedRows = 16;

struct UpdLayout {
  size_t cat, X, an, ssq, splitk, total;
  size_t splitk_floats;
  // self context: the layers' row state of a prefill step (q, own K/V,
  // attention output, x', SwiGLU rows, prefix ranges, attention partials of
  // one 256-row slice)
  size_t q, knew, vnew, ao, Xp, sb, ranges, part;
  int nch_ld;
};

UpdLayout upd_layout_of(const fe_config &c, size_t C) {
  UpdLayout U{};
  const size_t d = c.hidden, es = es_of(c), kvd = (size_t)c.n_kv_heads * c.head_dim;
  const size_t nan_ = c.dtype == FE_BF16 ? c.n_layers : 1;  // bf16: every layer's rows
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o += up256(bytes); return at; };
  U.cat = take(C * 2 * d * es);
  U.X = take(C * d * 4);
  U.an = take(nan_ * C * d * es);
  U.ssq = take(std::min<size_t>(kFusedRows, C) * (d / 16) * 4);
  const size_t rows = std::min<size_t>(kGemmMaxRows, C);
  const bool self = c.cascade_ctx == FE_CTX_SELF;
  const size_t qd = (size_t)c.n_q_heads * c.head_dim;
  const size_t cols = (std::max<size_t>(self ? qd + 2 * kvd : 2 * kvd, d) + 127) / 128 * 128;
  U.splitk_floats = rows > 16 ? 8 * rows * cols : 0;
  U.splitk = take(U.splitk_floats * 4);
  if (self) {
    const size_t D = c.head_dim;
    U.nch_ld = (c.max_prefix + kAttnChunk - 1) / kAttnChunk + 1;
    U.q = take(C * qd * 4);
    U.knew = take(C * kvd * 4);
    U.vnew = take(C * kvd * 4);
    U.ao = take(C * qd * es);
    U.Xp = take(C * d * 4);
    U.sb = take(C * (size_t)c.intermediate * es);
    U.ranges = take(C * 2 * 4);
    U.part = take(rows * c.n_q_heads * ((size_t)U.nch_ld * (D + 2) + 1) * 4);
  }
  U.total = o;
  return U;
}

fe_status check_config(const fe_config *c) {
  if (!c) return fail(FE_E_INVALID, "config is NULL");
  if (c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
      c->intermediate <= 0 || c->n_layers <= 0 || c->draft_vocab <= 0 || c->target_vocab <= 0 ||
      c->n_feat_levels <= 0 || c->max_batch <= 0 || c->max_topk <= 0 || c->max_prefix < 0)
    return fail(FE_E_INVALID, "config has a non-positive size");
  if (c->dtype != FE_F32 && c->dtype != FE_BF16) return fail(FE_E_INVALID, "unknown dtype %d", c->dtype);
  if (c->cascade_ctx != FE_CTX_CASCADE && c->cascade_ctx != FE_CTX_SELF &&
      c->cascade_ctx != FE_CTX_PARALLEL)
    return fail(FE_E_INVALID, "unknown cascade_ctx %d", c->cascade_ctx);
  if (!(c->rope_theta > 0.f) || !(c->rms_eps >= 0.f)) return fail(FE_E_INVALID, "bad rope_theta or rms_eps");
  if (c->n_q_heads % c->n_kv_heads) return fail(FE_E_INVALID, "n_q_heads must be a multiple of n_kv_heads");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(FE_E_UNSUPPORTED, "head_dim must be 64 or 128");
  if (c->n_layers > kMaxLayers) return fail(FE_E_UNSUPPORTED, "n_layers > %d", kMaxLayers);
  if (c->max_topk > kMaxTopk) return fail(FE_E_UNSUPPORTED, "max_topk > %d", kMaxTopk);
  if (c->max_topk > c->draft_vocab) return fail(FE_E_INVALID, "max_topk > draft_vocab");
  if ((long)c->max_batch * c->n_layers > kGemmMaxRows)
    return fail(FE_E_UNSUPPORTED, "max_batch * n_layers > %d", kGemmMaxRows);
  const int kstep = c->dtype == FE_BF16 ? 32 : 16;
  const long qd = (long)c->n_q_heads * c->head_dim;
  if (c->hidden % kstep || c->intermediate % kstep || qd % kstep)
    return fail(FE_E_UNSUPPORTED, "hidden, intermediate and n_q_heads*head_dim must be multiples of %d", kstep);
  if (c->hidden > 8192) return fail(FE_E_UNSUPPORTED, "hidden > 8192");
  if (c->draft_vocab % 16) return fail(FE_E_UNSUPPORTED, "draft_vocab must be a multiple of 16");
  if ((long)lmhead_tiles(c->draft_vocab) * c->max_topk > kMergeMaxCand)
    return fail(FE_E_UNSUPPORTED, "draft_vocab * max_topk too large for the top-k merge");
  if ((long)c->n_feat_levels * c->hidden > (1L << 30)) return fail(FE_E_UNSUPPORTED, "feature width too large");
  return FE_OK;
}

}  // namespace

struct fe_drafter {
  fe_config cfg;
  fe_weights w;
  std::vector<fe_layer_weights> layers;
  char *ws;
  Layout L;
  hipStream_t cap_stream = nullptr;
  bool graph_mode = false;
  int attn_split = 0;  // 64-key chunks per attention work unit (0 = automatic)
  bool table_ready = false;  // rotary table built (first pass on the handle)
  int pass_mode = 1;          // 1: one launch per stage; 0: persistent launches where the shape allows
  bool seg_ready = false;     // tagged words zeroed (first persistent pass on the handle)
  int seg_nwg = 0, seg_var = -2;  // workgroups (compute units) and variant of the persistent pass
  bool last_seg = false;      // the most recent pass ran as persistent launches
  bool img_ready = false;    // bitmask of d2t's image built (first sampling acceptance)
  // graph cache: key = every argument of the last captured call
  std::vector<uintptr_t> key;
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  // arguments of the most recent fe_draft_forward, for fe_time_stage
  bool have_last = false;
  int last_batch = 0, last_topk = 0;
  float last_inv_temp = 1.f;
  Draws last_draws;
  const void *last_features = nullptr;
  const int32_t *last_tokens = nullptr;
  std::vector<const void *> last_k, last_v;
  fe_kv_view last_kv{};
  fe_draft_out last_out{};
  fe_tree_out last_tree{};
  hipEvent_t ev_a = nullptr, ev_b = nullptr;
  // FE_CTX_PARALLEL: one stream per layer (default priority), fork and join events
  hipStream_t side[kMaxLayers] = {};
  hipEvent_t ev_fork = nullptr, ev_join[kMaxLayers] = {};
};

extern "C" {

const char *fe_last_error(void) { return g_err; }

size_t fe_workspace_bytes(const fe_config *cfg) {
  if (check_config(cfg) != FE_OK) return 0;
  return layout_of(*cfg).total;
}

fe_status fe_drafter_create(const fe_config *cfg, const fe_weights *w, void *workspace,
                            size_t workspace_bytes, void *stream, fe_drafter **out) {
  (void)stream;
  if (!out) return fail(FE_E_INVALID, "out is NULL");
  *out = nullptr;
  fe_status st = check_config(cfg);
  if (st != FE_OK) return st;
  if (!w || !w->layers) return fail(FE_E_INVALID, "weights or weights->layers is NULL");
  const void *top[] = {w->w_fuse, w->w_in, w->embed, w->final_norm, w->lm_head};
  const char *topn[] = {"w_fuse", "w_in", "embed", "final_norm", "lm_head"};
  for (int i = 0; i < 5; ++i) {
    if (!top[i]) return fail(FE_E_INVALID, "weight %s is NULL", topn[i]);
    if (!aligned16(top[i])) return fail(FE_E_ALIGN, "weight %s is not 16-byte aligned", topn[i]);
  }
  for (int l = 0; l < cfg->n_layers; ++l) {
    const fe_layer_weights &lw = w->layers[l];
    const void *p[] = {lw.attn_norm, lw.wq, lw.wk, lw.wv, lw.wo, lw.mlp_norm, lw.w_gate, lw.w_up, lw.w_down};
    for (int i = 0; i < 9; ++i) {
      if (!p[i]) return fail(FE_E_INVALID, "layer %d weight %d is NULL", l, i);
      if (!aligned16(p[i])) return fail(FE_E_ALIGN, "layer %d weight %d is not 16-byte aligned", l, i);
    }
  }
  const Layout L = layout_of(*cfg);
  if (!workspace || workspace_bytes < L.total)
    return fail(FE_E_WORKSPACE, "workspace needs %zu bytes, got %zu", L.total, workspace ? workspace_bytes : 0);
  if (((uintptr_t)workspace & 255u) != 0) return fail(FE_E_ALIGN, "workspace must be 256-byte aligned");
  fe_drafter *h = new (std::nothrow) fe_drafter();
  if (!h) return fail(FE_E_INVALID, "out of host memory");
  h->cfg = *cfg;
  h->w = *w;
  h->layers.assign(w->layers, w->layers + cfg->n_layers);
  h->w.layers = h->layers.data();
  h->ws = (char *)workspace;
  h->L = L;
  *out = h;
  return FE_OK;
}

fe_status fe_set_graph_mode(fe_drafter *h, int32_t on) {
  if (!h) return fail(FE_E_INVALID, "handle is NULL");
  h->graph_mode = on != 0;
  return FE_OK;
}

fe_status fe_set_pass_mode(fe_drafter *h, int32_t mode) {
  if (!h) return fail(FE_E_INVALID, "handle is NULL");
  if (mode != 0 && mode != 1) return fail(FE_E_INVALID, "pass mode %d is not 0 or 1", mode);
  if (mode == 0 && !kSegEnabled)
    return fail(FE_E_UNSUPPORTED, "the persistent batch-1 pass (mode 0) is switched off");
  h->pass_mode = mode;
  return FE_OK;
}

fe_status fe_pass_status(fe_drafter *h, void *stream, int32_t *status) {
  if (!h || !status) return fail(FE_E_INVALID, "handle or status is NULL");
  *status = h->last_seg ? (int32_t)kSegStatusPersistent : 0;
  if (!h->seg_ready) return FE_OK;  // no persistent pass has run
  hipStream_t s = (hipStream_t)stream;
  uint32_t *word = (uint32_t *)(h->ws + h->L.tagged) + kSegStatusWord;
  uint32_t v = 0;
  FE_TRY(hipStreamSynchronize(s));
  FE_TRY(hipMemcpy(&v, word, sizeof v, hipMemcpyDeviceToHost));
  if (v) FE_TRY(hipMemset(word, 0, sizeof v));
  *status |= (int32_t)v;
  return FE_OK;
}

fe_status fe_set_attention_split(fe_drafter *h, int32_t chunks_per_workgroup) {
  if (!h) return fail(FE_E_INVALID, "handle is NULL");
  if (chunks_per_workgroup < 0 || chunks_per_workgroup > (1 << 16))
    return fail(FE_E_INVALID, "chunks_per_workgroup %d outside [0, 65536]", chunks_per_workgroup);
  h->attn_split = chunks_per_workgroup;
  return FE_OK;
}

void fe_drafter_destroy(fe_drafter *h) {
  if (!h) return;
  if (h->ev_a) (void)hipEventDestroy(h->ev_a);
  if (h->ev_b) (void)hipEventDestroy(h->ev_b);
  if (h->exec) (void)hipGraphExecDestroy(h->exec);
  if (h->graph) (void)hipGraphDestroy(h->graph);
  if (h->cap_stream) (void)hipStreamDestroy(h->cap_stream);
  for (int i = 0; i < kMaxLayers; ++i) {
    if (h->side[i]) (void)hipStreamDestroy(h->side[i]);
    if (h->ev_join[i]) (void)hipEventDestroy(h->ev_join[i]);
  }
  if (h->ev_fork) (void)hipEventDestroy(h->ev_fork);
  delete h;
}

}  // extern "C"

namespace {


// With only_stage >= 0, a pass launches just the kernels of that stage (used
// to time them); every other launch is skipped.
#define FE_STAGE_RUN(stage, x)                       \
  do {                                               \
    if (only_stage < 0 || only_stage == (stage)) FE_TRY(x); \
  } while (0)
#define FE_OTHER(x)                  \
  do {                               \
    if (only_stage < 0) FE_TRY(x);   \
  } while (0)

// The per-layer streams and fork/join events of FE_CTX_PARALLEL, created once
// per handle before the first pass (never while a graph is being captured).
fe_status ensure_lanes(fe_drafter *h) {
  if (h->cfg.cascade_ctx != FE_CTX_PARALLEL || h->cfg.n_layers < 2) return FE_OK;
  if (!h->ev_fork) FE_TRY(hipEventCreateWithFlags(&h->ev_fork, hipEventDisableTiming));
  for (int i = 0; i < h->cfg.n_layers; ++i) {
    if (!h->side[i]) FE_TRY(hipStreamCreateWithFlags(&h->side[i], hipStreamNonBlocking));
    if (!h->ev_join[i]) FE_TRY(hipEventCreateWithFlags(&h->ev_join[i], hipEventDisableTiming));
  }
  return FE_OK;
}

// The whole pass: FCs of Eq. 1, N cascade layers (Eq. 2), LM head + top-k.
fe_status enqueue_forward(fe_drafter *h, int B, const void *features, const int32_t *next_tokens,
                          const fe_kv_view *kv, int topk, float inv_temp, Draws draws,
                          const fe_draft_out *out, hipStream_t s, int only_stage = -1) {
  const fe_config &c = h->cfg;
  const Layout &L = h->L;
  const int dt = c.dtype == FE_BF16 ? 1 : 0;
  const int d = c.hidden, N = c.n_layers, D = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads;
  const int I = c.intermediate, qd = Hq * D, F = c.n_feat_levels;
  char *ws = h->ws;
  void *cat = ws + L.cat;
  float *X = (float *)(ws + L.X);
  void *an = ws + L.an;  // lane 0: the final norm's rows after the layers
  const long xrow = (long)(N + 1) * d;  // stride between sequences in X
  const int esz = dt ? 2 : 4;
  const int nch = kv->max_prefix > 0 ? (kv->max_prefix + kAttnChunk - 1) / kAttnChunk : 0;
  const int nch_ld = L.nchmax;
  const int cpw = h->attn_split > 0 ? h->attn_split : attention_cpw(B, Hkv, 1, nch);
  const int ntile = d / 16;
  float *ssqX = (float *)(ws + L.ssqX);

  // g_t = FC(concat(l, m, h)) -> cat[:, :d]; e_{t+1} -> cat[:, d:]
  const SplitScratch ss{(float *)(ws + L.splitk), L.splitk_floats};
  FE_STAGE_RUN(FE_STAGE_FUSE, gemm_store(dt, features, F * d, B, F * d, h->w.w_fuse, d, cat, 2 * d, h->w.embed,
                    next_tokens, c.target_vocab, (char *)cat + (size_t)d * esz, 2 * d, d, B, s, &ss));
  // x_0 = FC(concat(g_t, e_{t+1}))  (Eq. 1)
  // Fused RMSNorm (up to 16 rows per GEMM): every producer of a residual row
  // also writes gamma * row for the later GEMMs that normalise it.  Above 16
  // sequences the producers' split-K row pass writes the normalised rows
  // themselves (rows_norm), for every consumer, and no RMSNorm launch remains.
  const bool cascade = c.cascade_ctx == FE_CTX_CASCADE;
  const bool parallel = c.cascade_ctx == FE_CTX_PARALLEL;  // every layer reads x_0
  char *AQ = ws + L.AQ, *AF = ws + L.AF;
  const size_t aq_layer = (size_t)c.max_batch * N * d * esz;  // bytes per layer block of AQ
  auto nctx_of = [&](int l) { return cascade ? l : 1; };
  const bool rows_norm = B > 16 && d <= 8192;
  const float norm_eps = rows_norm ? c.rms_eps : -1.f;
  auto fuse_q = [&](int l) { return rows_norm || B * nctx_of(l) <= 16; };
  const bool fuse_m = rows_norm || B <= 16, fuse_f = rows_norm || B * N <= 16;
  // copies of x_j (j = 0 from the input FC, j = i from layer i's down projection)
  auto x_copies = [&](int j) {
    GainCopies gc{};
    for (int l = j + 1; l <= N; ++l) {
      const bool uses = cascade ? j < l : parallel ? j == 0 : j == l - 1;  // layer l reads x_j
      if (!uses || !fuse_q(l)) continue;
      gc.gamma[gc.n] = h->layers[l - 1].attn_norm;
      gc.dst[gc.n] = AQ + (size_t)(l - 1) * aq_layer + (size_t)j * d * esz;
      gc.ld[gc.n] = (long)N * d;
      ++gc.n;
    }
    if (j >= 1 && fuse_f) {
      gc.gamma[gc.n] = h->w.final_norm;
      gc.dst[gc.n] = AF + (size_t)(j - 1) * d * esz;
      gc.ld[gc.n] = (long)N * d;
      ++gc.n;
    }
    return gc;
  };
  const GainCopies gc_x0 = x_copies(0);
  FE_STAGE_RUN(FE_STAGE_INPUT, gemm_resid(dt, cat, 2 * d, B, 2 * d, h->w.w_in, d, X, xrow, nullptr,
                                      0, rows_norm ? nullptr : ssqX, N + 1, 0, &gc_x0, s, &ss,
                                      norm_eps));

  // Under FE_CTX_PARALLEL the layers are independent (each reads x_0): each
  // runs on a stream of its own, forked from and joined back into `s`, with
  // its own buffers, so that their launches overlap (a captured pass holds
  // them as parallel branches).
  const bool fork = parallel && only_stage < 0 && N > 1;
  hipStream_t lane_stream[kMaxLayers];
  for (int i = 0; i < N; ++i) lane_stream[i] = s;
  if (fork) {
    FE_TRY(hipEventRecord(h->ev_fork, s));  // streams and events: ensure_lanes
    for (int i = 0; i < N; ++i) {
      FE_TRY(hipStreamWaitEvent(h->side[i], h->ev_fork, 0));
      lane_stream[i] = h->side[i];
    }
  }
  for (int i = 1; i <= N; ++i) {
    const Range range("fe.layer");
    const fe_layer_weights &lw = h->layers[i - 1];
    const int src = parallel ? 0 : i - 1;  // the layer's input state
    hipStream_t s = lane_stream[i - 1];
    // this layer's private buffers (lane i - 1 under FE_CTX_PARALLEL)
    const size_t ln = L.lanes > 1 ? (size_t)(i - 1) : 0;
    float *Xp = (float *)(ws + L.Xp + ln * L.Xp_l), *ssqP = (float *)(ws + L.ssqP + ln * L.ssqP_l);
    char *AM = ws + L.AM + ln * L.AM_l;
    void *an = ws + L.an + ln * L.an_l, *bn = ws + L.bn + ln * L.bn_l;
    float *q = (float *)(ws + L.q + ln * L.q_l), *knew = (float *)(ws + L.knew + ln * L.knew_l);
    float *vnew = (float *)(ws + L.vnew + ln * L.vnew_l), *part = (float *)(ws + L.part + ln * L.part_l);
    void *ao = ws + L.ao + ln * L.ao_l, *sbuf = ws + L.s + ln * L.s_l;
    const SplitScratch ss{(float *)(ws + L.splitk + ln * L.splitk_l), L.splitk_floats};
    const int nctx = nctx_of(i), j0 = cascade ? 0 : src;
    // pre-attention RMSNorm of the context rows: fused for up to 16 rows, a
    // separate pass otherwise
    QkvArgs qa{lw.wq, lw.wk, lw.wv, d, D, Hq, Hkv, nctx, j0, cascade ? 1 : 0, Seqs{kv->cu_prefix, 0},
               (const float *)(ws + L.rope), L.npos, q, knew, vnew, dt ? 0 : 1};
    if (fuse_q(i)) {
      const NormA na1{ssqX, ntile, nctx, j0, N + 1, d, c.rms_eps};
      FE_STAGE_RUN(FE_STAGE_QKV, gemm_qkv(dt, AQ + (size_t)(i - 1) * aq_layer, d, ARows{nctx, j0, N},
                                      B * nctx, qa, rows_norm ? nullptr : &na1, s, &ss));
    } else {
      FE_OTHER(rmsnorm_rows(dt, X, B * nctx, nctx, j0, xrow, d, lw.attn_norm, an, d, c.rms_eps, s));
      FE_STAGE_RUN(FE_STAGE_QKV, gemm_qkv(dt, an, d, kDenseRows, B * nctx, qa, nullptr, s, &ss));
    }
    // attention over the layer's prefix cache plus the cascade keys
    FE_STAGE_RUN(FE_STAGE_ATTN, attention(dt, kv->k[i - 1], kv->v[i - 1], Seqs{kv->cu_prefix, 0}, q, knew,
                                      vnew, nctx, part, nch, nch_ld, cpw, ao, B, Hq, Hkv, D,
                                      (const float *)(ws + L.rope), cascade ? 1 : 0,
                                      kv->max_prefix, s));
    // x' = x_{i-1} + W_o o
    GainCopies gc_p{};
    if (fuse_m) {
      gc_p.n = 1;
      gc_p.gamma[0] = lw.mlp_norm;
      gc_p.dst[0] = AM;
      gc_p.ld[0] = d;
    }
    FE_STAGE_RUN(FE_STAGE_OPROJ, gemm_resid(dt, ao, qd, B, qd, lw.wo, d, Xp, d,
                                        X + (size_t)src * d, xrow, rows_norm ? nullptr : ssqP, 1,
                                        0, &gc_p, s, &ss, norm_eps));
    // SwiGLU MLP on RMSNorm(x'), residual into x_i
    if (fuse_m) {
      const NormA na2{ssqP, ntile, 1, 0, 1, d, c.rms_eps};
      FE_STAGE_RUN(FE_STAGE_GATEUP, gemm_swiglu(dt, AM, d, kDenseRows, B, d, lw.w_gate, lw.w_up, I,
                                            sbuf, I, rows_norm ? nullptr : &na2, s));
    } else {
      FE_OTHER(rmsnorm_rows(dt, Xp, B, 1, 0, d, 0, lw.mlp_norm, bn, d, c.rms_eps, s));
      FE_STAGE_RUN(FE_STAGE_GATEUP, gemm_swiglu(dt, bn, d, kDenseRows, B, d, lw.w_gate, lw.w_up, I,
                                            sbuf, I, nullptr, s));
    }
    const GainCopies gc_xi = x_copies(i);
    FE_STAGE_RUN(FE_STAGE_DOWN, gemm_resid(dt, sbuf, I, B, I, lw.w_down, d, X + (size_t)i * d, xrow,
                                       Xp, d, rows_norm ? nullptr : ssqX, N + 1, i, &gc_xi, s, &ss,
                                       norm_eps));
  }
  if (fork)
    for (int i = 0; i < N; ++i) {
      FE_TRY(hipEventRecord(h->ev_join[i], h->side[i]));
      FE_TRY(hipStreamWaitEvent(s, h->ev_join[i], 0));
    }

  // shared LM head on every h_i (rows b*N + i-1), fused softmax statistics and top-k
  const NormA naf{ssqX, ntile, N, 1, N + 1, d, c.rms_eps};
  if (!fuse_f) FE_OTHER(rmsnorm_rows(dt, X, B * N, N, 1, xrow, d, h->w.final_norm, an, d, c.rms_eps, s));
  LmArgs la{h->w.lm_head, c.draft_vocab, topk, out->logits, (float *)(ws + L.pmax),
            (float *)(ws + L.psum), (float *)(ws + L.cval), (int32_t *)(ws + L.cidx), inv_temp,
            draws, (float *)(ws + L.cz)};
  int nwg = 0;
  FE_STAGE_RUN(FE_STAGE_LMHEAD, gemm_lmhead(dt, fuse_f ? (const void *)AF : an, d, kDenseRows, B * N,
                                        d, la, fuse_f && !rows_norm ? &naf : nullptr, &nwg, s));
  // with the Backbone Expansion tree of this pass (root = next token) written
  // by the same launch
  TreeRows tr{};
  if (out->tree) {
    const fe_tree_out *t = out->tree;
    tr = TreeRows{N, next_tokens, kv->cu_prefix, t->tokens, t->parents, t->depth, t->positions,
                  t->mask, t->retrieve};
  }
  FE_OTHER(topk_merge(la.part_max, la.part_sum, la.cand_val, la.cand_idx,
                      draws.on() ? la.cand_z : nullptr, B * N, nwg, topk, c.draft_vocab, h->w.d2t,
                      out->topk_ids, out->topk_draft, out->topk_probs, s,
                      out->tree ? &tr : nullptr));
  if (out->hidden)
    FE_OTHER(hipMemcpyAsync(out->hidden, X, (size_t)B * (N + 1) * d * sizeof(float),
                            hipMemcpyDeviceToDevice, s));
  return FE_OK;
}

// Can the persistent batch-1 pass run this call?  (Otherwise the pass runs as
// one launch per stage.)  Sets h->seg_var / h->seg_nwg on first use.
bool seg_supported(fe_drafter *h, int B, float inv_temp, Draws draws, int topk) {
  const fe_config &c = h->cfg;
  if (!kSegEnabled || h->pass_mode != 0 || B != 1 || draws.on() || inv_temp != 1.f || c.dtype != FE_BF16) return false;
  const long d = c.hidden, N = c.n_layers, I = c.intermediate, qd = (long)c.n_q_heads * c.head_dim;
  const long kvd = (long)c.n_kv_heads * c.head_dim, F = c.n_feat_levels, V = c.draft_vocab;
  if (N > kSegMaxRows || topk > kMaxTopk) return false;
  for (long K : {F * d, 2 * d, d, qd, I})
    if (K % 512) return false;
  if (h->seg_var == -2) {
    int dev = 0, cus = 0;
    h->seg_var = -1;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        cus >= 1 && cus <= kSegMaxWg) {
      const long xbytes = std::max({F * d, 2 * d, N * d, qd, d, I}) * 2;
      const int var = seg_variant((int)xbytes);
      int occ = 0;
      if (var >= 0 && seg_occupancy(var, &occ) == hipSuccess && occ >= 1) {
        h->seg_var = var;
        h->seg_nwg = cus;
      }
    }
    (void)hipGetLastError();
  }
  if (h->seg_var < 0) return false;
  const long nwg = h->seg_nwg;
  auto per_wg = [&](long C, long gran) { return (C / gran + nwg - 1) / nwg * gran; };
  if (d % 2 || per_wg(d, 2) > kSegResRows) return false;               // residual rows
  if (per_wg(V, 1) > kSegLmMaxCols || N * per_wg(V, 1) > kSegRedFloats / 2) return false;
  if (N * per_wg(qd + 2 * kvd, 1) > kSegRedFloats / 2) return false;
  if (per_wg(2 * I, 4) > kSegRedFloats / 2 || per_wg(F * d, 1) > kSegRedFloats / 2) return false;
  return true;
}

// The batch-1 pass as N + 1 persistent launches between the N attention
// launches: [fusion FC, input FC, Q/K/V of layer 1], attention 1, then per
// layer [O, gate/up + SwiGLU, down, Q/K/V of the next layer], attention, and
// finally [O, gate/up, down of layer N, LM head + top-k merge + tree].
fe_status enqueue_forward_seg(fe_drafter *h, const void *features, const int32_t *next_tokens,
                              const fe_kv_view *kv, int topk, const fe_draft_out *out,
                              hipStream_t s) {
  const fe_config &c = h->cfg;
  const Layout &L = h->L;
  const int d = c.hidden, N = c.n_layers, D = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads;
  const int I = c.intermediate, qd = Hq * D, kvd = Hkv * D, F = c.n_feat_levels;
  char *ws = h->ws;
  uint64_t *T = (uint64_t *)(ws + L.tagged);
  uint32_t *sync = (uint32_t *)(T + L.t_sync);
  float *X = (float *)(ws + L.X), *q = (float *)(ws + L.q);
  float *knew = (float *)(ws + L.knew), *vnew = (float *)(ws + L.vnew);
  float *part = (float *)(ws + L.part);
  const bf16_t *ao = (const bf16_t *)(ws + L.ao);
  const bool cascade = c.cascade_ctx == FE_CTX_CASCADE;
  const bool parallel = c.cascade_ctx == FE_CTX_PARALLEL;
  const int nch = kv->max_prefix > 0 ? (kv->max_prefix + kAttnChunk - 1) / kAttnChunk : 0;
  const int cpw = h->attn_split > 0 ? h->attn_split : attention_cpw(1, Hkv, 1, nch);
  auto copy_of = [&](int j, int l) { return T + L.t_copy + ((size_t)j * (N + 1) + l) * (d / 2); };
  auto ssq_of = [&](int j) { return T + L.t_ssq + (size_t)j * kSegMaxWg; };
  auto ssqp_of = [&](int i) { return T + L.t_ssqp + (size_t)(i - 1) * kSegMaxWg; };
  auto xp_of = [&](int i) { return T + L.t_xp + (size_t)(i - 1) * (d / 2); };
  auto s_of = [&](int i) { return T + L.t_s + (size_t)(i - 1) * (I / 2); };
  auto nctx_of = [&](int l) { return cascade ? l : 1; };
  const bf16_t *const *dummy = nullptr;
  (void)dummy;

  SegArgs base{};
  base.nwg = h->seg_nwg;
  base.d = d;
  base.V = c.draft_vocab;
  base.topk = topk;
  base.eps = c.rms_eps;
  base.sync = sync;
  base.cand_t = T + L.t_cand;
  base.d2t = h->w.d2t;
  base.ids = out->topk_ids;
  base.draft_ids = out->topk_draft;
  base.probs = out->topk_probs;
  base.logits = out->logits;
  if (out->tree) {
    const fe_tree_out *t = out->tree;
    base.tree = TreeRows{N, next_tokens, kv->cu_prefix, t->tokens, t->parents, t->depth,
                         t->positions, t->mask, t->retrieve};
  }
  auto src = [](const void *p, int kind, int m, int e0, int n) {
    SegSrc r{};
    r.p = p;
    r.kind = kind;
    r.m = m;
    r.e0 = e0;
    r.n = n;
    return r;
  };
  // normalised copies of x_j for its consumers: the Q/K/V GEMVs of the layers
  // that read it and (j >= 1) the LM head
  auto copies_x = [&](SegStage &st, int j) {
    st.ncopy = 0;
    for (int l = j + 1; l <= N; ++l) {
      const bool uses = cascade ? true : parallel ? j == 0 : l == j + 1;
      if (!uses) continue;
      st.gamma[st.ncopy] = (const bf16_t *)h->layers[l - 1].attn_norm;
      st.copy_t[st.ncopy] = copy_of(j, l);
      ++st.ncopy;
    }
    if (j >= 1) {
      st.gamma[st.ncopy] = (const bf16_t *)h->w.final_norm;
      st.copy_t[st.ncopy] = copy_of(j, 0);
      ++st.ncopy;
    }
  };
  auto qkv = [&](int l) {
    const fe_layer_weights &lw = h->layers[l - 1];
    SegStage st{};
    st.kind = kSegQkv;
    st.C = qd + 2 * kvd;
    st.K = d;
    st.mr = nctx_of(l);
    st.gran = 1;
    st.w0 = (const bf16_t *)lw.wq;
    st.w1 = (const bf16_t *)lw.wk;
    st.w2 = (const bf16_t *)lw.wv;
    st.split1 = qd;
    st.split2 = qd + kvd;
    st.qrow = st.mr - 1;
    st.nsrc = st.mr;
    for (int t = 0; t < st.mr; ++t) {
      const int j = cascade ? t : parallel ? 0 : l - 1;
      st.src[t] = src(copy_of(j, l), kSrcTagged, t, 0, d);
      st.ssq[t] = ssq_of(j);
    }
    st.x_out = q;
    st.k_out = knew;
    st.v_out = vnew;
    return st;
  };
  auto oproj = [&](int i) {
    const fe_layer_weights &lw = h->layers[i - 1];
    SegStage st{};
    st.kind = kSegO;
    st.C = d;
    st.K = qd;
    st.mr = 1;
    st.gran = 2;
    st.w0 = (const bf16_t *)lw.wo;
    st.nsrc = 1;
    st.src[0] = src(ao, kSrcPlain, 0, 0, qd);
    st.resid = X + (size_t)(parallel ? 0 : i - 1) * d;
    st.ssq_out = ssqp_of(i);
    st.ncopy = 1;
    st.gamma[0] = (const bf16_t *)lw.mlp_norm;
    st.copy_t[0] = xp_of(i);
    return st;
  };
  auto gateup = [&](int i) {
    const fe_layer_weights &lw = h->layers[i - 1];
    SegStage st{};
    st.kind = kSegGu;
    st.C = 2 * I;
    st.K = d;
    st.mr = 1;
    st.gran = 4;
    st.w0 = (const bf16_t *)lw.w_gate;
    st.w1 = (const bf16_t *)lw.w_up;
    st.nsrc = 1;
    st.src[0] = src(xp_of(i), kSrcTagged, 0, 0, d);
    st.ssq[0] = ssqp_of(i);
    st.out_t = s_of(i);
    return st;
  };
  auto down = [&](int i) {
    const fe_layer_weights &lw = h->layers[i - 1];
    SegStage st{};
    st.kind = kSegDown;
    st.C = d;
    st.K = I;
    st.mr = 1;
    st.gran = 2;
    st.w0 = (const bf16_t *)lw.w_down;
    st.nsrc = 1;
    st.src[0] = src(s_of(i), kSrcTagged, 0, 0, I);
    st.x_out = X + (size_t)i * d;
    st.ssq_out = ssq_of(i);
    copies_x(st, i);
    return st;
  };
  auto attn = [&](int l) -> fe_status {
    FE_TRY(attention(1, kv->k[l - 1], kv->v[l - 1], Seqs{kv->cu_prefix, 0}, q, knew, vnew, nctx_of(l),
                     part, nch, L.nchmax, cpw, (void *)ao, 1, Hq, Hkv, D,
                     (const float *)(ws + L.rope), cascade ? 1 : 0, kv->max_prefix, s));
    return FE_OK;
  };
  auto launch = [&](std::initializer_list<SegStage> stages, int last) -> fe_status {
    SegArgs a = base;
    a.nst = 0;
    for (const SegStage &st : stages) a.st[a.nst++] = st;
    a.last = last;
    FE_TRY(seg_launch(h->seg_var, a, s));
    return FE_OK;
  };

  // [g_t = FC(l, m, h); x_0 = FC(g_t, e_{t+1}) (Eq. 1); Q/K/V of layer 1]
  SegStage fuse{};
  fuse.kind = kSegFuse;
  fuse.C = d;
  fuse.K = F * d;
  fuse.mr = 1;
  fuse.gran = 2;
  fuse.w0 = (const bf16_t *)h->w.w_fuse;
  fuse.nsrc = 1;
  fuse.src[0] = src(features, kSrcPlain, 0, 0, F * d);
  fuse.out_t = T + L.t_g;
  SegStage input{};
  input.kind = kSegInput;
  input.C = d;
  input.K = 2 * d;
  input.mr = 1;
  input.gran = 2;
  input.w0 = (const bf16_t *)h->w.w_in;
  input.nsrc = 2;
  input.src[0] = src(T + L.t_g, kSrcTagged, 0, 0, d);
  input.src[1] = src(h->w.embed, kSrcEmbed, 0, d, d);
  input.src[1].tok = next_tokens;
  input.src[1].vocab = c.target_vocab;
  input.x_out = X;
  input.ssq_out = ssq_of(0);
  copies_x(input, 0);
  fe_status st = launch({fuse, input, qkv(1)}, 0);
  if (st != FE_OK) return st;
  for (int i = 1; i <= N; ++i) {
    if ((st = attn(i)) != FE_OK) return st;
    if (i < N) {
      st = launch({oproj(i), gateup(i), down(i), qkv(i + 1)}, 0);
    } else {
      SegStage lm{};
      lm.kind = kSegLm;
      lm.C = c.draft_vocab;
      lm.K = d;
      lm.mr = N;
      lm.gran = 1;
      lm.w0 = (const bf16_t *)h->w.lm_head;
      lm.nsrc = N;
      for (int t = 0; t < N; ++t) {
        lm.src[t] = src(copy_of(t + 1, 0), kSrcTagged, t, 0, d);
        lm.ssq[t] = ssq_of(t + 1);
      }
      lm.out_t = T + L.t_cand;
      st = launch({oproj(i), gateup(i), down(i), lm}, 1);
    }
    if (st != FE_OK) return st;
  }
  if (out->hidden)
    FE_TRY(hipMemcpyAsync(out->hidden, X, (size_t)(N + 1) * d * sizeof(float),
                          hipMemcpyDeviceToDevice, s));
  return FE_OK;
}

}  // namespace

extern "C" fe_status fe_draft_forward(fe_drafter *h, int32_t batch, const void *features,
                                      const int32_t *next_tokens, const fe_kv_view *kv,
                                      int32_t topk, const fe_draft_out *out, void *stream) {
  return fe_draft_sample(h, batch, features, next_tokens, kv, topk, 1.0f, nullptr, out, stream);
}

namespace {
fe_status draft_sample_impl(fe_drafter *h, int32_t batch, const void *features,
                            const int32_t *next_tokens, const fe_kv_view *kv, int32_t topk,
                            float temperature, Draws draws, const fe_draft_out *out, void *stream);
}  // namespace

extern "C" fe_status fe_draft_sample(fe_drafter *h, int32_t batch, const void *features,
                                     const int32_t *next_tokens, const fe_kv_view *kv,
                                     int32_t topk, float temperature, const float *uniforms,
                                     const fe_draft_out *out, void *stream) {
  if (uniforms && ((uintptr_t)uniforms & 3u)) return fail(FE_E_ALIGN, "uniforms must be 4-byte aligned");
  Draws dr;
  dr.u = uniforms;
  return draft_sample_impl(h, batch, features, next_tokens, kv, topk, temperature, dr, out, stream);
}

extern "C" fe_status fe_draft_sample_seeded(fe_drafter *h, int32_t batch, const void *features,
                                            const int32_t *next_tokens, const fe_kv_view *kv,
                                            int32_t topk, float temperature,
                                            const uint64_t *seed_offset, const fe_draft_out *out,
                                            void *stream) {
  if (!seed_offset) return fail(FE_E_INVALID, "seed_offset is NULL");
  if ((uintptr_t)seed_offset & 7u) return fail(FE_E_ALIGN, "seed_offset must be 8-byte aligned");
  Draws dr;
  dr.so = seed_offset;
  return draft_sample_impl(h, batch, features, next_tokens, kv, topk, temperature, dr, out, stream);
}

namespace {
fe_status draft_sample_impl(fe_drafter *h, int32_t batch, const void *features,
                            const int32_t *next_tokens, const fe_kv_view *kv, int32_t topk,
                            float temperature, Draws draws, const fe_draft_out *out, void *stream) {
  const Range range("fe_draft_sample");
  if (!h) return fail(FE_E_INVALID, "handle is NULL");
  const fe_config &c = h->cfg;
  if (!(temperature > 0.f) || !(temperature < INFINITY))
    return fail(FE_E_INVALID, "temperature must be positive and finite");
  const float inv_temp = 1.0f / temperature;
  if (!(inv_temp < INFINITY)) return fail(FE_E_INVALID, "temperature %g is too small", temperature);
  if (batch < 0 || batch > c.max_batch) return fail(FE_E_INVALID, "batch %d outside [0, %d]", batch, c.max_batch);
  if (topk < 1 || topk > c.max_topk || topk > c.draft_vocab)
    return fail(FE_E_INVALID, "topk %d outside [1, %d]", topk, c.max_topk);
  if (!out || !out->topk_ids || !out->topk_probs) return fail(FE_E_INVALID, "out, out->topk_ids and out->topk_probs are required");
  if (!kv || !kv->k || !kv->v || !kv->cu_prefix) return fail(FE_E_INVALID, "kv view is incomplete");
  if (kv->max_prefix < 0 || kv->max_prefix > c.max_prefix)
    return fail(FE_E_INVALID, "kv->max_prefix %d outside [0, %d]", kv->max_prefix, c.max_prefix);
  if (batch == 0) return FE_OK;
  if (!features || !next_tokens) return fail(FE_E_INVALID, "features and next_tokens are required");
  if (!aligned16(features)) return fail(FE_E_ALIGN, "features must be 16-byte aligned");
  for (int l = 0; l < c.n_layers; ++l) {
    if (kv->max_prefix > 0 && (!kv->k[l] || !kv->v[l]))
      return fail(FE_E_INVALID, "kv cache pointer of layer %d is NULL", l);
    if (!aligned16(kv->k[l]) || !aligned16(kv->v[l]))
      return fail(FE_E_ALIGN, "kv cache of layer %d is not 16-byte aligned", l);
  }
  if (out->logits && ((uintptr_t)out->logits & 3u)) return fail(FE_E_ALIGN, "logits misaligned");
  if (out->tree) {
    const fe_tree_out *t = out->tree;
    if (!t->tokens || !t->parents || !t->depth || !t->positions || !t->mask || !t->retrieve)
      return fail(FE_E_INVALID, "every tree output is required when out->tree is set");
  }
  hipStream_t s = (hipStream_t)stream;
  if (!h->table_ready) {  // first pass on this handle: the rotary table
    FE_TRY(rope_table((float *)(h->ws + h->L.rope), h->L.npos, c.head_dim, (double)c.rope_theta, s));
    h->table_ready = true;
  }
  {
    const fe_status st = ensure_lanes(h);
    if (st != FE_OK) return st;
  }

  // remember the call for fe_time_stage
  h->have_last = true;
  h->last_batch = batch;
  h->last_topk = topk;
  h->last_inv_temp = inv_temp;
  h->last_draws = draws;
  h->last_features = features;
  h->last_tokens = next_tokens;
  h->last_k.assign(kv->k, kv->k + c.n_layers);
  h->last_v.assign(kv->v, kv->v + c.n_layers);
  h->last_kv = *kv;
  h->last_kv.k = h->last_k.data();
  h->last_kv.v = h->last_v.data();
  h->last_out = *out;
  if (out->tree) {
    h->last_tree = *out->tree;
    h->last_out.tree = &h->last_tree;
  }

  const bool seg = seg_supported(h, batch, inv_temp, draws, topk);
  h->last_seg = seg;
  if (seg && !h->seg_ready) {  // tagged words start at tag 0, below every pass's tag
    FE_TRY(seg_zero((uint64_t *)(h->ws + h->L.tagged), h->L.t_words, s));
    h->seg_ready = true;
  }
  auto enqueue = [&](hipStream_t st) {
    return seg ? enqueue_forward_seg(h, features, next_tokens, kv, topk, out, st)
               : enqueue_forward(h, batch, features, next_tokens, kv, topk, inv_temp, draws,
                                 out, st);
  };
  if (!h->graph_mode) return enqueue(s);

  std::vector<uintptr_t> key = {(uintptr_t)batch, (uintptr_t)features, (uintptr_t)next_tokens,
                                (uintptr_t)kv->cu_prefix, (uintptr_t)kv->max_prefix,
                                (uintptr_t)topk, (uintptr_t)out->topk_ids,
                                (uintptr_t)out->topk_probs, (uintptr_t)out->topk_draft,
                                (uintptr_t)(out->tree ? out->tree->tokens : nullptr),
                                (uintptr_t)(out->tree ? out->tree->parents : nullptr),
                                (uintptr_t)(out->tree ? out->tree->depth : nullptr),
                                (uintptr_t)(out->tree ? out->tree->positions : nullptr),
                                (uintptr_t)(out->tree ? out->tree->mask : nullptr),
                                (uintptr_t)(out->tree ? out->tree->retrieve : nullptr),
                                (uintptr_t)out->logits, (uintptr_t)out->hidden,
                                (uintptr_t)h->attn_split, (uintptr_t)__builtin_bit_cast(uint32_t, inv_temp),
                                (uintptr_t)draws.u, (uintptr_t)draws.so, (uintptr_t)seg};
  for (int l = 0; l < c.n_layers; ++l) {
    key.push_back((uintptr_t)kv->k[l]);
    key.push_back((uintptr_t)kv->v[l]);
  }
  if (!h->exec || key != h->key) {
    if (!h->cap_stream) FE_TRY(hipStreamCreateWithFlags(&h->cap_stream, hipStreamNonBlocking));
    if (h->exec) { (void)hipGraphExecDestroy(h->exec); h->exec = nullptr; }
    if (h->graph) { (void)hipGraphDestroy(h->graph); h->graph = nullptr; }
    h->key.clear();
    FE_TRY(hipStreamBeginCapture(h->cap_stream, hipStreamCaptureModeThreadLocal));
    fe_status st = enqueue(h->cap_stream);
    hipGraph_t g = nullptr;
    hipError_t ec = hipStreamEndCapture(h->cap_stream, &g);
    if (st != FE_OK) { if (g) (void)hipGraphDestroy(g); return st; }
    if (ec != hipSuccess) return fail(FE_E_HIP, "hipStreamEndCapture: %s", hipGetErrorString(ec));
    h->graph = g;
    FE_TRY(hipGraphInstantiate(&h->exec, g, nullptr, nullptr, 0));
    h->key = key;
  }
  FE_TRY(hipGraphLaunch(h->exec, s));
  return FE_OK;
}
}  // namespace

extern "C" fe_status fe_time_stage(fe_drafter *h, int32_t stage, int32_t repeats, void *stream,
                                   float *ms_per_launch, int32_t *launches) {
  const Range range("fe_time_stage");
  if (!h || !ms_per_launch || !launches) return fail(FE_E_INVALID, "bad arguments");
  if (stage < FE_STAGE_FUSE || stage > FE_STAGE_PASS) return fail(FE_E_INVALID, "unknown stage %d", stage);
  if (repeats < 1) return fail(FE_E_INVALID, "repeats must be >= 1");
  if (!h->have_last) return fail(FE_E_INVALID, "no fe_draft_forward call to replay yet");
  const int N = h->cfg.n_layers;
  const int per_pass = (stage == FE_STAGE_FUSE || stage == FE_STAGE_INPUT || stage == FE_STAGE_LMHEAD ||
                        stage == FE_STAGE_PASS) ? 1 : N;
  const bool seg = stage == FE_STAGE_PASS &&
                   seg_supported(h, h->last_batch, h->last_inv_temp, h->last_draws, h->last_topk);
  hipStream_t s = (hipStream_t)stream;
  if (!h->ev_a) FE_TRY(hipEventCreate(&h->ev_a));
  if (!h->ev_b) FE_TRY(hipEventCreate(&h->ev_b));
  FE_TRY(hipEventRecord(h->ev_a, s));
  for (int r = 0; r < repeats; ++r) {
    const fe_status st =
        seg ? enqueue_forward_seg(h, h->last_features, h->last_tokens, &h->last_kv, h->last_topk,
                                  &h->last_out, s)
            : enqueue_forward(h, h->last_batch, h->last_features, h->last_tokens, &h->last_kv,
                              h->last_topk, h->last_inv_temp, h->last_draws, &h->last_out, s,
                              stage == FE_STAGE_PASS ? -1 : stage);
    if (st != FE_OK) return st;
  }
  FE_TRY(hipEventRecord(h->ev_b, s));
  FE_TRY(hipEventSynchronize(h->ev_b));
  float ms = 0.f;
  FE_TRY(hipEventElapsedTime(&ms, h->ev_a, h->ev_b));
  *ms_per_launch = ms / (float)(repeats * per_pass);
  *launches = per_pass;
  return FE_OK;
}

// Test export (host only, no device work): the pieces the persistent bf16
// attention's waves take for the given prefix lengths, from the same split
// arithmetic the kernel runs (AttnSplit, attn_prefix, attn_seg_chunks).
// Test export: one layer's attention exactly as the pass launches it, on
// caller buffers, with its own (allocated and freed) rotary table and partials.
extern "C" fe_status fe_test_attention(int32_t dtype, int32_t batch, int32_t n_q_heads,
                                       int32_t n_kv_heads, int32_t head_dim, const void *k_cache,
                                       const void *v_cache, const int32_t *cu_prefix,
                                       int32_t max_prefix, const float *q, const float *knew,
                                       const float *vnew, int32_t nctx, int32_t cascade,
                                       double rope_theta, int32_t chunks_per_workgroup, void *out,
                                       void *stream) {
  if (dtype != FE_BF16 && dtype != FE_F32) return fail(FE_E_INVALID, "dtype %d", dtype);
  if (batch < 0 || n_kv_heads < 1 || n_q_heads % n_kv_heads || max_prefix < 0 ||
      chunks_per_workgroup < 0 || nctx < 1 || nctx > kMaxLayers)
    return fail(FE_E_INVALID, "bad attention shape");
  if (head_dim != 64 && head_dim != 128) return fail(FE_E_UNSUPPORTED, "head_dim %d", head_dim);
  if (batch == 0) return FE_OK;
  if (!cu_prefix || !q || !knew || !vnew || !out || (max_prefix > 0 && (!k_cache || !v_cache)))
    return fail(FE_E_INVALID, "attention inputs are required");
  const int dt = dtype == FE_BF16 ? 1 : 0, D = head_dim, Hq = n_q_heads, Hkv = n_kv_heads;
  const int nch = max_prefix > 0 ? (max_prefix + kAttnChunk - 1) / kAttnChunk : 0;
  const int nch_ld = (max_prefix > 0 ? nch : 1) + 1;
  const int npos = max_prefix + nctx;
  const int cpw = chunks_per_workgroup > 0 ? chunks_per_workgroup : attention_cpw(batch, Hkv, 1, nch);
  hipStream_t s = (hipStream_t)stream;
  float *rope = nullptr, *part = nullptr;
  const size_t part_floats = (size_t)batch * Hq * ((size_t)nch_ld * (D + 2) + 1);
  FE_TRY(hipMalloc(&rope, (size_t)npos * (D / 2) * 2 * sizeof(float)));
  hipError_t e = hipMalloc(&part, part_floats * sizeof(float));
  if (e == hipSuccess) e = rope_table(rope, npos, D, rope_theta, s);
  if (e == hipSuccess)
    e = attention(dt, k_cache, v_cache, Seqs{cu_prefix, 0}, q, knew, vnew, nctx, part, nch, nch_ld,
                  cpw, out, batch, Hq, Hkv, D, rope, cascade ? 1 : 0, max_prefix, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  (void)hipFree(part);
  (void)hipFree(rope);
  if (e != hipSuccess) return fail(FE_E_HIP, "fe_test_attention: %s", hipGetErrorString(e));
  return FE_OK;
}

// Test export: the standalone RMSNorm launch (fp32 rows in, storage dtype out).
extern "C" fe_status fe_test_rmsnorm(int32_t dtype, const float *x, int32_t rows, int32_t d,
                                     const void *gamma, float eps, void *out, void *stream) {
  if (dtype != FE_BF16 && dtype != FE_F32) return fail(FE_E_INVALID, "dtype %d", dtype);
  if (rows < 0 || d < 4 || d % 4 || d > 8192) return fail(FE_E_INVALID, "bad shape");
  if (rows == 0) return FE_OK;
  if (!x || !gamma || !out) return fail(FE_E_INVALID, "inputs are required");
  FE_TRY(rmsnorm_rows(dtype == FE_BF16 ? 1 : 0, x, rows, 1, 0, d, 0, gamma, out, d, eps,
                      (hipStream_t)stream));
  return FE_OK;
}

extern "C" fe_status fe_test_attn_split(const int32_t *prefix_lens, int32_t batch, int32_t ncols,
                                        int32_t nch_ld, int32_t pmax, int32_t waves,
                                        int32_t *pieces, int32_t max_pieces, int32_t *n_pieces) {
  if (!prefix_lens || (!pieces && max_pieces > 0) || !n_pieces || batch < 1 || batch > 256 || ncols < 1 ||
      nch_ld < 1 || waves < 1 || max_pieces < 0)
    return fail(FE_E_INVALID, "bad arguments");
  std::vector<int32_t> cu(batch + 1, 0);
  for (int b = 0; b < batch; ++b) cu[b + 1] = cu[b] + prefix_lens[b];
  std::vector<long> uend(batch);
  std::vector<int> ucnt(batch);
  long run = 0;
  for (int b = 0; b < batch; ++b) {
    bool bad;
    ucnt[b] = attn_seg_chunks(attn_prefix(Seqs{cu.data(), 0}, b, pmax, bad), nch_ld) * ncols;
    run += ucnt[b];
    uend[b] = run;
  }
  const AttnSplit eq{run, std::min<long>(waves, run)};
  int np_out = 0;
  for (long w = 0; w < eq.W; ++w) {
    int x = eq.begin(w);
    const int xe = eq.begin(w + 1);
    while (x < xe) {
      int b = 0;
      while (b < batch && uend[b] <= x) ++b;  // sequences wholly before chunk x
      if (b >= batch) return fail(FE_E_INVALID, "split walked past the last sequence");
      int col, ch0, n, slot, np;
      eq.piece(x, xe, (int)(uend[b] - ucnt[b]), ucnt[b], ncols, col, ch0, n, slot, np);
      if (np_out < max_pieces) {
        int32_t *r = pieces + (size_t)np_out * 7;
        r[0] = (int32_t)w; r[1] = b; r[2] = col; r[3] = ch0; r[4] = n; r[5] = slot; r[6] = np;
      }
      ++np_out;
      if (n < 1) return fail(FE_E_INVALID, "empty piece");
      x += n;
    }
  }
  *n_pieces = np_out;
  return FE_OK;
}

extern "C" fe_status fe_accept_greedy(fe_drafter *h, int32_t batch, int32_t topk,
                                      const int32_t *tokens, const int32_t *retrieve,
                                      const int32_t *target_next, int32_t *accept_len,
                                      int32_t *accept_path, int32_t *accepted, void *stream) {
  const Range range("fe_accept_greedy");
  if (!h) return fail(FE_E_INVALID, "handle is NULL");
  const fe_config &c = h->cfg;
  if (batch < 0 || batch > c.max_batch) return fail(FE_E_INVALID, "batch %d outside [0, %d]", batch, c.max_batch);
  if (topk < 1 || topk > c.max_topk) return fail(FE_E_INVALID, "topk %d outside [1, %d]", topk, c.max_topk);
  if (batch == 0) return FE_OK;
  if (!tokens || !retrieve || !target_next || !accept_len || !accept_path || !accepted)
    return fail(FE_E_INVALID, "every acceptance input and output is required");
  const void *ptrs[] = {tokens, retrieve, target_next, accept_len, accept_path, accepted};
  for (const void *q : ptrs)
    if ((uintptr_t)q & 3u) return fail(FE_E_ALIGN, "acceptance arrays must be 4-byte aligned");
  FE_TRY(accept_greedy(batch, c.n_layers, topk, tokens, retrieve, target_next, accept_len,
                       accept_path, accepted, (hipStream_t)stream));
  return FE_OK;
}

extern "C" size_t fe_kv_update_workspace_bytes(const fe_config *cfg, int32_t chunk_rows) {
  if (check_config(cfg) != FE_OK) return 0;
  if (chunk_rows < 1) {
    fail(FE_E_INVALID, "chunk_rows must be positive");
    return 0;
  }
  return upd_layout_of(*cfg, (size_t)chunk_rows).total;
}

// Drafter cache rows of verified positions (Section 2.4 update step, cascade
// context): x_0 of every row as in the pass (Eq. 1), then per layer its
// RMSNorm and the rotated K / V projections, scattered into the caches.
namespace {
// The N layers over Mc new rows of the self context, whose x_0 rows are in U.X:
// layer by layer, every row's Q/K/V, its K/V into the cache, then its attention
// over its sequence's rows of earlier positions (the rows this step just wrote
// included) plus its own key, the O projection, the MLP, x_i into U.X.  Rows
// go in slices of at most kGemmMaxRows per launch.
fe_status prefill_layers(fe_drafter *h, const UpdLayout &U, char *ws, int Mc,
                         const int32_t *positions, const int32_t *dst_rows,
                         const fe_kv_cache *cache, const SplitScratch *ss, hipStream_t s) {
  const fe_config &c = h->cfg;
  const int dt = c.dtype == FE_BF16 ? 1 : 0, es = es_of(c);
  const int d = c.hidden, D = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads, I = c.intermediate;
  const int qd = Hq * D, kvd = Hkv * D;
  float *X = (float *)(ws + U.X), *Xp = (float *)(ws + U.Xp);
  float *q = (float *)(ws + U.q), *knew = (float *)(ws + U.knew), *vnew = (float *)(ws + U.vnew);
  char *an = ws + U.an, *ao = ws + U.ao, *sb = ws + U.sb;
  int32_t *ranges = (int32_t *)(ws + U.ranges);
  float *part = (float *)(ws + U.part);
  const float *rope = (const float *)(h->ws + h->L.rope);
  const int pmax = c.max_prefix;
  const int nch = (pmax + kAttnChunk - 1) / kAttnChunk;
  FE_TRY(prefill_ranges(positions, dst_rows, Mc, (long)cache->rows, c.max_prefix, pmax, ranges, s));
  // bf16 chunks of more rows than one batched launch takes: every GEMM as one
  // 2-D tiled launch over all rows (each weight matrix streamed once per chunk)
  const bool tiled = dt && Mc >= kTiledRows;
  for (int l = 0; l < c.n_layers; ++l) {
    const Range range("fe.prefill_layer");
    const fe_layer_weights &lw = h->layers[l];
    FE_TRY(rmsnorm_rows(dt, X, Mc, 1, 0, d, 0, lw.attn_norm, an, d, c.rms_eps, s));
    if (tiled) {
      // q, K, V of every row (fp32, unrotated: the attention rotates them)
      FE_TRY(gemm_resid_rows(an, d, Mc, d, lw.wq, qd, q, qd, s));
      FE_TRY(gemm_resid_rows(an, d, Mc, d, lw.wk, kvd, knew, kvd, s));
      FE_TRY(gemm_resid_rows(an, d, Mc, d, lw.wv, kvd, vnew, kvd, s));
    }
    for (int s0 = 0; s0 < Mc && !tiled; s0 += kGemmMaxRows) {
      const int Ms = std::min(kGemmMaxRows, Mc - s0);
      const QkvArgs qa{lw.wq, lw.wk, lw.wv, d, D, Hq, Hkv, 1, 0, 0, Seqs{ranges + 2 * s0, 1},
                       rope, h->L.npos, q + (size_t)s0 * qd, knew + (size_t)s0 * kvd,
                       vnew + (size_t)s0 * kvd, dt ? 0 : 1};
      FE_TRY(gemm_qkv(dt, an + (size_t)s0 * d * es, d, kDenseRows, Ms, qa, nullptr, s, ss));
    }
    // every row's K/V is in the cache before any row's attention reads it
    FE_TRY(kv_scatter(dt, knew, vnew, Mc, Hkv, D, positions, dst_rows, (long)cache->rows,
                      c.max_prefix, rope, dt ? 0 : 1, cache->k[l], cache->v[l], s));
    for (int s0 = 0; s0 < Mc; s0 += kGemmMaxRows) {
      const int Ms = std::min(kGemmMaxRows, Mc - s0);
      const int cpw = h->attn_split > 0 ? h->attn_split : attention_cpw(Ms, Hkv, 1, nch);
      FE_TRY(attention(dt, cache->k[l], cache->v[l], Seqs{ranges + 2 * s0, 1},
                       q + (size_t)s0 * qd, knew + (size_t)s0 * kvd, vnew + (size_t)s0 * kvd, 1,
                       part, nch, U.nch_ld, cpw, ao + (size_t)s0 * qd * es, Ms, Hq, Hkv, D, rope,
                       0, pmax, s));
    }
    if (tiled) {  // x' = x_{i-1} + W_o o
      FE_TRY(gemm_resid_rows(ao, qd, Mc, qd, lw.wo, d, Xp, d, s, X, d));
    }
    for (int s0 = 0; s0 < Mc && !tiled; s0 += kGemmMaxRows) {
      const int Ms = std::min(kGemmMaxRows, Mc - s0);
      // x' = x_{i-1} + W_o o
      FE_TRY(gemm_resid(dt, ao + (size_t)s0 * qd * es, qd, Ms, qd, lw.wo, d, Xp + (size_t)s0 * d,
                        d, X + (size_t)s0 * d, d, nullptr, 1, 0, nullptr, s, ss));
    }
    FE_TRY(rmsnorm_rows(dt, Xp, Mc, 1, 0, d, 0, lw.mlp_norm, an, d, c.rms_eps, s));
    if (tiled) {  // SwiGLU rows, then x_i = x' + W_d s (Eq. 2)
      FE_TRY(gemm_swiglu_rows(an, d, Mc, d, lw.w_gate, lw.w_up, I, sb, I, s));
      FE_TRY(gemm_resid_rows(sb, I, Mc, I, lw.w_down, d, X, d, s, Xp, d));
    }
    for (int s0 = 0; s0 < Mc && !tiled; s0 += kGemmMaxRows) {
      const int Ms = std::min(kGemmMaxRows, Mc - s0);
      FE_TRY(gemm_swiglu(dt, an + (size_t)s0 * d * es, d, kDenseRows, Ms, d, lw.w_gate, lw.w_up, I,
                         sb + (size_t)s0 * I * es, I, nullptr, s));
      // x_i = x' + W_d s (Eq. 2)
      FE_TRY(gemm_resid(dt, sb + (size_t)s0 * I * es, I, Ms, I, lw.w_down, d, X + (size_t)s0 * d,
                        d, Xp + (size_t)s0 * d, d, nullptr, 1, 0, nullptr, s, ss));
    }
  }
  return FE_OK;
}

fe_status kv_update_impl(fe_drafter *h, int32_t n_rows, const void *features,
                         const int32_t *tokens, const int32_t *positions,
                         const int32_t *dst_rows, const fe_kv_cache *cache, void *workspace,
                         size_t ws_bytes, void *stream) {
  const Range range("fe_kv_update");
  if (!h) return fail(FE_E_INVALID, "handle is NULL");
  const fe_config &c = h->cfg;
  if (n_rows < 0) return fail(FE_E_INVALID, "n_rows %d is negative", n_rows);
  if (!cache || !cache->k || !cache->v) return fail(FE_E_INVALID, "cache and its pointer arrays are required");
  if (cache->rows < 0) return fail(FE_E_INVALID, "cache->rows is negative");
  if (n_rows == 0) return FE_OK;
  if (c.max_prefix < 1) return fail(FE_E_INVALID, "config max_prefix is 0: no cache position is valid");
  if (!features || !tokens || !positions || !dst_rows)
    return fail(FE_E_INVALID, "features, tokens, positions and dst_rows are required");
  if (!aligned16(features)) return fail(FE_E_ALIGN, "features must be 16-byte aligned");
  const void *ip[] = {tokens, positions, dst_rows};
  for (const void *q : ip)
    if ((uintptr_t)q & 3u) return fail(FE_E_ALIGN, "tokens, positions and dst_rows must be 4-byte aligned");
  for (int l = 0; l < c.n_layers; ++l) {
    if (!cache->k[l] || !cache->v[l]) return fail(FE_E_INVALID, "cache pointer of layer %d is NULL", l);
    if (!aligned16(cache->k[l]) || !aligned16(cache->v[l]))
      return fail(FE_E_ALIGN, "cache of layer %d is not 16-byte aligned", l);
  }
  if (!workspace) return fail(FE_E_WORKSPACE, "workspace is NULL");
  if (((uintptr_t)workspace & 255u)) return fail(FE_E_ALIGN, "workspace must be 256-byte aligned");
  // rows per chunk: the most that fit the workspace, up to n_rows
  size_t lo = 1, hi = (size_t)n_rows;
  if (upd_layout_of(c, 1).total > ws_bytes)
    return fail(FE_E_WORKSPACE, "workspace of %zu bytes is below the %zu bytes of one row", ws_bytes,
                upd_layout_of(c, 1).total);
  while (lo < hi) {
    const size_t mid = (lo + hi + 1) / 2;
    if (upd_layout_of(c, mid).total <= ws_bytes) lo = mid;
    else hi = mid - 1;
  }
  const int C = (int)lo;
  const UpdLayout U = upd_layout_of(c, (size_t)C);
  hipStream_t s = (hipStream_t)stream;
  if (!h->table_ready) {
    FE_TRY(rope_table((float *)(h->ws + h->L.rope), h->L.npos, c.head_dim, (double)c.rope_theta, s));
    h->table_ready = true;
  }
  const int dt = c.dtype == FE_BF16 ? 1 : 0, es = es_of(c);
  const int d = c.hidden, F = c.n_feat_levels, kvd = c.n_kv_heads * c.head_dim;
  char *ws = (char *)workspace;
  char *cat = ws + U.cat, *an = ws + U.an;
  float *X = (float *)(ws + U.X);
  const SplitScratch ss{(float *)(ws + U.splitk), U.splitk_floats};
  // bf16: every layer's K/V projection in one launch
  auto layer_args = [&](int r0, KvCacheArgs *la) {
    for (int l = 0; l < c.n_layers; ++l) {
      const fe_layer_weights &lw = h->layers[l];
      la[l] = KvCacheArgs{lw.wk, lw.wv, d, c.head_dim, c.n_kv_heads, positions + r0,
                          dst_rows + r0, (long)cache->rows, c.max_prefix,
                          (const float *)(h->ws + h->L.rope), cache->k[l], cache->v[l]};
    }
  };
  const bool self = c.cascade_ctx == FE_CTX_SELF;
  for (int r0 = 0; r0 < n_rows; r0 += C) {
    const int Mc = std::min(C, n_rows - r0);
    if (dt && Mc <= kFusedRows && !self) {
      // few rows: the input FC also writes gamma_l * x_0 for every layer and
      // the rows' sums of squares, and the K/V launch applies 1/rms
      FE_TRY(gemm_store(dt, (const char *)features + (size_t)r0 * F * d * es, F * d, Mc, F * d,
                        h->w.w_fuse, d, cat, 2 * d, h->w.embed, tokens + r0, c.target_vocab,
                        cat + (size_t)d * es, 2 * d, d, Mc, s, &ss));
      GainCopies gc{};
      gc.n = c.n_layers;
      for (int l = 0; l < c.n_layers; ++l) {
        gc.gamma[l] = h->layers[l].attn_norm;
        gc.dst[l] = an + (size_t)l * C * d * es;
        gc.ld[l] = d;
      }
      float *ssq = (float *)(ws + U.ssq);
      FE_TRY(gemm_resid(dt, cat, 2 * d, Mc, 2 * d, h->w.w_in, d, X, d, nullptr, 0, ssq, 1, 0, &gc,
                        s, &ss));
      KvCacheArgs la[kMaxLayers];
      layer_args(r0, la);
      const NormA na{ssq, d / 16, 1, 0, 1, d, c.rms_eps};
      FE_TRY(gemm_kv_rows(an, d, (long)C * d, Mc, c.n_layers, la, &na, s));
      continue;
    }
    if (dt && Mc >= kTiledRows) {
      // many rows: one launch per stage over 128 x 64 output tiles
      // (matrix-core bound from a few hundred rows)
      FE_TRY(gemm_store_rows((const char *)features + (size_t)r0 * F * d * es, F * d, Mc, F * d,
                             h->w.w_fuse, d, cat, 2 * d, h->w.embed, tokens + r0, c.target_vocab,
                             cat + (size_t)d * es, 2 * d, d, s));
      FE_TRY(gemm_resid_rows(cat, 2 * d, Mc, 2 * d, h->w.w_in, d, X, d, s));
    } else {
      // stage by stage over the chunk, so that each weight matrix is read by
      // consecutive launches
      for (int s0 = 0; s0 < Mc; s0 += kGemmMaxRows) {
        const int Ms = std::min(kGemmMaxRows, Mc - s0);
        FE_TRY(gemm_store(dt, (const char *)features + (size_t)(r0 + s0) * F * d * es, F * d, Ms,
                          F * d, h->w.w_fuse, d, cat + (size_t)s0 * 2 * d * es, 2 * d, h->w.embed,
                          tokens + r0 + s0, c.target_vocab, cat + ((size_t)s0 * 2 * d + d) * es,
                          2 * d, d, Ms, s, &ss));
      }
      for (int s0 = 0; s0 < Mc; s0 += kGemmMaxRows) {
        const int Ms = std::min(kGemmMaxRows, Mc - s0);
        FE_TRY(gemm_resid(dt, cat + (size_t)s0 * 2 * d * es, 2 * d, Ms, 2 * d, h->w.w_in, d,
                          X + (size_t)s0 * d, d, nullptr, 0, nullptr, 1, 0, nullptr, s, &ss));
      }
    }
    if (self) {
      const fe_status st = prefill_layers(h, U, ws, Mc, positions + r0, dst_rows + r0, cache, &ss, s);
      if (st != FE_OK) return st;
      continue;
    }
    if (dt) {
      // every layer's normalised rows from one RMS per row (one launch)
      RmsCopies rc{};
      rc.n = c.n_layers;
      for (int l = 0; l < c.n_layers; ++l) {
        rc.gamma[l] = h->layers[l].attn_norm;
        rc.out[l] = an + (size_t)l * C * d * es;
      }
      FE_TRY(rmsnorm_copies(dt, X, Mc, rc, d, c.rms_eps, s));
      KvCacheArgs la[kMaxLayers];
      layer_args(r0, la);
      FE_TRY(gemm_kv_rows(an, d, (long)C * d, Mc, c.n_layers, la, nullptr, s));
      continue;
    }
    for (int l = 0; l < c.n_layers; ++l) {
      const fe_layer_weights &lw = h->layers[l];
      FE_TRY(rmsnorm_rows(dt, X, Mc, 1, 0, d, 0, lw.attn_norm, an, d, c.rms_eps, s));
      for (int s0 = 0; s0 < Mc; s0 += kGemmMaxRows) {
        const int Ms = std::min(kGemmMaxRows, Mc - s0);
        const KvCacheArgs ka{lw.wk, lw.wv, d, c.head_dim, c.n_kv_heads,
                             positions + r0 + s0, dst_rows + r0 + s0, (long)cache->rows,
                             c.max_prefix, (const float *)(h->ws + h->L.rope),
                             cache->k[l], cache->v[l]};
        FE_TRY(gemm_kvcache(dt, an + (size_t)s0 * d * es, d, Ms, ka, s, &ss));
      }
    }
  }
  (void)kvd;
  return FE_OK;
}
}  // namespace

extern "C" fe_status fe_kv_update(fe_drafter *h, int32_t n_rows, const void *features,
                                  const int32_t *tokens, const int32_t *positions,
                                  const int32_t *dst_rows, const fe_kv_cache *cache,
                                  void *workspace, size_t ws_bytes, void *stream) {
  return kv_update_impl(h, n_rows, features, tokens, positions, dst_rows, cache, workspace,
                        ws_bytes, stream);
}

// Workspace of fe_kv_update_noalloc: a file-scope device array, one copy per
// GPU, held until the process ends.  Host code never passes the array's name
// to a kernel or a copy: it stands for a host-side symbol, not a device
// address; the device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) char scratch[FE_KV_UPDATE_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
void *g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];
std::once_flag g_scratch_once[kMaxDevices];
}  // namespace

extern "C" fe_status fe_kv_update_noalloc(fe_drafter *h, int32_t n_rows, const void *features,
                                          const int32_t *tokens, const int32_t *positions,
                                          const int32_t *dst_rows, const fe_kv_cache *cache,
                                          void *stream) {
  if (!h) return fail(FE_E_INVALID, "handle is NULL");
  const size_t one_row = upd_layout_of(h->cfg, 1).total;
  if (one_row > (size_t)FE_KV_UPDATE_SCRATCH_BYTES)
    return fail(FE_E_UNSUPPORTED,
                "one row of this config needs %zu bytes of workspace, above the %d bytes of "
                "fe_kv_update_noalloc's device array; use fe_kv_update", one_row,
                (int)FE_KV_UPDATE_SCRATCH_BYTES);
  int dev = 0;
  FE_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(FE_E_INVALID, "device %d outside [0, %d)", dev, kMaxDevices);
  std::call_once(g_scratch_once[dev], [dev] {
    g_scratch_err[dev] = hipGetSymbolAddress(&g_scratch_ptr[dev], HIP_SYMBOL(scratch));
  });
  if (g_scratch_err[dev] != hipSuccess || !g_scratch_ptr[dev])
    return fail(FE_E_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                hipGetErrorString(g_scratch_err[dev]));
  return kv_update_impl(h, n_rows, features, tokens, positions, dst_rows, cache,
                        g_scratch_ptr[dev], (size_t)FE_KV_UPDATE_SCRATCH_BYTES, stream);
}

namespace {
fe_status accept_sample_impl(fe_drafter *h, int32_t batch, int32_t topk, const int32_t *tokens,
                             const int32_t *retrieve, const int32_t *topk_draft,
                             const float *draft_logits, float temperature, Draws draft_draws,
                             const float *target_probs, const float *uniforms,
                             int32_t *accept_len, int32_t *accept_path, int32_t *accepted,
                             void *stream) {
  const Range range("fe_accept_sample");
  if (!h) return fail(FE_E_INVALID, "handle is NULL");
  const fe_config &c = h->cfg;
  if (batch < 0 || batch > c.max_batch) return fail(FE_E_INVALID, "batch %d outside [0, %d]", batch, c.max_batch);
  if (topk < 1 || topk > c.max_topk) return fail(FE_E_INVALID, "topk %d outside [1, %d]", topk, c.max_topk);
  if (!(temperature > 0.f) || !(temperature < INFINITY) || !(1.0f / temperature < INFINITY))
    return fail(FE_E_INVALID, "temperature must be positive and finite");
  if (c.draft_vocab > kAccSampleMaxV || c.target_vocab > kAccSampleMaxVt)
    return fail(FE_E_UNSUPPORTED, "sampling acceptance needs draft_vocab <= %d and target_vocab <= %d",
                kAccSampleMaxV, kAccSampleMaxVt);
  if (batch == 0) return FE_OK;
  if (!tokens || !retrieve || !topk_draft || !draft_logits || !target_probs || !uniforms ||
      !accept_len || !accept_path || !accepted)
    return fail(FE_E_INVALID, "every acceptance input and output except draft_uniforms is required");
  const void *ptrs[] = {tokens, retrieve, topk_draft, draft_logits, draft_draws.u, target_probs,
                        uniforms, accept_len, accept_path, accepted};
  for (const void *q : ptrs)
    if ((uintptr_t)q & 3u) return fail(FE_E_ALIGN, "acceptance arrays must be 4-byte aligned");
  uint32_t *img = (uint32_t *)(h->ws + h->L.img);
  if (!h->img_ready) {
    FE_TRY(accept_img(h->w.d2t, c.draft_vocab, c.target_vocab, img, (hipStream_t)stream));
    h->img_ready = true;
  }
  AccPre pre;
  pre.p = (float *)(h->ws + h->L.acc_pre);
  pre.max_batch = h->L.acc_pre_batch;
  FE_TRY(accept_sample(batch, c.n_layers, topk, c.draft_vocab, c.target_vocab, tokens, retrieve,
                       topk_draft, draft_logits, 1.0f / temperature, draft_draws, h->w.d2t,
                       target_probs, uniforms, img, accept_len, accept_path, accepted,
                       (hipStream_t)stream, pre));
  return FE_OK;
}
}  // namespace

extern "C" fe_status fe_accept_sample(fe_drafter *h, int32_t batch, int32_t topk,
                                      const int32_t *tokens, const int32_t *retrieve,
                                      const int32_t *topk_draft, const float *draft_logits,
                                      float temperature, const float *draft_uniforms,
                                      const float *target_probs, const float *uniforms,
                                      int32_t *accept_len, int32_t *accept_path,
                                      int32_t *accepted, void *stream) {
  Draws dr;
  dr.u = draft_uniforms;
  return accept_sample_impl(h, batch, topk, tokens, retrieve, topk_draft, draft_logits,
                            temperature, dr, target_probs, uniforms, accept_len, accept_path,
                            accepted, stream);
}

extern "C" fe_status fe_accept_sample_seeded(fe_drafter *h, int32_t batch, int32_t topk,
                                             const int32_t *tokens, const int32_t *retrieve,
                                             const int32_t *topk_draft, const float *draft_logits,
                                             float temperature, const uint64_t *draft_seed_offset,
                                             const float *target_probs, const float *uniforms,
                                             int32_t *accept_len, int32_t *accept_path,
                                             int32_t *accepted, void *stream) {
  if (!draft_seed_offset) return fail(FE_E_INVALID, "draft_seed_offset is NULL");
  if ((uintptr_t)draft_seed_offset & 7u) return fail(FE_E_ALIGN, "draft_seed_offset must be 8-byte aligned");
  Draws dr;
  dr.so = draft_seed_offset;
  return accept_sample_impl(h, batch, topk, tokens, retrieve, topk_draft, draft_logits,
                            temperature, dr, target_probs, uniforms, accept_len, accept_path,
                            accepted, stream);
}

extern "C" fe_status fe_test_philox_uniforms(const uint64_t *seed_offset, uint64_t first,
                                             int64_t n, float *out, void *stream) {
  if (n < 0) return fail(FE_E_INVALID, "n is negative");
  if (n == 0) return FE_OK;
  if (!seed_offset || !out) return fail(FE_E_INVALID, "seed_offset and out are required");
  if ((uintptr_t)seed_offset & 7u) return fail(FE_E_ALIGN, "seed_offset must be 8-byte aligned");
  if ((uintptr_t)out & 3u) return fail(FE_E_ALIGN, "out must be 4-byte aligned");
  FE_TRY(philox_fill(seed_offset, first, (long)n, out, (hipStream_t)stream));
  return FE_OK;
}

extern "C" fe_status fe_build_tree(fe_drafter *h, int32_t batch, int32_t topk,
                                   const int32_t *root_tokens, const int32_t *topk_ids,
                                   const int32_t *prefix_lens, const fe_tree_out *out,
                                   void *stream) {
  const Range range("fe_build_tree");
  if (!h) return fail(FE_E_INVALID, "handle is NULL");
  const fe_config &c = h->cfg;
  if (batch < 0 || batch > c.max_batch) return fail(FE_E_INVALID, "batch %d outside [0, %d]", batch, c.max_batch);
  if (topk < 1 || topk > c.max_topk) return fail(FE_E_INVALID, "topk %d outside [1, %d]", topk, c.max_topk);
  if (batch == 0) return FE_OK;
  if (!root_tokens || !topk_ids || !prefix_lens) return fail(FE_E_INVALID, "tree inputs are required");
  if (!out || !out->tokens || !out->parents || !out->depth || !out->positions || !out->mask ||
      !out->retrieve)
    return fail(FE_E_INVALID, "every tree output is required");
  FE_TRY(build_tree(batch, c.n_layers, topk, root_tokens, topk_ids, prefix_lens, nullptr, out->tokens,
                    out->parents, out->depth, out->positions, out->mask, out->retrieve,
                    (hipStream_t)stream));
  return FE_OK;
}
