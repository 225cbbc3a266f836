/*
 * fe.h -- C ABI of the MI355X (gfx950) FastEagle drafting library, libfe.so.
 *
 * FastEagle (arXiv 2509.20416) replaces N sequential EAGLE drafting passes by
 * ONE pass through N lightweight decoder layers in series (Section 2.1,
 * Eq. 1-2), reads a distribution for position t+i off every layer through the
 * target's shared LM head, and turns the N distributions into a linear-size
 * "Backbone Expansion" draft tree for tree-attention verification
 * (Sections 2.2 and 2.4).  This library computes exactly that pass and that
 * tree on one GPU.
 *
 * Conventions for every call
 *  - Pointers are DEVICE pointers unless a field says HOST.
 *  - Every tensor (weights, KV caches, inputs, outputs, workspace) is allocated
 *    by the caller and BORROWED.  The library frees nothing it did not
 *    allocate; the only library-owned allocations are the handle (host memory)
 *    and, if graph replay is on, the HIP graphs it captures.  Weights and the
 *    workspace must outlive the handle.
 *  - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *    Calls are asynchronous on `stream`; device-side faults surface at the
 *    caller's next synchronisation.
 *  - Every call validates its arguments on the host BEFORE enqueueing
 *    anything: a non-OK status has no device side effect.  No C++ exception
 *    crosses the ABI.  fe_last_error() gives a message for the last non-OK
 *    status of the calling thread.
 *  - Calls on one handle must be serialised by the caller.  Outputs are
 *    bitwise deterministic for identical inputs (fixed reduction order, no
 *    floating-point atomics).
 *  - Matrices are row-major [out, in] (nn.Linear convention), no biases.
 *    Weight, feature and KV storage is FE_BF16 (bf16 bit patterns) or FE_F32
 *    for all of them; every pointer must be 16-byte aligned.
 */
#ifndef FE_H
#define FE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FE_OK = 0,
  FE_E_INVALID = 1,     /* bad pointer, size or enum value */
  FE_E_UNSUPPORTED = 2, /* shape the kernels do not implement (see fe_drafter_create) */
  FE_E_ALIGN = 3,       /* a pointer is not 16-byte aligned */
  FE_E_WORKSPACE = 4,   /* workspace missing or smaller than fe_workspace_bytes() */
  FE_E_HIP = 5          /* a HIP runtime call failed */
} fe_status;

typedef enum { FE_F32 = 0, FE_BF16 = 1 } fe_dtype;

/* What cascade layer i attends to, besides its prefix KV cache (the paper's
 * architecture figure is not available; Eq. 2 and Section 2.1 are read as):
 *  FE_CTX_CASCADE: the query is x_{i-1} at position P+i-1; keys/values are
 *    layer i's own projections of x_0..x_{i-1} at positions P..P+i-1;
 *  FE_CTX_SELF: query, key and value come from x_{i-1} alone, at position P.
 * FE_CTX_PARALLEL is the ablation without the cascade (Section 3.2, Table 2,
 * "parallel instead of serial"): every layer reads x_0, x_i = L_i(x_0), with
 * query, key and value from x_0 at position P and x_0 as the residual. */
typedef enum { FE_CTX_CASCADE = 0, FE_CTX_SELF = 1, FE_CTX_PARALLEL = 2 } fe_cascade_ctx;

typedef struct {
  int32_t hidden;        /* d */
  int32_t n_q_heads;     /* H_q */
  int32_t n_kv_heads;    /* H_kv, divides H_q (q head h reads KV head h / (H_q/H_kv)) */
  int32_t head_dim;      /* D: 64 or 128 */
  int32_t intermediate;  /* SwiGLU width I */
  int32_t n_layers;      /* N cascade layers (1..16) */
  int32_t draft_vocab;   /* V: rows of the LM head */
  int32_t target_vocab;  /* V_t: rows of the embedding table, range of d2t */
  int32_t n_feat_levels; /* number of target features fused (3: low, mid, high) */
  int32_t max_batch;     /* largest batch any call will pass */
  int32_t max_topk;      /* largest k any call will pass (1..16) */
  int32_t max_prefix;    /* largest prefix length P_b any call will pass */
  float rope_theta;      /* rotary base: angle of pair m at position p is p*theta^(-2m/D) */
  float rms_eps;         /* RMSNorm epsilon */
  int32_t dtype;         /* fe_dtype of weights, features and KV caches */
  int32_t cascade_ctx;   /* fe_cascade_ctx */
} fe_config;

/* One cascade layer L_i (Section 2.1: every layer has its own parameters). */
typedef struct {
  const void *attn_norm; /* [d] */
  const void *wq;        /* [H_q*D, d] */
  const void *wk;        /* [H_kv*D, d] */
  const void *wv;        /* [H_kv*D, d] */
  const void *wo;        /* [d, H_q*D] */
  const void *mlp_norm;  /* [d] */
  const void *w_gate;    /* [I, d] */
  const void *w_up;      /* [I, d] */
  const void *w_down;    /* [d, I] */
} fe_layer_weights;

typedef struct {
  const void *w_fuse;     /* [d, n_feat_levels*d]: g_t = FC(concat(l_t, m_t, h_t)) */
  const void *w_in;       /* [d, 2d]: x_0 = FC(concat(g_t, e_{t+1})) (Eq. 1) */
  const void *embed;      /* [V_t, d]: the target's (frozen) embedding table */
  const void *final_norm; /* [d]: RMSNorm applied before the LM head */
  const void *lm_head;    /* [V, d]: the target's frozen LM head (draft vocabulary rows) */
  const int32_t *d2t;     /* [V] draft id -> target id, or NULL for the identity */
  const fe_layer_weights *layers; /* HOST array [n_layers] */
} fe_weights;

/* Prefix KV caches of the N cascade layers for a batch (packed, ragged). */
typedef struct {
  const void *const *k;      /* HOST array [n_layers] of device pointers, each
                                [sum_b P_b, H_kv, D], keys ALREADY rotary-embedded */
  const void *const *v;      /* HOST array [n_layers], each [sum_b P_b, H_kv, D] */
  const int32_t *cu_prefix;  /* device [B+1]: sequence b owns rows cu[b]..cu[b+1]-1 */
  int32_t max_prefix;        /* HOST bound: every P_b <= max_prefix <= cfg.max_prefix.  On the
                                device, a sequence whose P_b lies outside [0, max_prefix] reads
                                no cache row and its outputs are NaN (ids -1) */
} fe_kv_view;

typedef struct fe_tree_out fe_tree_out;

typedef struct {
  int32_t *topk_ids;  /* [B, N, k]: target-vocabulary ids, rank order (largest logit
                         first; equal logits -> lower draft id first) */
  float *topk_probs;  /* [B, N, k]: temperature-1 softmax probability over the draft vocab */
  int32_t *topk_draft;/* optional [B, N, k] draft-vocabulary ids; NULL = not written */
  float *logits;      /* optional [B, N, V] fp32; NULL = never materialised */
  float *hidden;      /* optional [B, N+1, d] fp32 cascade states x_0..x_N; NULL = not written */
  const fe_tree_out *tree; /* optional: also build the Backbone Expansion tree of this pass
                         (root = next_tokens, P_b from kv->cu_prefix), as fe_build_tree would,
                         in the same launch sequence; NULL = no tree */
} fe_draft_out;

struct fe_tree_out {
  int32_t *tokens;    /* [B, T], T = 1 + N*k: root token, then level by level in rank order */
  int32_t *parents;   /* [B, T]: parent node index, -1 for the root */
  int32_t *depth;     /* [B, T]: 0 for the root, level l for level-l nodes */
  int32_t *positions; /* [B, T]: P_b + depth */
  uint8_t *mask;      /* [B, T, T]: mask[a][c] = 1 iff c is on the root->a path (inclusive) */
  int32_t *retrieve;  /* [B, N*(k-1)+1, N+1]: root->leaf node paths of the leaves in node
                         order, -1 padded */
};

typedef struct fe_drafter fe_drafter;

/* Device workspace the handle needs for `cfg` (bytes; 0 if cfg is invalid). */
size_t fe_workspace_bytes(const fe_config *cfg);

/* Creates a drafter over borrowed weights and workspace (Section 2.1).
 * Supported shapes: head_dim 64 or 128; d <= 8192; d, I, H_q*D multiples of 32
 * (bf16) or 16 (fp32); V a multiple of 16 with ceil(V/64)*max_topk <= 8192;
 * 1 <= n_layers <= 16; 1 <= max_topk <= 16; H_q % H_kv == 0;
 * max_batch*n_layers <= 256.  `workspace` (256-byte aligned) must hold
 * fe_workspace_bytes(cfg) bytes; the first fe_draft_forward builds the rotary
 * table in it, which persists between calls.  Creation makes no HIP call;
 * `stream` is unused.  On success *out receives the handle. */
fe_status fe_drafter_create(const fe_config *cfg, const fe_weights *w, void *workspace,
                            size_t workspace_bytes, void *stream, fe_drafter **out);

/* One drafting pass (Section 2.4, "Non-Autoregressive Drafting"): from the
 * target features of the last verified token and the next token t+1, produce
 * the N distributions q_{t+1..t+N} in a single pass and write their top-k.
 *  features    [B, n_feat_levels*d] (dtype): l_t, m_t, h_t concatenated
 *  next_tokens [B] int32: token t+1 in the target vocabulary (its embedding row is read)
 *  kv          prefix caches of the N layers
 *  topk        1..cfg.max_topk, <= V
 * The KV caches are read only. */
fe_status fe_draft_forward(fe_drafter *h, int32_t batch, const void *features,
                           const int32_t *next_tokens, const fe_kv_view *kv, int32_t topk,
                           const fe_draft_out *out, void *stream);

/* fe_draft_forward at temperature T with stochastic candidates: Section 2.2
 * samples k candidates per level from q_{t+i} (Section 3 evaluates at
 * temperature 0 and 1).  Here q_{t+i} = softmax(z_i / T).  With uniforms ==
 * NULL the candidates are the k most probable tokens (fe_draft_forward is
 * this call with T = 1).  With uniforms, [B, N, V] fp32 values in the open
 * interval (0, 1), one per draft-vocabulary entry of every LM-head row
 * (b, i-1), the k candidates are drawn without replacement from q_{t+i}: the
 * k largest z_v / T - log(-log(u_v)) (Gumbel-top-k; ties to the lower id).
 * Either way topk_ids / topk_draft list them most probable first (larger
 * z, then lower id), so the tree's backbone takes the most probable sampled
 * token, and topk_probs holds q_{t+i} of each.  `logits` (if asked) are the
 * raw z.  The caller draws the uniforms (e.g. a counter-based generator on
 * the device); a u of 0 excludes its token, a u of 1 forces it in.
 * Errors as fe_draft_forward, plus FE_E_INVALID for a temperature that is
 * not positive and finite (or whose reciprocal overflows) and FE_E_ALIGN for
 * uniforms not 4-byte aligned.  With graph replay on, the temperature and
 * the uniforms pointer are part of the captured arguments. */
fe_status fe_draft_sample(fe_drafter *h, int32_t batch, const void *features,
                          const int32_t *next_tokens, const fe_kv_view *kv, int32_t topk,
                          float temperature, const float *uniforms, const fe_draft_out *out,
                          void *stream);

/* fe_draft_sample with the uniforms drawn inside the pass from a counter-based
 * generator instead of read from an array (Section 2.2's sampled candidates;
 * Section 3 evaluates T = 1): uniform e = (b*N + i - 1) * V + v -- the index
 * the uniforms array of fe_draft_sample would give it -- is word e mod 4 of
 * the Philox4x64-10 block (Salmon, Moraes, Dror and Shaw, SC 2011) at
 * counter (e / 4, offset, 0, 0) under key (seed, 0), its top 23 bits j giving
 * u = (j + 1/2) / 2^23.  seed_offset: device memory holding the two uint64
 * values (seed, offset), 8-byte aligned, read by the kernels when they run,
 * so a captured pass (graph mode) replays with whatever the caller wrote
 * there: advance the offset per cycle to draw fresh candidates.  The pass
 * reads no [B, N, V] array (28.7 MB at the 8B batch-32 shapes).  Outputs,
 * tree and errors as fe_draft_sample, plus FE_E_INVALID for a NULL
 * seed_offset and FE_E_ALIGN for a misaligned one. */
fe_status fe_draft_sample_seeded(fe_drafter *h, int32_t batch, const void *features,
                                 const int32_t *next_tokens, const fe_kv_view *kv, int32_t topk,
                                 float temperature, const uint64_t *seed_offset,
                                 const fe_draft_out *out, void *stream);

/* Backbone Expansion tree (Section 2.2) of every sequence in one launch:
 * level 1 hangs the k candidates of q_{t+1} under the root; the most probable
 * extends the backbone, the other k-1 are side branches; every later level hangs
 * its k candidates under the previous backbone node.
 *  root_tokens [B] (the root is token t+1), topk_ids [B, N, k] (rank order, as
 *  written by fe_draft_forward), prefix_lens [B] (node positions are P_b + depth). */
fe_status fe_build_tree(fe_drafter *h, int32_t batch, int32_t topk, const int32_t *root_tokens,
                        const int32_t *topk_ids, const int32_t *prefix_lens,
                        const fe_tree_out *out, void *stream);

/* Greedy acceptance of a drafting cycle (Section 2.4, parallel verification,
 * read at temperature 0) for every sequence in one launch.  target_next[b][n]
 * is the target model's greedy next token after the tree path that ends at
 * node n (what tree-attention verification produces).  Along a root->leaf path
 * r_0 = root, r_1, ..., node r_m is accepted when every r_t (t <= m) carries
 * the token predicted after r_{t-1}; the path with the most accepted nodes
 * wins, the first in retrieve order on a tie.
 *  tokens      [B, T] int32, retrieve [B, N*(k-1)+1, N+1] int32: a tree from
 *              fe_build_tree (or fe_draft_out.tree) with the same topk
 *  target_next [B, T] int32
 *  accept_len  [B] out: accepted draft tokens, 0..N
 *  accept_path [B] out: the winning row of retrieve
 *  accepted    [B, N+1] out: the accepted draft tokens in path order, then the
 *              target's token after the last accepted node, then -1
 * All device pointers, 4-byte aligned, owned by the caller.  Errors:
 * FE_E_INVALID (NULL handle or array, batch outside [0, max_batch], topk
 * outside [1, max_topk]), FE_E_ALIGN; nothing is launched on an error.  Node
 * indices outside the tree end a path's walk. */
fe_status fe_accept_greedy(fe_drafter *h, int32_t batch, int32_t topk, const int32_t *tokens,
                           const int32_t *retrieve, const int32_t *target_next,
                           int32_t *accept_len, int32_t *accept_path, int32_t *accepted,
                           void *stream);

/* Destination of fe_kv_update: the N per-layer caches, each an array of
 * `rows` rows of [H_kv, D] elements in the config's dtype (row r at element
 * offset r * H_kv * D). */
typedef struct {
  void *const *k;  /* HOST array [n_layers] of device pointers, 16-byte aligned */
  void *const *v;  /* HOST array [n_layers] of device pointers, 16-byte aligned */
  int64_t rows;    /* rows of every cache array */
} fe_kv_cache;

/* Device workspace (bytes) fe_kv_update needs to process `chunk_rows` rows per
 * chunk (0 if cfg is invalid or chunk_rows < 1).  Larger chunks let every
 * weight matrix serve more rows per read. */
size_t fe_kv_update_workspace_bytes(const fe_config *cfg, int32_t chunk_rows);

/* Drafter cache update after verification (Section 2.4's update step).  Row m
 * is a verified position: the target's features there, features[m]
 * (n_feat_levels * d, as for fe_draft_forward), and the token after it,
 * tokens[m], with x_0(m) = FC(concat(FC(features[m]), e_{tokens[m]})) (Eq. 1).
 * What a layer keys depends on the context (Section 2.1, Eq. 2):
 *  FE_CTX_CASCADE / FE_CTX_PARALLEL: every layer i writes, at cache row
 *   dst_rows[m],
 *     k = RoPE(W_k^i RMSNorm(x_0(m); attn_norm_i), positions[m])   (rotated)
 *     v = W_v^i RMSNorm(x_0(m); attn_norm_i)
 *   the projections the pass applies to its own cascade entry x_0.
 *  FE_CTX_SELF: layer i's row is its key and value of its own input
 *   x_{i-1}(m), the state the pass at prefix positions[m] computes, so the
 *   update runs the N layers over the new rows (a multi-position prefill):
 *   layer by layer, each row attends to its sequence's rows of positions
 *   0 .. p-1, which sit at cache rows dst_rows[m] - p .. dst_rows[m] - 1
 *   (p = positions[m]; the rows this call writes included), plus its own key.
 *   Rows are taken in chunks (as many as the workspace holds): within a chunk
 *   every row sees the others' rows of the same layer, across chunks the
 *   earlier chunk's rows of every layer; rows of one sequence must therefore
 *   come in increasing position order, and no row may need a row of a later
 *   one.  A row whose rows of position 0 would lie before cache row 0 gets
 *   NaN state from its first attention on.
 * Rows are written in the storage dtype, so a later pass over the grown prefix
 * reads them as cached keys/values; nothing else in the caches is written.
 *  features  [n_rows, n_feat_levels*d] dtype, 16-byte aligned
 *  tokens, positions, dst_rows  [n_rows] int32, 4-byte aligned
 *  workspace caller-owned device memory, 256-byte aligned, at least
 *            fe_kv_update_workspace_bytes(cfg, 1); the rows are processed in
 *            chunks of the most rows that fit (work on the stream, no
 *            allocation).  The workspace of the handle is not touched.
 * Device-side values the host cannot check: a dst_rows entry outside
 * [0, cache->rows) is not written; a position outside [0, cfg.max_prefix) or a
 * token outside [0, target_vocab) writes NaN rows.  Rows that share a
 * destination race.  Errors: FE_E_INVALID (NULL handle, cache or array,
 * n_rows < 0, cfg.max_prefix == 0), FE_E_ALIGN, FE_E_WORKSPACE (workspace
 * NULL or below one row); nothing is launched on an error.  n_rows == 0 is a
 * no-op. */
fe_status fe_kv_update(fe_drafter *h, int32_t n_rows, const void *features,
                       const int32_t *tokens, const int32_t *positions, const int32_t *dst_rows,
                       const fe_kv_cache *cache, void *workspace, size_t ws_bytes, void *stream);

/* Bytes of the device array fe_kv_update_noalloc works in (8 MiB per GPU). */
#define FE_KV_UPDATE_SCRATCH_BYTES (8 << 20)

/* fe_kv_update for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same computation, rows and errors, but its workspace is a file-scope device
 * array of FE_KV_UPDATE_SCRATCH_BYTES bytes inside the library, one per GPU,
 * held until the process ends, instead of a caller buffer.  The rows are
 * processed in chunks of the most rows that fit it, exactly as fe_kv_update
 * does with a workspace of that size (so the two give bitwise equal caches).
 * The call allocates nothing: no hipMalloc, no hipFree; its first call on a
 * device looks up that device's array address (hipGetSymbolAddress).
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents (nothing in it needs to start at zero): calls that overlap on one
 * GPU, on any streams or handles, race and must be serialised by the caller.
 * Errors as fe_kv_update, without the workspace ones, plus FE_E_UNSUPPORTED
 * when one row of the config needs more than the array holds. */
fe_status fe_kv_update_noalloc(fe_drafter *h, int32_t n_rows, const void *features,
                               const int32_t *tokens, const int32_t *positions,
                               const int32_t *dst_rows, const fe_kv_cache *cache, void *stream);

/* Speculative-sampling acceptance of a drafting cycle at temperature T
 * (Section 2.4, parallel verification, with the sampling of Section 3 at
 * T > 0), one workgroup per sequence.  Walking from the root, the children of
 * a node are tested against the target's distribution p there:
 *  - children drawn by fe_draft_sample (draft_uniforms = the uniforms given to
 *    it) in the order of their draws (their Gumbel keys), by recursive
 *    rejection sampling: child x is accepted when u <= p(x) / q(x), with q the
 *    level's draft distribution softmax(z / T) mapped through d2t; on a
 *    rejection p becomes the normalised positive part of p - q and x leaves q
 *    (renormalised);
 *  - children chosen without randomness (draft_uniforms NULL, e.g. the top-k
 *    list of fe_draft_forward) in listing order against a point mass: accepted
 *    when u <= p(x), else x leaves p.
 * When every child is rejected, or the accepted node has no children, one more
 * token is drawn from the current p by inverse CDF, enumerating first the
 * target ids that draft ids map to (in draft-id order), then the others in
 * increasing order.  The emitted tokens then follow the target's distributions
 * exactly, whatever the draft (the speculative-sampling guarantee).  d2t must
 * be one-to-one.
 *  tokens, retrieve  the tree (fe_build_tree / fe_draft_out.tree), [B, T] and
 *                    [B, N*(k-1)+1, N+1] int32, T = 1 + N*k
 *  topk_draft        [B, N, k] int32: the children's draft ids (fe_draft_out)
 *  draft_logits      [B, N, V] fp32: the raw logits z of the pass (fe_draft_out)
 *  draft_uniforms    [B, N, V] fp32 or NULL (see above)
 *  target_probs      [B, T, V_t] fp32: the target's next-token distribution
 *                    after each node's path, at temperature T (what tree-
 *                    attention verification yields); rows need not be normalised
 *  uniforms          [B, N*k + 1] fp32 in (0, 1): accept test number j (in the
 *                    order the walk makes them) uses uniforms[j], the final
 *                    draw the last one
 *  accept_len, accept_path, accepted   as fe_accept_greedy (accept_path: the
 *                    first retrieve row that holds the accepted nodes)
 * The residual distribution lives in on-chip memory: draft_vocab <= 32768
 * and target_vocab <= 131072.  All device pointers 4-byte aligned.  Errors:
 * FE_E_INVALID (NULL handle or required array, batch outside [0, max_batch],
 * topk outside [1, max_topk], temperature not positive and finite),
 * FE_E_UNSUPPORTED (vocabulary sizes), FE_E_ALIGN; nothing is launched on an
 * error. */
fe_status fe_accept_sample(fe_drafter *h, int32_t batch, int32_t topk, const int32_t *tokens,
                           const int32_t *retrieve, const int32_t *topk_draft,
                           const float *draft_logits, float temperature,
                           const float *draft_uniforms, const float *target_probs,
                           const float *uniforms, int32_t *accept_len, int32_t *accept_path,
                           int32_t *accepted, void *stream);

/* fe_accept_sample for children drawn by fe_draft_sample_seeded: the drafting
 * uniforms of the children come from the same counter-based stream (the
 * (seed, offset) pair in device memory at draft_seed_offset, as given to the
 * pass) instead of a [B, N, V] array.  Everything else as fe_accept_sample,
 * plus FE_E_INVALID for a NULL draft_seed_offset and FE_E_ALIGN for a
 * misaligned one. */
fe_status fe_accept_sample_seeded(fe_drafter *h, int32_t batch, int32_t topk,
                                  const int32_t *tokens, const int32_t *retrieve,
                                  const int32_t *topk_draft, const float *draft_logits,
                                  float temperature, const uint64_t *draft_seed_offset,
                                  const float *target_probs, const float *uniforms,
                                  int32_t *accept_len, int32_t *accept_path, int32_t *accepted,
                                  void *stream);

/* Replays fe_draft_forward through a captured HIP graph when on != 0 (the
 * default is off).  A graph is captured on the first call with a given set of
 * arguments and replayed while they stay the same. */
fe_status fe_set_graph_mode(fe_drafter *h, int32_t on);

/* Attention work split: each attention work unit covers this many 64-key
 * chunks of one sequence's prefix (0 = automatic, the default, which sizes the
 * units to keep every compute unit streaming).  A sequence longer than one
 * unit's span leaves partial softmax states that a second launch merges;
 * every split gives the same result up to rounding.  Meant for tuning and
 * testing.  Errors: FE_E_INVALID for a NULL handle or a value outside
 * [0, 65536]. */
fe_status fe_set_attention_split(fe_drafter *h, int32_t chunks_per_workgroup);

/* How a batch-1 pass is launched.  Mode 1 (the default): every stage is its
 * own launch.  Mode 0 runs, when the shape allows (bf16, batch 1, greedy
 * top-k, n_layers <= 8, the fusion/input/hidden/intermediate/H_q*D widths
 * multiples of 512), the stages between two attention launches as ONE launch
 * of resident workgroups, one per compute unit, passing results to each other
 * through tagged words in the workspace (the pass of Section 2.4 as N + 1
 * launches besides the N attention launches); other calls still run mode 1.
 * Errors: FE_E_INVALID for a NULL handle or another mode, FE_E_UNSUPPORTED for
 * mode 0 in a build that has the persistent launches switched off. */
fe_status fe_set_pass_mode(fe_drafter *h, int32_t mode);

/* Waits for `stream`, then reports and clears the persistent pass's status
 * word: 0 when every wait of every persistent launch so far completed; bit 0
 * set when a workgroup gave up waiting for another's results (a bounded
 * wait; the kernel still ended normally, but that pass's outputs are
 * unspecified), which happens only when the workgroups of one launch cannot
 * all be resident at once (the launch uses one per compute unit).  Bit 16 is
 * set when the most recent pass on the handle ran as persistent launches.
 * Errors: FE_E_INVALID for NULL arguments, FE_E_HIP. */
fe_status fe_pass_status(fe_drafter *h, void *stream, int32_t *status);

/* Stages of the pass whose kernel launches can be timed with HIP events. */
typedef enum {
  FE_STAGE_FUSE = 0,     /* g_t = FC(l, m, h) and the embedding gather (one launch) */
  FE_STAGE_INPUT = 1,    /* x_0 = FC(g_t, e_{t+1}) (one launch) */
  FE_STAGE_QKV = 2,      /* per layer: Q/K/V projections + rotary embedding */
  FE_STAGE_ATTN = 3,     /* per layer: attention over the prefix cache and cascade keys */
  FE_STAGE_OPROJ = 4,    /* per layer: output projection + residual */
  FE_STAGE_GATEUP = 5,   /* per layer: gate/up projections + SwiGLU */
  FE_STAGE_DOWN = 6,     /* per layer: down projection + residual */
  FE_STAGE_LMHEAD = 7,   /* LM head on all N states + tile softmax statistics and top-k */
  FE_STAGE_PASS = 8      /* the whole pass as fe_draft_forward runs it (one "launch" = one pass) */
} fe_stage;

/* Kernel timing for roofline measurements: replays every launch of `stage`
 * (stages 0..7 in their one-launch-per-stage form; FE_STAGE_PASS: the whole
 * pass as fe_draft_forward launches it) from the most recent fe_draft_forward
 * on this handle, `repeats` times back to
 * back on `stream`, between two HIP events recorded on that stream, waits for
 * them, and writes the mean duration of one launch (ms) to *ms_per_launch and
 * the number of launches of the stage in one pass to *launches.  The buffers
 * of that fe_draft_forward call must still be valid.  The replays rewrite
 * workspace scratch (and `logits`, with the same values), so the workspace is
 * unspecified until the next fe_draft_forward. */
fe_status fe_time_stage(fe_drafter *h, int32_t stage, int32_t repeats, void *stream,
                        float *ms_per_launch, int32_t *launches);

/* Test export (device work on `stream`, synchronised; allocates and frees its
 * own scratch, so not for production paths): one layer's attention as the
 * pass runs it (Section 2.1: the GQA attention of a decoder layer over its
 * prefix cache plus the cascade keys).  Query b, heads 0..Hq-1: keys/values
 * are the prefix rows cu_prefix[b] .. cu_prefix[b+1]-1 of k_cache / v_cache
 * ([rows, Hkv, D], storage dtype, keys rotated at their positions) followed by
 * the nctx rows knew/vnew[b, t] ([B, nctx, Hkv, D] fp32) at positions P_b + t
 * (cascade != 0) or P_b (cascade == 0, nctx == 1); the query q[b] ([B, Hq, D]
 * fp32) sits at the last of those positions.  bf16: q and knew unrotated (the
 * kernel rotates them); fp32: already rotated.  Head h reads KV head
 * h / (Hq/Hkv).  out [B, Hq, D] in the storage dtype.  chunks_per_workgroup
 * as fe_set_attention_split (0 = automatic).  Errors: FE_E_INVALID,
 * FE_E_UNSUPPORTED (head_dim not 64 or 128), FE_E_HIP. */
fe_status fe_test_attention(int32_t dtype, int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                            int32_t head_dim, const void *k_cache, const void *v_cache,
                            const int32_t *cu_prefix, int32_t max_prefix, const float *q,
                            const float *knew, const float *vnew, int32_t nctx, int32_t cascade,
                            double rope_theta, int32_t chunks_per_workgroup, void *out,
                            void *stream);

/* Test export (device work on `stream`): the standalone RMSNorm launch,
 * out[r] = gamma * x[r] / sqrt(mean(x[r]^2) + eps) for rows x [rows, d] fp32,
 * gamma [d] and out [rows, d] in the storage dtype.  Errors: FE_E_INVALID,
 * FE_E_HIP. */
fe_status fe_test_rmsnorm(int32_t dtype, const float *x, int32_t rows, int32_t d,
                          const void *gamma, float eps, void *out, void *stream);

/* Test export (device work on `stream`): uniforms first .. first+n-1 of the
 * counter-based stream of fe_draft_sample_seeded ((seed, offset) in device
 * memory at seed_offset) into the device array out [n] fp32, so the generator
 * can be checked on its own.  Errors: FE_E_INVALID (n < 0, NULL pointers with
 * n > 0), FE_E_ALIGN, FE_E_HIP. */
fe_status fe_test_philox_uniforms(const uint64_t *seed_offset, uint64_t first, int64_t n,
                                  float *out, void *stream);

/* Test export, host only (no device work, no handle): the work pieces of the
 * persistent bf16 attention for a batch whose prefix lengths are
 * prefix_lens[0..batch) (HOST array), `ncols` (KV head, head group) columns
 * per sequence, `nch_ld` partial slots per (sequence, head) and `waves`
 * resident waves, from the same split arithmetic the kernel runs.  Row p of
 * `pieces` (HOST, [max_pieces, 7] int32) is (wave, sequence, column, first
 * 64-key chunk, chunks, partial slot, pieces of the segment if this is its
 * first piece else 0); *n_pieces gets the total (rows past max_pieces are not
 * written; `pieces` may be NULL when max_pieces is 0).  A P_b outside
 * [0, pmax] counts as an empty prefix.  Errors: FE_E_INVALID for NULL arrays,
 * batch outside [1, 256] or non-positive sizes. */
fe_status fe_test_attn_split(const int32_t *prefix_lens, int32_t batch, int32_t ncols,
                             int32_t nch_ld, int32_t pmax, int32_t waves, int32_t *pieces,
                             int32_t max_pieces, int32_t *n_pieces);

void fe_drafter_destroy(fe_drafter *h);

/* Message for the last non-OK status returned on the calling thread. */
const char *fe_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* FE_H */
