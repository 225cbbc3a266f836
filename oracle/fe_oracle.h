/*
 * fe_oracle.h -- CPU oracle of the FastEagle cascaded drafter and its
 * Backbone Expansion tree (FastEagle, Sections 2.1, 2.2 and 2.4).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's
 * CPU-baseline leg may load this library.  It shares no code, header, table or
 * helper with the GPU library and must never be on the product path.
 *
 * Everything is computed in double precision on the host, one sequence at a
 * time, in the order the paper states the steps.  Stored inputs (fp32 or bf16
 * bit patterns) are widened exactly to double.
 */
#ifndef FE_ORACLE_H
#define FE_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { FEO_F32 = 0, FEO_BF16 = 1 };
/* What layer i reads: CASCADE and SELF are the two readings of Eq. 2 (see
 * feo_draft_forward); PARALLEL is the ablation "w/o cascaded structure"
 * (Section 3.2, Table 2): every layer takes x_0, x_i = L_i(x_0). */
enum { FEO_CTX_CASCADE = 0, FEO_CTX_SELF = 1, FEO_CTX_PARALLEL = 2 };

typedef struct {
  int32_t hidden, n_q_heads, n_kv_heads, head_dim, intermediate, n_layers;
  int32_t draft_vocab, target_vocab, n_feat_levels;
  int32_t dtype;        /* storage of weights, features and prefix KV: FEO_F32 / FEO_BF16 */
  int32_t cascade_ctx;  /* FEO_CTX_CASCADE / FEO_CTX_SELF */
  double rope_theta, rms_eps;
} feo_config;

typedef struct {
  const void *attn_norm, *wq, *wk, *wv, *wo, *mlp_norm, *w_gate, *w_up, *w_down;
} feo_layer;

typedef struct {
  const void *w_fuse, *w_in, *embed, *final_norm, *lm_head;
  const int32_t *d2t;       /* [V] draft id -> target id; NULL = identity */
  const feo_layer *layers;  /* [n_layers] */
} feo_weights;

/* Threads used by the matrix-vector loops (OpenMP over output rows). */
void feo_set_threads(int n);
int feo_get_threads(void);

/* y = gamma * x / sqrt(mean(x^2) + eps), n elements. */
void feo_rmsnorm(const double *x, const void *gamma, int32_t dtype, int32_t n, double eps,
                 double *y);

/* Rotate-half rotary embedding of one head vector v[D] in place at position pos:
 * pairs (m, m + D/2), angle pos * theta^(-2m/D). */
void feo_rope(double *v, int32_t D, int64_t pos, double theta);

/* One query head against L key/value rows (row stride `stride` doubles):
 * out[D] = sum_j softmax_j(q.k_j / sqrt(D)) v_j.  L == 0 writes zeros. */
void feo_attend(const double *q, const double *keys, const double *vals, int32_t L,
                int32_t D, int64_t stride, double *out);

/*
 * The drafting pass for `batch` sequences.
 *  features  [B, n_feat_levels*d]  (dtype)   l_t, m_t, h_t concatenated
 *  next_tok  [B] int32                       token t+1 (target vocabulary)
 *  kcache/vcache  [n_layers] pointers, each [sum P_b, H_kv, D] (dtype), K already rotated
 *  prefix_lens [B] int32
 * Outputs (any may be NULL):
 *  hidden [B, N+1, d]  x_0 .. x_N;   logits [B, N, V]
 *  topk_draft [B, N, k] int32 draft ids;  topk_ids [B, N, k] int32 target ids;
 *  topk_probs [B, N, k] double.
 * Returns 0, or -1 on invalid arguments.
 */
int feo_draft_forward(const feo_config *cfg, const feo_weights *w, int32_t batch,
                      const void *features, const int32_t *next_tok,
                      const void *const *kcache, const void *const *vcache,
                      const int32_t *prefix_lens, int32_t topk, double *hidden, double *logits,
                      int32_t *topk_draft, int32_t *topk_ids, double *topk_probs);

/*
 * The drafting pass at temperature T with stochastic candidates (Section 2.2
 * samples k candidates per level; Section 3 reports temperature 1):
 * q_{t+i} = softmax(z_i / T).  With uniforms == NULL the candidates are the k
 * most probable tokens (feo_draft_forward is this call with T = 1).  With
 * uniforms [B, N, V] (fp32 in (0, 1), one per draft-vocabulary entry) the k
 * candidates are drawn without replacement from q_{t+i}: the k largest
 * z_v / T - log(-log(u_v)) (ties to the lower id).  Either way they are
 * listed most probable first (larger z, then lower id) and topk_probs holds
 * q_{t+i} of each.  logits are the raw z.  Returns 0, or -1 on invalid
 * arguments (also T <= 0).
 */
int feo_draft_sample(const feo_config *cfg, const feo_weights *w, int32_t batch,
                     const void *features, const int32_t *next_tok,
                     const void *const *kcache, const void *const *vcache,
                     const int32_t *prefix_lens, int32_t topk, double temperature,
                     const float *uniforms, double *hidden, double *logits, int32_t *topk_draft,
                     int32_t *topk_ids, double *topk_probs);

/*
 * Backbone Expansion tree for `batch` sequences, T = 1 + N*k nodes each.
 *  root_tokens [B], topk_ids [B, N, k] (rank order), prefix_lens [B]
 * Outputs: tokens/parents/depth/positions [B, T] int32, mask [B, T, T] uint8
 * (mask[a][c] = 1 iff c is on the root->a path), retrieve [B, N*(k-1)+1, N+1]
 * (root->leaf node paths, -1 padded).  Returns 0, or -1 on invalid arguments.
 */
int feo_build_tree(int32_t batch, int32_t n_layers, int32_t topk, const int32_t *root_tokens,
                   const int32_t *topk_ids, const int32_t *prefix_lens, int32_t *tokens,
                   int32_t *parents, int32_t *depth, int32_t *positions, uint8_t *mask,
                   int32_t *retrieve);

/*
 * Greedy acceptance of one drafting cycle (Section 2.4, parallel verification,
 * read at temperature 0): target_next[b][n] is the target model's greedy next
 * token after the tree path that ends at node n.  Along a root->leaf path
 * r_0 = root, r_1, ..., node r_m is accepted when every r_t, t <= m, carries
 * the token the target predicts after r_{t-1}.  Per sequence the path with
 * the most accepted nodes wins (the first such path in retrieve order on a
 * tie).  Inputs: tokens [B, T], retrieve [B, NL, N+1] as built above,
 * target_next [B, T].  Outputs: accept_len [B] (accepted draft tokens, 0..N),
 * accept_path [B] (row of retrieve), accepted [B, N+1]: the accepted draft
 * tokens in path order, then the target's token after the last accepted node,
 * then -1.  Returns 0, or -1 on invalid arguments.
 */
int feo_accept_greedy(int32_t batch, int32_t n_layers, int32_t topk, const int32_t *tokens,
                      const int32_t *retrieve, const int32_t *target_next, int32_t *accept_len,
                      int32_t *accept_path, int32_t *accepted);

/*
 * Drafter KV-cache rows for verified positions (Section 2.4 update step, read
 * under FEO_CTX_CASCADE, where it equals FEO_CTX_PARALLEL's; FEO_CTX_SELF is
 * rejected).  Row m carries the
 * target's features at position positions[m], features [n_rows,
 * n_feat_levels*d] (dtype), and the token that follows it, tokens[m].  With
 * x_0(m) = FC(concat(FC(f_m), e_{tokens[m]})) as in Eq. 1, every layer i
 * gets a = RMSNorm(x_0(m); attn_norm_i), k = RoPE(W_k^i a, positions[m]) and
 * v = W_v^i a.  k_out / v_out: [n_layers] pointers, each [n_rows, H_kv, D]
 * double.  Returns 0, or -1 on invalid arguments (a token outside
 * [0, target_vocab), a negative position).
 */
int feo_kv_update(const feo_config *cfg, const feo_weights *w, int32_t n_rows,
                  const void *features, const int32_t *tokens, const int32_t *positions,
                  double *const *k_out, double *const *v_out);

/*
 * Drafter KV-cache rows under FEO_CTX_SELF (Section 2.4 update step, read
 * under the self context).  Layer i's row at position p is its rotated key and
 * value of its own input x_{i-1}(p), the state the pass at prefix p computes,
 * so the rows are produced by running the pass at each new position in turn
 * (a multi-position prefill of the N layers).  Row m (features, tokens as in
 * feo_kv_update) sits at position positions[m] and is written at cache row
 * dst_rows[m]; its sequence's row of position j < p is cache row
 * dst_rows[m] - (positions[m] - j), taken from an earlier row of this call
 * that wrote it (fp64) or else from kcache / vcache ([n_layers] pointers, each
 * [cache_rows, H_kv, D] in cfg->dtype, keys rotated).  Outputs as
 * feo_kv_update.  Returns 0, or -1 on invalid arguments (not FEO_CTX_SELF, a
 * token outside [0, target_vocab), a negative position, dst_rows[m] outside
 * [positions[m], cache_rows)).
 */
int feo_kv_update_self(const feo_config *cfg, const feo_weights *w, int32_t n_rows,
                       const void *features, const int32_t *tokens, const int32_t *positions,
                       const int32_t *dst_rows, const void *const *kcache,
                       const void *const *vcache, int64_t cache_rows, double *const *k_out,
                       double *const *v_out);

/*
 * Counter-based uniforms for stochastic drafting (the randomness of Section
 * 2.2's sampled candidates, drawn from a seed and an offset instead of a
 * stored array).  feo_philox4x64_10: one block of the Philox4x64-10 generator
 * (Salmon et al., SC 2011) for counter ctr and key.  feo_philox_uniforms:
 * uniforms first .. first+n-1 of the stream (seed, offset); uniform e is word
 * e mod 4 of the block at counter (e / 4, offset, 0, 0), key (seed, 0), its
 * top 23 bits j giving (j + 1/2) / 2^23.  Uniform e of a drafting pass is the
 * one of row b*N + i - 1, draft id v: e = (b*N + i - 1) * V + v, as the
 * uniforms array of feo_draft_sample is laid out.
 */
void feo_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]);
void feo_philox_uniforms(uint64_t seed, uint64_t offset, uint64_t first, int64_t n, float *out);

/*
 * Speculative-sampling acceptance of one cycle at temperature T (Section 2.4).
 * For the tree of feo_build_tree (tokens [B, T] target ids, retrieve) with
 * topk_draft [B, N, k] the children's draft ids, draft_logits [B, N, V] the
 * raw z of each level (q = softmax(z / T)), draft_uniforms [B, N, V] the
 * uniforms the candidates were drawn with (feo_draft_sample; NULL for
 * candidates chosen without randomness), d2t [V] (NULL = identity),
 * target_probs [B, T, V_t] the target's next-token distribution after each
 * node's path, and uniforms [B, N*k + 1] in (0, 1): accept test number j uses
 * uniforms[j], the final draw uses the last one.  Sampled children are tested
 * in draw order by recursive rejection sampling, unsampled ones in listing
 * order against a point mass; the final draw enumerates the target ids that
 * draft ids map to first, in draft-id order, then the others in increasing
 * order (see fe_oracle.c).  Outputs as
 * feo_accept_greedy; accept_path is the first retrieve row that holds the
 * accepted nodes.  margin [B] (optional): the smallest relative distance of a
 * decision from its threshold.  Returns 0, or -1 on invalid arguments.
 */
int feo_accept_sample(int32_t batch, int32_t n_layers, int32_t topk, int32_t draft_vocab,
                      int32_t target_vocab, const int32_t *tokens, const int32_t *retrieve,
                      const int32_t *topk_draft, const float *draft_logits, double temperature,
                      const float *draft_uniforms, const int32_t *d2t, const float *target_probs,
                      const float *uniforms, int32_t *accept_len, int32_t *accept_path,
                      int32_t *accepted, double *margin);

#ifdef __cplusplus
}
#endif
#endif
