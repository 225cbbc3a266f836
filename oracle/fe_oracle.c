/*
 * fe_oracle.c -- CPU oracle of the FastEagle drafting pass and tree.
 *
 * TEST INFRASTRUCTURE ONLY (tests, smoke check, bench CPU-baseline leg).  It
 * is deliberately plain: double precision, one sequence at a time, straight
 * loops over rows, no blocking or fusion, steps in the paper's order.  It
 * shares no code with the GPU library.
 *
 * Paper passages followed (FastEagle):
 *   Section 2.1, first paragraph: multi-level features l_t, m_t, h_t of the
 *     target are concatenated and fused by an FC layer into g_t; g_t is
 *     concatenated with the embedding e_{t+1} of the next token.
 *   Section 2.1, Eq. 1: h_1 = L_1(FC(concat(g_t, e_{t+1}))).
 *   Section 2.1, Eq. 2: h_i = L_i(h_{i-1}) for i = 2..N, each L_i with its own
 *     parameters; every h_i goes through the target's frozen LM head to give
 *     the distribution for position t+i.
 *   Section 2.1 (EAGLE-style drafter): each L_i is one lightweight decoder
 *     layer; its internals are a pre-norm LLaMA layer (RMSNorm, rotary GQA
 *     attention over the prefix KV cache plus the cascade entries, SwiGLU).
 *   Section 2.2: Backbone Expansion tree.
 *   Section 2.4: one pass yields all N distributions, then the tree is built.
 *
 * Readings where the paper is silent (they are listed with reasons in the
 * design notes of the repository):
 *   - cascade context: layer i's query is x_{i-1} at position P+i-1 and its
 *     keys/values are its own prefix cache plus its own projections of
 *     x_0..x_{i-1} at positions P..P+i-1 (FEO_CTX_CASCADE); FEO_CTX_SELF lets
 *     layer i see the prefix plus its own input only, at position P;
 *   - two FC layers (3d->d fusion, then 2d->d input), no biases;
 *   - one shared final RMSNorm before the LM head;
 *   - k candidates per level are the k largest logits, ties to the lower
 *     draft id;  probabilities are the temperature-1 softmax over the draft
 *     vocabulary;
 *   - rotary embedding in rotate-half form, frequencies theta^(-2m/D);
 *   - q head h reads KV head floor(h / (H_q/H_kv)).
 */
#include "fe_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

static int g_threads = 1;

void feo_set_threads(int n) { g_threads = n < 1 ? 1 : n; }
int feo_get_threads(void) { return g_threads; }

/* Storage code of prefix rows the oracle assembles itself (fp64). */
enum { KV_F64 = 2 };

/* Exact widening of one stored element. */
static double widen(const void *p, int32_t dtype, size_t i) {
  if (dtype == KV_F64) return ((const double *)p)[i];
  if (dtype == FEO_BF16) {
    uint32_t bits = (uint32_t)((const uint16_t *)p)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
  }
  return (double)((const float *)p)[i];
}

/* y[o] = sum_k W[o][k] * x[k] with W stored row-major [rows][cols]
 * (an FC layer without bias, nn.Linear convention). */
static void matvec(const void *W, int32_t dtype, int64_t rows, int64_t cols, const double *x,
                   double *y) {
  if (dtype == FEO_BF16) {
    const uint16_t *w = (const uint16_t *)W;
#pragma omp parallel for num_threads(g_threads) schedule(static)
    for (int64_t o = 0; o < rows; ++o) {
      const uint16_t *row = w + (size_t)o * (size_t)cols;
      double acc = 0.0;
      for (int64_t k = 0; k < cols; ++k) {
        uint32_t bits = (uint32_t)row[k] << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        acc += (double)f * x[k];
      }
      y[o] = acc;
    }
  } else {
    const float *w = (const float *)W;
#pragma omp parallel for num_threads(g_threads) schedule(static)
    for (int64_t o = 0; o < rows; ++o) {
      const float *row = w + (size_t)o * (size_t)cols;
      double acc = 0.0;
      for (int64_t k = 0; k < cols; ++k) acc += (double)row[k] * x[k];
      y[o] = acc;
    }
  }
}

void feo_rmsnorm(const double *x, const void *gamma, int32_t dtype, int32_t n, double eps,
                 double *y) {
  double ss = 0.0;
  for (int32_t i = 0; i < n; ++i) ss += x[i] * x[i];
  const double inv = 1.0 / sqrt(ss / (double)n + eps);
  for (int32_t i = 0; i < n; ++i) y[i] = widen(gamma, dtype, (size_t)i) * (x[i] * inv);
}

void feo_rope(double *v, int32_t D, int64_t pos, double theta) {
  const int32_t half = D / 2;
  for (int32_t m = 0; m < half; ++m) {
    const double freq = pow(theta, -2.0 * (double)m / (double)D);
    const double ang = (double)pos * freq;
    const double c = cos(ang), s = sin(ang);
    const double a = v[m], b = v[m + half];
    v[m] = a * c - b * s;
    v[m + half] = b * c + a * s;
  }
}

void feo_attend(const double *q, const double *keys, const double *vals, int32_t L, int32_t D,
                int64_t stride, double *out) {
  for (int32_t d = 0; d < D; ++d) out[d] = 0.0;
  if (L <= 0) return;
  double *s = (double *)malloc(sizeof(double) * (size_t)L);
  const double scale = 1.0 / sqrt((double)D);
  double mx = -INFINITY;
  for (int32_t j = 0; j < L; ++j) {
    double dot = 0.0;
    for (int32_t d = 0; d < D; ++d) dot += q[d] * keys[(size_t)j * stride + d];
    s[j] = dot * scale;
    if (s[j] > mx) mx = s[j];
  }
  double den = 0.0;
  for (int32_t j = 0; j < L; ++j) {
    s[j] = exp(s[j] - mx);
    den += s[j];
  }
  for (int32_t j = 0; j < L; ++j)
    for (int32_t d = 0; d < D; ++d) out[d] += s[j] * vals[(size_t)j * stride + d];
  for (int32_t d = 0; d < D; ++d) out[d] /= den;
  free(s);
}

typedef struct {
  double z;
  int32_t id;
} scored;

/* Order: larger logit first, equal logits by lower draft id. */
static int by_logit_desc(const void *pa, const void *pb) {
  const scored *a = (const scored *)pa, *b = (const scored *)pb;
  if (a->z > b->z) return -1;
  if (a->z < b->z) return 1;
  return (a->id > b->id) - (a->id < b->id);
}

static double silu(double u) { return u / (1.0 + exp(-u)); }

/* One decoder layer L_i of the cascade for one sequence (Section 2.1, Eq. 1-2).
 * xs[0..i-1] are the cascade states produced so far (x_0 = fused input);
 * writes x_i into xs[i].  Under FEO_CTX_PARALLEL (the ablation of Section 3.2
 * that replaces the series by parallel heads) every layer reads x_0 instead:
 * x_i = L_i(x_0), attending to its prefix plus x_0 at position P.  The prefix
 * keys/values are rows prefix_off .. prefix_off + P - 1 of kc / vc, stored as
 * kv_dtype (FEO_F32, FEO_BF16 or KV_F64).  k_own / v_own (optional, [H_kv*D]):
 * the layer's rotated key and value of its own input x_src. */
static void cascade_layer(const feo_config *c, const feo_layer *L, int32_t i, double *xs,
                          const void *kc, const void *vc, int32_t kv_dtype, int64_t prefix_off,
                          int32_t P, double *k_own, double *v_own) {
  const int32_t d = c->hidden, D = c->head_dim, Hq = c->n_q_heads, Hkv = c->n_kv_heads;
  const int32_t G = Hq / Hkv, I = c->intermediate;
  const int32_t qd = Hq * D, kvd = Hkv * D;
  /* the layer's input: x_{i-1} in series, x_0 for parallel heads */
  const int32_t src = (c->cascade_ctx == FEO_CTX_PARALLEL) ? 0 : i - 1;
  const int32_t j0 = (c->cascade_ctx == FEO_CTX_CASCADE) ? 0 : src;
  const int32_t nctx = (c->cascade_ctx == FEO_CTX_CASCADE) ? i : 1;

  /* Pre-attention RMSNorm and projections of every context row. */
  double *a = (double *)malloc(sizeof(double) * (size_t)d);
  double *kn = (double *)malloc(sizeof(double) * (size_t)nctx * kvd);
  double *vn = (double *)malloc(sizeof(double) * (size_t)nctx * kvd);
  double *q = (double *)malloc(sizeof(double) * (size_t)qd);
  for (int32_t t = 0; t < nctx; ++t) {
    const int32_t j = j0 + t;
    const int64_t pos = (c->cascade_ctx == FEO_CTX_CASCADE) ? (int64_t)P + j : (int64_t)P;
    feo_rmsnorm(xs + (size_t)j * d, L->attn_norm, c->dtype, d, c->rms_eps, a);
    matvec(L->wk, c->dtype, kvd, d, a, kn + (size_t)t * kvd);
    matvec(L->wv, c->dtype, kvd, d, a, vn + (size_t)t * kvd);
    for (int32_t h = 0; h < Hkv; ++h) feo_rope(kn + (size_t)t * kvd + (size_t)h * D, D, pos, c->rope_theta);
    if (j == src) {
      matvec(L->wq, c->dtype, qd, d, a, q);
      for (int32_t h = 0; h < Hq; ++h) feo_rope(q + (size_t)h * D, D, pos, c->rope_theta);
      if (k_own) memcpy(k_own, kn + (size_t)t * kvd, sizeof(double) * (size_t)kvd);
      if (v_own) memcpy(v_own, vn + (size_t)t * kvd, sizeof(double) * (size_t)kvd);
    }
  }

  /* GQA attention: q head h reads KV head h / G over [prefix ; context rows]. */
  const int32_t Lk = P + nctx;
  double *o = (double *)malloc(sizeof(double) * (size_t)qd);
#pragma omp parallel for num_threads(g_threads) schedule(static)
  for (int32_t ch = 0; ch < Hkv; ++ch) {
    double *K = (double *)malloc(sizeof(double) * ((size_t)Lk * D + 1));
    double *V = (double *)malloc(sizeof(double) * ((size_t)Lk * D + 1));
    for (int32_t t = 0; t < P; ++t)
      for (int32_t e = 0; e < D; ++e) {
        const size_t src = ((size_t)(prefix_off + t) * Hkv + ch) * D + e;
        K[(size_t)t * D + e] = widen(kc, kv_dtype, src);
        V[(size_t)t * D + e] = widen(vc, kv_dtype, src);
      }
    for (int32_t t = 0; t < nctx; ++t)
      for (int32_t e = 0; e < D; ++e) {
        K[(size_t)(P + t) * D + e] = kn[(size_t)t * kvd + (size_t)ch * D + e];
        V[(size_t)(P + t) * D + e] = vn[(size_t)t * kvd + (size_t)ch * D + e];
      }
    for (int32_t g = 0; g < G; ++g) {
      const int32_t h = ch * G + g;
      feo_attend(q + (size_t)h * D, K, V, Lk, D, D, o + (size_t)h * D);
    }
    free(K);
    free(V);
  }

  /* Output projection and residual. */
  double *xp = (double *)malloc(sizeof(double) * (size_t)d);
  matvec(L->wo, c->dtype, d, qd, o, xp);
  for (int32_t e = 0; e < d; ++e) xp[e] += xs[(size_t)src * d + e];

  /* Post-attention RMSNorm, SwiGLU MLP and residual. */
  double *bn = (double *)malloc(sizeof(double) * (size_t)d);
  double *gt = (double *)malloc(sizeof(double) * (size_t)I);
  double *up = (double *)malloc(sizeof(double) * (size_t)I);
  double *dn = (double *)malloc(sizeof(double) * (size_t)d);
  feo_rmsnorm(xp, L->mlp_norm, c->dtype, d, c->rms_eps, bn);
  matvec(L->w_gate, c->dtype, I, d, bn, gt);
  matvec(L->w_up, c->dtype, I, d, bn, up);
  for (int32_t e = 0; e < I; ++e) gt[e] = silu(gt[e]) * up[e];
  matvec(L->w_down, c->dtype, d, I, gt, dn);
  for (int32_t e = 0; e < d; ++e) xs[(size_t)i * d + e] = xp[e] + dn[e];

  free(a); free(kn); free(vn); free(q); free(o); free(xp);
  free(bn); free(gt); free(up); free(dn);
}

/* x_0 of one row (Section 2.1, Eq. 1): g_t = FC(concat(l_t, m_t, h_t)) from
 * row `row` of the features, then x_0 = FC(concat(g_t, e_{t+1})) with e_{t+1}
 * the embedding of token `tok`.  f [F*d] and ge [2d] are scratch. */
static void fused_input(const feo_config *c, const feo_weights *w, const void *features,
                        size_t row, int32_t tok, double *f, double *ge, double *x0) {
  const int32_t d = c->hidden, F = c->n_feat_levels;
  for (int64_t e = 0; e < (int64_t)F * d; ++e)
    f[e] = widen(features, c->dtype, row * F * d + (size_t)e);
  matvec(w->w_fuse, c->dtype, d, (int64_t)F * d, f, ge);
  for (int32_t e = 0; e < d; ++e) ge[d + e] = widen(w->embed, c->dtype, (size_t)tok * d + e);
  matvec(w->w_in, c->dtype, d, 2 * d, ge, x0);
}

int feo_draft_forward(const feo_config *c, const feo_weights *w, int32_t batch,
                      const void *features, const int32_t *next_tok,
                      const void *const *kcache, const void *const *vcache,
                      const int32_t *prefix_lens, int32_t topk, double *hidden, double *logits,
                      int32_t *topk_draft, int32_t *topk_ids, double *topk_probs) {
  return feo_draft_sample(c, w, batch, features, next_tok, kcache, vcache, prefix_lens, topk, 1.0,
                          NULL, hidden, logits, topk_draft, topk_ids, topk_probs);
}

/* Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC 2011): ten rounds of the 4x64 Philox S-box over the
 * counter, the two-word key bumped by the Weyl constants between rounds.  A
 * round multiplies counter words 0 and 2 by the two round multipliers and
 * rebuilds the counter as (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1,
 * lo(M0 c0)). */
void feo_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
  uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3], k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += W0;
      k1 += W1;
    }
    const unsigned __int128 p0 = (unsigned __int128)M0 * c0, p1 = (unsigned __int128)M1 * c2;
    const uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    const uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    c0 = hi1 ^ c1 ^ k0;
    c1 = lo1;
    c2 = hi0 ^ c3 ^ k1;
    c3 = lo0;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Uniforms first .. first+n-1 of the draw stream (seed, offset): uniform e is
 * word e mod 4 of the Philox4x64-10 block at counter (floor(e / 4), offset, 0,
 * 0) under key (seed, 0), its top 23 bits j mapped to (j + 1/2) / 2^23, which
 * is exact in float and lies in (0, 1). */
void feo_philox_uniforms(uint64_t seed, uint64_t offset, uint64_t first, int64_t n, float *out) {
  const uint64_t key[2] = {seed, 0};
  for (int64_t i = 0; i < n; ++i) {
    const uint64_t e = first + (uint64_t)i;
    const uint64_t ctr[4] = {e >> 2, offset, 0, 0};
    uint64_t blk[4];
    feo_philox4x64_10(ctr, key, blk);
    const uint64_t j = blk[e & 3] >> 41;
    out[i] = (float)(((double)j + 0.5) / 8388608.0);
  }
}

/* -log(-log(u)): a standard Gumbel variate from a uniform u in (0, 1). */
static double gumbel(float u) { return -log(-log((double)u)); }

int feo_draft_sample(const feo_config *c, const feo_weights *w, int32_t batch,
                     const void *features, const int32_t *next_tok,
                     const void *const *kcache, const void *const *vcache,
                     const int32_t *prefix_lens, int32_t topk, double temperature,
                     const float *uniforms, double *hidden, double *logits, int32_t *topk_draft,
                     int32_t *topk_ids, double *topk_probs) {
  if (!c || !w || batch < 0 || topk < 1 || topk > c->draft_vocab || c->n_layers < 1) return -1;
  if (!(temperature > 0.0)) return -1;
  if (c->cascade_ctx < FEO_CTX_CASCADE || c->cascade_ctx > FEO_CTX_PARALLEL) return -1;
  if (c->n_q_heads % c->n_kv_heads != 0 || c->head_dim % 2 != 0) return -1;
  const int32_t d = c->hidden, N = c->n_layers, V = c->draft_vocab, F = c->n_feat_levels;
  int64_t prefix_off = 0;
  double *xs = (double *)malloc(sizeof(double) * (size_t)(N + 1) * d);
  double *f = (double *)malloc(sizeof(double) * (size_t)F * d);
  double *ge = (double *)malloc(sizeof(double) * (size_t)2 * d);
  double *hn = (double *)malloc(sizeof(double) * (size_t)d);
  double *z = (double *)malloc(sizeof(double) * (size_t)V);
  scored *ord = (scored *)malloc(sizeof(scored) * (size_t)V);

  for (int32_t b = 0; b < batch; ++b) {
    const int32_t P = prefix_lens[b];
    if (P < 0 || next_tok[b] < 0 || next_tok[b] >= c->target_vocab) {
      free(xs); free(f); free(ge); free(hn); free(z); free(ord);
      return -1;
    }
    fused_input(c, w, features, b, next_tok[b], f, ge, xs);
    /* h_i = L_i(h_{i-1}) (Eq. 1-2) */
    for (int32_t i = 1; i <= N; ++i)
      cascade_layer(c, &w->layers[i - 1], i, xs, kcache[i - 1], vcache[i - 1], c->dtype, prefix_off,
                    P, NULL, NULL);
    if (hidden) memcpy(hidden + (size_t)b * (N + 1) * d, xs, sizeof(double) * (size_t)(N + 1) * d);

    /* q_{t+i} = softmax(LMHead(RMSNorm(h_i)) / T) and its k candidates
     * (Section 2.2): the k most probable tokens (uniforms == NULL), or k
     * tokens sampled without replacement from q_{t+i} (the Gumbel-top-k
     * construction: the k largest z/T + Gumbel noise), listed most probable
     * first so that the backbone takes the most probable sampled token. */
    for (int32_t i = 1; i <= N; ++i) {
      feo_rmsnorm(xs + (size_t)i * d, w->final_norm, c->dtype, d, c->rms_eps, hn);
      matvec(w->lm_head, c->dtype, V, d, hn, z);
      const size_t row = (size_t)b * N + (size_t)(i - 1);
      if (logits) memcpy(logits + row * V, z, sizeof(double) * (size_t)V);
      for (int32_t v = 0; v < V; ++v) z[v] /= temperature;
      double mx = -INFINITY;
      for (int32_t v = 0; v < V; ++v) mx = z[v] > mx ? z[v] : mx;
      double den = 0.0;
      for (int32_t v = 0; v < V; ++v) den += exp(z[v] - mx);
      const float *u = uniforms ? uniforms + row * (size_t)V : NULL;
      for (int32_t v = 0; v < V; ++v) { ord[v].z = u ? z[v] + gumbel(u[v]) : z[v]; ord[v].id = v; }
      qsort(ord, (size_t)V, sizeof(scored), by_logit_desc);
      for (int32_t r = 0; r < topk; ++r) { ord[r].z = z[ord[r].id]; }
      qsort(ord, (size_t)topk, sizeof(scored), by_logit_desc);
      for (int32_t r = 0; r < topk; ++r) {
        const int32_t id = ord[r].id;
        if (topk_draft) topk_draft[row * topk + r] = id;
        if (topk_ids) topk_ids[row * topk + r] = w->d2t ? w->d2t[id] : id;
        if (topk_probs) topk_probs[row * topk + r] = exp(ord[r].z - mx) / den;
      }
    }
    prefix_off += P;
  }
  free(xs); free(f); free(ge); free(hn); free(z); free(ord);
  return 0;
}

/* Backbone Expansion (Section 2.2): level 1 takes the k candidates of
 * q_{t+1} as children of the root; the most probable one becomes the
 * backbone node and the other k-1 are side branches.  Every later level takes
 * its k candidates as children of the previous backbone node and again extends
 * the backbone with the most probable one.  Nodes are numbered level by level,
 * rank by rank, after the root. */
int feo_build_tree(int32_t batch, int32_t n_layers, int32_t topk, const int32_t *root_tokens,
                   const int32_t *topk_ids, const int32_t *prefix_lens, int32_t *tokens,
                   int32_t *parents, int32_t *depth, int32_t *positions, uint8_t *mask,
                   int32_t *retrieve) {
  if (batch < 0 || n_layers < 1 || topk < 1) return -1;
  const int32_t N = n_layers, k = topk, T = 1 + N * k, NL = N * (k - 1) + 1;
  int32_t *path = (int32_t *)malloc(sizeof(int32_t) * (size_t)(N + 1));
  for (int32_t b = 0; b < batch; ++b) {
    int32_t *tok = tokens + (size_t)b * T, *par = parents + (size_t)b * T;
    int32_t *dep = depth + (size_t)b * T, *pos = positions + (size_t)b * T;
    uint8_t *msk = mask + (size_t)b * T * T;
    int32_t *ret = retrieve + (size_t)b * NL * (N + 1);
    tok[0] = root_tokens[b];
    par[0] = -1;
    dep[0] = 0;
    int32_t backbone = 0, next = 1;
    for (int32_t lvl = 1; lvl <= N; ++lvl) {
      const int32_t *cand = topk_ids + ((size_t)b * N + (size_t)(lvl - 1)) * k;
      int32_t new_backbone = -1;
      for (int32_t r = 0; r < k; ++r) {
        tok[next] = cand[r];
        par[next] = backbone;
        dep[next] = dep[backbone] + 1;
        if (r == 0) new_backbone = next;
        ++next;
      }
      backbone = new_backbone;
    }
    for (int32_t n = 0; n < T; ++n) pos[n] = prefix_lens[b] + dep[n];
    /* ancestor-or-self mask: walk each node's parent chain */
    memset(msk, 0, (size_t)T * T);
    for (int32_t a = 0; a < T; ++a)
      for (int32_t cur = a; cur >= 0; cur = par[cur]) msk[(size_t)a * T + cur] = 1;
    /* leaves (nodes with no children) in node order, with their root paths */
    int32_t leaf = 0;
    for (int32_t n = 0; n < T; ++n) {
      int has_child = 0;
      for (int32_t m = 0; m < T; ++m) has_child |= (par[m] == n);
      if (has_child) continue;
      int32_t len = 0;
      for (int32_t cur = n; cur >= 0; cur = par[cur]) path[len++] = cur;
      int32_t *row = ret + (size_t)leaf * (N + 1);
      for (int32_t t = 0; t < N + 1; ++t) row[t] = t < len ? path[len - 1 - t] : -1;
      ++leaf;
    }
    if (leaf != NL) {
      free(path);
      return -1;
    }
  }
  free(path);
  return 0;
}

/* Greedy acceptance (Section 2.4, parallel verification at temperature 0):
 * every root->leaf path is walked from the root while each next node carries
 * the token the target predicts after its predecessor; the longest accepted
 * prefix wins, the first such path on a tie. */
int feo_accept_greedy(int32_t batch, int32_t n_layers, int32_t topk, const int32_t *tokens,
                      const int32_t *retrieve, const int32_t *target_next, int32_t *accept_len,
                      int32_t *accept_path, int32_t *accepted) {
  if (batch < 0 || n_layers < 1 || topk < 1) return -1;
  const int32_t N = n_layers, T = 1 + N * topk, NL = N * (topk - 1) + 1;
  for (int32_t b = 0; b < batch; ++b) {
    const int32_t *tok = tokens + (size_t)b * T, *nxt = target_next + (size_t)b * T;
    const int32_t *ret = retrieve + (size_t)b * NL * (N + 1);
    int32_t best = -1, best_len = -1;
    for (int32_t p = 0; p < NL; ++p) {
      const int32_t *path = ret + (size_t)p * (N + 1);
      int32_t m = 0;
      while (m < N && path[m + 1] >= 0 && tok[path[m + 1]] == nxt[path[m]]) ++m;
      if (m > best_len) {
        best_len = m;
        best = p;
      }
    }
    const int32_t *path = ret + (size_t)best * (N + 1);
    int32_t *acc = accepted + (size_t)b * (N + 1);
    for (int32_t t = 0; t <= N; ++t) acc[t] = -1;
    for (int32_t t = 1; t <= best_len; ++t) acc[t - 1] = tok[path[t]];
    acc[best_len] = nxt[path[best_len]];
    accept_len[b] = best_len;
    accept_path[b] = best;
  }
  return 0;
}

/* Drafter cache rows of verified positions (Section 2.4: after verification
 * the accepted tokens' target features become the drafter's new context; the
 * cache step is read under the cascade context of Section 2.1).  Every layer
 * i keeps, for position p, its own key and value of the fused input x_0(p):
 * the same projections it applies to the cascade entry x_0 of a pass whose
 * prefix ends at p. */
int feo_kv_update(const feo_config *c, const feo_weights *w, int32_t n_rows, const void *features,
                  const int32_t *tokens, const int32_t *positions, double *const *k_out,
                  double *const *v_out) {
  if (!c || !w || n_rows < 0 || c->n_layers < 1 || c->cascade_ctx == FEO_CTX_SELF) return -1;
  if (c->n_q_heads % c->n_kv_heads != 0 || c->head_dim % 2 != 0) return -1;
  const int32_t d = c->hidden, F = c->n_feat_levels, D = c->head_dim, Hkv = c->n_kv_heads;
  const int32_t kvd = Hkv * D;
  for (int32_t m = 0; m < n_rows; ++m)
    if (tokens[m] < 0 || tokens[m] >= c->target_vocab || positions[m] < 0) return -1;
  double *f = (double *)malloc(sizeof(double) * (size_t)F * d);
  double *ge = (double *)malloc(sizeof(double) * (size_t)2 * d);
  double *x0 = (double *)malloc(sizeof(double) * (size_t)d);
  double *a = (double *)malloc(sizeof(double) * (size_t)d);
  for (int32_t m = 0; m < n_rows; ++m) {
    fused_input(c, w, features, (size_t)m, tokens[m], f, ge, x0);
    for (int32_t i = 1; i <= c->n_layers; ++i) {
      const feo_layer *L = &w->layers[i - 1];
      double *k = k_out[i - 1] + (size_t)m * kvd, *v = v_out[i - 1] + (size_t)m * kvd;
      feo_rmsnorm(x0, L->attn_norm, c->dtype, d, c->rms_eps, a);
      matvec(L->wk, c->dtype, kvd, d, a, k);
      matvec(L->wv, c->dtype, kvd, d, a, v);
      for (int32_t h = 0; h < Hkv; ++h) feo_rope(k + (size_t)h * D, D, positions[m], c->rope_theta);
    }
  }
  free(f); free(ge); free(x0); free(a);
  return 0;
}

/* Drafter cache rows under FEO_CTX_SELF (Section 2.4 update step, read under
 * the self context of Eq. 2: layer i's context is its prefix plus its own
 * input).  The row of layer i at position p is layer i's key and value of its
 * own input x_{i-1}(p) -- what the pass at prefix p attends to as that input
 * -- so filling it means running the pass itself at every new position, one
 * position after the other: row m at position p = positions[m] goes to cache
 * row r = dst_rows[m], its sequence's row of position j < p being cache row
 * r - (p - j): the row an earlier row of this call wrote there (its fp64
 * result), else that row of kcache / vcache (storage precision, keys
 * rotated).  For row m, x_0 is the fused input (Eq. 1); layer i takes x_{i-1},
 * emits its key and value at position p as row m's output and computes x_i
 * over the prefix rows 0..p-1 plus its own. */
int feo_kv_update_self(const feo_config *c, const feo_weights *w, int32_t n_rows,
                       const void *features, const int32_t *tokens, const int32_t *positions,
                       const int32_t *dst_rows, const void *const *kcache,
                       const void *const *vcache, int64_t cache_rows, double *const *k_out,
                       double *const *v_out) {
  if (!c || !w || n_rows < 0 || c->n_layers < 1 || c->cascade_ctx != FEO_CTX_SELF) return -1;
  if (c->n_q_heads % c->n_kv_heads != 0 || c->head_dim % 2 != 0 || cache_rows < 0) return -1;
  const int32_t d = c->hidden, F = c->n_feat_levels, N = c->n_layers;
  const int32_t kvd = c->n_kv_heads * c->head_dim;
  for (int32_t m = 0; m < n_rows; ++m) {
    if (tokens[m] < 0 || tokens[m] >= c->target_vocab || positions[m] < 0) return -1;
    if (dst_rows[m] < positions[m] || dst_rows[m] >= cache_rows) return -1;
  }
  double *xs = (double *)malloc(sizeof(double) * (size_t)(N + 1) * d);
  double *f = (double *)malloc(sizeof(double) * (size_t)F * d);
  double *ge = (double *)malloc(sizeof(double) * (size_t)2 * d);
  for (int32_t m = 0; m < n_rows; ++m) {
    const int32_t p = positions[m];
    const int64_t r0 = (int64_t)dst_rows[m] - p;  /* cache row of position 0 */
    double *pk = (double *)malloc(sizeof(double) * ((size_t)p * kvd + 1));
    double *pv = (double *)malloc(sizeof(double) * ((size_t)p * kvd + 1));
    fused_input(c, w, features, (size_t)m, tokens[m], f, ge, xs);
    for (int32_t i = 1; i <= N; ++i) {
      /* layer i's rows of positions 0..p-1 */
      for (int32_t j = 0; j < p; ++j) {
        const int64_t row = r0 + j;
        int32_t from = -1;  /* the last earlier row of this call written there */
        for (int32_t e = 0; e < m; ++e)
          if (dst_rows[e] == row) from = e;
        for (int32_t x = 0; x < kvd; ++x) {
          if (from >= 0) {
            pk[(size_t)j * kvd + x] = k_out[i - 1][(size_t)from * kvd + x];
            pv[(size_t)j * kvd + x] = v_out[i - 1][(size_t)from * kvd + x];
          } else {
            pk[(size_t)j * kvd + x] = widen(kcache[i - 1], c->dtype, (size_t)row * kvd + x);
            pv[(size_t)j * kvd + x] = widen(vcache[i - 1], c->dtype, (size_t)row * kvd + x);
          }
        }
      }
      cascade_layer(c, &w->layers[i - 1], i, xs, pk, pv, KV_F64, 0, p,
                    k_out[i - 1] + (size_t)m * kvd, v_out[i - 1] + (size_t)m * kvd);
    }
    free(pk);
    free(pv);
  }
  free(xs); free(f); free(ge);
  return 0;
}

/* Speculative-sampling acceptance of one drafting cycle at temperature T
 * (Section 2.4, parallel verification; Section 3 reports temperature 1).
 * Children drawn without replacement from the level's draft distribution q
 * (draft_uniforms given: their Gumbel keys fix the order of the draws) are
 * tested in draw order by recursive rejection sampling: child x is accepted
 * when u <= p(x) / q(x); on a rejection the target's distribution becomes the
 * normalised positive part of p - q and x leaves q (which is renormalised).
 * Children chosen without randomness (draft_uniforms NULL: the top-k list) are
 * tested in listing order against q = a point mass on x: accepted when
 * u <= p(x), else x leaves p.  When every child is rejected, or the accepted
 * node has no children, one more token is drawn from the current p by inverse
 * CDF (target ids that draft ids map to first, in draft-id order, then the
 * others in increasing order).  Either way the emitted tokens follow the
 * target's distributions exactly. */
int feo_accept_sample(int32_t batch, int32_t n_layers, int32_t topk, int32_t draft_vocab,
                      int32_t target_vocab, const int32_t *tokens, const int32_t *retrieve,
                      const int32_t *topk_draft, const float *draft_logits, double temperature,
                      const float *draft_uniforms, const int32_t *d2t, const float *target_probs,
                      const float *uniforms, int32_t *accept_len, int32_t *accept_path,
                      int32_t *accepted, double *margin) {
  if (batch < 0 || n_layers < 1 || n_layers > 63 || topk < 1 || topk > 64 || draft_vocab < topk ||
      target_vocab < 1)
    return -1;
  if (!(temperature > 0.0)) return -1;
  const int32_t N = n_layers, k = topk, V = draft_vocab, Vt = target_vocab;
  const int32_t T = 1 + N * k, NL = N * (k - 1) + 1, NU = N * k + 1;
  double *r = (double *)malloc(sizeof(double) * (size_t)Vt);
  double *q0 = (double *)malloc(sizeof(double) * (size_t)V);
  char *gone = (char *)malloc((size_t)V);
  for (int32_t b = 0; b < batch; ++b) {
    const int32_t *tok = tokens + (size_t)b * T;
    const float *u = uniforms + (size_t)b * NU;
    int32_t path[64], len = 0, node = 0, t = 0;
    double mg = INFINITY, Z = 0.0;
    path[0] = 0;
    for (;;) {
      /* the target's distribution after the path so far */
      const float *p = target_probs + ((size_t)b * T + (size_t)node) * Vt;
      Z = 0.0;
      for (int32_t x = 0; x < Vt; ++x) { r[x] = (double)p[x]; Z += r[x]; }
      /* children: the k level-(len+1) nodes under the root or a backbone node */
      const int32_t lvl = len + 1;
      const int has_children = lvl <= N && (node == 0 || node == 1 + (lvl - 2) * k);
      if (!has_children) break;
      const size_t lrow = (size_t)b * N + (size_t)(lvl - 1);
      const float *z = draft_logits + lrow * V;
      const int32_t *cd = topk_draft + lrow * k;
      /* test order: the draws' order (Gumbel keys, larger first, lower id on
       * ties), or the listing order for unsampled children */
      scored ordk[64];
      for (int32_t rho = 0; rho < k; ++rho) {
        ordk[rho].id = rho;
        ordk[rho].z = draft_uniforms
            ? z[cd[rho]] / temperature + gumbel(draft_uniforms[lrow * V + (size_t)cd[rho]])
            : -(double)rho;
      }
      for (int32_t i = 1; i < k; ++i)   /* insertion sort: keys desc, draft id asc */
        for (int32_t j = i; j > 0; --j) {
          const scored a = ordk[j - 1], c = ordk[j];
          const int swap = c.z > a.z || (c.z == a.z && cd[c.id] < cd[a.id]);
          if (!swap) break;
          ordk[j - 1] = c;
          ordk[j] = a;
        }
      if (draft_uniforms)   /* how close the draw order came to a tie */
        for (int32_t j = 1; j < k; ++j) {
          const double sc = fabs(ordk[j].z) > 1.0 ? fabs(ordk[j].z) : 1.0;
          const double m = (ordk[j - 1].z - ordk[j].z) / sc;
          if (m < mg) mg = m;
        }
      /* q_{t+lvl} = softmax(z / T) over the draft vocabulary */
      double mx = -INFINITY, S = 0.0;
      for (int32_t v = 0; v < V; ++v) mx = z[v] / temperature > mx ? z[v] / temperature : mx;
      for (int32_t v = 0; v < V; ++v) { q0[v] = exp(z[v] / temperature - mx); S += q0[v]; }
      for (int32_t v = 0; v < V; ++v) { q0[v] /= S; gone[v] = 0; }
      double R = 0.0;  /* q mass of the rejected children */
      int accepted_child = 0;
      for (int32_t j = 0; j < k; ++j) {
        const int32_t rho = ordk[j].id;
        const int32_t child = 1 + (lvl - 1) * k + rho, vd = cd[rho], x = tok[child];
        const double qi = draft_uniforms ? q0[vd] / (1.0 - R) : 1.0, pi = r[x] / Z;
        const double ut = (double)u[t++];
        const double m = fabs(ut * qi - pi) / (qi > pi ? qi : pi);
        if (m < mg) mg = m;
        if (ut * qi <= pi) {
          node = child;
          path[++len] = child;
          accepted_child = 1;
          break;
        }
        if (!draft_uniforms) {   /* q is a point mass on x: x leaves p */
          Z -= r[x];
          r[x] = 0.0;
          continue;
        }
        /* p <- (p - q)^+ / Z', q <- q without x */
        double dec = 0.0;
        for (int32_t v = 0; v < V; ++v) {
          if (gone[v]) continue;
          const int32_t xt = d2t ? d2t[v] : v;
          const double nv = r[xt] - Z * q0[v] / (1.0 - R);
          const double nr = nv > 0.0 ? nv : 0.0;
          dec += r[xt] - nr;
          r[xt] = nr;
        }
        Z -= dec;
        gone[vd] = 1;
        R += q0[vd];
      }
      if (!accepted_child) break;
    }
    /* one token from the current p by inverse CDF, enumerating the target ids
     * in a fixed order: those the draft vocabulary maps to, in draft-id order,
     * then every other target id in increasing order */
    const double target = (double)u[NU - 1] * Z;
    double cum = 0.0;
    int32_t pick = -1, last = -1;
    char *img = (char *)calloc((size_t)Vt, 1);
    for (int32_t v = 0; v < V; ++v) img[d2t ? d2t[v] : v] = 1;
    for (int32_t e = 0; e < V + Vt; ++e) {
      int32_t x;
      if (e < V) x = d2t ? d2t[e] : e;
      else if (!img[e - V]) x = e - V;
      else continue;
      if (r[x] > 0.0) last = x;
      const double prev = cum;
      cum += r[x];
      if (pick < 0 && cum > target) {
        pick = x;
        const double m1 = (target - prev) / Z, m2 = (cum - target) / Z;
        const double m = m1 < m2 ? m1 : m2;
        if (m < mg) mg = m;
      }
    }
    free(img);
    if (pick < 0) pick = last;
    int32_t *acc = accepted + (size_t)b * (N + 1);
    for (int32_t i = 0; i <= N; ++i) acc[i] = -1;
    for (int32_t i = 1; i <= len; ++i) acc[i - 1] = tok[path[i]];
    acc[len] = pick;
    accept_len[b] = len;
    /* the first root->leaf path that holds the accepted nodes */
    const int32_t *ret = retrieve + (size_t)b * NL * (N + 1);
    accept_path[b] = -1;
    for (int32_t row = 0; row < NL && accept_path[b] < 0; ++row) {
      int ok = 1;
      for (int32_t i = 0; i <= len; ++i) ok &= ret[(size_t)row * (N + 1) + i] == path[i];
      if (ok) accept_path[b] = row;
    }
    if (margin) margin[b] = mg;
  }
  free(r); free(q0); free(gone);
  return 0;
}
