// fe_misc.hip -- RMSNorm rows, LM-head top-k merge and the Backbone Expansion
// tree (gfx950).
#include "fe_internal.h"
#include "fe_tree.h"

namespace fe {

// ---------------------------------------------------------------------------
// RMSNorm (pre-attention, pre-MLP and final norm of the LLaMA-style layer):
// y = gamma * x / sqrt(mean(x^2) + eps), fp32 statistics, storage-type output.
// One workgroup per row; fixed-order reductions.
// ---------------------------------------------------------------------------
// One workgroup per row; the row (NV float4 per thread, d <= 1024*NV) and its
// gains are loaded once, up front, and stay in registers.
template <typename T, int NV>
__global__ __launch_bounds__(256) void k_rmsnorm(const float *__restrict__ X, int per, int j0,
                                                 long outer, long inner,
                                                 const T *__restrict__ gamma, T *__restrict__ out,
                                                 int d, float eps) {
  __shared__ float red[4];
  const int r = blockIdx.x, tid = threadIdx.x;
  const float *x = X + (long)(r / per) * outer + (long)(j0 + r % per) * inner;
  f32x4 xv[NV];
  float gv[NV][4];
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int e = 4 * (tid + 256 * u);
    const int ec = min(e, d - 4);
    xv[u] = *reinterpret_cast<const f32x4 *>(x + ec);
#pragma unroll
    for (int q = 0; q < 4; ++q) gv[u][q] = Elt<T>::to_f(gamma[ec + q]);
    if (e >= d) xv[u] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < NV; ++u) ss += xv[u].x * xv[u].x + xv[u].y * xv[u].y + xv[u].z * xv[u].z + xv[u].w * xv[u].w;
  ss = group_sum<64>(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  T *y = out + (long)r * d;
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int e = 4 * (tid + 256 * u);
    if (e < d) {
      const float v0 = gv[u][0] * (xv[u].x * inv), v1 = gv[u][1] * (xv[u].y * inv);
      const float v2 = gv[u][2] * (xv[u].z * inv), v3 = gv[u][3] * (xv[u].w * inv);
      if constexpr (sizeof(T) == 2)  // four values in one 8-byte store
        *reinterpret_cast<u32x2 *>(y + e) = u32x2{f2bf2(v0, v1), f2bf2(v2, v3)};
      else
        *reinterpret_cast<f32x4 *>(y + e) = f32x4{v0, v1, v2, v3};
    }
  }
}

template <typename T>
static void launch_rmsnorm(const float *X, int rows, int per, int j0, long outer, long inner,
                           const void *gamma, void *out, int d, float eps, hipStream_t s) {
#define FE_RMS(NVV)                                                                         \
  hipLaunchKernelGGL((k_rmsnorm<T, NVV>), dim3(rows), dim3(256), 0, s, X, per, j0, outer, inner, \
                     (const T *)gamma, (T *)out, d, eps)
  if (d <= 1024) FE_RMS(1);
  else if (d <= 2048) FE_RMS(2);
  else if (d <= 4096) FE_RMS(4);
  else FE_RMS(8);
#undef FE_RMS
}

// One RMS per row, several gains: copy q of row r is gamma_q * x / rms(x) at
// out_q + r * d (the cache update's per-layer K/V operands from one x_0).
template <typename T, int NV>
__global__ __launch_bounds__(256) void k_rmsnorm_copies(const float *__restrict__ X, RmsCopies c,
                                                        int d, float eps) {
  __shared__ float red[4];
  const int r = blockIdx.x, tid = threadIdx.x;
  const float *x = X + (long)r * d;
  f32x4 xv[NV];
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int e = 4 * (tid + 256 * u);
    xv[u] = e < d ? *reinterpret_cast<const f32x4 *>(x + e) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < NV; ++u) ss += xv[u].x * xv[u].x + xv[u].y * xv[u].y + xv[u].z * xv[u].z + xv[u].w * xv[u].w;
  ss = group_sum<64>(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int e = 4 * (tid + 256 * u);
    if (e >= d) continue;
    for (int q = 0; q < c.n; ++q) {
      const T *g = (const T *)c.gamma[q];
      T *y = (T *)c.out[q] + (long)r * d + e;
      float v[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = Elt<T>::to_f(g[e + k]) * (xv[u][k] * inv);
      if constexpr (sizeof(T) == 2)  // four values in one 8-byte store
        *reinterpret_cast<u32x2 *>(y) = u32x2{f2bf2(v[0], v[1]), f2bf2(v[2], v[3])};
      else
        *reinterpret_cast<f32x4 *>(y) = f32x4{v[0], v[1], v[2], v[3]};
    }
  }
}

hipError_t rmsnorm_copies(int dt, const float *X, int rows, const RmsCopies &c, int d, float eps,
                          hipStream_t s) {
  if (rows <= 0 || c.n <= 0) return hipSuccess;
  if (d > 8192 || d % 4 || c.n > kMaxLayers) return hipErrorInvalidValue;
#define FE_RMSC(TV, NVV) \
  hipLaunchKernelGGL((k_rmsnorm_copies<TV, NVV>), dim3(rows), dim3(256), 0, s, X, c, d, eps)
#define FE_RMSC_T(TV)                \
  if (d <= 1024) FE_RMSC(TV, 1);     \
  else if (d <= 2048) FE_RMSC(TV, 2); \
  else if (d <= 4096) FE_RMSC(TV, 4); \
  else FE_RMSC(TV, 8)
  if (dt) { FE_RMSC_T(bf16_t); } else { FE_RMSC_T(float); }
#undef FE_RMSC_T
#undef FE_RMSC
  return hipGetLastError();
}

hipError_t rmsnorm_rows(int dt, const float *X, int rows, int per, int j0, long outer, long inner,
                        const void *gamma, void *out, int d, float eps, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d > 8192 || d % 4) return hipErrorInvalidValue;
  if (dt) launch_rmsnorm<bf16_t>(X, rows, per, j0, outer, inner, gamma, out, d, eps, s);
  else launch_rmsnorm<float>(X, rows, per, j0, outer, inner, gamma, out, d, eps, s);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Top-k merge: the LM-head tiles left, per row, a (max, sum exp) pair and k
// candidates each.  The row's softmax statistics are mu = max_t m_t and
// S = sum_t s_t exp(m_t - mu); the global top-k is the best k of all tile
// candidates (larger logit first, lower draft id on ties); p = exp(z - mu)/S.
// ---------------------------------------------------------------------------

// One workgroup (4 waves) per row.  Each wave selects the top-k of the
// candidates its lanes hold (k rounds of butterfly max over ordering keys, no
// block barrier), then wave 0 selects the top-k of the 4k wave winners and
// writes them.

template <bool SAMPLED, int CAP>
__global__ __launch_bounds__(256) void k_topk_merge(const float *__restrict__ pmax,
                                                    const float *__restrict__ psum,
                                                    const float *__restrict__ cval,
                                                    const int32_t *__restrict__ cidx,
                                                    const float *__restrict__ cz, int nwg,
                                                    int topk, int V, const int32_t *__restrict__ d2t,
                                                    int32_t *ids, int32_t *draft_ids,
                                                    float *probs, TreeRows tr) {
  static_assert(256 * CAP <= kMergeMaxCand, "candidates per thread");
  __shared__ float sv[4];
  __shared__ uint64_t s_key[4][kMaxTopk];
  __shared__ float s_z[4][kMaxTopk];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // the tree of sequence b (rows b*N .. b*N+N-1 are its levels): the level-1
  // row's workgroup writes its root and structure, every row its level's nodes
  const int tb = tr.tokens ? row / tr.N : 0, tl = tr.tokens ? row % tr.N : 0;
  const int tT = 1 + tr.N * topk;
  if (tr.tokens && tl == 0) {
    if (tid == 0) tr.tokens[(size_t)tb * tT] = tr.root[tb];
    tree_structure(tb, tr.N, topk, tr.cu_prefix[tb + 1] - tr.cu_prefix[tb], tr.parents, tr.depth,
                   tr.positions, tr.mask, tr.retrieve);
  }
  const float *pm = pmax + (size_t)row * nwg;
  const float *ps = psum + (size_t)row * nwg;
  // every candidate of the row into registers (thread t holds t, t+256, ...):
  // unconditional loads at clamped indices (one memory round trip), masked after
  const int ncand = nwg * topk;
  float cv[CAP];
  int ci[CAP];
#pragma unroll
  for (int j = 0; j < CAP; ++j) {
    const int c = min(tid + 256 * j, ncand - 1);
    const size_t o = ((size_t)row * nwg + c / topk) * kMaxTopk + c % topk;
    cv[j] = cval[o];
    ci[j] = cidx[o];
  }
  // softmax statistics: mu = max_t m_t, S = sum_t s_t exp(m_t - mu), fixed
  // order; the tile statistics are loaded with the candidates (kStatLoads per
  // thread cover nwg <= 1024; a loop covers the rest)
  constexpr int kStatLoads = 4;
  float pmv[kStatLoads], psv[kStatLoads];
#pragma unroll
  for (int u = 0; u < kStatLoads; ++u) {
    const int t = min(tid + 256 * u, nwg - 1);
    pmv[u] = pm[t];
    psv[u] = ps[t];
  }
  uint64_t key[CAP];
#pragma unroll
  for (int j = 0; j < CAP; ++j) key[j] = tid + 256 * j < ncand ? topk_key(cv[j], ci[j]) : kNoKey;
  float m = -INFINITY;
#pragma unroll
  for (int u = 0; u < kStatLoads; ++u)
    if (tid + 256 * u < nwg) m = fmaxf(m, pmv[u]);
  for (int t = tid + 256 * kStatLoads; t < nwg; t += 256) m = fmaxf(m, pm[t]);
  m = group_max<64>(m);
  if (lane == 0) sv[wave] = m;
  __syncthreads();
  const float mu = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
  __syncthreads();
  float S = 0.f;
#pragma unroll
  for (int u = 0; u < kStatLoads; ++u)
    if (tid + 256 * u < nwg) S += psv[u] * expf(pmv[u] - mu);
  for (int t = tid + 256 * kStatLoads; t < nwg; t += 256) S += ps[t] * expf(pm[t] - mu);
  S = group_sum<64>(S);
  if (lane == 0) sv[wave] = S;
  // sampled candidates: their z / T, loaded beside the keys
  float czv[SAMPLED ? CAP : 1];
  if constexpr (SAMPLED) {
#pragma unroll
    for (int j = 0; j < CAP; ++j) {
      const int c = min(tid + 256 * j, ncand - 1);
      czv[j] = cz[((size_t)row * nwg + c / topk) * kMaxTopk + c % topk];
    }
  }
  // per-wave top-k
  for (int r = 0; r < topk; ++r) {
    uint64_t best = kNoKey;
#pragma unroll
    for (int j = 0; j < CAP; ++j) best = key[j] > best ? key[j] : best;
    best = wave_max_u64(best);
    float zb = -INFINITY;
#pragma unroll
    for (int j = 0; j < CAP; ++j) {
      if constexpr (SAMPLED) {
        if (key[j] == best && best != kNoKey) zb = czv[j];
      }
      key[j] = key[j] == best ? kNoKey : key[j];
    }
    if constexpr (SAMPLED) zb = group_max<64>(zb);  // one lane held the winner
    if (lane == 0) {
      s_key[wave][r] = best;
      if constexpr (SAMPLED) s_z[wave][r] = zb;
    }
  }
  __syncthreads();
  if (wave == 0) {
    const float Ssum = (sv[0] + sv[1]) + (sv[2] + sv[3]);
    uint64_t k = lane < 4 * topk ? s_key[lane / topk][lane % topk] : kNoKey;
    const float kz = SAMPLED && lane < 4 * topk ? s_z[lane / topk][lane % topk] : -INFINITY;
    uint64_t mine = kNoKey;
    float mz = -INFINITY;
    for (int r = 0; r < topk; ++r) {
      const uint64_t best = wave_max_u64(k);
      // the lane holding the winner (keys are distinct) gives its z / T
      float bz = -INFINITY;
      if constexpr (SAMPLED) {
        const uint64_t hit = __builtin_amdgcn_ballot_w64(k == best && best != kNoKey);
        bz = hit ? __shfl(kz, __builtin_ctzll(hit)) : -INFINITY;
      }
      k = k == best ? kNoKey : k;
      if (lane == r) {
        mine = best;
        mz = bz;
      }
    }
    const int i = topk_key_id(mine);
    const bool valid = lane < topk && mine != kNoKey && i >= 0 && i < V;  // none left (NaN row): -1
    const float z = SAMPLED ? mz : topk_key_value(mine);
    // listing position: key order, or for sampled candidates the order of z / T
    // (larger first, lower id on ties, NaN after numbers, invalid entries last
    // in lane order): the rank of the lane's ordering key among the winners
    int pos = lane;
    if constexpr (SAMPLED) {
      const uint64_t zk = valid ? topk_key(z, i) : kNoKey;
      pos = 0;
      for (int t = 0; t < topk; ++t) {
        const uint64_t kt = ((uint64_t)(uint32_t)__shfl((int)(uint32_t)(zk >> 32), t) << 32) |
                            (uint32_t)__shfl((int)(uint32_t)zk, t);
        pos += (kt > zk || (kt == zk && t < lane)) ? 1 : 0;
      }
    }
    if (lane < topk) {
      const size_t o = (size_t)row * topk + pos;
      const int32_t id = valid ? (d2t ? d2t[i] : i) : -1;
      ids[o] = id;
      if (tr.tokens) tr.tokens[(size_t)tb * tT + 1 + tl * topk + pos] = id;
      if (draft_ids) draft_ids[o] = valid ? i : -1;
      probs[o] = valid ? expf(z - mu) / Ssum : __int_as_float(0x7fc00000);
    }
  }
}

hipError_t topk_merge(const float *part_max, const float *part_sum, const float *cand_val,
                      const int32_t *cand_idx, const float *cand_z, int rows, int nwg, int topk,
                      int V, const int32_t *d2t, int32_t *ids, int32_t *draft_ids, float *probs,
                      hipStream_t s, const TreeRows *tree) {
  const TreeRows tr = tree ? *tree : TreeRows{};
  if (tr.tokens && (tr.N < 1 || rows % tr.N)) return hipErrorInvalidValue;
  if (rows <= 0) return hipSuccess;
  const long ncand = (long)nwg * topk;
  if (ncand > kMergeMaxCand) return hipErrorInvalidValue;
  // candidates per thread: the fewest registers that hold the row (the k
  // selection rounds scan all of them)
#define FE_MERGE(SV, CAPV)                                                                         \
  hipLaunchKernelGGL((k_topk_merge<SV, CAPV>), dim3(rows), dim3(256), 0, s, part_max, part_sum,    \
                     cand_val, cand_idx, cand_z, nwg, topk, V, d2t, ids, draft_ids, probs, tr)
#define FE_MERGE_CAP(SV)                                     \
  if (ncand <= 256 * 8) FE_MERGE(SV, 8);                     \
  else if (ncand <= 256 * 16) FE_MERGE(SV, 16);              \
  else FE_MERGE(SV, kMergeMaxCand / 256)
  if (cand_z) { FE_MERGE_CAP(true); }
  else { FE_MERGE_CAP(false); }
#undef FE_MERGE_CAP
#undef FE_MERGE
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Backbone Expansion tree (Section 2.2), one workgroup per sequence.  With
// nodes numbered root first and then level by level in rank order, node
// n >= 1 sits at level l = 1 + (n-1)/k with rank rho = (n-1)%k; its parent is
// the root for l = 1 and the level-(l-1) backbone node 1 + (l-2)k otherwise.
// Its ancestors are the root, the backbone nodes of the levels above it, and
// itself.  Leaves are the side branches (rho != 0) and the level-N backbone
// node.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_build_tree(int N, int k,
                                                    const int32_t *__restrict__ root_tokens,
                                                    const int32_t *__restrict__ topk_ids,
                                                    const int32_t *__restrict__ prefix_lens,
                                                    const int32_t *__restrict__ cu_prefix,
                                                    int32_t *tokens, int32_t *parents,
                                                    int32_t *depth, int32_t *positions,
                                                    uint8_t *mask, int32_t *retrieve) {
  const int b = blockIdx.x, T = 1 + N * k;
  const int P = prefix_lens ? prefix_lens[b] : cu_prefix[b + 1] - cu_prefix[b];
  for (int n = threadIdx.x; n < T; n += blockDim.x) {
    int tok = root_tokens[b];
    if (n > 0) {
      const int lvl = 1 + (n - 1) / k, rho = (n - 1) % k;
      tok = topk_ids[((size_t)b * N + (lvl - 1)) * k + rho];
    }
    tokens[(size_t)b * T + n] = tok;
  }
  tree_structure(b, N, k, P, parents, depth, positions, mask, retrieve);
}

hipError_t build_tree(int B, int N, int k, const int32_t *root_tokens, const int32_t *topk_ids,
                      const int32_t *prefix_lens, const int32_t *cu_prefix, int32_t *tokens,
                      int32_t *parents, int32_t *depth, int32_t *positions, uint8_t *mask,
                      int32_t *retrieve, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_build_tree, dim3(B), dim3(256), 0, s, N, k, root_tokens, topk_ids,
                     prefix_lens, cu_prefix, tokens, parents, depth, positions, mask, retrieve);
  return hipGetLastError();
}

// ---- greedy acceptance of a drafting cycle --------------------------------------
// Section 2.4 (parallel verification) at temperature 0: along a root->leaf path
// of the tree, node r_t is accepted while every node up to it carries the token
// the target predicts after its predecessor.  One wave per sequence, one lane
// per path (64 at a time): the accepted length, then a wave max over the key
// (length << 16 | 0xffff - path), so ties go to the first path.  Node indices
// outside the tree end a walk (they cannot occur in a tree built here).
__global__ __launch_bounds__(64) void k_accept_greedy(int N, int k, const int32_t *__restrict__ tokens,
                                                      const int32_t *__restrict__ retrieve,
                                                      const int32_t *__restrict__ target_next,
                                                      int32_t *__restrict__ accept_len,
                                                      int32_t *__restrict__ accept_path,
                                                      int32_t *__restrict__ accepted) {
  const int b = blockIdx.x, lane = threadIdx.x;
  const int T = 1 + N * k, NL = N * (k - 1) + 1;
  const int32_t *tok = tokens + (size_t)b * T, *nxt = target_next + (size_t)b * T;
  const int32_t *ret = retrieve + (size_t)b * NL * (N + 1);
  uint32_t best = 0;
  for (int p = lane; p < NL; p += 64) {
    const int32_t *path = ret + (size_t)p * (N + 1);
    int m = 0, prev = path[0];
    while (m < N && prev >= 0 && prev < T) {
      const int nn = path[m + 1];
      if (nn < 0 || nn >= T || tok[nn] != nxt[prev]) break;
      prev = nn;
      ++m;
    }
    best = max(best, ((uint32_t)m << 16) | (uint32_t)(0xffff - p));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) best = max(best, (uint32_t)__shfl_xor((int)best, o, 64));
  const int m = (int)(best >> 16), p = 0xffff - (int)(best & 0xffffu);
  const int32_t *path = ret + (size_t)p * (N + 1);
  for (int t = lane; t <= N; t += 64) {
    int32_t v = -1;
    if (t < m) {
      v = tok[path[t + 1]];
    } else if (t == m) {
      const int last = path[m];
      v = last >= 0 && last < T ? nxt[last] : -1;
    }
    accepted[(size_t)b * (N + 1) + t] = v;
  }
  if (lane == 0) {
    accept_len[b] = m;
    accept_path[b] = p;
  }
}
hipError_t accept_greedy(int B, int N, int k, const int32_t *tokens, const int32_t *retrieve,
                         const int32_t *target_next, int32_t *accept_len, int32_t *accept_path,
                         int32_t *accepted, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_accept_greedy, dim3(B), dim3(64), 0, s, N, k, tokens, retrieve, target_next,
                     accept_len, accept_path, accepted);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Speculative-sampling acceptance at temperature T (Section 2.4), one
// 1024-thread workgroup per sequence walking its tree from the root.  The
// target's distribution p at the current node changes only where the draft
// distribution q lives, i.e. at the target ids the draft ids map to, so the
// residual is kept per draft id in LDS (rd[v] = r(d2t[v])) while every other
// target id keeps p(x) in memory; an LDS bitmask marks the mapped target ids.
// Sampled children are tested in draw order (their Gumbel keys, recomputed
// from the drafting uniforms) by recursive rejection sampling (accept when
// u * q_i(x) <= r(x) / Z; on a rejection rd <- (rd - Z q_i)^+ and x leaves q),
// unsampled ones in listing order against point masses (accept when
// u <= r(x) / Z, else rd(x) <- 0).  The last uniform draws one token by
// inverse CDF: mapped ids first in draft-id order, then the other target ids
// in increasing order.  Each wave owns a contiguous chunk of the ids and
// reads it 64 consecutive ids per step (coalesced): one pass per visited node
// sums p (Z) and the unmapped part of every chunk; chunk sums are added in
// order, the chunks' ranges tile the line exactly, and the owning wave walks
// its chunk with wave scans to the drawn id.  Loads are issued kAccBatch at a
// time.  Every decision is taken on block-reduced values, so control flow is
// uniform across the workgroup.
// ---------------------------------------------------------------------------
constexpr int kAccThreads = 1024;
constexpr int kAccBatch = 32;  // floats per lane in flight in a pass over a target row
constexpr int kAccMaxV = kAccSampleMaxV;    // draft ids whose residual fits the LDS
constexpr int kAccMaxVt = kAccSampleMaxVt;  // target ids the LDS bitmask covers
constexpr int kAccWaves = kAccThreads / 64;

__device__ __forceinline__ float acc_sum(float v, float *red) {
  v = group_sum<64>(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int w = 0; w < kAccWaves; ++w) t += red[w];
  return t;
}
__device__ __forceinline__ float acc_max(float v, float *red) {
  v = group_max<64>(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float t = -INFINITY;
#pragma unroll
  for (int w = 0; w < kAccWaves; ++w) t = fmaxf(t, red[w]);
  return t;
}
// Inclusive scan over the 64 lanes of a wave (fixed order of additions).
__device__ __forceinline__ float wave_incl_scan(float x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

// The owning wave's walk of its chunk [c0, c1) for the running sum (from
// `start`) to pass `target`: val(e) per id, W consecutive ids per lane and
// 64 * W per step, kAccBatch / W steps' loads in flight.  Returns the id, or
// -1 if rounding kept the running sum at or below target through the chunk.
template <int W, class Load>
__device__ int acc_walk(int c0, int c1, float start, float target, const Load &load) {
  constexpr int NB = kAccBatch / W;
  const int lane = threadIdx.x & 63;
  float run = start;
#pragma unroll 1
  for (int e = c0; e < c1; e += 64 * W * NB) {
    float a[NB][W];
#pragma unroll
    for (int j = 0; j < NB; ++j) load(e + 64 * W * j + W * lane, a[j]);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      float sl = 0.f;
#pragma unroll
      for (int q = 0; q < W; ++q) sl += a[j][q];
      const float incl = wave_incl_scan(sl);
      const uint64_t hit = __builtin_amdgcn_ballot_w64(run + incl > target);
      if (hit) {
        const int L = __builtin_ctzll(hit);
        float ex = __shfl_up(incl, 1);
        if (lane == 0) ex = 0.f;
        float c = run + ex;
        int pk = -1;
#pragma unroll
        for (int q = 0; q < W; ++q) {   // first q whose running sum passes
          c += a[j][q];
          if (pk < 0 && c > target) pk = q;
        }
        if (pk < 0) pk = W - 1;
        return e + 64 * W * j + W * L + __shfl(pk, L);
      }
      run += __shfl(incl, 63);
    }
  }
  return -1;
}

// Bitmask of the target ids that draft ids map to: bit x of img is set when
// x = d2t[v] for some v (built in LDS by one workgroup, then stored).
__global__ __launch_bounds__(kAccThreads) void k_build_img(const int32_t *__restrict__ d2t, int V,
                                                           int Vt, uint32_t *img) {
  __shared__ uint32_t s_img[kAccMaxVt / 32];
  const int tid = threadIdx.x, nw = (Vt + 31) / 32;
  for (int w = tid; w < nw; w += kAccThreads) s_img[w] = 0u;
  __syncthreads();
  for (int v = tid; v < V; v += kAccThreads) {
    const int x = d2t ? d2t[v] : v;
    if (x >= 0 && x < Vt) atomicOr(&s_img[x >> 5], 1u << (x & 31));
  }
  __syncthreads();
  for (int w = tid; w < nw; w += kAccThreads) img[w] = s_img[w];
}

// Chunks of a target row as the walk's waves own them: kAccWaves contiguous
// ranges of CW ids (CW a multiple of 64 W).
__host__ __device__ inline int acc_chunk_width(int Vt, int W) {
  return ((Vt + kAccWaves - 1) / kAccWaves + 64 * W - 1) / (64 * W) * (64 * W);
}

// Few sequences: before the walk, every node's target row is reduced by
// workgroups of its own instead of by the one walking workgroup when (and if)
// it gets there.  Row (sequence b, node n), workgroup y < kAccWaves: chunk y's
// sum of p, its unmapped part (ids no draft id maps to) and its last unmapped
// id with mass; y >= kAccWaves: p at the mapped ids of draft ids
// [(y - kAccWaves) * VP, ...) (the walk's residual row, compact).
constexpr int kAccPreThreads = 256, kAccPreGather = 16;
template <int W>
__global__ __launch_bounds__(kAccPreThreads) void k_accept_rows(
    int Vt, int V, const int32_t *__restrict__ d2t, const float *__restrict__ target_probs,
    const uint32_t *__restrict__ img, float *__restrict__ agg, int32_t *__restrict__ agg_last,
    float *__restrict__ gathered) {
  __shared__ float red[kAccPreThreads / 64];
  __shared__ int redi[kAccPreThreads / 64];
  const int row = blockIdx.x, y = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float *p = target_probs + (size_t)row * Vt;
  if (y >= kAccWaves) {
    const int VP = (V + kAccPreGather - 1) / kAccPreGather;
    const int v0 = (y - kAccWaves) * VP, v1 = min(v0 + VP, V);
    for (int v = v0 + tid; v < v1; v += kAccPreThreads) {
      const int x = d2t ? d2t[v] : v;
      gathered[(size_t)row * V + v] = (x >= 0 && x < Vt) ? p[x] : 0.f;
    }
    return;
  }
  const int CW = acc_chunk_width(Vt, W);
  const int c0 = min(y * CW, Vt), c1 = min(c0 + CW, Vt);
  float zs = 0.f, cn = 0.f;
  int last = -1;
  for (int x0 = c0 + tid * W; x0 < c1; x0 += kAccPreThreads * W) {
    float a[W];
    if constexpr (W == 4) {
      const f32x4 q = *reinterpret_cast<const f32x4 *>(p + x0);  // W | CW, rows 16-byte aligned
      a[0] = q.x; a[1] = q.y; a[2] = q.z; a[3] = q.w;
    } else {
      a[0] = p[x0];
    }
#pragma unroll
    for (int q = 0; q < W; ++q) {
      const int x = x0 + q;
      if (x >= c1) continue;
      zs += a[q];
      if (!((img[x >> 5] >> (x & 31)) & 1u)) {
        cn += a[q];
        if (a[q] > 0.f) last = x;
      }
    }
  }
  zs = group_sum<64>(zs);
  cn = group_sum<64>(cn);
  last = (int)group_max<64>((float)last);
  if (lane == 0) {
    red[wave] = zs;
    redi[wave] = last;
  }
  __syncthreads();
  if (tid == 0) {
    float z = 0.f;
    int l = -1;
    for (int w = 0; w < kAccPreThreads / 64; ++w) {
      z += red[w];
      l = max(l, redi[w]);
    }
    agg[((size_t)row * kAccWaves + y) * 2] = z;
    agg_last[(size_t)row * kAccWaves + y] = l;
  }
  __syncthreads();
  if (lane == 0) red[wave] = cn;
  __syncthreads();
  if (tid == 0) {
    float c = 0.f;
    for (int w = 0; w < kAccPreThreads / 64; ++w) c += red[w];
    agg[((size_t)row * kAccWaves + y) * 2 + 1] = c;
  }
}

// VEC: target rows read four ids per lane (Vt % 4 == 0, 16-byte aligned rows).
// agg / agg_last / gathered (k_accept_rows, or null): the nodes' rows reduced
// beforehand; the walk then reads them instead of the target rows.
template <bool VEC>
__global__ __launch_bounds__(kAccThreads) void k_accept_sample(
    int N, int k, int V, int Vt, const int32_t *__restrict__ tokens,
    const int32_t *__restrict__ retrieve, const int32_t *__restrict__ topk_draft,
    const float *__restrict__ draft_logits, float inv_temp,
    Draws draft_draws, const int32_t *__restrict__ d2t,
    const float *__restrict__ target_probs, const float *__restrict__ uniforms,
    const uint32_t *__restrict__ img, int32_t *accept_len, int32_t *accept_path,
    int32_t *accepted, const float *__restrict__ agg, const int32_t *__restrict__ agg_last,
    const float *__restrict__ gathered) {
  constexpr int W = VEC ? 4 : 1;  // target ids per lane per load
  __shared__ float s_rd[kAccMaxV];
  __shared__ uint32_t s_img[kAccMaxVt / 32];
  __shared__ float red[kAccWaves];
  __shared__ int s_path[kMaxLayers + 1];
  __shared__ int s_cd[kMaxTopk], s_ord[kMaxTopk];
  __shared__ float s_cn[kAccWaves];
  __shared__ float s_zc[kMaxTopk], s_key[kMaxTopk], s_uc[kMaxTopk];
  __shared__ int s_pick;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = 1 + N * k, NU = N * k + 1, NL = N * (k - 1) + 1;
  const int32_t *tok = tokens + (size_t)b * T;
  const float *u = uniforms + (size_t)b * NU;
  auto tgt = [&](int v) { return d2t ? d2t[v] : v; };
  auto in_img = [&](int x) { return (s_img[x >> 5] >> (x & 31)) & 1u; };
  constexpr int kZ = (kAccMaxV + kAccThreads - 1) / kAccThreads;  // draft ids per thread
  // bitmask of the target ids that draft ids map to (k_build_img)
  {
    constexpr int kW = kAccMaxVt / 32 / kAccThreads;
    const int nw = (Vt + 31) / 32;
    uint32_t m[kW];
#pragma unroll
    for (int j = 0; j < kW; ++j) {
      const int w = tid + j * kAccThreads;
      m[j] = w < nw ? img[w] : 0u;
    }
#pragma unroll
    for (int j = 0; j < kW; ++j) {
      const int w = tid + j * kAccThreads;
      if (w < nw) s_img[w] = m[j];
    }
  }
  __syncthreads();
  // this wave's contiguous chunk of target ids
  const int CW = acc_chunk_width(Vt, W);
  const int c0 = min(wave * CW, Vt), c1 = min(c0 + CW, Vt);
  int node = 0, len = 0, t = 0;
  float Z = 0.f;
  int lastn = -1;  // last unmapped id with mass in this lane's share of the chunk
  const float *p = target_probs + (size_t)b * T * Vt;
  // loads W consecutive target ids at x of row p (zeros past the chunk)
  auto loadp = [&](int x, float *a) {
    if constexpr (VEC) {
      f32x4 q = {0.f, 0.f, 0.f, 0.f};
      if (x < c1) q = *reinterpret_cast<const f32x4 *>(p + x);
      a[0] = q.x; a[1] = q.y; a[2] = q.z; a[3] = q.w;
    } else {
      a[0] = x < c1 ? p[x] : 0.f;
    }
  };
  if (tid == 0) s_path[0] = 0;
  for (;;) {
    p = target_probs + ((size_t)b * T + node) * Vt;
    // the draft ids of the next level's children, fetched early (lane j)
    const int lvl = len + 1;
    const size_t lrow = (size_t)b * N + (lvl - 1);
    const int cdv = (tid < k && lvl <= N) ? topk_draft[lrow * k + tid] : 0;
    float zs = 0.f, cn = 0.f;
    lastn = -1;
    constexpr int NB = kAccBatch / W;
    if (agg) {  // reduced beforehand: chunk sums (summed in chunk order) and rd
      const size_t r = (size_t)b * T + node;
      float z = 0.f;
      for (int w = 0; w < kAccWaves; ++w) z += agg[(r * kAccWaves + w) * 2];
      if (lane == 0) s_cn[wave] = agg[(r * kAccWaves + wave) * 2 + 1];
      lastn = agg_last[r * kAccWaves + wave];
      for (int v = tid; v < V; v += kAccThreads) s_rd[v] = gathered[r * V + v];
      __syncthreads();
      Z = z;
    }
#pragma unroll 1
    for (int e = c0; e < c1 && !agg; e += 64 * W * NB) {
      float a[NB][W];
#pragma unroll
      for (int j = 0; j < NB; ++j) loadp(e + 64 * W * j + W * lane, a[j]);
#pragma unroll
      for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int q = 0; q < W; ++q) {
          const int x = e + 64 * W * j + W * lane + q;
          zs += a[j][q];
          if (x < c1 && !in_img(x)) {
            cn += a[j][q];
            if (a[j][q] > 0.f) lastn = x;
          }
        }
    }
    if (!agg) {
    cn = group_sum<64>(cn);
    if (lane == 0) s_cn[wave] = cn;  // read after the barriers below
    }
    // rd = p at the mapped ids: the map, then the values, half the ids at a time
#pragma unroll 1
    for (int h = 0; h < kZ && !agg; h += kZ / 2) {
      int xs[kZ / 2];
      float g[kZ / 2];
#pragma unroll
      for (int j = 0; j < kZ / 2; ++j) {
        const int v = tid + (h + j) * kAccThreads;
        const int x = v < V ? tgt(v) : -1;
        xs[j] = (x >= 0 && x < Vt) ? x : -1;
      }
#pragma unroll
      for (int j = 0; j < kZ / 2; ++j) g[j] = xs[j] >= 0 ? p[xs[j]] : 0.f;
#pragma unroll
      for (int j = 0; j < kZ / 2; ++j) {
        const int v = tid + (h + j) * kAccThreads;
        if (v < V) s_rd[v] = g[j];
      }
    }
    if (!agg) Z = acc_sum(zs, red);  // its barriers also publish s_rd
    const bool has_children = lvl <= N && (node == 0 || node == 1 + (lvl - 2) * k);
    if (!has_children) break;
    const float *z = draft_logits + lrow * V;
    // the children: draft ids, tempered logits, keys and the uniforms of the
    // tests this level can make (lane j), then their test order (thread 0);
    // their loads go out with this thread's tempered logits of the level
    const int cd = min(max(cdv, 0), V - 1);
    float zc = 0.f, ud = 0.5f, uj = 0.f;
    if (tid < k) {
      zc = z[cd];
      if (draft_draws.on()) ud = draft_draws.at((uint64_t)lrow * V + cd);
      uj = u[t + tid];
    }
    float zr[kZ];
#pragma unroll
    for (int j = 0; j < kZ; ++j) {
      const int v = tid + j * kAccThreads;
      zr[j] = v < V ? z[v] * inv_temp : -INFINITY;
    }
    if (tid < k) {
      zc *= inv_temp;
      s_cd[tid] = cd;
      s_zc[tid] = zc;
      s_key[tid] = draft_draws.on() ? zc - logf(-logf(ud)) : -(float)tid;
      s_uc[tid] = uj;
    }
    __syncthreads();
    if (tid == 0) {
      for (int j = 0; j < k; ++j) s_ord[j] = j;
      for (int i = 1; i < k; ++i)
        for (int j = i; j > 0; --j) {
          const int a = s_ord[j - 1], c = s_ord[j];
          const bool swap = s_key[c] > s_key[a] || (s_key[c] == s_key[a] && s_cd[c] < s_cd[a]);
          if (!swap) break;
          s_ord[j - 1] = c;
          s_ord[j] = a;
        }
    }
    // q = softmax(z / T) over the draft vocabulary: zr becomes exp(z/T - mx)
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < kZ; ++j) mx = fmaxf(mx, zr[j]);
    mx = acc_max(mx, red);  // its barriers also publish s_ord
    float se = 0.f;
#pragma unroll
    for (int j = 0; j < kZ; ++j) {
      zr[j] = expf(zr[j] - mx);  // 0 past V
      se += zr[j];
    }
    const float S = acc_sum(se, red);
    float R = 0.f;  // q mass of the rejected children
    bool took = false;
    for (int j = 0; j < k; ++j) {
      const int rho = s_ord[j];
      const int child = 1 + (lvl - 1) * k + rho;
      const int vd = s_cd[rho];
      const float q0v = expf(s_zc[rho] - mx) / S;
      const float qi = draft_draws.on() ? q0v / (1.f - R) : 1.f;
      const float rx = s_rd[vd];
      const float ut = s_uc[j];
      ++t;
      __syncthreads();  // every thread has read rd(x) before it changes
      if (ut * qi <= rx / Z) {
        node = child;
        ++len;
        if (tid == 0) s_path[len] = child;
        took = true;
        break;
      }
      if (!draft_draws.on()) {  // point mass on x: x leaves p
        if (tid == 0) s_rd[vd] = 0.f;
        Z -= rx;
        __syncthreads();
        continue;
      }
      // rd <- (rd - Z q_i)^+.  A rejected x had r(x) / Z < q_i(x), so its rd
      // is now 0 and stays 0 in later passes: leaving x out of q changes
      // nothing further but the renormalisation 1 / (1 - R).
      const float scale = Z / (1.f - R);
      float dec = 0.f;
#pragma unroll
      for (int jj = 0; jj < kZ; ++jj) {
        const int v = tid + jj * kAccThreads;
        if (v >= V) continue;
        const float old = s_rd[v];
        const float nr = fmaxf(old - scale * (zr[jj] / S), 0.f);
        s_rd[v] = nr;
        dec += old - nr;
      }
      Z -= acc_sum(dec, red);
      R += q0v;
    }
    if (!took) break;
  }
  // one token from the current p: mapped ids in draft-id order, then the rest;
  // chunk sums added in order (the same float expression for a chunk's end
  // and the next chunk's start), the owning wave walks its chunk
  const int CV = ((V + kAccWaves - 1) / kAccWaves + 63) / 64 * 64;
  const int d0 = min(wave * CV, V), d1 = min(d0 + CV, V);
  float ci = 0.f;
  int lasti = -1;
  for (int v = d0 + lane; v < d1; v += 64) {
    ci += s_rd[v];
    if (s_rd[v] > 0.f) lasti = v;
  }
  ci = group_sum<64>(ci);
  __syncthreads();
  if (lane == 0) red[wave] = ci;
  if (tid == 0) s_pick = -1;
  __syncthreads();
  const float target = u[NU - 1] * Z;
  float Mimg = 0.f, wi = 0.f, wn = 0.f;
  for (int w = 0; w < kAccWaves; ++w) {
    if (w == wave) wi = Mimg;
    Mimg += red[w];
  }
  if (target < Mimg) {
    if (wi <= target && target < wi + red[wave]) {
      const int e = acc_walk<1>(d0, d1, wi, target, [&](int v, float *a) {
        a[0] = v < d1 ? s_rd[v] : 0.f;
      });
      if (lane == 0) s_pick = tgt(e >= 0 ? e : d1 - 1);
    }
  } else {
    const float t2 = target - Mimg;
    float tn = 0.f;
    for (int w = 0; w < kAccWaves; ++w) {
      if (w == wave) wn = tn;
      tn += s_cn[w];
    }
    if (wn <= t2 && t2 < wn + s_cn[wave]) {
      const int e = acc_walk<W>(c0, c1, wn, t2, [&](int x, float *a) {
        loadp(x, a);
#pragma unroll
        for (int q = 0; q < W; ++q)
          if (x + q >= c1 || in_img(x + q)) a[q] = 0.f;
      });
      const int ln = (int)group_max<64>((float)lastn);
      if (lane == 0) s_pick = e >= 0 ? e : ln;
    }
  }
  const int lo = (int)acc_max((float)lastn, red);   // its barriers publish s_pick
  const int li = (int)acc_max((float)lasti, red);
  int pick = s_pick;
  if (pick < 0) pick = lo >= 0 ? lo : (li >= 0 ? tgt(li) : -1);  // past the total (rounding)
  if (tid <= N) {
    int32_t *acc = accepted + (size_t)b * (N + 1);
    acc[tid] = tid < len ? tok[s_path[tid + 1]] : (tid == len ? pick : -1);
  }
  if (tid == 0) {
    accept_len[b] = len;
    const int32_t *ret = retrieve + (size_t)b * NL * (N + 1);
    int row = -1;
    for (int w = 0; w < NL && row < 0; ++w) {
      bool ok = true;
      for (int i = 0; i <= len; ++i) ok &= ret[(size_t)w * (N + 1) + i] == s_path[i];
      if (ok) row = w;
    }
    accept_path[b] = row;
  }
}

hipError_t accept_img(const int32_t *d2t, int V, int Vt, uint32_t *img, hipStream_t s) {
  if (V > kAccMaxV || Vt > kAccMaxVt) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_build_img, dim3(1), dim3(kAccThreads), 0, s, d2t, V, Vt, img);
  return hipGetLastError();
}

hipError_t accept_sample(int B, int N, int k, int V, int Vt, const int32_t *tokens,
                         const int32_t *retrieve, const int32_t *topk_draft,
                         const float *draft_logits, float inv_temp, Draws draft_draws,
                         const int32_t *d2t, const float *target_probs, const float *uniforms,
                         const uint32_t *img, int32_t *accept_len, int32_t *accept_path,
                         int32_t *accepted, hipStream_t s, AccPre pre) {
  if (B <= 0) return hipSuccess;
  if (k > kMaxTopk || N > kMaxLayers || V > kAccMaxV || Vt > kAccMaxVt) return hipErrorInvalidValue;
  const bool vec = Vt % 4 == 0 && ((uintptr_t)target_probs & 15u) == 0;
  float *agg = nullptr, *gathered = nullptr;
  int32_t *agg_last = nullptr;
  if (pre.p && B <= pre.max_batch) {  // few sequences: reduce every node's row first
    const int T = 1 + N * k;
    agg = pre.p;
    agg_last = (int32_t *)(agg + (size_t)B * T * kAccWaves * 2);
    gathered = (float *)(agg_last + (size_t)B * T * kAccWaves);
    const dim3 grid(B * T, kAccWaves + kAccPreGather);
    if (vec)
      hipLaunchKernelGGL(k_accept_rows<4>, grid, dim3(kAccPreThreads), 0, s, Vt, V, d2t,
                         target_probs, img, agg, agg_last, gathered);
    else
      hipLaunchKernelGGL(k_accept_rows<1>, grid, dim3(kAccPreThreads), 0, s, Vt, V, d2t,
                         target_probs, img, agg, agg_last, gathered);
  }
  if (vec)
    hipLaunchKernelGGL(k_accept_sample<true>, dim3(B), dim3(kAccThreads), 0, s, N, k, V, Vt,
                       tokens, retrieve, topk_draft, draft_logits, inv_temp, draft_draws, d2t,
                       target_probs, uniforms, img, accept_len, accept_path, accepted, agg,
                       agg_last, gathered);
  else
    hipLaunchKernelGGL(k_accept_sample<false>, dim3(B), dim3(kAccThreads), 0, s, N, k, V, Vt,
                       tokens, retrieve, topk_draft, draft_logits, inv_temp, draft_draws, d2t,
                       target_probs, uniforms, img, accept_len, accept_path, accepted, agg,
                       agg_last, gathered);
  return hipGetLastError();
}

__global__ void k_rope_table(float *tab, int npos, int D, double theta) {
  const int half = D / 2;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < npos * half; i += gridDim.x * blockDim.x) {
    const int p = i / half, m = i % half;
    const double ang = (double)p * pow(theta, -2.0 * (double)m / (double)D);
    double sn, cs;
    sincos(ang, &sn, &cs);
    tab[2 * (size_t)i] = (float)cs;
    tab[2 * (size_t)i + 1] = (float)sn;
  }
}

// ---- multi-position prefill under the self context --------------------------
// Prefix rows of each new row m: its sequence's rows of positions 0..p-1, at
// cache rows dst - p .. dst - 1 (pairs for Seqs).  A row whose position or
// cache rows are out of range gets an empty range marked bad (length pmax + 1),
// so its attention output, and everything after it, is NaN.
__global__ void k_prefill_ranges(const int32_t *__restrict__ positions,
                                 const int32_t *__restrict__ dst_rows, int M, long cache_rows,
                                 int pos_limit, int pmax, int32_t *__restrict__ ranges) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= M) return;
  const int p = positions[m], r = dst_rows[m];
  const bool ok = p >= 0 && p < pos_limit && p <= pmax && r - p >= 0 && r < cache_rows;
  ranges[2 * m] = ok ? r - p : 0;
  ranges[2 * m + 1] = ok ? r : pmax + 1;
}

// Row m's key (rotated at positions[m] unless `rotated`) and value into cache
// row dst_rows[m] in the storage type; rows outside [0, cache_rows) are not
// written, positions outside [0, pos_limit) give NaN rows.  One workgroup per
// row, rotate-half pairs (e, e + D/2).
template <typename T>
__global__ __launch_bounds__(256) void k_kv_scatter(const float *__restrict__ knew,
                                                    const float *__restrict__ vnew, int Hkv, int D,
                                                    const int32_t *__restrict__ positions,
                                                    const int32_t *__restrict__ dst_rows,
                                                    long cache_rows, int pos_limit,
                                                    const float *__restrict__ rope, int rotated,
                                                    T *__restrict__ kc, T *__restrict__ vc) {
  const int m = blockIdx.x, kvd = Hkv * D, half = D / 2;
  const long r = dst_rows[m];
  if (r < 0 || r >= cache_rows) return;
  const int p = positions[m];
  const bool bad = p < 0 || p >= pos_limit;
  const float qnan = __int_as_float(0x7fc00000);
  const float *kr = knew + (size_t)m * kvd, *vr = vnew + (size_t)m * kvd;
  for (int i = threadIdx.x; i < Hkv * half; i += blockDim.x) {
    const int h = i / half, e = i % half, o0 = h * D + e, o1 = o0 + half;
    float k0 = kr[o0], k1 = kr[o1];
    if (!rotated && !bad) {
      const float cs = rope[((size_t)p * half + e) * 2], sn = rope[((size_t)p * half + e) * 2 + 1];
      const float a = k0 * cs - k1 * sn, b = k1 * cs + k0 * sn;
      k0 = a;
      k1 = b;
    }
    kc[(size_t)r * kvd + o0] = Elt<T>::from_f(bad ? qnan : k0);
    kc[(size_t)r * kvd + o1] = Elt<T>::from_f(bad ? qnan : k1);
    vc[(size_t)r * kvd + o0] = Elt<T>::from_f(bad ? qnan : vr[o0]);
    vc[(size_t)r * kvd + o1] = Elt<T>::from_f(bad ? qnan : vr[o1]);
  }
}

hipError_t prefill_ranges(const int32_t *positions, const int32_t *dst_rows, int M,
                          long cache_rows, int pos_limit, int pmax, int32_t *ranges, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_prefill_ranges, dim3((M + 255) / 256), dim3(256), 0, s, positions, dst_rows,
                     M, cache_rows, pos_limit, pmax, ranges);
  return hipGetLastError();
}

hipError_t kv_scatter(int dt, const float *knew, const float *vnew, int M, int Hkv, int D,
                      const int32_t *positions, const int32_t *dst_rows, long cache_rows,
                      int pos_limit, const float *rope, int rotated, void *kc, void *vc,
                      hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (dt)
    hipLaunchKernelGGL((k_kv_scatter<bf16_t>), dim3(M), dim3(256), 0, s, knew, vnew, Hkv, D,
                       positions, dst_rows, cache_rows, pos_limit, rope, rotated, (bf16_t *)kc,
                       (bf16_t *)vc);
  else
    hipLaunchKernelGGL((k_kv_scatter<float>), dim3(M), dim3(256), 0, s, knew, vnew, Hkv, D,
                       positions, dst_rows, cache_rows, pos_limit, rope, rotated, (float *)kc,
                       (float *)vc);
  return hipGetLastError();
}

__global__ void k_philox_fill(const uint64_t *__restrict__ so, uint64_t first, long n,
                              float *__restrict__ out) {
  const Draws dr{nullptr, so};
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    out[i] = dr.at(first + (uint64_t)i);
}

hipError_t philox_fill(const uint64_t *seed_offset, uint64_t first, long n, float *out,
                       hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const long blocks = (n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096;
  hipLaunchKernelGGL(k_philox_fill, dim3((unsigned)blocks), dim3(256), 0, s, seed_offset, first, n, out);
  return hipGetLastError();
}

hipError_t rope_table(float *tab, int npos, int D, double theta, hipStream_t s) {
  const long n = (long)npos * (D / 2);
  const int grid = (int)((n + 255) / 256 < 2048 ? (n + 255) / 256 : 2048);
  hipLaunchKernelGGL(k_rope_table, dim3(grid), dim3(256), 0, s, tab, npos, D, theta);
  return hipGetLastError();
}

}  // namespace fe
