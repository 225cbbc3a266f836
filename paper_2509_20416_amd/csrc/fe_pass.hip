// fe_pass.hip -- the batch-1 drafting pass as a few persistent launches (gfx950).
//
// At batch 1 every FC of the pass (Eq. 1, the cascade layers of Eq. 2, the
// shared LM head) streams its weight matrix once against one to N activation
// rows: the pass is a chain of weight streams tied together by small data
// dependencies.  Between two attention launches, every stage of that chain
// (O projection, gate/up + SwiGLU, down projection, the next layer's Q/K/V;
// the fusion and input FCs before the first attention; the LM head, its top-k
// merge and the draft tree after the last) runs inside ONE launch of resident
// workgroups, one per compute unit:
//  * Every wave streams its share of the stage's weight rows in 1 KB pieces
//    (64 lanes x 16 bytes of one row) through two register banks of DEP
//    pieces: one bank is in flight while the other is consumed, so up to
//    2 * DEP KB per wave (W waves per compute unit) are on their way from
//    memory.  Every bank slot issues its load, also past the end of the
//    stream (it then re-reads the last piece, and nothing consumes it), so the
//    compiler's own wait counts stay exact.  The issue cursor runs ahead
//    across stage boundaries: the next stage's first weights are in flight
//    while a stage's results are published and the next inputs collected.
//  * A stage's results reach the other workgroups as 64-bit words holding a
//    32-bit payload and the pass's tag (device-scope stores and loads, which
//    bypass the non-coherent L2 of each XCD).  A consumer polls its input
//    words until every tag matches: no barrier, counter or acknowledgement
//    round trip sits between stages.  Each input is written once per pass.
//  * A workgroup owns the same output rows in every stage of the same width,
//    so residuals never leave it, and each row's dot product is summed in a
//    fixed order (deterministic, no atomics on data).
// Every wait is bounded: a poll that gives up sets a status bit and the
// kernel runs on to its normal end.
// On the 8B-, 13B- and 70B-shaped drafters these launches are slower than one
// launch per stage (their one-workgroup-per-CU streaming loop reads the
// weights at about 4 TB/s, the per-stage GEMVs at up to 5.7), so a pass takes
// this path only when the caller selects it (fe_set_pass_mode(h, 0)).
#include <type_traits>

#include "fe_internal.h"
#include "fe_tree.h"

namespace fe {

namespace {

constexpr int kPieceElems = 512;       // bf16 elements per 1 KB piece
constexpr int kSpinLimit = 1 << 17;    // polls before a wait gives up (about 0.1 s)
constexpr int kMaxStat = 2 + 2 * kMaxTopk;  // LM-head words per (row, workgroup)

__device__ __forceinline__ void tag_put(uint64_t *p, uint32_t v, uint32_t tag) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t tag_get(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void set_status(uint32_t *sync, uint32_t bit) {
  __hip_atomic_fetch_or(sync + kSegStatusWord, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float dot8(u32x4 w, u32x4 x, float acc) {
  const uint32_t w0 = w[0], w1 = w[1], w2 = w[2], w3 = w[3];
  const uint32_t x0 = x[0], x1 = x[1], x2 = x[2], x3 = x[3];
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, w0), __builtin_bit_cast(bf16x2_v, x0), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, w1), __builtin_bit_cast(bf16x2_v, x1), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, w2), __builtin_bit_cast(bf16x2_v, x2), acc, false);
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, w3), __builtin_bit_cast(bf16x2_v, x3), acc, false);
}

__device__ __forceinline__ u32x4 ld_piece(const bf16_t *p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}
__device__ __forceinline__ void wg_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Sum over the 64 lanes, in every lane (fixed order: the same bits in every
// workgroup for the same inputs).
__device__ __forceinline__ float wave_sum(float x) { return group_sum<64>(x); }

// The rows of stage s this workgroup owns: [r0, r1), whole granules.
struct Rows {
  int r0, r1;
};
__device__ __forceinline__ Rows rows_of(const SegStage &s, int g, int nwg) {
  const int units = s.C / s.gran;
  return Rows{s.gran * (int)((long)units * g / nwg), s.gran * (int)((long)units * (g + 1) / nwg)};
}
// The pieces of this workgroup's rows a wave streams: [t0, t1) of T = rows *
// ppr, split over the first `act` waves (each gets at least ppr pieces, so a
// row is shared by at most two waves).
struct Range {
  int t0, t1, act;
};
__device__ __forceinline__ Range range_of(int T, int ppr, int W, int w) {
  int act = T / ppr;
  act = act < 1 ? 1 : (act > W ? W : act);
  if (T == 0 || w >= act) return Range{0, 0, act};
  return Range{(int)((long)T * w / act), (int)((long)T * (w + 1) / act), act};
}
// weight row of virtual row r
__device__ __forceinline__ const bf16_t *wrow(const SegStage &s, int r) {
  if (s.kind == kSegGu) return ((r & 1) ? s.w1 : s.w0) + (size_t)(r >> 1) * s.K;
  if (s.kind == kSegQkv) {
    if (r >= s.split2) return s.w2 + (size_t)(r - s.split2) * s.K;
    if (r >= s.split1) return s.w1 + (size_t)(r - s.split1) * s.K;
  }
  return s.w0 + (size_t)r * s.K;
}

template <int W, int DEP, int XB>
struct SegLds {
  // the stage's input rows; after the last stage, the LM-head candidates of
  // every workgroup for the merge
  bf16_t x[XB / 2];
  float red[kSegRedFloats];
  union {  // epilogue values; the next stage's partial sums of squares (not at once)
    float tmp[kSegMaxRows * kSegLmMaxCols];
    uint32_t part[kSegMaxRows][kSegMaxWg];
  };
  float xres[kSegResRows];
  float inv[kSegMaxRows];
  uint64_t key[W][kMaxTopk];
  float stat[2];
  int aborted;  // a wait of this workgroup gave up
};

// Polls `nw` tagged words into dst (their payloads), spread over the
// workgroup's threads; words whose tag is not yet `tag` are read again.  After
// one wait of this workgroup has given up (*aborted), later ones do not wait.
__device__ void poll_words(const uint64_t *src, int nw, uint32_t *dst, uint32_t tag,
                           uint32_t *sync, int *aborted) {
  constexpr int U = 8;
  const int nt = blockDim.x;
  for (int i0 = threadIdx.x; i0 < nw; i0 += U * nt) {
    uint64_t v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * nt;
      v[u] = i < nw ? tag_get(src + i) : ((uint64_t)tag << 32);
    }
    for (int spins = 0;; ++spins) {
      bool ok = true;
#pragma unroll
      for (int u = 0; u < U; ++u) ok = ok && (uint32_t)(v[u] >> 32) == tag;
      if (ok) break;
      if (spins >= kSpinLimit || *aborted) {
        if (!*aborted) set_status(sync, kSegStatusTimeout);
        *aborted = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * nt;
        if (i < nw && (uint32_t)(v[u] >> 32) != tag) v[u] = tag_get(src + i);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + u * nt;
      if (i < nw) dst[i] = (uint32_t)v[u];
    }
  }
}

// The inputs of stage s: its rows (bf16) into lds.x at row m * K, and the
// 1/rms of every normalised row into lds.inv.
template <int W, int DEP, int XB>
__device__ void collect(const SegArgs &a, const SegStage &s, SegLds<W, DEP, XB> &lds,
                        uint32_t tag) {
  const int nt = blockDim.x;
  for (int j = 0; j < s.nsrc; ++j) {
    const SegSrc &src = s.src[j];
    bf16_t *dst = lds.x + (size_t)src.m * s.K + src.e0;
    if (src.kind == kSrcTagged) {
      poll_words((const uint64_t *)src.p, src.n / 2, reinterpret_cast<uint32_t *>(dst), tag,
                 a.sync, &lds.aborted);
    } else {
      const bf16_t *p = (const bf16_t *)src.p;
      bool nan_row = false;
      if (src.kind == kSrcEmbed) {  // row tokens[0] of the table; an id outside it gives NaN
        const int tok = src.tok[0];
        nan_row = tok < 0 || tok >= src.vocab;
        p += (size_t)(nan_row ? 0 : tok) * src.n;
      }
      for (int e = threadIdx.x * 8; e < src.n; e += nt * 8) {
        u32x4 v = *reinterpret_cast<const u32x4 *>(p + e);
        if (nan_row) v = u32x4{0x7fc07fc0u, 0x7fc07fc0u, 0x7fc07fc0u, 0x7fc07fc0u};
        *reinterpret_cast<u32x4 *>(dst + e) = v;
      }
    }
  }
  // 1/rms of the normalised rows: the producers' per-workgroup partial sums
  // of squares, summed in a fixed order (wave m, lane l: partials l, l + 64, ...)
  uint32_t (*s_part)[kSegMaxWg] = lds.part;
  for (int m = 0; m < s.mr; ++m)
    if (s.ssq[m]) poll_words(s.ssq[m], a.nwg, s_part[m], tag, a.sync, &lds.aborted);
  wg_sync();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int m = wave; m < s.mr; m += W) {
    if (!s.ssq[m]) continue;
    float acc = 0.f;
    for (int i = lane; i < a.nwg; i += 64) acc += __uint_as_float(s_part[m][i]);
    acc = wave_sum(acc);
    if (lane == 0) lds.inv[m] = 1.0f / sqrtf(acc / (float)a.d + a.eps);
  }
}

// row-sum of output (m, rl): its first part, plus the second when a wave range
// starts inside the row
template <int W, int DEP, int XB>
__device__ __forceinline__ float row_value(const SegLds<W, DEP, XB> &lds, int RW, int m, int rl,
                                           int T, int ppr, int act) {
  float v = lds.red[(m * RW + rl) * 2];
  for (int w = 1; w < act; ++w) {
    const int tw = (int)((long)T * w / act);
    if (tw % ppr != 0 && tw / ppr == rl) v += lds.red[(m * RW + rl) * 2 + 1];
  }
  return v;
}

// Sum of squares of the fp32 values lds.tmp[0..n) (wave 0, fixed order),
// published as this workgroup's partial.
template <int W, int DEP, int XB>
__device__ void publish_ssq(const SegArgs &a, SegLds<W, DEP, XB> &lds, int n, uint64_t *dst,
                            uint32_t tag) {
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  float acc = 0.f;
  for (int i = lane; i < n; i += 64) acc += lds.tmp[i] * lds.tmp[i];
  acc = wave_sum(acc);
  if (lane == 0) tag_put(dst + blockIdx.x, __float_as_uint(acc), tag);
}

// gamma_q * x of this workgroup's rows [r0, r0 + n) (x in lds.tmp) as bf16 pairs
template <int W, int DEP, int XB>
__device__ void publish_copies(const SegStage &s, SegLds<W, DEP, XB> &lds, int r0, int n,
                               uint32_t tag) {
  for (int idx = threadIdx.x; idx < s.ncopy * (n / 2); idx += blockDim.x) {
    const int q = idx / (n / 2), pr = idx % (n / 2), rl = 2 * pr, r = r0 + rl;
    const bf16_t *gm = s.gamma[q];
    const float v0 = bf2f(gm[r]) * lds.tmp[rl], v1 = bf2f(gm[r + 1]) * lds.tmp[rl + 1];
    tag_put(s.copy_t[q] + r / 2, f2bf2(v0, v1), tag);
  }
}

// What stage s produces, from the row sums in lds.red.
template <int W, int DEP, int XB>
__device__ void epilogue(const SegArgs &a, const SegStage &s, SegLds<W, DEP, XB> &lds,
                         uint32_t tag) {
  const int g = blockIdx.x, nt = blockDim.x, tid = threadIdx.x;
  const Rows rw = rows_of(s, g, a.nwg);
  const int RW = rw.r1 - rw.r0, ppr = s.K / kPieceElems, T = RW * ppr;
  const int act = range_of(T, ppr, W, 0).act;
  auto val = [&](int m, int rl) { return row_value(lds, RW, m, rl, T, ppr, act); };
  switch (s.kind) {
    case kSegFuse:  // g_t, bf16 pairs
      for (int pr = tid; pr < RW / 2; pr += nt)
        tag_put(s.out_t + (rw.r0 / 2 + pr), f2bf2(val(0, 2 * pr), val(0, 2 * pr + 1)), tag);
      break;
    case kSegInput:
    case kSegO:
    case kSegDown: {
      // x_0 = FC(..) (Eq. 1); x' = x_{i-1} + W_o o; x_i = x' + W_d s (Eq. 2)
      for (int rl = tid; rl < RW; rl += nt) {
        float x = val(0, rl);
        if (s.kind == kSegO) x += s.resid[rw.r0 + rl];
        if (s.kind == kSegDown) x += lds.xres[rl];
        if (s.kind == kSegO) lds.xres[rl] = x;
        if (s.x_out) s.x_out[rw.r0 + rl] = x;
        lds.tmp[rl] = x;
      }
      wg_sync();
      publish_ssq(a, lds, RW, s.ssq_out, tag);
      publish_copies(s, lds, rw.r0, RW, tag);
      break;
    }
    case kSegQkv: {
      const int kvd = s.split2 - s.split1;
      for (int idx = tid; idx < s.mr * RW; idx += nt) {
        const int m = idx / RW, rl = idx % RW, r = rw.r0 + rl;
        const float v = val(m, rl) * lds.inv[m];
        if (r < s.split1) {
          if (m == s.qrow) s.x_out[r] = v;
        } else if (r < s.split2) {
          s.k_out[(size_t)m * kvd + r - s.split1] = v;
        } else {
          s.v_out[(size_t)m * kvd + r - s.split2] = v;
        }
      }
      break;
    }
    case kSegGu: {  // rows (gate c, up c, gate c+1, up c+1) -> s[c], s[c+1]
      const float inv = lds.inv[0];
      for (int qd = tid; qd < RW / 4; qd += nt) {
        const int rl = 4 * qd;
        const float g0 = val(0, rl) * inv, u0 = val(0, rl + 1) * inv;
        const float g1 = val(0, rl + 2) * inv, u1 = val(0, rl + 3) * inv;
        const float s0 = g0 / (1.f + expf(-g0)) * u0, s1 = g1 / (1.f + expf(-g1)) * u1;
        tag_put(s.out_t + (rw.r0 + rl) / 4, f2bf2(s0, s1), tag);
      }
      break;
    }
    case kSegLm: {
      // z = W_lm RMSNorm(h_i): per row, this workgroup's max, sum of exp(z - max)
      // and its top-k by (z desc, id asc), one wave per row
      for (int idx = tid; idx < s.mr * RW; idx += nt) {
        const int m = idx / RW, rl = idx % RW;
        const float z = val(m, rl) * lds.inv[m];
        lds.tmp[idx] = z;
        if (a.logits) a.logits[(size_t)m * a.V + rw.r0 + rl] = z;
      }
      wg_sync();
      const int wave = tid >> 6, lane = tid & 63;
      for (int m = wave; m < s.mr; m += W) {
        float mx = -INFINITY;
        for (int rl = lane; rl < RW; rl += 64) mx = fmaxf(mx, lds.tmp[m * RW + rl]);
        mx = group_max<64>(mx);
        float se = 0.f;
        for (int rl = lane; rl < RW; rl += 64) se += expf(lds.tmp[m * RW + rl] - mx);
        se = wave_sum(se);
        uint64_t *dst = s.out_t + ((size_t)m * a.nwg + g) * kMaxStat;
        if (lane == 0) {
          tag_put(dst, __float_as_uint(mx), tag);
          tag_put(dst + 1, __float_as_uint(se), tag);
        }
        constexpr int C = kSegLmMaxCols / 64;
        uint64_t key[C];
#pragma unroll
        for (int c = 0; c < C; ++c) {
          const int rl = lane + 64 * c;
          key[c] = rl < RW ? topk_key(lds.tmp[m * RW + rl], rw.r0 + rl) : kNoKey;
        }
        for (int r = 0; r < a.topk; ++r) {
          uint64_t best = kNoKey;
#pragma unroll
          for (int c = 0; c < C; ++c) best = key[c] > best ? key[c] : best;
          best = wave_max_u64(best);
#pragma unroll
          for (int c = 0; c < C; ++c) key[c] = key[c] == best ? kNoKey : key[c];
          if (lane == 0) {
            tag_put(dst + 2 + 2 * r, (uint32_t)(best >> 32), tag);
            tag_put(dst + 3 + 2 * r, (uint32_t)best, tag);
          }
        }
        // the merge reads every slot: the ranks past k hold no key
        for (int r = a.topk + lane; r < kMaxTopk; r += 64) {
          tag_put(dst + 2 + 2 * r, (uint32_t)(kNoKey >> 32), tag);
          tag_put(dst + 3 + 2 * r, (uint32_t)kNoKey, tag);
        }
      }
      break;
    }
    default:
      break;
  }
}

// Global top-k of LM-head row m from every workgroup's candidates, softmax
// statistics, vocabulary map and (row 0) the tree structure: what the
// multi-launch pass's top-k merge computes, for batch 1.
template <int W, int DEP, int XB>
__device__ void merge_row(const SegArgs &a, SegLds<W, DEP, XB> &lds, int m, uint32_t tag) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int k = a.topk, nwg = a.nwg, nw = nwg * kMaxStat;
  static_assert(XB >= kSegMaxWg * kMaxStat * 4, "candidate words fit the input rows' space");
  uint32_t *buf = reinterpret_cast<uint32_t *>(lds.x);  // no stage reads its inputs any more
  poll_words(a.cand_t + (size_t)m * nw, nw, buf, tag, a.sync, &lds.aborted);
  const TreeRows &tr = a.tree;
  if (tr.tokens && m == 0) {
    if (tid == 0) tr.tokens[0] = tr.root[0];
    tree_structure(0, tr.N, k, tr.cu_prefix[1] - tr.cu_prefix[0], tr.parents, tr.depth,
                   tr.positions, tr.mask, tr.retrieve);
  }
  wg_sync();
  // statistics: mu = max_g m_g, S = sum_g s_g exp(m_g - mu) (wave 0, fixed order)
  if (wave == 0) {
    float mu = -INFINITY;
    for (int i = lane; i < nwg; i += 64) mu = fmaxf(mu, __uint_as_float(buf[i * kMaxStat]));
    mu = group_max<64>(mu);
    float S = 0.f;
    for (int i = lane; i < nwg; i += 64)
      S += __uint_as_float(buf[i * kMaxStat + 1]) * expf(__uint_as_float(buf[i * kMaxStat]) - mu);
    S = wave_sum(S);
    if (lane == 0) {
      lds.stat[0] = mu;
      lds.stat[1] = S;
    }
  }
  // per-wave top-k over the candidates (thread t: candidates t, t + nt, ...)
  const int ncand = nwg * k;
  constexpr int CAP = kSegMaxWg * kMaxTopk / (64 * W) + 1;
  uint64_t key[CAP];
#pragma unroll
  for (int j = 0; j < CAP; ++j) {
    const int c = tid + j * 64 * W;
    key[j] = kNoKey;
    if (c < ncand) {
      const uint32_t *w = buf + (c / k) * kMaxStat + 2 + 2 * (c % k);
      key[j] = ((uint64_t)w[0] << 32) | w[1];
    }
  }
  for (int r = 0; r < k; ++r) {
    uint64_t best = kNoKey;
#pragma unroll
    for (int j = 0; j < CAP; ++j) best = key[j] > best ? key[j] : best;
    best = wave_max_u64(best);
#pragma unroll
    for (int j = 0; j < CAP; ++j) key[j] = key[j] == best ? kNoKey : key[j];
    if (lane == 0) lds.key[wave][r] = best;
  }
  wg_sync();
  if (wave == 0) {
    uint64_t mine = kNoKey, kk[(W * kMaxTopk + 63) / 64];
#pragma unroll
    for (int j = 0; j < (W * kMaxTopk + 63) / 64; ++j) {
      const int c = lane + 64 * j;
      kk[j] = c < W * k ? lds.key[c / k][c % k] : kNoKey;
    }
    for (int r = 0; r < k; ++r) {
      uint64_t best = kNoKey;
#pragma unroll
      for (int j = 0; j < (W * kMaxTopk + 63) / 64; ++j) best = kk[j] > best ? kk[j] : best;
      best = wave_max_u64(best);
#pragma unroll
      for (int j = 0; j < (W * kMaxTopk + 63) / 64; ++j) kk[j] = kk[j] == best ? kNoKey : kk[j];
      if (lane == r) mine = best;
    }
    const int i = topk_key_id(mine);
    const bool valid = lane < k && mine != kNoKey && i >= 0 && i < a.V;  // none left: -1
    if (lane < k) {
      const size_t o = (size_t)m * k + lane;
      const int32_t id = valid ? (a.d2t ? a.d2t[i] : i) : -1;
      a.ids[o] = id;
      if (tr.tokens) tr.tokens[1 + m * k + lane] = id;
      if (a.draft_ids) a.draft_ids[o] = valid ? i : -1;
      a.probs[o] = valid ? expf(topk_key_value(mine) - lds.stat[0]) / lds.stat[1]
                         : __int_as_float(0x7fc00000);
    }
  }
}

template <int W, int DEP, int XB>
__global__ __launch_bounds__(64 * W) void k_seg(SegArgs args) {
  // The arguments are read in place from the kernel-argument segment (constant
  // memory, scalar loads): indexing a copy of them by the run-time stage
  // number would put that copy in per-lane scratch memory.
  (void)args;
  const SegArgs &a = *(const SegArgs *)__builtin_amdgcn_kernarg_segment_ptr();
  __shared__ __align__(16) SegLds<W, DEP, XB> lds;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, g = blockIdx.x;
  const int sw = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t tag =
      __hip_atomic_load(a.sync + kSegEpochWord, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u;
  if (threadIdx.x == 0) lds.aborted = 0;
  wg_sync();
  const int nst = a.nst;

  // ---- issue cursor: a bank never spans two stages ----
  // The wave's pieces of a stage are [it, iend) of the row-major piece list of
  // its rows.  Within one weight matrix consecutive pieces are 1 KB apart, so
  // the cursor walks runs of contiguous pieces with one add per piece and only
  // maps a piece back to its row where a run ends (a gate/up row pair, a
  // Q/K/V matrix boundary).
  int ist = 0, it = 0, iend = 0, irun = 0, ippr = 1, ir0 = 0;
  const char *iptr = reinterpret_cast<const char *>(a.st[0].w0);
  const char *ilast = iptr;  // last piece issued (first row of stage 0 before any)
  auto run_init = [&]() {
    const SegStage &s = a.st[ist];
    const int r = ir0 + it / ippr;
    iptr = reinterpret_cast<const char *>(wrow(s, r)) + (size_t)(it % ippr) * (kPieceElems * 2);
    int rend = s.C;  // first row past this matrix-contiguous run
    if (s.kind == kSegGu) rend = r + 1;
    else if (s.kind == kSegQkv) rend = r < s.split1 ? s.split1 : (r < s.split2 ? s.split2 : s.C);
    irun = min(iend, (rend - ir0) * ippr);
  };
  auto issue_stage_init = [&]() {
    while (ist < nst) {
      const SegStage &s = a.st[ist];
      const Rows rw = rows_of(s, g, a.nwg);
      ir0 = rw.r0;
      ippr = s.K / kPieceElems;
      const Range q = range_of((rw.r1 - rw.r0) * ippr, ippr, W, sw);
      it = q.t0;
      iend = q.t1;
      if (it < iend) {
        run_init();
        return;
      }
      ++ist;
    }
  };
  issue_stage_init();
  // Fills a bank with the next pieces of the current stage (at most DEP);
  // returns how many slots hold pieces.  Every slot issues a load.
  auto issue_bank = [&](u32x4(&bank)[DEP]) -> int {
    int n = 0;
    const bool live = ist < nst;
#pragma unroll
    for (int i = 0; i < DEP; ++i) {
      if (live && it < iend) {
        ilast = iptr;
        iptr += kPieceElems * 2;
        ++n;
        if (++it == irun && it < iend) run_init();
      }
      bank[i] = ld_piece(reinterpret_cast<const bf16_t *>(ilast) + lane * 8);
    }
    if (live && it >= iend) {
      ++ist;
      issue_stage_init();
    }
    return n;
  };
  u32x4 b0[DEP], b1[DEP];
  int n0 = issue_bank(b0);
  int n1 = issue_bank(b1);

  // ---- consume cursor ----
  int cst = 0, ct = 0, cend = 0, crow = 0, cp = 0, cppr = 1, cK = 0, cmr = 1, frow = 0, RW = 0;
  bool fsplit = false;
  auto consume_stage_init = [&]() {
    const SegStage &s = a.st[cst];
    const Rows rw = rows_of(s, g, a.nwg);
    RW = rw.r1 - rw.r0;
    cppr = s.K / kPieceElems;
    cK = s.K;
    cmr = s.mr;
    const Range q = range_of(RW * cppr, cppr, W, sw);
    ct = q.t0;
    cend = q.t1;
    crow = q.t0 / cppr;
    cp = q.t0 % cppr;
    frow = crow;
    fsplit = cp != 0;
  };
  collect(a, a.st[0], lds, tag);
  wg_sync();
  consume_stage_init();
  // Runs the stage ends this wave has reached (epilogue, next inputs); false
  // once every stage is done.
  auto ready = [&]() -> bool {
    while (ct >= cend) {
      wg_sync();
      epilogue(a, a.st[cst], lds, tag);
      wg_sync();
      if (++cst >= nst) return false;
      collect(a, a.st[cst], lds, tag);
      wg_sync();
      consume_stage_init();
    }
    return true;
  };
  float acc[kSegMaxRows];
#pragma unroll
  for (int m = 0; m < kSegMaxRows; ++m) acc[m] = 0.f;
  // The n pieces of a bank (all of stage cst) into the row sums; MR rows at
  // compile time (1: the single-row stages), else cmr <= kSegMaxRows.
  auto consume_rows = [&](const u32x4(&bank)[DEP], int n, auto mr_tag) {
    constexpr int MR = decltype(mr_tag)::value;
    const int mr = MR == 1 ? 1 : cmr;
    const bf16_t *xl = lds.x + lane * 8;
#pragma unroll
    for (int i = 0; i < DEP; ++i) {
      if (i < n) {
        const bf16_t *xp = xl + cp * kPieceElems;
#pragma unroll
        for (int m = 0; m < MR; ++m)
          if (MR == 1 || m < mr)
            acc[m] = dot8(bank[i], *reinterpret_cast<const u32x4 *>(xp + (size_t)m * cK), acc[m]);
        ++ct;
        const bool row_end = ++cp == cppr;
        if (row_end || ct == cend) {
          const int slot = (crow == frow && fsplit) ? 1 : 0;
#pragma unroll
          for (int m = 0; m < MR; ++m) {
            if (MR == 1 || m < mr) {
              const float v = wave_sum(acc[m]);
              if (lane == 0) lds.red[(m * RW + crow) * 2 + slot] = v;
            }
            acc[m] = 0.f;
          }
          if (row_end) {
            cp = 0;
            ++crow;
          }
        }
      } else {
        // a slot past the stream: its load is waited for here, so that no
        // path reaches the bank's refill with a load still pending on its
        // registers (the compiler would otherwise wait before every refill
        // load, draining the other bank)
        asm volatile("" ::"v"(bank[i]));
      }
    }
  };
  auto consume = [&](const u32x4(&bank)[DEP], int n) {
    if (cmr == 1) consume_rows(bank, n, std::integral_constant<int, 1>{});
    else consume_rows(bank, n, std::integral_constant<int, kSegMaxRows>{});
  };
  // banks alternate: b0, b1, b0, ...; each is refilled as soon as it is consumed
  for (;;) {
    if (!ready()) break;
    consume(b0, n0);
    n0 = issue_bank(b0);
    if (!ready()) break;
    consume(b1, n1);
    n1 = issue_bank(b1);
  }

  if (a.last) {
    // the LM head's rows: row m merged by workgroup m
    wg_sync();
    const int mr = a.st[nst - 1].mr;
    for (int m = g; m < mr; m += a.nwg) merge_row(a, lds, m, tag);
    // every workgroup has finished: the last one advances the pass tag
    wg_sync();
    if (threadIdx.x == 0) {
      const uint32_t old = __hip_atomic_fetch_add(a.sync + kSegDepartWord, 1u, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
      if (old == (uint32_t)a.nwg - 1) {
        __hip_atomic_store(a.sync + kSegDepartWord, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(a.sync + kSegEpochWord, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
}

// zero fill (the tagged words before their first pass)
__global__ void k_zero_words(uint64_t *p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

}  // namespace

// Workgroup shapes by the activation bytes a stage holds in LDS.
int seg_variant(int xbytes) {
  if (xbytes <= 40960) return 0;
  if (xbytes <= 65536) return 1;
  if (xbytes <= 81920) return 2;
  return -1;
}

// (waves, bank depth, activation bytes) per variant
#ifndef FE_SEG_VARIANTS
#define FE_SEG_VARIANTS(X) X(0, 16, 4, 40960) X(1, 16, 4, 65536) X(2, 16, 4, 81920)
#endif

hipError_t seg_occupancy(int variant, int *blocks_per_cu) {
#define FE_SEG_OCC(V, W, DEP, XB) \
  if (variant == V) return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, k_seg<W, DEP, XB>, W * 64, 0);
  FE_SEG_VARIANTS(FE_SEG_OCC)
#undef FE_SEG_OCC
  return hipErrorInvalidValue;
}

hipError_t seg_launch(int variant, const SegArgs &a, hipStream_t s) {
#define FE_SEG_LAUNCH(V, W, DEP, XB)                                               \
  if (variant == V) {                                                             \
    hipLaunchKernelGGL((k_seg<W, DEP, XB>), dim3(a.nwg), dim3(W * 64), 0, s, a);  \
    return hipGetLastError();                                                     \
  }
  FE_SEG_VARIANTS(FE_SEG_LAUNCH)
#undef FE_SEG_LAUNCH
  return hipErrorInvalidValue;
}

hipError_t seg_zero(uint64_t *words, size_t n, hipStream_t s) {
  hipLaunchKernelGGL(k_zero_words, dim3(256), dim3(256), 0, s, words, n);
  return hipGetLastError();
}

}  // namespace fe
