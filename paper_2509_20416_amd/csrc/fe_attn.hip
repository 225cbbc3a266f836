// fe_attn.hip -- GQA decode attention of a cascade layer over its prefix KV
// cache plus the cascade entries, in one launch (gfx950).
//
// Layer i's query (one row per sequence, H_q heads) attends to the P_b cached
// prefix keys of its own cache and to the nctx keys it projected from the
// cascade states (Section 2.1; the cache is per layer because every L_i has
// its own parameters).
//
//  * fp32 caches (k_attn): one workgroup (4 waves) per (sequence, KV head,
//    head group, span of chunks of kAttnChunk prefix keys), heads fastest in
//    the grid; the GH query heads sharing a KV head are done together so every
//    K/V byte is read once.  A key row is split in 16-byte pieces over
//    RL = D*sizeof(T)/16 lanes, so one load instruction covers 64/RL whole
//    rows; K and V are loaded together.  A score is reduced over its RL lanes
//    with DPP row operations and leaves every lane of the row with the same
//    value, which is exactly what the value pass needs: each lane accumulates
//    p*V for its own dims and key rows, so the value sums need no cross-lane
//    traffic.  Row-group maxima use gfx950's permlane swaps.  The
//    per-(wave, row group) sums meet in LDS.  Chunk 0 also takes the nctx
//    cascade keys (fp32, one extra load per lane).
//  * bf16 caches (k_attn_mma): one-wave workgroups on the matrix cores with a
//    direct-to-LDS ring; see the comment above that kernel.
//  * A span that is not the whole sequence leaves o[D] (scaled to its max)
//    and (max, sum) per head in the workspace, and a second launch
//    (k_attn_merge) combines them in a fixed order: no atomics, no fences, the
//    result does not depend on scheduling.  A sequence with an empty prefix
//    still runs chunk 0 for its cascade keys.
#include "fe_attn_unit.h"

namespace fe {

constexpr int kWaveKeys = kAttnChunk / 4;   // keys per wave

__device__ __forceinline__ float scaled_exp(float m, float M) {
  return m == -INFINITY ? 0.f : expf(m - M);
}

// element e of a 16-byte piece holding 16/sizeof(T) values
template <typename T> __device__ __forceinline__ float piece_at(const u32x4 &w, int e) {
  const uint32_t u = (e >> (sizeof(T) == 2 ? 1 : 0)) == 0   ? w.x
                     : (e >> (sizeof(T) == 2 ? 1 : 0)) == 1 ? w.y
                     : (e >> (sizeof(T) == 2 ? 1 : 0)) == 2 ? w.z
                                                            : w.w;
  if constexpr (sizeof(T) == 2) return (e & 1) ? __uint_as_float(u & 0xffff0000u) : __uint_as_float(u << 16);
  else return __uint_as_float(u);
}

template <typename T, int D, int GH>
__global__ __launch_bounds__(256) void k_attn(const T *__restrict__ Kc, const T *__restrict__ Vc,
                                              Seqs cu,
                                              const float *__restrict__ q,
                                              const float *__restrict__ knew,
                                              const float *__restrict__ vnew, int nctx,
                                              float *__restrict__ part, int nch, int nch_ld,
                                              int cpw,
                                              T *__restrict__ out, int Hq, int Hkv, int pmax) {
  constexpr int RL = D * (int)sizeof(T) / 16;  // lanes per key row
  constexpr int KPL = 64 / RL;                  // key rows per load instruction
  constexpr int DPL = 16 / (int)sizeof(T);      // dims per lane
  constexpr int NLD = kWaveKeys / KPL;          // K (and V) loads per lane per sub-chunk
  constexpr int CW = DPL / 4;                   // fp32 16-byte pieces per lane of a cascade row
  constexpr int NCX = (kMaxLayers + 4 * KPL - 1) / (4 * KPL);  // cascade rows per lane (chunk 0)
  __shared__ float s_o[4][KPL][GH][D];
  __shared__ float s_l[4][KPL][GH];
  __shared__ float s_m[4][GH];

  const int G = Hq / Hkv, ngrp = G / GH;
  // heads fastest: the workgroups that run side by side read neighbouring
  // head segments of the same token rows
  const int ch = blockIdx.y, c = blockIdx.x / ngrp, hg = blockIdx.x % ngrp, b = blockIdx.z;
  bool bad;
  const int start = cu.start(b), P = attn_prefix(cu, b, pmax, bad);
  const int span = kAttnChunk * cpw;  // prefix keys per workgroup
  const int nv = max(1, min((P + span - 1) / span, nch));
  if (ch >= nv) return;  // chunk beyond this sequence's prefix
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, kg = lane / RL, dl = lane % RL;
  const int h0 = c * G + hg * GH;
  const float scale = rsqrtf((float)D);
  const int base = ch * span;
  // sub-chunks of kAttnChunk keys this workgroup visits (0 for an empty prefix)
  const int nsc = P > 0 ? min(cpw, (P - base + kAttnChunk - 1) / kAttnChunk) : 0;
  const int lkey = wave * kWaveKeys + kg;  // this lane's first key within a sub-chunk; step KPL
  const bool casc = ch == 0;
  float *part_o = part;
  float *part_ml = part + (size_t)gridDim.z * Hq * nch_ld * D;

  const size_t rs = (size_t)Hkv * D;
  const T *kb = Kc + ((size_t)start * Hkv + c) * D + dl * DPL;
  const T *vb = Vc + ((size_t)start * Hkv + c) * D + dl * DPL;
  // rows of sub-chunk `sc` at clamped in-bounds keys (masked when scored)
  auto load_rows = [&](int sc, u32x4 (&kr)[NLD], u32x4 (&vr)[NLD]) {
#pragma unroll
    for (int t = 0; t < NLD; ++t) {
      const size_t key = (size_t)min(base + sc * kAttnChunk + lkey + t * KPL, P - 1);
      kr[t] = *reinterpret_cast<const u32x4 *>(kb + key * rs);
      vr[t] = *reinterpret_cast<const u32x4 *>(vb + key * rs);
    }
  };
  u32x4 kr[NLD], vr[NLD];
  if (nsc > 0) load_rows(0, kr, vr);
  float qv[GH][DPL];
#pragma unroll
  for (int gh = 0; gh < GH; ++gh) {
    const f32x4 *qp = reinterpret_cast<const f32x4 *>(q + ((size_t)b * Hq + h0 + gh) * D + dl * DPL);
#pragma unroll
    for (int w = 0; w < DPL / 4; ++w) {
      const f32x4 v = qp[w];
      qv[gh][4 * w + 0] = v.x;
      qv[gh][4 * w + 1] = v.y;
      qv[gh][4 * w + 2] = v.z;
      qv[gh][4 * w + 3] = v.w;
    }
  }

  // running softmax state of this lane's row group, per head: m (uniform over
  // the wave), l and o (the group's own keys)
  float m[GH], l[GH], o[GH][DPL];
#pragma unroll
  for (int gh = 0; gh < GH; ++gh) {
    m[gh] = -INFINITY;
    l[gh] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[gh][e] = 0.f;
  }
  // online update with NS scored keys: s[t][gh] (masked -inf), value dims val(t, e)
  auto absorb = [&](auto &s, auto val) {
    constexpr int NS = sizeof(s) / sizeof(s[0]);
#pragma unroll
    for (int gh = 0; gh < GH; ++gh) {
      float mx = m[gh];
#pragma unroll
      for (int t = 0; t < NS; ++t) mx = fmaxf(mx, s[t][gh]);
      mx = across_groups_max<RL>(mx);
      const float alpha = scaled_exp(m[gh], mx);
      m[gh] = mx;
      float sum = l[gh] * alpha;
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[gh][e] *= alpha;
#pragma unroll
      for (int t = 0; t < NS; ++t) {
        s[t][gh] = scaled_exp(s[t][gh], mx);
        sum += s[t][gh];
      }
      l[gh] = sum;
    }
#pragma unroll
    for (int t = 0; t < NS; ++t)
#pragma unroll
      for (int e = 0; e < DPL; ++e) {
        const float ve = val(t, e);
#pragma unroll
        for (int gh = 0; gh < GH; ++gh) o[gh][e] += s[t][gh] * ve;  // weight 0 when masked
      }
  };

  // ---- chunk 0: the cascade keys (fp32) --------------------------------------
  if (casc) {
    f32x4 kx[NCX][CW], vx[NCX][CW];
#pragma unroll
    for (int t = 0; t < NCX; ++t) {
      const int j = min((t * 4 + wave) * KPL + kg, nctx - 1);
      const size_t off = (((size_t)b * nctx + j) * Hkv + c) * D + dl * DPL;
#pragma unroll
      for (int w = 0; w < CW; ++w) {
        kx[t][w] = reinterpret_cast<const f32x4 *>(knew + off)[w];
        vx[t][w] = reinterpret_cast<const f32x4 *>(vnew + off)[w];
      }
    }
    float sx[NCX][GH];
#pragma unroll
    for (int t = 0; t < NCX; ++t)
#pragma unroll
      for (int gh = 0; gh < GH; ++gh) {
        float acc = 0.f;
#pragma unroll
        for (int w = 0; w < CW; ++w)
          acc += qv[gh][4 * w] * kx[t][w].x + qv[gh][4 * w + 1] * kx[t][w].y +
                 qv[gh][4 * w + 2] * kx[t][w].z + qv[gh][4 * w + 3] * kx[t][w].w;
        acc = group_sum<RL>(acc);
        sx[t][gh] = (t * 4 + wave) * KPL + kg < nctx ? acc * scale : -INFINITY;
      }
    absorb(sx, [&](int t, int e) {
      const f32x4 &v = vx[t][e >> 2];
      return (e & 3) == 0 ? v.x : (e & 3) == 1 ? v.y : (e & 3) == 2 ? v.z : v.w;
    });
  }

  // ---- prefix keys, sub-chunk by sub-chunk (next rows in flight) -------------
  // The prefetch is unconditional (the last one re-reads clamped in-bounds
  // rows): under a branch the compiler would wait for it before the compute.
  for (int sc = 0; sc < nsc; ++sc) {
    u32x4 kn[NLD], vn[NLD];
    load_rows(sc + 1, kn, vn);
    const int key0 = base + sc * kAttnChunk + lkey;
    float s[NLD][GH];
#pragma unroll
    for (int t = 0; t < NLD; ++t)
#pragma unroll
      for (int gh = 0; gh < GH; ++gh) {
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc += qv[gh][e] * piece_at<T>(kr[t], e);
        acc = group_sum<RL>(acc);
        s[t][gh] = key0 + t * KPL < P ? acc * scale : -INFINITY;
      }
    absorb(s, [&](int t, int e) { return piece_at<T>(vr[t], e); });
#pragma unroll
    for (int t = 0; t < NLD; ++t) {
      kr[t] = kn[t];
      vr[t] = vn[t];
    }
  }

#pragma unroll
  for (int gh = 0; gh < GH; ++gh) {
#pragma unroll
    for (int w = 0; w < DPL / 4; ++w)
      *reinterpret_cast<f32x4 *>(&s_o[wave][kg][gh][dl * DPL + 4 * w]) =
          f32x4{o[gh][4 * w], o[gh][4 * w + 1], o[gh][4 * w + 2], o[gh][4 * w + 3]};
    if (dl == 0) s_l[wave][kg][gh] = l[gh];
    if (lane == 0) s_m[wave][gh] = m[gh];
  }
  __syncthreads();

  // ---- this workgroup's result: the output row when it holds the whole
  //      sequence, else its partial (o scaled to its max, (max, sum))
  const bool whole = nv == 1;
  for (int idx = tid; idx < GH * D; idx += 256) {
    const int gh = idx / D, e = idx % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, s_m[w][gh]);
    float acc = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      float g = 0.f, gl = 0.f;
#pragma unroll
      for (int k = 0; k < KPL; ++k) {
        g += s_o[w][k][gh][e];
        gl += s_l[w][k][gh];
      }
      const float sw = scaled_exp(s_m[w][gh], M);
      acc += sw * g;
      L += sw * gl;
    }
    if (bad) {  // P_b outside [0, pmax]: the sequence's output is NaN
      acc = __int_as_float(0x7fc00000);
      L = whole ? 1.f : acc;
      M = 0.f;
    }
    if (whole) {
      out[(size_t)b * Hq * D + (size_t)(h0 + gh) * D + e] = Elt<T>::from_f(acc / L);
    } else {
      part_o[(((size_t)b * Hq + h0 + gh) * nch_ld + ch) * D + e] = acc;
      if (e == 0) {
        float *ml = part_ml + (((size_t)b * Hq + h0 + gh) * nch_ld + ch) * 2;
        ml[0] = M;
        ml[1] = L;
      }
    }
  }
}


// ---- bf16 caches: both contractions on the matrix cores -------------------------
//
// One wave per workgroup, so up to four run on a CU side by side and the set-up
// and write-out of one overlap the streaming of the others; each covers a span
// of prefix keys of one (sequence, KV head, head group).  K and V rows reach
// LDS by direct-to-LDS loads through a per-wave ring of DEPTH stages of 16 keys
// (DEPTH-1 stages in flight), with an XOR swizzle of the 16-byte pieces that
// keeps both operand gathers free of bank conflicts.
// Per stage, QK^T runs with the keys as MFMA rows (A = 16-byte pieces of K
// rows) and the GH query heads as columns (B = q, zero-padded to 16 heads).  q
// is split into a bf16 high part and a bf16 remainder, two MFMAs each, which
// keeps the scores at fp32-level accuracy against the bf16 keys.  q is
// pre-scaled by log2(e)/sqrt(D), so scores are in log2 units and every
// exponential is one v_exp_f32.  The result leaves each lane with 4 scores of
// one head, which is exactly the B operand of the 16-key value product
// O^T = V^T P^T, so the probabilities never move between lanes; V^T is
// gathered from the ring with 16-bit reads.  The probabilities enter the
// product as bf16 and the running sum adds the same rounded values, so the
// output is an exact weighted mean of V.  The running maximum is raised only
// when a score exceeds it by more than kLazyMax (probabilities stay below
// 2^kLazyMax), so the accumulators are rescaled on few stages.
// The nctx cascade keys (fp32) are done on the vector ALU by chunk 0 and merged
// into its result at the end.



template <int D, int GH, int DEPTH, int NCX>
__global__ __launch_bounds__(64) void k_attn_mma(const bf16_t *__restrict__ Kc,
                                                 const bf16_t *__restrict__ Vc,
                                                 Seqs cu,
                                                 const float *__restrict__ q,
                                                 const float *__restrict__ knew,
                                                 const float *__restrict__ vnew, int nctx,
                                                 float *__restrict__ part, int nch, int nch_ld,
                                                 int cpw, bf16_t *__restrict__ out, int Hq,
                                                 int Hkv, const float *__restrict__ rope,
                                                 int cascade, int nseq, int persist,
                                                 int csplit, int pmax) {
  __shared__ AttnLds<D, GH, DEPTH> lds;
  const int G = Hq / Hkv, ngrp = G / GH, ncols = Hkv * ngrp;
  const int lane = threadIdx.x;
  const int span = kAttnChunk * cpw;
  float *part_o = part;
  float *part_ml = part + (size_t)nseq * Hq * nch_ld * D;

  // One piece of work: prefix chunks [ch0, ch0 + nchunk) (kAttnChunk keys
  // each) of sequence b for the query heads of column col (KV head c, head
  // group hg), plus the (at most NCX) cascade keys when casc.  The result goes
  // to the output when `whole`, else to partial slot `slot`; npieces > 0
  // (given to the first piece of a segment) is stored as the segment's
  // partial count.
  auto unit = [&](const int b, const int col, const int ch0, const int nchunk, const int slot,
                  const bool whole, const int npieces, const bool casc) {
    const int c = col / ngrp, hg = col % ngrp;
    const int h0 = c * G + hg * GH;
    bool bad;
    const int start = cu.start(b), P = attn_prefix(cu, b, pmax, bad);
    const size_t row0 = (size_t)b * Hq + h0;
    attn_unit<D, GH, DEPTH, NCX>(
        Kc + ((size_t)start * Hkv + c) * D, Vc + ((size_t)start * Hkv + c) * D, (size_t)Hkv * D,
        P, bad, q + row0 * D, knew + ((size_t)b * nctx * Hkv + c) * D,
        vnew + ((size_t)b * nctx * Hkv + c) * D, (size_t)Hkv * D, nctx, rope, cascade, ch0, nchunk,
        whole, casc, part_o + (row0 * nch_ld + slot) * D, nch_ld * D,
        part_ml + (row0 * nch_ld + slot) * 2, nch_ld * 2, out + row0 * D,
        part_ml + (size_t)nseq * Hq * nch_ld * 2 + row0, npieces, lds);
  };


  if (!persist) {
    // one workgroup per span of cpw chunks: grid (columns, spans, sequences),
    // heads fastest so the workgroups that run side by side read neighbouring
    // head segments of the same token rows; partial slot = span index
    const int b = blockIdx.z, col = blockIdx.x, ch = blockIdx.y;
    bool bad;
    const int P = attn_prefix(cu, b, pmax, bad);
    const int nv = max(1, min((P + span - 1) / span, nch));
    if (csplit) {
      // the cascade keys as a unit of their own (grid y = nch), off the
      // prefix units' critical path; every sequence leaves nv + 1 partials,
      // the cascade's last
      if (ch == nch) unit(b, col, 0, 0, nv, false, 0, true);
      else if (ch < nv) unit(b, col, ch * cpw, cpw, ch, false, 0, false);
      return;
    }
    if (ch < nv) unit(b, col, ch * cpw, cpw, ch, nv == 1, 0, ch == 0);
    return;
  }
  // Persistent: a grid of resident waves, each taking one range of the
  // equal-chunk split (AttnSplit; W = the grid, or the chunk count if
  // smaller), so the waves finish together however ragged the sequences are.
  // Up to 256 sequences (4 per lane).
  int ucnt[4], uend[4];  // chunks of sequence lane + 64 i (all columns), running total
  int run = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int b = lane + 64 * i;
    int n = 0;
    if (b < nseq) {
      bool bad;
      n = attn_seg_chunks(attn_prefix(cu, b, pmax, bad), nch_ld) * ncols;
    }
    // inclusive scan over the wave, then add the totals of earlier blocks
    int x = n;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    ucnt[i] = n;
    uend[i] = run + x;
    run += __shfl(x, 63, 64);
  }
  const AttnSplit eq{run, min((long)gridDim.x, (long)run)};
  if ((long)blockIdx.x >= eq.W) return;
  int x = eq.begin(blockIdx.x);
  const int xe = eq.begin(blockIdx.x + 1);
  while (x < xe) {
    // sequence b: the number of sequences whose chunks all come before x
    int b = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) b += __popcll(__ballot(uend[i] <= x));
    int first = 0, cnt = 0;  // chunks before sequence b, and its own
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = __shfl(uend[i], b & 63, 64), n = __shfl(ucnt[i], b & 63, 64);
      if ((b >> 6) == i) {
        first = e - n;
        cnt = n;
      }
    }
    int col, ch0, n, slot, np;
    eq.piece(x, xe, first, cnt, ncols, col, ch0, n, slot, np);
    // items [ch0, ch0 + n) of the segment: prefix chunks below its last item,
    // which stands for the cascade keys
    const int items = cnt / ncols, pre = min(ch0 + n, items - 1) - ch0;
    unit(b, col, ch0, pre > 0 ? pre : 0, slot, false, np, ch0 + n == items);
    x += n;
  }
}


// ---- chunk merge (second launch) -------------------------------------------------
// A sequence whose prefix spans several workgroups leaves one partial per
// workgroup: o (scaled to that workgroup's max), max and sum per head.  This
// launch combines them in chunk order, 32 per round trip.  Sequences that fit
// one workgroup wrote their rows directly and are skipped.  Keeping the merge in
// its own launch means no workgroup ever waits on another: the kernel boundary
// publishes the partials once, where per-workgroup device-scope fences would
// write back the L2 once per workgroup.  LOG2: maxima in log2 units.
template <typename T, bool LOG2>
__global__ __launch_bounds__(256) void k_attn_merge(const float *__restrict__ part, int nch_ld,
                                                    Seqs cu, int span,
                                                    int nwg, T *__restrict__ out, int Hq, int D,
                                                    int counted, int csplit, int pmax) {
  const int b = blockIdx.y;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= Hq * D / 2) return;
  const int h = (2 * idx) / D, e = (2 * idx) % D;
  // partials of (b, h): one per span (sequences within one span wrote their
  // rows directly) and, with csplit, the cascade keys' one after them, or as
  // counted by the persistent attention
  int nv;
  if (counted) {
    nv = (int)part[(size_t)gridDim.y * Hq * nch_ld * (D + 2) + (size_t)b * Hq + h];
  } else {
    bool bad;
    const int P = attn_prefix(cu, b, pmax, bad);
    nv = max(1, min((P + span - 1) / span, nwg)) + csplit;
    if (nv == 1) return;
  }
  const float *po = part + ((size_t)b * Hq + h) * nch_ld * D + e;
  const float *pml = part + (size_t)gridDim.y * Hq * nch_ld * D + ((size_t)b * Hq + h) * nch_ld * 2;
  auto ex = [](float m, float M) {
    return m == -INFINITY ? 0.f : (LOG2 ? __builtin_amdgcn_exp2f(m - M) : expf(m - M));
  };
  float M = -INFINITY, L = 0.f, ax = 0.f, ay = 0.f;
  constexpr int R = 32;  // partials per round trip
  for (int c0 = 0; c0 < nv; c0 += R) {
    float2 ov[R], ml[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int k = min(c0 + u, nv - 1);
      ov[u] = *reinterpret_cast<const float2 *>(po + (size_t)k * D);
      ml[u] = *reinterpret_cast<const float2 *>(pml + 2 * k);
    }
    float Mn = M;
#pragma unroll
    for (int u = 0; u < R; ++u)
      if (c0 + u < nv) Mn = fmaxf(Mn, ml[u].x);
    const float rr = ex(M, Mn);
    L *= rr;
    ax *= rr;
    ay *= rr;
#pragma unroll
    for (int u = 0; u < R; ++u)
      if (c0 + u < nv) {
        const float w = ex(ml[u].x, Mn);
        L += w * ml[u].y;
        ax += w * ov[u].x;
        ay += w * ov[u].y;
      }
    M = Mn;
  }
  T *op = out + (size_t)b * Hq * D + (size_t)h * D + e;
  op[0] = Elt<T>::from_f(ax / L);
  op[1] = Elt<T>::from_f(ay / L);
}

template <typename T, int D>
static hipError_t attn_t(const void *K, const void *V, Seqs cu, const float *q,
                         const float *knew, const float *vnew, int nctx, float *part, int nch,
                         int nch_ld, int cpw, void *out, int B, int Hq, int Hkv, int pmax,
                         hipStream_t s) {
  const int G = Hq / Hkv;
  const int GH = (G % 4 == 0) ? 4 : (G % 2 == 0 ? 2 : 1);
  const int nwg = nch < 1 ? 1 : (nch + cpw - 1) / cpw;
  const dim3 grid(Hkv * (G / GH), nwg, B);
#define FE_ATTN(GHV)                                                                            \
  hipLaunchKernelGGL((k_attn<T, D, GHV>), grid, dim3(256), 0, s, (const T *)K, (const T *)V, cu, \
                     q, knew, vnew, nctx, part, nwg, nch_ld, cpw, (T *)out, Hq, Hkv, pmax)
  if (GH == 4) FE_ATTN(4);
  else if (GH == 2) FE_ATTN(2);
  else FE_ATTN(1);
#undef FE_ATTN
  return hipGetLastError();
}

// Waves that stay resident at once: four one-wave workgroups per CU.
static int resident_waves() {
  static int n[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1024;
  if (n[dev] == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
    n[dev] = 4 * cus;
  }
  return n[dev];
}

template <int D>
static hipError_t attn_mma_t(const void *K, const void *V, Seqs cu, const float *q,
                             const float *knew, const float *vnew, int nctx, float *part, int nch,
                             int nch_ld, int cpw, void *out, int B, int Hq, int Hkv,
                             const float *rope, int cascade, int pmax, int *persisted,
                             int *csplit, hipStream_t s) {
  const int G = Hq / Hkv;
  // query heads per wave (the MFMA tiles have 16 columns; more than 8 heads
  // would spill the cascade step's registers)
  const int GH = G % 8 == 0 ? 8 : G % 4 == 0 ? 4 : G % 2 == 0 ? 2 : 1;
  const int nwg = nch < 1 ? 1 : (nch + cpw - 1) / cpw;
  const int ncols = Hkv * (G / GH);
  // persistent waves when the units outnumber the resident waves
  const int waves = resident_waves();
  const int persist = B <= 256 && (long)B * ncols * nwg > waves ? 1 : 0;
  *persisted = persist;
  // a launch whose partials are merged anyway gives the cascade keys units of
  // their own (one more partial slot per sequence)
  const int split = !persist && nwg > 1 ? 1 : 0;
  *csplit = split;
  const dim3 grid = persist ? dim3(waves) : dim3(ncols, nwg + split, B);
  // a span of at most 4 stages is requested whole by the ring's prologue
  const bool short_span = cpw * (kAttnChunk / 16) <= 4;
#define FE_ATTN(GHV, DEP, NCXV)                                                                  \
  hipLaunchKernelGGL((k_attn_mma<D, GHV, DEP, NCXV>), grid, dim3(64), 0, s, (const bf16_t *)K,   \
                     (const bf16_t *)V, cu, q, knew, vnew, nctx, part, nwg, nch_ld, cpw,         \
                     (bf16_t *)out, Hq, Hkv, rope, cascade, B, persist, split, pmax)
#define FE_ATTN_NCX(GHV, DEP)                                                                    \
  if (nctx <= 8) FE_ATTN(GHV, DEP, 8);                                                           \
  else FE_ATTN(GHV, DEP, kMaxLayers)
#define FE_ATTN_GH(GHV)                                                                          \
  if (short_span) { FE_ATTN_NCX(GHV, 5); }                                                       \
  else { FE_ATTN_NCX(GHV, 4); }
  switch (GH) {
    case 8: FE_ATTN_GH(8); break;
    case 4: FE_ATTN_GH(4); break;
    case 2: FE_ATTN_GH(2); break;
    default: FE_ATTN_GH(1); break;
  }
#undef FE_ATTN_GH
#undef FE_ATTN_NCX
#undef FE_ATTN
  return hipGetLastError();
}

// Enough workgroups to keep every CU busy with several at a time until the
// end (one-wave workgroups, four per CU) and no more: a sequence split over
// more workgroups only adds set-up work and partials to merge.
// A launch of at most a few rounds of resident waves (batch 1 at every model
// shape) instead takes the fewest chunks per unit that keep it to one round
// and its merge to one round trip (32 partials per head): measured at batch 1,
// 13B-shaped (40 KV heads, P 2048) 16.3 us per layer against 31.1 with one
// chunk per unit, 70B-shaped (P 4096) 16.2 against 19.0, 8B-shaped unchanged.
int attention_cpw(int B, int Hkv, int ngroups, int nch) {
  constexpr long kTargetWorkgroups = 4096;
  const long cols = (long)B * Hkv * ngroups, units = cols * nch;
  long cpw = (units + kTargetWorkgroups - 1) / kTargetWorkgroups;
  if (units <= kTargetWorkgroups) {
    const long waves = resident_waves();
    const long one_round = (units + waves - 1) / waves, one_trip = (nch + 31) / 32;
    cpw = one_round > one_trip ? one_round : one_trip;
  }
  if (cpw > nch) cpw = nch;
  return cpw < 1 ? 1 : (int)cpw;
}

hipError_t attention(int dt, const void *K, const void *V, Seqs cu, const float *q,
                     const float *knew, const float *vnew, int nctx, float *part, int nch,
                     int nch_ld, int cpw, void *out, int B, int Hq, int Hkv, int D,
                     const float *rope, int cascade, int pmax, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (cpw < 1) cpw = 1;
  hipError_t e;
  int persisted = 0, csplit = 0;
  if (nctx < 1 || nctx > kMaxLayers) return hipErrorInvalidValue;
  if (dt)
    e = D == 128 ? attn_mma_t<128>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld, cpw, out, B,
                                   Hq, Hkv, rope, cascade, pmax, &persisted, &csplit, s)
                 : attn_mma_t<64>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld, cpw, out, B,
                                  Hq, Hkv, rope, cascade, pmax, &persisted, &csplit, s);
  else
    e = D == 128 ? attn_t<float, 128>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld, cpw, out,
                                      B, Hq, Hkv, pmax, s)
                 : attn_t<float, 64>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld, cpw, out,
                                     B, Hq, Hkv, pmax, s);
  if (e != hipSuccess) return e;
  const int nwg = nch < 1 ? 1 : (nch + cpw - 1) / cpw;
  if (nwg == 1 && !persisted) return hipSuccess;  // every sequence fits one workgroup
  const dim3 grid((Hq * D / 2 + 255) / 256, B);
  if (dt)
    hipLaunchKernelGGL((k_attn_merge<bf16_t, true>), grid, dim3(256), 0, s, part, nch_ld, cu,
                       kAttnChunk * cpw, nwg, (bf16_t *)out, Hq, D, persisted, csplit, pmax);
  else
    hipLaunchKernelGGL((k_attn_merge<float, false>), grid, dim3(256), 0, s, part, nch_ld, cu,
                       kAttnChunk * cpw, nwg, (float *)out, Hq, D, 0, 0, pmax);
  return hipGetLastError();
}

}  // namespace fe
