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
#include "fe_internal.h"

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
                                              const int32_t *__restrict__ cu,
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
  const int start = cu[b], P = attn_prefix(cu, b, pmax, bad);
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
__device__ __forceinline__ float sexp2(float m, float M) {
  return m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M);
}
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) { return f2bf2(lo, hi); }
constexpr float kLazyMax = 8.f;

// vmcnt wait for the ring's last stages: n (0..MAXN) stages of PER loads each
// may stay in flight.
template <int MAXN, int PER> __device__ __forceinline__ void wait_tail(int n) {
  if constexpr (MAXN > 0) {
    if (n >= MAXN) {
      wait_vmcnt<MAXN * PER>();
      return;
    }
    wait_tail<MAXN - 1, PER>(n);
  } else {
    wait_vmcnt<0>();
  }
}

// Direct-to-LDS load issued as inline assembly: the compiler does not track it,
// so it adds no waits of its own before reads of the ring (its alias-based
// tracking otherwise drains every outstanding load at some of them); the
// kernel orders the ring with explicit vmcnt/lgkmcnt waits instead.  lds must
// be wave-uniform.  M0 is set here without a clobber (the compiler reserves
// it); the kernel that uses this has no other M0 users.
__device__ __forceinline__ void ring_dma16(const void *src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds) : "memory");
}

template <int D, int GH, int DEPTH, int NCX>
__global__ __launch_bounds__(64) void k_attn_mma(const bf16_t *__restrict__ Kc,
                                                 const bf16_t *__restrict__ Vc,
                                                 const int32_t *__restrict__ cu,
                                                 const float *__restrict__ q,
                                                 const float *__restrict__ knew,
                                                 const float *__restrict__ vnew, int nctx,
                                                 float *__restrict__ part, int nch, int nch_ld,
                                                 int cpw, bf16_t *__restrict__ out, int Hq,
                                                 int Hkv, const float *__restrict__ rope,
                                                 int cascade, int nseq, int persist,
                                                 int csplit, int pmax) {
  static_assert(D == 64 || D == 128, "head dims 64 and 128");
  static_assert(NCX <= kMaxLayers, "cascade keys per layer");
  constexpr int NKC = D / 32;          // 32-dim steps of QK^T
  constexpr int NDT = D / 16;          // 16-dim tiles of the value product
  constexpr int VPR = D / 8;           // 16-byte pieces per K or V row
  constexpr int RB = 2 * D;            // bytes per K or V row
  constexpr int RPW = 256 / RB;        // rows per 256-byte span of the LDS banks
  constexpr int SK = 16;               // keys per stage
  constexpr int HALF = SK * RB;        // K rows of a stage, then as many V rows
  constexpr int STAGE = 2 * HALF;
  constexpr int NDMA = STAGE / 1024;   // 1 KB direct-to-LDS loads per stage
  constexpr int NOFF = NDMA / 2;       // of which K (the rest V, same layout)
  // DEPTH ring slots: DEPTH-1 stages in flight
  static_assert(DEPTH * NDMA <= 63, "outstanding loads stay within the vmcnt range");
  static_assert(kAttnChunk % SK == 0, "whole stages per chunk");
  constexpr int HD = D / 2;            // rotary pairs (m, m + D/2)
  __shared__ __align__(16) unsigned char s_ring[DEPTH][STAGE];
  __shared__ __align__(16) float s_oc[GH][D];  // cascade partial: o, max, sum per head
  __shared__ float s_mc[GH], s_lc[GH];

  const int G = Hq / Hkv, ngrp = G / GH, ncols = Hkv * ngrp;
  const int lane = threadIdx.x, r = lane & 15, g = lane >> 4;
  const float qscale = 1.4426950408889634f * rsqrtf((float)D);
  const int span = kAttnChunk * cpw;

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

  // Loads that do not depend on the prefix bounds go first, so their latency
  // overlaps the read of cu: q (B-operand layout), and in chunk 0 the cascade
  // rows.
  f32x4 qraw[NKC][2];
  {
    const float *qp = q + ((size_t)b * Hq + h0 + min(r, GH - 1)) * D;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      qraw[kc][0] = *reinterpret_cast<const f32x4 *>(qp + 32 * kc + 8 * g);
      qraw[kc][1] = *reinterpret_cast<const f32x4 *>(qp + 32 * kc + 8 * g + 4);
    }
  }
  // cascade step: lane l < D/2 holds the rotary pair (m, m + D/2), m = l
  const int m2 = min(lane, HD - 1);
  const bool cact = lane < HD;
  float kj[NCX][2], vj[NCX][2], qc[GH][2];
  if (casc) {
#pragma unroll
    for (int gh = 0; gh < GH; ++gh)
#pragma unroll
      for (int e = 0; e < 2; ++e) qc[gh][e] = q[((size_t)b * Hq + h0 + gh) * D + m2 + e * HD];
#pragma unroll
    for (int j = 0; j < NCX; ++j) {
      const size_t off = (((size_t)b * nctx + min(j, nctx - 1)) * Hkv + c) * D + m2;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        kj[j][e] = knew[off + e * HD];
        vj[j][e] = vnew[off + e * HD];
      }
    }
  }

  bool bad;
  const int start = cu[b], P = attn_prefix(cu, b, pmax, bad);
  // rotary coefficients (Section 2.1's decoder layers use RoPE; the cached
  // prefix keys are stored rotated): the query sits at the last cascade
  // position, cascade key j at P + j (one position, P, per layer otherwise).
  const int pos_q = cascade ? P + nctx - 1 : P;
  f32x4 rq[NKC / 2][4];
#pragma unroll
  for (int kc = 0; kc < NKC / 2; ++kc)
#pragma unroll
    for (int w = 0; w < 4; ++w)
      rq[kc][w] = *reinterpret_cast<const f32x4 *>(rope + ((size_t)pos_q * HD + 32 * kc + 8 * g) * 2 + 4 * w);
  float2 rcj[NCX], rcq;
  if (casc) {
#pragma unroll
    for (int j = 0; j < NCX; ++j)
      rcj[j] = *reinterpret_cast<const float2 *>(rope + ((size_t)(cascade ? P + min(j, nctx - 1) : P) * HD + m2) * 2);
    rcq = *reinterpret_cast<const float2 *>(rope + ((size_t)pos_q * HD + m2) * 2);
  }
  const int base = ch0 * kAttnChunk;
  // stages of SK keys; past P the loads are clamped in bounds and the scores masked
  const int nst = P > base ? min(nchunk * (kAttnChunk / SK), (P - base + SK - 1) / SK) : 0;
  float *part_o = part;
  float *part_ml = part + (size_t)nseq * Hq * nch_ld * D;

  // Stage st: keys base + SK st + R, R < SK, K rows then V rows, loaded straight
  // into ring slot `slot`.  Load i moves 1 KB: lane l the 16 bytes at 16 l of
  // it, i.e. row R, position sl of that row, which holds 16-byte piece
  // sl ^ swz(R).  The swizzle spreads the pieces that one MFMA operand read
  // gathers from 16 rows (K: one piece of rows 0..15; V: two pieces of rows
  // 4g + e) over distinct banks.
  const size_t rs = (size_t)Hkv * D;
  const bf16_t *kb = Kc + ((size_t)start * Hkv + c) * D;
  const bf16_t *vb = Vc + ((size_t)start * Hkv + c) * D;
  // row R's 16-byte pieces are rotated by swz(R), a bijection on the rows of one
  // bank span's worth of pieces that also sends the 8 rows one transposing read
  // of V meets (two pieces each) to distinct bank groups
  constexpr int LQ = VPR == 16 ? 3 : 2;
  auto swz = [](int R) {
    const int Q = R / RPW;
    return (2 * Q + (Q >> LQ)) & (VPR - 1);
  };
  int lrow[NOFF], loff[NOFF];  // this lane's row and element offset in it, per load
#pragma unroll
  for (int i = 0; i < NOFF; ++i) {
    const int o = i * 1024 + 16 * lane, R = o / RB, sl = (o % RB) / 16;
    lrow[i] = R;
    loff[i] = 8 * (sl ^ swz(R));
  }
  const uint32_t ring0 = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)((__attribute__((address_space(3))) unsigned char *)&s_ring[0][0]));
  auto load_stage = [&](int st, int slot) {
    const int k0 = base + st * SK;
    const uint32_t dst = ring0 + slot * STAGE;
    if (k0 + SK <= P) {  // whole stage inside the prefix: one row base for all lanes
      const bf16_t *ks = kb + (size_t)k0 * rs, *vs = vb + (size_t)k0 * rs;
#pragma unroll
      for (int i = 0; i < NOFF; ++i) ring_dma16(ks + lrow[i] * rs + loff[i], dst + i * 1024);
#pragma unroll
      for (int i = 0; i < NOFF; ++i) ring_dma16(vs + lrow[i] * rs + loff[i], dst + HALF + i * 1024);
    } else {
#pragma unroll
      for (int i = 0; i < NOFF; ++i)
        ring_dma16(kb + (size_t)min(k0 + lrow[i], P - 1) * rs + loff[i], dst + i * 1024);
#pragma unroll
      for (int i = 0; i < NOFF; ++i)
        ring_dma16(vb + (size_t)min(k0 + lrow[i], P - 1) * rs + loff[i], dst + HALF + i * 1024);
    }
  };
  // prologue: the first DEPTH-1 stages (fewer if there are fewer); the ring's
  // reads by a previous unit have returned
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int d = 0; d < DEPTH - 1; ++d)
    if (d < nst) load_stage(d, d);

  // q as B operands: column r = head h0 + r (zero for r >= GH), high and low parts
  // rotate-half: dims 32kc + 8g + e and their partners D/2 later (kc + NKC/2)
  float qf[NKC][8];
#pragma unroll
  for (int kc = 0; kc < NKC; ++kc) {
    qf[kc][0] = qraw[kc][0].x; qf[kc][1] = qraw[kc][0].y; qf[kc][2] = qraw[kc][0].z; qf[kc][3] = qraw[kc][0].w;
    qf[kc][4] = qraw[kc][1].x; qf[kc][5] = qraw[kc][1].y; qf[kc][6] = qraw[kc][1].z; qf[kc][7] = qraw[kc][1].w;
  }
#pragma unroll
  for (int kc = 0; kc < NKC / 2; ++kc)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const f32x4 cw = rq[kc][e >> 1];
      const float cs = (e & 1) ? cw.z : cw.x, sn = (e & 1) ? cw.w : cw.y;
      const float x1 = qf[kc][e], x2 = qf[kc + NKC / 2][e];
      qf[kc][e] = x1 * cs - x2 * sn;
      qf[kc + NKC / 2][e] = x2 * cs + x1 * sn;
    }
  u32x4 qh[NKC], ql[NKC];
#pragma unroll
  for (int kc = 0; kc < NKC; ++kc) {
    const float *x = qf[kc];
    uint32_t hw[4], lw[4];
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const float a0 = r < GH ? x[e] * qscale : 0.f, a1 = r < GH ? x[e + 1] * qscale : 0.f;
      hw[e / 2] = pack_bf16(a0, a1);
      lw[e / 2] = pack_bf16(a0 - __uint_as_float(hw[e / 2] << 16),
                            a1 - __uint_as_float(hw[e / 2] & 0xffff0000u));
    }
    qh[kc] = u32x4{hw[0], hw[1], hw[2], hw[3]};
    ql[kc] = u32x4{lw[0], lw[1], lw[2], lw[3]};
  }

  // ---- prefix keys: online softmax over stages, DEPTH-1 in flight ------------------
  float m = -INFINITY, l = 0.f;  // head r: running max (uniform over g), this lane's sum
  f32x4 oacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) oacc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // unrolled by DEPTH so that stage st = s0 + u sits in ring slot u
  for (int s0 = 0; s0 < nst; s0 += DEPTH) {
#pragma unroll
    for (int u = 0; u < DEPTH; ++u) {
      const int st = s0 + u;
      if (st >= nst) break;
      // refill the slot that stage st-1 left (its reads have returned), then
      // wait until stage st has landed in slot u: the loads of the stages
      // after it may stay in flight
      if (st + DEPTH - 1 < nst) {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        load_stage(st + DEPTH - 1, (u + DEPTH - 1) % DEPTH);
        wait_vmcnt<(DEPTH - 1) * NDMA>();
      } else {
        wait_tail<DEPTH - 2, NDMA>(nst - 1 - st);
      }
      const unsigned char *kr = s_ring[u], *vr = kr + HALF;
      // S^T = K q: A = K (key r, dims 32kc + 8g..), B = q (hi and lo parts)
      // two accumulation chains (q high and low parts), summed at the end
      f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc) {
        const u32x4 ka = *reinterpret_cast<const u32x4 *>(kr + r * RB + 16 * ((4 * kc + g) ^ swz(r)));
        sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka),
                                                     __builtin_bit_cast(bf16x8, qh[kc]), sa, 0, 0, 0);
        sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka),
                                                     __builtin_bit_cast(bf16x8, ql[kc]), sb, 0, 0, 0);
      }
      sa += sb;
      // V^T (independent of the scores): lane (r, g) needs dim 16dt + r of keys
      // 4g + e, e < 4.  gfx950's transposing read does it in one instruction
      // per dt: within each 16-lane group, lane 4e + q names 4 consecutive
      // 16-bit values and lane i receives value i % 4 of lanes i / 4 + 4e, so
      // lane 4e + q points at key 4g + e, dims 16dt + 4q .. + 3.
      i16x4 av[NDT];
      {
        const int R = 4 * g + (r >> 2), q4 = r & 3;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const int pc = 2 * dt + (q4 >> 1);
          av[dt] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) i16x4 *)(vr + R * RB + 16 * (pc ^ swz(R)) + 8 * (q4 & 1)));
        }
      }
      // lane holds S[key 4g + v][head r]; keys past P (last stage only) are masked
      const int kq = base + st * SK + 4 * g;
      float sv4[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) sv4[v] = kq + v < P ? sa[v] : -INFINITY;
      float mx = fmaxf(fmaxf(sv4[0], sv4[1]), fmaxf(sv4[2], sv4[3]));
      mx = xor32_max(xor16_max(mx));
      const bool up = mx > m + kLazyMax;  // same for the 4 lanes of a head
      if (__builtin_amdgcn_ballot_w64(up)) {
        const float mn = up ? mx : m;
        const float alpha = sexp2(m, mn);
        m = mn;
        l *= alpha;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) oacc[dt] *= alpha;
      }
      // P is already in the B layout of the 16-key value product: key 4g + e, head r
      const u32x2 pb = {pack_bf16(sexp2(sv4[0], m), sexp2(sv4[1], m)),
                        pack_bf16(sexp2(sv4[2], m), sexp2(sv4[3], m))};
      l += (__uint_as_float(pb.x << 16) + __uint_as_float(pb.x & 0xffff0000u)) +
           (__uint_as_float(pb.y << 16) + __uint_as_float(pb.y & 0xffff0000u));
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
        oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(av[dt],
                                                             __builtin_bit_cast(i16x4, pb),
                                                             oacc[dt], 0, 0, 0);
    }
  }

  // ---- chunk 0: the cascade keys, fp32 on the vector ALU -> s_oc, s_mc, s_lc ----
  // Done after the prefix loop: its inputs were loaded at the start and have
  // long arrived, and waiting for them earlier would also wait for the ring.
  if (casc) {
    // rotate-half on the pair (m, m + D/2); all nctx-bound work is masked rather
    // than branched, so the reductions of different keys and heads interleave
    float kr2[NCX][2];
#pragma unroll
    for (int j = 0; j < NCX; ++j) {
      kr2[j][0] = kj[j][0] * rcj[j].x - kj[j][1] * rcj[j].y;
      kr2[j][1] = kj[j][1] * rcj[j].x + kj[j][0] * rcj[j].y;
    }
    constexpr int HB = GH < 4 ? GH : 4;  // heads per batch of reductions
#pragma unroll
    for (int g0 = 0; g0 < GH; g0 += HB) {
    float sj[HB][NCX];
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
      const float qa = qc[g0 + hb][0], qb = qc[g0 + hb][1];
      const float q0 = cact ? (qa * rcq.x - qb * rcq.y) * qscale : 0.f;
      const float q1 = cact ? (qb * rcq.x + qa * rcq.y) * qscale : 0.f;
#pragma unroll
      for (int j = 0; j < NCX; ++j) sj[hb][j] = q0 * kr2[j][0] + q1 * kr2[j][1];
    }
#pragma unroll
    for (int hb = 0; hb < HB; ++hb)
#pragma unroll
      for (int j = 0; j < NCX; ++j) {
        const float t = group_sum<64>(sj[hb][j]);
        sj[hb][j] = j < nctx ? t : -INFINITY;
      }
#pragma unroll
    for (int hb = 0; hb < HB; ++hb) {
      const int gh = g0 + hb;
      float mc = -INFINITY;
#pragma unroll
      for (int j = 0; j < NCX; ++j) mc = fmaxf(mc, sj[hb][j]);
      float L = 0.f, o[2] = {0.f, 0.f};
#pragma unroll
      for (int j = 0; j < NCX; ++j) {
        const float pj = sexp2(sj[hb][j], mc);
        L += pj;
#pragma unroll
        for (int e = 0; e < 2; ++e) o[e] += pj * vj[j][e];
      }
      if (cact) {
        s_oc[gh][m2] = o[0];
        s_oc[gh][m2 + HD] = o[1];
      }
      if (lane == 0) {
        s_mc[gh] = mc;
        s_lc[gh] = L;
      }
    }
    }
  }

  // ---- result: O^T[16dt + 4g + v][head r], merged with the cascade partial ----
  l = xor32_sum(xor16_sum(l));
  float M = m, L = l, sp = 1.f, sc = 0.f;
  if (casc) {
    const int rr = min(r, GH - 1);
    const float mc = s_mc[rr];
    M = fmaxf(m, mc);
    sp = sexp2(m, M);
    sc = sexp2(mc, M);
    L = l * sp + s_lc[rr] * sc;
  }
  if (bad) {  // P_b outside [0, pmax]: the sequence's output is NaN
    M = 0.f;
    L = __int_as_float(0x7fc00000);
    sp = L;
  }
  if (npieces > 0 && g == 0 && r < GH)
    part_ml[(size_t)nseq * Hq * nch_ld * 2 + (size_t)b * Hq + h0 + r] = (float)npieces;
  if (r >= GH) return;  // padding columns of the MFMA tiles
  const size_t row = (size_t)b * Hq + h0 + r;
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) {
    const int d0 = 16 * dt + 4 * g;
    f32x4 o = oacc[dt] * sp;
    if (casc) {
      const f32x4 oc = *reinterpret_cast<const f32x4 *>(&s_oc[r][d0]);
      o += oc * sc;
    }
    if (whole) {
      const float inv = 1.f / L;
      const u32x2 w = {pack_bf16(o[0] * inv, o[1] * inv), pack_bf16(o[2] * inv, o[3] * inv)};
      *reinterpret_cast<u32x2 *>(out + row * D + d0) = w;
    } else {
      *reinterpret_cast<f32x4 *>(part_o + (row * nch_ld + slot) * D + d0) = o;
    }
  }
  if (!whole && g == 0) {
    float *ml = part_ml + (row * nch_ld + slot) * 2;
    ml[0] = M;
    ml[1] = L;
  }
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
    unit(b, col, ch0, n, slot, false, np, ch0 == 0);
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
                                                    const int32_t *__restrict__ cu, int span,
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
static hipError_t attn_t(const void *K, const void *V, const int32_t *cu, const float *q,
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
static hipError_t attn_mma_t(const void *K, const void *V, const int32_t *cu, const float *q,
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
int attention_cpw(int B, int Hkv, int ngroups, int nch) {
  constexpr long kTargetWorkgroups = 4096;
  const long cols = (long)B * Hkv * ngroups;
  long cpw = (cols * nch + kTargetWorkgroups - 1) / kTargetWorkgroups;
  if (cpw > nch) cpw = nch;
  return cpw < 1 ? 1 : (int)cpw;
}

hipError_t attention(int dt, const void *K, const void *V, const int32_t *cu, const float *q,
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
