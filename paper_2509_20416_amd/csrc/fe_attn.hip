// fe_attn.hip -- GQA decode attention of a cascade layer over its prefix KV
// cache plus the cascade entries, in one launch (gfx950).
//
// Layer i's query (one row per sequence, H_q heads) attends to the P_b cached
// prefix keys of its own cache and to the nctx keys it projected from the
// cascade states (Section 2.1; the cache is per layer because every L_i has
// its own parameters).
//
//  * One workgroup (4 waves) per (sequence, KV head, head group, chunk of
//    kAttnChunk prefix keys); the GH query heads sharing a KV head are done
//    together so every K/V byte is read once.  Each wave takes 32 keys.  A key
//    row is split in 16-byte pieces over RL = D*sizeof(T)/16 lanes, so one
//    load instruction covers 64/RL whole rows; K and V are loaded together.
//  * A score is reduced over its RL lanes with DPP row operations and leaves
//    every lane of the row with the same value, which is exactly what the
//    value pass needs: each lane accumulates p*V for its own dims and key
//    rows, so the value sums need no cross-lane traffic.  Row-group maxima use
//    gfx950's permlane swaps.  The per-(wave, row group) sums meet in LDS.
//  * Chunk 0 also takes the nctx cascade keys (fp32, one extra load per lane).
//  * Each chunk leaves o[D] (scaled to the chunk max) and (max, sum) per head
//    in the workspace; every chunk workgroup bumps a counter after a release
//    fence and the last one (acquire fence) merges the chunks in a fixed
//    order, writes the output row and resets the counter for the next launch.
//    A sequence with an empty prefix still runs chunk 0 for its cascade keys.
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
                                              T *__restrict__ out, int Hq, int Hkv) {
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
  const int ch = blockIdx.x, c = blockIdx.y / ngrp, hg = blockIdx.y % ngrp, b = blockIdx.z;
  const int start = cu[b], P = cu[b + 1] - start;
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
// Per wave and sub-chunk: 32 keys as two 16-key tiles.  QK^T runs with the keys
// as MFMA rows (A = 16-byte pieces of K rows, straight from HBM) and the GH
// query heads as columns (B = q, zero-padded to 16 heads).  q is split into a
// bf16 high part and a bf16 remainder, two MFMAs each, which keeps the scores
// at fp32-level accuracy against the bf16 keys.  q is pre-scaled by
// log2(e)/sqrt(D), so scores are in log2 units and every exponential is one
// v_exp_f32.  The result leaves each lane with 8 scores of one head, which is
// exactly the B operand of the value product O^T = V^T P^T (keys as the
// contraction index, in the order the score tiles produced them), so the
// probabilities never move between lanes; V goes through LDS (padded rows,
// conflict-free transposed 16-bit reads) to form the A operand.  The
// probabilities enter the product as bf16 and the running sum adds the same
// rounded values, so the output is an exact weighted mean of V.
// The nctx cascade keys (fp32) are done on the vector ALU by chunk 0 and enter
// the workgroup merge as a fifth partial.
__device__ __forceinline__ float sexp2(float m, float M) {
  return m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M);
}
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return (uint32_t)f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
}

template <int D, int GH>
__global__ __launch_bounds__(256) void k_attn_mma(const bf16_t *__restrict__ Kc,
                                                  const bf16_t *__restrict__ Vc,
                                                  const int32_t *__restrict__ cu,
                                                  const float *__restrict__ q,
                                                  const float *__restrict__ knew,
                                                  const float *__restrict__ vnew, int nctx,
                                                  float *__restrict__ part, int nch, int nch_ld,
                                                  int cpw, bf16_t *__restrict__ out, int Hq,
                                                  int Hkv, const float *__restrict__ rope,
                                                  int cascade) {
  constexpr int NKC = D / 32;         // 32-dim steps of QK^T
  constexpr int NDT = D / 16;         // 16-dim tiles of the value product
  constexpr int VPR = D / 8;          // 16-byte pieces per V row
  constexpr int NVL = 32 * VPR / 64;  // V pieces per lane per sub-chunk
  constexpr int RSB = 2 * D + 16;     // LDS bytes per staged V row
  constexpr int HD = D / 2;           // rotary pairs (m, m + D/2)
  __shared__ __align__(16) unsigned char s_v[4][32 * RSB];
  __shared__ float s_o[5][GH][D];
  __shared__ float s_l[5][GH], s_m[5][GH];

  const int G = Hq / Hkv, ngrp = G / GH;
  const int ch = blockIdx.x, c = blockIdx.y / ngrp, hg = blockIdx.y % ngrp, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r = lane & 15, g = lane >> 4;
  const int h0 = c * G + hg * GH;
  const float qscale = 1.4426950408889634f * rsqrtf((float)D);
  const bool casc = ch == 0;
  constexpr int GHW = (GH + 3) / 4;  // cascade-step heads per wave

  // Loads that do not depend on the prefix bounds go first, so their latency
  // overlaps the read of cu: q (B-operand layout), and in chunk 0 the cascade
  // rows and this wave's cascade-step q.
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
  float kj[kMaxLayers][2], vj[kMaxLayers][2], qc[GHW][2];
  if (casc) {
#pragma unroll
    for (int j = 0; j < kMaxLayers; ++j) {
      const size_t off = (((size_t)b * nctx + min(j, nctx - 1)) * Hkv + c) * D + m2;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        kj[j][e] = knew[off + e * HD];
        vj[j][e] = vnew[off + e * HD];
      }
    }
#pragma unroll
    for (int i = 0; i < GHW; ++i) {
      const int gh = min(wave + 4 * i, GH - 1);
#pragma unroll
      for (int e = 0; e < 2; ++e) qc[i][e] = q[((size_t)b * Hq + h0 + gh) * D + m2 + e * HD];
    }
  }

  const int start = cu[b], P = cu[b + 1] - start;
  // rotary coefficients (Section 2.1's decoder layers use RoPE; the cached
  // prefix keys are stored rotated): the query sits at the last cascade
  // position, cascade key j at P + j (one position, P, per layer otherwise).
  // Loaded with the first K/V rows: no round trip of their own.
  const int pos_q = cascade ? P + nctx - 1 : P;
  f32x4 rq[NKC / 2][4];
#pragma unroll
  for (int kc = 0; kc < NKC / 2; ++kc)
#pragma unroll
    for (int w = 0; w < 4; ++w)
      rq[kc][w] = *reinterpret_cast<const f32x4 *>(rope + ((size_t)pos_q * HD + 32 * kc + 8 * g) * 2 + 4 * w);
  float2 rcj[kMaxLayers], rcq;
  if (casc) {
#pragma unroll
    for (int j = 0; j < kMaxLayers; ++j)
      rcj[j] = *reinterpret_cast<const float2 *>(rope + ((size_t)(cascade ? P + min(j, nctx - 1) : P) * HD + m2) * 2);
    rcq = *reinterpret_cast<const float2 *>(rope + ((size_t)pos_q * HD + m2) * 2);
  }
  const int span = kAttnChunk * cpw;
  const int nv = max(1, min((P + span - 1) / span, nch));
  if (ch >= nv) return;  // chunk beyond this sequence's prefix
  const int base = ch * span;
  const int nsc = P > 0 ? min(cpw, (P - base + kAttnChunk - 1) / kAttnChunk) : 0;
  float *part_o = part;
  float *part_ml = part + (size_t)gridDim.z * Hq * nch_ld * D;

  const size_t rs = (size_t)Hkv * D;
  const bf16_t *kb = Kc + ((size_t)start * Hkv + c) * D;
  const bf16_t *vb = Vc + ((size_t)start * Hkv + c) * D;
  // sub-chunk sc: K pieces (key 16t + r of the wave's 32, dims 32kc + 8g) and V
  // pieces (row p / VPR, piece p % VPR for p = lane + 64i), clamped in bounds
  auto load_rows = [&](int sc, u32x4 (&ka)[2][NKC], u32x4 (&vv)[NVL]) {
    const int k0 = base + sc * kAttnChunk + wave * kWaveKeys;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const size_t key = (size_t)min(k0 + 16 * t + r, P - 1);
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc)
        ka[t][kc] = *reinterpret_cast<const u32x4 *>(kb + key * rs + 32 * kc + 8 * g);
    }
#pragma unroll
    for (int i = 0; i < NVL; ++i) {
      const int pc = lane + 64 * i;
      const size_t key = (size_t)min(k0 + pc / VPR, P - 1);
      vv[i] = *reinterpret_cast<const u32x4 *>(vb + key * rs + 8 * (pc % VPR));
    }
  };
  u32x4 ka[2][NKC], vv[NVL];
  if (nsc > 0) load_rows(0, ka, vv);

  // ---- chunk 0: the cascade keys, fp32 on the vector ALU -> partial slot 4 ----
  if (casc) {
#pragma unroll
    for (int i = 0; i < GHW; ++i) {
      const int gh = wave + 4 * i;
      if (gh >= GH) break;
      // rotate-half on the pair (m, m + D/2)
      const float q0 = qc[i][0] * rcq.x - qc[i][1] * rcq.y, q1 = qc[i][1] * rcq.x + qc[i][0] * rcq.y;
      float sj[kMaxLayers];
#pragma unroll
      for (int j = 0; j < kMaxLayers; ++j) {
        const float k0 = kj[j][0] * rcj[j].x - kj[j][1] * rcj[j].y;
        const float k1 = kj[j][1] * rcj[j].x + kj[j][0] * rcj[j].y;
        float d = cact ? (q0 * k0 + q1 * k1) * qscale : 0.f;
        d = group_sum<64>(d);
        sj[j] = j < nctx ? d : -INFINITY;
      }
      float m = -INFINITY;
#pragma unroll
      for (int j = 0; j < kMaxLayers; ++j) m = fmaxf(m, sj[j]);
      float L = 0.f, o[2] = {0.f, 0.f};
#pragma unroll
      for (int j = 0; j < kMaxLayers; ++j) {
        const float pj = sexp2(sj[j], m);
        L += pj;
#pragma unroll
        for (int e = 0; e < 2; ++e) o[e] += pj * vj[j][e];
      }
      if (cact) {
        s_o[4][gh][m2] = o[0];
        s_o[4][gh][m2 + HD] = o[1];
      }
      if (lane == 0) {
        s_m[4][gh] = m;
        s_l[4][gh] = L;
      }
    }
  }

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
      const uint16_t h0b = f2bf(a0), h1b = f2bf(a1);
      hw[e / 2] = (uint32_t)h0b | ((uint32_t)h1b << 16);
      lw[e / 2] = pack_bf16(a0 - bf2f(h0b), a1 - bf2f(h1b));
    }
    qh[kc] = u32x4{hw[0], hw[1], hw[2], hw[3]};
    ql[kc] = u32x4{lw[0], lw[1], lw[2], lw[3]};
  }

  // ---- prefix keys: online softmax over sub-chunks, next rows in flight ----------
  float m = -INFINITY, l = 0.f;  // head r: running max (uniform over g), this lane's sum
  f32x4 oacc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) oacc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  unsigned char *sv = s_v[wave];
  for (int sc = 0; sc < nsc; ++sc) {
    u32x4 kn[2][NKC], vn[NVL];
    load_rows(sc + 1, kn, vn);  // unconditional: clamped rows past the end
    // V rows of this sub-chunk -> LDS (LDS ops of one wave complete in order, so
    // the previous sub-chunk's reads are done before these writes land)
#pragma unroll
    for (int i = 0; i < NVL; ++i) {
      const int pc = lane + 64 * i;
      *reinterpret_cast<u32x4 *>(sv + (pc / VPR) * RSB + 16 * (pc % VPR)) = vv[i];
    }
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka[0][kc]),
                                                   __builtin_bit_cast(bf16x8, qh[kc]), s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka[1][kc]),
                                                   __builtin_bit_cast(bf16x8, qh[kc]), s1, 0, 0, 0);
      s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka[0][kc]),
                                                   __builtin_bit_cast(bf16x8, ql[kc]), s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka[1][kc]),
                                                   __builtin_bit_cast(bf16x8, ql[kc]), s1, 0, 0, 0);
    }
    // lane holds S[key 4g+v (+16 for s1)][head r]; mask keys past P
    const int kq = base + sc * kAttnChunk + wave * kWaveKeys + 4 * g;
    float sv8[8];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      sv8[v] = kq + v < P ? s0[v] : -INFINITY;
      sv8[4 + v] = kq + 16 + v < P ? s1[v] : -INFINITY;
    }
    float mx = m;
#pragma unroll
    for (int v = 0; v < 8; ++v) mx = fmaxf(mx, sv8[v]);
    mx = xor32_max(xor16_max(mx));
    const float alpha = sexp2(m, mx);
    m = mx;
    uint32_t pw[4];
    float ps = 0.f;
#pragma unroll
    for (int v = 0; v < 8; v += 2) {
      const uint16_t p0 = f2bf(sexp2(sv8[v], mx)), p1 = f2bf(sexp2(sv8[v + 1], mx));
      ps += bf2f(p0) + bf2f(p1);
      pw[v / 2] = (uint32_t)p0 | ((uint32_t)p1 << 16);
    }
    l = l * alpha + ps;
    const u32x4 pb = {pw[0], pw[1], pw[2], pw[3]};
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      // A = V^T: dim 16dt + r, keys (4g + j) and (16 + 4g + j), j < 4
      const unsigned char *col = sv + 2 * (16 * dt + r);
      uint32_t aw[4];
#pragma unroll
      for (int j = 0; j < 4; j += 2) {
        const uint16_t v0 = *reinterpret_cast<const uint16_t *>(col + (4 * g + j) * RSB);
        const uint16_t v1 = *reinterpret_cast<const uint16_t *>(col + (4 * g + j + 1) * RSB);
        const uint16_t v2 = *reinterpret_cast<const uint16_t *>(col + (16 + 4 * g + j) * RSB);
        const uint16_t v3 = *reinterpret_cast<const uint16_t *>(col + (17 + 4 * g + j) * RSB);
        aw[j / 2] = (uint32_t)v0 | ((uint32_t)v1 << 16);
        aw[2 + j / 2] = (uint32_t)v2 | ((uint32_t)v3 << 16);
      }
      const u32x4 av = {aw[0], aw[1], aw[2], aw[3]};
      oacc[dt] *= alpha;
      oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av),
                                                         __builtin_bit_cast(bf16x8, pb), oacc[dt],
                                                         0, 0, 0);
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc) ka[t][kc] = kn[t][kc];
#pragma unroll
    for (int i = 0; i < NVL; ++i) vv[i] = vn[i];
  }
  // wave partial: O^T[16dt + 4g + v][head r], max m, sum over the 4 lanes of head r
  l = xor32_sum(xor16_sum(l));
  if (r < GH) {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int v = 0; v < 4; ++v) s_o[wave][r][16 * dt + 4 * g + v] = oacc[dt][v];
    if (g == 0) {
      s_m[wave][r] = m;
      s_l[wave][r] = l;
    }
  }
  __syncthreads();

  // ---- this workgroup's result: the output row, or its partial ----------------
  const bool whole = nv == 1;
  const int nslot = casc ? 5 : 4;
  for (int idx = tid; idx < GH * D; idx += 256) {
    const int gh = idx / D, e = idx % D;
    float M = -INFINITY;
    for (int w = 0; w < nslot; ++w) M = fmaxf(M, s_m[w][gh]);
    float acc = 0.f, L = 0.f;
    for (int w = 0; w < nslot; ++w) {
      const float sw = sexp2(s_m[w][gh], M);
      acc += sw == 0.f ? 0.f : sw * s_o[w][gh][e];
      L += sw * s_l[w][gh];
    }
    if (whole) {
      out[(size_t)b * Hq * D + (size_t)(h0 + gh) * D + e] = f2bf(acc / L);
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


// ---- chunk merge (second launch) -------------------------------------------------
// A sequence whose prefix spans several workgroups leaves one partial per
// workgroup: o (scaled to that workgroup's max), max and sum per head.  This
// launch combines them in chunk order, 16 per round trip.  Sequences that fit
// one workgroup wrote their rows directly and are skipped.  Keeping the merge in
// its own launch means no workgroup ever waits on another: the kernel boundary
// publishes the partials once, where per-workgroup device-scope fences would
// write back the L2 once per workgroup.  LOG2: maxima in log2 units.
template <typename T, bool LOG2>
__global__ __launch_bounds__(256) void k_attn_merge(const float *__restrict__ part, int nch_ld,
                                                    const int32_t *__restrict__ cu, int span,
                                                    int nwg, T *__restrict__ out, int Hq, int D) {
  const int b = blockIdx.y;
  const int P = cu[b + 1] - cu[b];
  const int nv = max(1, min((P + span - 1) / span, nwg));
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (nv == 1 || idx >= Hq * D / 2) return;
  const int h = (2 * idx) / D, e = (2 * idx) % D;
  const float *po = part + ((size_t)b * Hq + h) * nch_ld * D + e;
  const float *pml = part + (size_t)gridDim.y * Hq * nch_ld * D + ((size_t)b * Hq + h) * nch_ld * 2;
  auto ex = [](float m, float M) {
    return m == -INFINITY ? 0.f : (LOG2 ? __builtin_amdgcn_exp2f(m - M) : expf(m - M));
  };
  float M = -INFINITY, L = 0.f, ax = 0.f, ay = 0.f;
  for (int c0 = 0; c0 < nv; c0 += 16) {
    float2 ov[16], ml[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int k = min(c0 + u, nv - 1);
      ov[u] = *reinterpret_cast<const float2 *>(po + (size_t)k * D);
      ml[u] = *reinterpret_cast<const float2 *>(pml + 2 * k);
    }
    float Mn = M;
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (c0 + u < nv) Mn = fmaxf(Mn, ml[u].x);
    const float rr = ex(M, Mn);
    L *= rr;
    ax *= rr;
    ay *= rr;
#pragma unroll
    for (int u = 0; u < 16; ++u)
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
                         int nch_ld, int cpw, void *out, int B, int Hq, int Hkv,
                         hipStream_t s) {
  const int G = Hq / Hkv;
  const int GH = (G % 4 == 0) ? 4 : (G % 2 == 0 ? 2 : 1);
  const int nwg = nch < 1 ? 1 : (nch + cpw - 1) / cpw;
  const dim3 grid(nwg, Hkv * (G / GH), B);
#define FE_ATTN(GHV)                                                                            \
  hipLaunchKernelGGL((k_attn<T, D, GHV>), grid, dim3(256), 0, s, (const T *)K, (const T *)V, cu, \
                     q, knew, vnew, nctx, part, nwg, nch_ld, cpw, (T *)out, Hq, Hkv)
  if (GH == 4) FE_ATTN(4);
  else if (GH == 2) FE_ATTN(2);
  else FE_ATTN(1);
#undef FE_ATTN
  return hipGetLastError();
}

template <int D>
static hipError_t attn_mma_t(const void *K, const void *V, const int32_t *cu, const float *q,
                             const float *knew, const float *vnew, int nctx, float *part, int nch,
                             int nch_ld, int cpw, void *out, int B, int Hq, int Hkv,
                             const float *rope, int cascade, hipStream_t s) {
  const int G = Hq / Hkv;
  const int GH = G % 16 == 0 ? 16 : G % 8 == 0 ? 8 : G % 4 == 0 ? 4 : G % 2 == 0 ? 2 : 1;
  const int nwg = nch < 1 ? 1 : (nch + cpw - 1) / cpw;
  const dim3 grid(nwg, Hkv * (G / GH), B);
#define FE_ATTN(GHV)                                                                             \
  hipLaunchKernelGGL((k_attn_mma<D, GHV>), grid, dim3(256), 0, s, (const bf16_t *)K,             \
                     (const bf16_t *)V, cu, q, knew, vnew, nctx, part, nwg, nch_ld, cpw, \
                     (bf16_t *)out, Hq, Hkv, rope, cascade)
  switch (GH) {
    case 16: FE_ATTN(16); break;
    case 8: FE_ATTN(8); break;
    case 4: FE_ATTN(4); break;
    case 2: FE_ATTN(2); break;
    default: FE_ATTN(1); break;
  }
#undef FE_ATTN
  return hipGetLastError();
}

// Enough workgroups to keep every CU streaming (about one each) and no more:
// a sequence split over more workgroups only adds partials to merge.
int attention_cpw(int B, int Hkv, int ngroups, int nch) {
  constexpr long kTargetWorkgroups = 256;
  const long cols = (long)B * Hkv * ngroups;
  long cpw = (cols * nch + kTargetWorkgroups - 1) / kTargetWorkgroups;
  if (cpw > nch) cpw = nch;
  return cpw < 1 ? 1 : (int)cpw;
}

hipError_t attention(int dt, const void *K, const void *V, const int32_t *cu, const float *q,
                     const float *knew, const float *vnew, int nctx, float *part, int nch,
                     int nch_ld, int cpw, void *out, int B, int Hq, int Hkv, int D,
                     const float *rope, int cascade, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (cpw < 1) cpw = 1;
  hipError_t e;
  if (dt)
    e = D == 128 ? attn_mma_t<128>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld, cpw, out, B,
                                   Hq, Hkv, rope, cascade, s)
                 : attn_mma_t<64>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld, cpw, out, B,
                                  Hq, Hkv, rope, cascade, s);
  else
    e = D == 128 ? attn_t<float, 128>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld, cpw, out,
                                      B, Hq, Hkv, s)
                 : attn_t<float, 64>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld, cpw, out,
                                     B, Hq, Hkv, s);
  if (e != hipSuccess) return e;
  const int nwg = nch < 1 ? 1 : (nch + cpw - 1) / cpw;
  if (nwg == 1) return hipSuccess;  // every sequence fits one workgroup
  const dim3 grid((Hq * D / 2 + 255) / 256, B);
  if (dt)
    hipLaunchKernelGGL((k_attn_merge<bf16_t, true>), grid, dim3(256), 0, s, part, nch_ld, cu,
                       kAttnChunk * cpw, nwg, (bf16_t *)out, Hq, D);
  else
    hipLaunchKernelGGL((k_attn_merge<float, false>), grid, dim3(256), 0, s, part, nch_ld, cu,
                       kAttnChunk * cpw, nwg, (float *)out, Hq, D);
  return hipGetLastError();
}

}  // namespace fe
