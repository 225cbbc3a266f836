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
//    together so every K/V byte is read once.  Each wave takes 32 keys: 8 lanes
//    per key row (D/8 dims each, 16-byte loads, the row contiguous), 8 keys
//    per load step, K and V loads issued together.
//  * Dot products reduce over the 8 lanes of a key with xor-shuffles; the
//    softmax max/sum and the value sums reduce across key slots with
//    xor-shuffles, then across the 4 waves in LDS.  Each chunk leaves
//    (sum, max, o[D]) per head in the workspace.
//  * Split-K completion: every chunk workgroup bumps a counter after a
//    release fence; the last one (acquire fence) merges all chunk partials and
//    the nctx cascade keys, held in fp32, in a fixed order, writes the output
//    row and resets the counter for the next launch.  A sequence with an empty
//    prefix still runs chunk 0, which carries no keys.
#include "fe_internal.h"

namespace fe {

template <typename T, int D> struct KvRow {
  static constexpr int DL = D / 8;                      // dims per lane
  static constexpr int NV = DL * sizeof(T) / 16;        // 16-byte loads per lane
  uint32_t w[NV * 4];  // plain words: element access by index never touches a vector
  __device__ __forceinline__ void load(const T *p) {
    const u32x4 *q = reinterpret_cast<const u32x4 *>(p);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const u32x4 v = q[i];
      w[4 * i + 0] = v.x;
      w[4 * i + 1] = v.y;
      w[4 * i + 2] = v.z;
      w[4 * i + 3] = v.w;
    }
  }
  __device__ __forceinline__ float at(int e) const {
    if constexpr (sizeof(T) == 2) {
      const uint32_t u = w[e / 2];
      return (e & 1) ? __uint_as_float(u & 0xffff0000u) : __uint_as_float(u << 16);
    } else {
      return __uint_as_float(w[e]);
    }
  }
};

constexpr int kWaveKeys = kAttnChunk / 4;   // keys per wave
constexpr int kSteps = kWaveKeys / 8;       // load steps per wave

__device__ __forceinline__ float scaled_exp(float m, float M) {
  return m == -INFINITY ? 0.f : expf(m - M);
}

template <typename T, int D, int GH>
__global__ __launch_bounds__(256) void k_attn(const T *__restrict__ Kc, const T *__restrict__ Vc,
                                              const int32_t *__restrict__ cu,
                                              const float *__restrict__ q,
                                              const float *__restrict__ knew,
                                              const float *__restrict__ vnew, int nctx,
                                              float *__restrict__ part, int nch, int nch_ld,
                                              int *__restrict__ counters, T *__restrict__ out,
                                              int Hq, int Hkv) {
  constexpr int DL = D / 8;
  __shared__ float s_m[4][GH], s_l[4][GH];
  __shared__ float s_o[4][GH][D];
  __shared__ float s_sc[GH][kMaxLayers];
  __shared__ int s_last;

  const int G = Hq / Hkv, ngrp = G / GH;
  const int ch = blockIdx.x, c = blockIdx.y / ngrp, hg = blockIdx.y % ngrp, b = blockIdx.z;
  const int start = cu[b], P = cu[b + 1] - start;
  const int nv = max(1, min((P + kAttnChunk - 1) / kAttnChunk, nch));
  if (ch >= nv) return;  // chunk beyond this sequence's prefix
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, slot = lane >> 3, dp = lane & 7;
  const int h0 = c * G + hg * GH;
  const float scale = rsqrtf((float)D);
  const int key0 = ch * kAttnChunk + wave * kWaveKeys;

  // ---- this wave's 32 keys -------------------------------------------------
  const size_t rowstride = (size_t)Hkv * D;
  const T *kbase = Kc + ((size_t)start * Hkv + c) * D + dp * DL;
  const T *vbase = Vc + ((size_t)start * Hkv + c) * D + dp * DL;
  // Rows are loaded unconditionally at clamped keys (missing keys get weight 0
  // below); an empty prefix reads nothing.
  KvRow<T, D> kr[kSteps], vr[kSteps];
  if (P > 0) {
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      const int key = min(key0 + st * 8 + slot, P - 1);
      kr[st].load(kbase + (size_t)key * rowstride);
      vr[st].load(vbase + (size_t)key * rowstride);
    }
  }
  float qv[GH][DL];
#pragma unroll
  for (int gh = 0; gh < GH; ++gh)
#pragma unroll
    for (int e = 0; e < DL; ++e) qv[gh][e] = q[((size_t)b * Hq + h0 + gh) * D + dp * DL + e];
  // cascade keys of head group member `wave` (waves < GH): loaded now, scored
  // below, so that the final merge needs no further inputs but the partials
  constexpr int DPL = D / 64;
  float qd[DPL], kd[kMaxLayers][DPL];
  if (wave < GH) {
#pragma unroll
    for (int t = 0; t < DPL; ++t) qd[t] = q[((size_t)b * Hq + h0 + wave) * D + lane * DPL + t];
#pragma unroll
    for (int j = 0; j < kMaxLayers; ++j)
#pragma unroll
      for (int t = 0; t < DPL; ++t)
        kd[j][t] = knew[(((size_t)b * nctx + min(j, nctx - 1)) * Hkv + c) * D + lane * DPL + t];
  }

  float s[kSteps][GH];
#pragma unroll
  for (int st = 0; st < kSteps; ++st)
#pragma unroll
    for (int gh = 0; gh < GH; ++gh) {
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < DL; ++e) acc += qv[gh][e] * kr[st].at(e);
      acc += __shfl_xor(acc, 1);
      acc += __shfl_xor(acc, 2);
      acc += __shfl_xor(acc, 4);
      const int key = key0 + st * 8 + slot;
      s[st][gh] = key < P ? acc * scale : -INFINITY;
    }
  float mx[GH], l[GH], o[GH][DL];
#pragma unroll
  for (int gh = 0; gh < GH; ++gh) {
    float m = -INFINITY;
#pragma unroll
    for (int st = 0; st < kSteps; ++st) m = fmaxf(m, s[st][gh]);
    m = fmaxf(m, __shfl_xor(m, 8));
    m = fmaxf(m, __shfl_xor(m, 16));
    m = fmaxf(m, __shfl_xor(m, 32));
    mx[gh] = m;
    float sum = 0.f;
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      const float p = scaled_exp(s[st][gh], m);
      s[st][gh] = p;
      sum += p;
    }
    sum += __shfl_xor(sum, 8);
    sum += __shfl_xor(sum, 16);
    sum += __shfl_xor(sum, 32);
    l[gh] = sum;
#pragma unroll
    for (int e = 0; e < DL; ++e) o[gh][e] = 0.f;
  }
  if (P > 0) {
#pragma unroll
    for (int st = 0; st < kSteps; ++st)
#pragma unroll
      for (int e = 0; e < DL; ++e) {
        const float ve = vr[st].at(e);
#pragma unroll
        for (int gh = 0; gh < GH; ++gh) o[gh][e] += s[st][gh] * ve;  // weight 0 past P
      }
  }
#pragma unroll
  for (int gh = 0; gh < GH; ++gh)
#pragma unroll
    for (int e = 0; e < DL; ++e) {
      float v = o[gh][e];
      v += __shfl_xor(v, 8);
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      o[gh][e] = v;
    }
  if (slot == 0) {
#pragma unroll
    for (int gh = 0; gh < GH; ++gh) {
#pragma unroll
      for (int e = 0; e < DL; ++e) s_o[wave][gh][dp * DL + e] = o[gh][e];
      if (dp == 0) {
        s_m[wave][gh] = mx[gh];
        s_l[wave][gh] = l[gh];
      }
    }
  }
  if (wave < GH) {  // scores of the cascade keys for head h0 + wave
#pragma unroll
    for (int j = 0; j < kMaxLayers; ++j) {
      float v = 0.f;
#pragma unroll
      for (int t = 0; t < DPL; ++t) v += qd[t] * kd[j][t];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
      if (lane == 0) s_sc[wave][j] = j < nctx ? v * scale : -INFINITY;
    }
  }
  __syncthreads();

  // ---- merge the 4 waves into this chunk's partial: [o[D], max, sum] --------
  for (int idx = tid; idx < GH * (D + 2); idx += 256) {
    const int gh = idx / (D + 2), e = idx % (D + 2);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, s_m[w][gh]);
    float acc = 0.f;
    if (e == D) {
      acc = M;
    } else {
#pragma unroll
      for (int w = 0; w < 4; ++w)
        acc += scaled_exp(s_m[w][gh], M) * (e < D ? s_o[w][gh][e] : s_l[w][gh]);
    }
    part[(((size_t)b * Hq + h0 + gh) * nch_ld + ch) * (D + 2) + e] = acc;
  }

  // ---- split-K completion ---------------------------------------------------
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const int old = atomicAdd(&counters[((size_t)b * Hkv + c) * ngrp + hg], 1);
    s_last = (old == nv - 1);
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();

  // ---- last chunk workgroup: merge every chunk and the cascade keys ---------
  // Thread (gh, e) reads what it needs in one round trip (8 chunks per group,
  // clamped in-bounds indices, unused values masked) and merges with a running
  // max in a fixed order.
  for (int idx = tid; idx < GH * D; idx += 256) {
    const int gh = idx / D, e = idx % D, h = h0 + gh;
    const float *pp = part + ((size_t)b * Hq + h) * nch_ld * (D + 2);
    float vv[kMaxLayers];
#pragma unroll
    for (int j = 0; j < kMaxLayers; ++j)
      vv[j] = vnew[(((size_t)b * nctx + min(j, nctx - 1)) * Hkv + c) * D + e];
    float M = -INFINITY;
#pragma unroll
    for (int j = 0; j < kMaxLayers; ++j) M = fmaxf(M, s_sc[gh][j]);
    float L = 0.f, acc = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxLayers; ++j) {
      const float w = scaled_exp(s_sc[gh][j], M);
      L += w;
      acc += w * vv[j];
    }
    for (int k0 = 0; k0 < nv; k0 += 8) {
      float ov[8], mv[8], lv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float *pk = pp + (size_t)min(k0 + u, nv - 1) * (D + 2);
        ov[u] = pk[e];
        mv[u] = pk[D];
        lv[u] = pk[D + 1];
      }
      float Mn = M;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (k0 + u < nv) Mn = fmaxf(Mn, mv[u]);
      const float rs = scaled_exp(M, Mn);
      L *= rs;
      acc *= rs;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (k0 + u < nv) {
          const float w = scaled_exp(mv[u], Mn);
          L += lv[u] * w;
          acc += ov[u] * w;
        }
      M = Mn;
    }
    out[(size_t)b * Hq * D + (size_t)h * D + e] = Elt<T>::from_f(acc / L);
  }
  if (tid == 0) counters[((size_t)b * Hkv + c) * ngrp + hg] = 0;
}

template <typename T, int D>
static hipError_t attn_t(const void *K, const void *V, const int32_t *cu, const float *q,
                         const float *knew, const float *vnew, int nctx, float *part, int nch,
                         int nch_ld, int *counters, void *out, int B, int Hq, int Hkv,
                         hipStream_t s) {
  const int G = Hq / Hkv;
  const int GH = (G % 4 == 0) ? 4 : (G % 2 == 0 ? 2 : 1);
  const int nchl = nch < 1 ? 1 : nch;
  const dim3 grid(nchl, Hkv * (G / GH), B);
#define FE_ATTN(GHV)                                                                            \
  hipLaunchKernelGGL((k_attn<T, D, GHV>), grid, dim3(256), 0, s, (const T *)K, (const T *)V, cu, \
                     q, knew, vnew, nctx, part, nchl, nch_ld, counters, (T *)out, Hq, Hkv)
  if (GH == 4) FE_ATTN(4);
  else if (GH == 2) FE_ATTN(2);
  else FE_ATTN(1);
#undef FE_ATTN
  return hipGetLastError();
}

hipError_t attention(int dt, const void *K, const void *V, const int32_t *cu, const float *q,
                     const float *knew, const float *vnew, int nctx, float *part, int nch,
                     int nch_ld, int *counters, void *out, int B, int Hq, int Hkv, int D,
                     hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (dt)
    return D == 128 ? attn_t<bf16_t, 128>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld,
                                          counters, out, B, Hq, Hkv, s)
                    : attn_t<bf16_t, 64>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld,
                                         counters, out, B, Hq, Hkv, s);
  return D == 128 ? attn_t<float, 128>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld,
                                       counters, out, B, Hq, Hkv, s)
                  : attn_t<float, 64>(K, V, cu, q, knew, vnew, nctx, part, nch, nch_ld, counters,
                                      out, B, Hq, Hkv, s);
}

}  // namespace fe
