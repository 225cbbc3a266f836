// fe_attn.hip -- GQA decode attention of a cascade layer over its prefix KV
// cache plus the cascade entries (gfx950).
//
// Layer i's query (one row per sequence, H_q heads) attends to the P_b cached
// prefix keys of its own cache and to the nctx keys it projected from the
// cascade states (Section 2.1; the cache is per layer because every L_i has
// its own parameters).  The prefix part is flash-decoding:
//
//  * one wave per (sequence, KV head, head group, chunk of 64 keys); the GH
//    query heads that share a KV head are processed together, so every K/V
//    byte is loaded once per chunk;
//  * 8 lanes cover one key row (D/8 dims each, 16-byte vector loads, a whole
//    row contiguous), 8 keys per load step;
//  * dot products are reduced over the 8 lanes of a key with xor-shuffles,
//    the softmax max/sum over the chunk with xor-shuffles across key slots,
//    and the value accumulation likewise; the chunk leaves (max, sum, o[D])
//    per head.
//
// The combine kernel merges the chunk partials and the nctx cascade keys (held
// in fp32) with the usual max-rescaling, in a fixed order.
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

template <typename T, int D, int GH>
__global__ __launch_bounds__(64) void k_attn_prefix(const T *__restrict__ Kc,
                                                    const T *__restrict__ Vc,
                                                    const int32_t *__restrict__ cu,
                                                    const float *__restrict__ q,
                                                    float *__restrict__ part, int Hq, int Hkv,
                                                    int nch_ld) {
  constexpr int DL = D / 8;
  constexpr int STEPS = kAttnChunk / 8;
  const int G = Hq / Hkv, ngrp = G / GH;
  const int ch = blockIdx.x, c = blockIdx.y / ngrp, hg = blockIdx.y % ngrp, b = blockIdx.z;
  const int start = cu[b], P = cu[b + 1] - start;
  const int key0 = ch * kAttnChunk;
  if (key0 >= P) return;  // chunk beyond this sequence's prefix: nothing to write
  const int lane = threadIdx.x, slot = lane >> 3, dp = lane & 7;
  const int h0 = c * G + hg * GH;
  const float scale = rsqrtf((float)D);

  float qv[GH][DL];
#pragma unroll
  for (int gh = 0; gh < GH; ++gh)
#pragma unroll
    for (int e = 0; e < DL; ++e) qv[gh][e] = q[((size_t)b * Hq + h0 + gh) * D + dp * DL + e];

  const size_t rowstride = (size_t)Hkv * D;
  const T *kbase = Kc + ((size_t)start * Hkv + c) * D + dp * DL;
  const T *vbase = Vc + ((size_t)start * Hkv + c) * D + dp * DL;

  KvRow<T, D> kr[STEPS];
#pragma unroll
  for (int st = 0; st < STEPS; ++st) {
    const int key = key0 + st * 8 + slot;
    if (key < P) kr[st].load(kbase + (size_t)key * rowstride);
  }
  float s[STEPS][GH];
#pragma unroll
  for (int st = 0; st < STEPS; ++st) {
#pragma unroll
    for (int gh = 0; gh < GH; ++gh) {
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < DL; ++e) acc += qv[gh][e] * kr[st].at(e);
      s[st][gh] = acc;
    }
  }
#pragma unroll
  for (int st = 0; st < STEPS; ++st)
#pragma unroll
    for (int gh = 0; gh < GH; ++gh) {
      float v = s[st][gh];
      v += __shfl_xor(v, 1);
      v += __shfl_xor(v, 2);
      v += __shfl_xor(v, 4);
      const int key = key0 + st * 8 + slot;
      s[st][gh] = key < P ? v * scale : -INFINITY;
    }
  float mx[GH], l[GH];
#pragma unroll
  for (int gh = 0; gh < GH; ++gh) {
    float m = -INFINITY;
#pragma unroll
    for (int st = 0; st < STEPS; ++st) m = fmaxf(m, s[st][gh]);
    m = fmaxf(m, __shfl_xor(m, 8));
    m = fmaxf(m, __shfl_xor(m, 16));
    m = fmaxf(m, __shfl_xor(m, 32));
    mx[gh] = m;
    float sum = 0.f;
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
      const float p = expf(s[st][gh] - m);  // exp(-inf) = 0 for missing keys
      s[st][gh] = p;
      sum += p;
    }
    sum += __shfl_xor(sum, 8);
    sum += __shfl_xor(sum, 16);
    sum += __shfl_xor(sum, 32);
    l[gh] = sum;
  }
  float o[GH][DL];
#pragma unroll
  for (int gh = 0; gh < GH; ++gh)
#pragma unroll
    for (int e = 0; e < DL; ++e) o[gh][e] = 0.f;
#pragma unroll
  for (int st = 0; st < STEPS; ++st) {
    const int key = key0 + st * 8 + slot;
    if (key < P) {
      KvRow<T, D> vr;
      vr.load(vbase + (size_t)key * rowstride);
#pragma unroll
      for (int e = 0; e < DL; ++e) {
        const float ve = vr.at(e);
#pragma unroll
        for (int gh = 0; gh < GH; ++gh) o[gh][e] += s[st][gh] * ve;
      }
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
      float *dst = part + (((size_t)b * Hq + h0 + gh) * nch_ld + ch) * (D + 2);
#pragma unroll
      for (int e = 0; e < DL; ++e) dst[dp * DL + e] = o[gh][e];
      if (dp == 0) {
        dst[D] = mx[gh];
        dst[D + 1] = l[gh];
      }
    }
  }
}

// One workgroup of D threads per (query head, sequence); thread e owns dim e.
template <typename T, int D>
__global__ __launch_bounds__(D) void k_attn_combine(const float *__restrict__ part, int nch,
                                                    int nch_ld,
                                                    const int32_t *__restrict__ cu,
                                                    const float *__restrict__ q,
                                                    const float *__restrict__ knew,
                                                    const float *__restrict__ vnew, int nctx,
                                                    T *__restrict__ out, int Hq, int Hkv) {
  __shared__ float red[D / 64][kMaxLayers];
  __shared__ float sc[kMaxLayers];
  const int h = blockIdx.x, b = blockIdx.y, e = threadIdx.x;
  const int G = Hq / Hkv, c = h / G;
  const int P = cu[b + 1] - cu[b];
  const int nv = min((P + kAttnChunk - 1) / kAttnChunk, nch);
  const float scale = rsqrtf((float)D);
  const float qe = q[((size_t)b * Hq + h) * D + e];
  // scores of the cascade keys
  for (int j = 0; j < nctx; ++j) {
    float v = qe * knew[(((size_t)b * nctx + j) * Hkv + c) * D + e];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    if ((e & 63) == 0) red[e >> 6][j] = v;
  }
  __syncthreads();
  if (e < nctx) {
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < D / 64; ++w) v += red[w][e];
    sc[e] = v * scale;
  }
  __syncthreads();
  const float *pp = part + ((size_t)b * Hq + h) * nch_ld * (D + 2);
  float M = -INFINITY;
  for (int ch = 0; ch < nv; ++ch) M = fmaxf(M, pp[(size_t)ch * (D + 2) + D]);
  for (int j = 0; j < nctx; ++j) M = fmaxf(M, sc[j]);
  float L = 0.f, acc = 0.f;
  for (int ch = 0; ch < nv; ++ch) {
    const float *p = pp + (size_t)ch * (D + 2);
    const float w = expf(p[D] - M);
    L += p[D + 1] * w;
    acc += p[e] * w;
  }
  for (int j = 0; j < nctx; ++j) {
    const float w = expf(sc[j] - M);
    L += w;
    acc += w * vnew[(((size_t)b * nctx + j) * Hkv + c) * D + e];
  }
  out[(size_t)b * Hq * D + (size_t)h * D + e] = Elt<T>::from_f(acc / L);
}

template <typename T, int D>
static hipError_t attn_prefix_t(const void *K, const void *V, const int32_t *cu, const float *q,
                                float *part, int B, int Hq, int Hkv, int nch, int nch_ld,
                                hipStream_t s) {
  const int G = Hq / Hkv;
  const int GH = (G % 4 == 0) ? 4 : (G % 2 == 0 ? 2 : 1);
  const dim3 grid(nch, Hkv * (G / GH), B);
  if (GH == 4)
    hipLaunchKernelGGL((k_attn_prefix<T, D, 4>), grid, dim3(64), 0, s, (const T *)K, (const T *)V,
                       cu, q, part, Hq, Hkv, nch_ld);
  else if (GH == 2)
    hipLaunchKernelGGL((k_attn_prefix<T, D, 2>), grid, dim3(64), 0, s, (const T *)K, (const T *)V,
                       cu, q, part, Hq, Hkv, nch_ld);
  else
    hipLaunchKernelGGL((k_attn_prefix<T, D, 1>), grid, dim3(64), 0, s, (const T *)K, (const T *)V,
                       cu, q, part, Hq, Hkv, nch_ld);
  return hipGetLastError();
}

hipError_t attn_prefix(int dt, const void *K, const void *V, const int32_t *cu, const float *q,
                       float *part, int B, int Hq, int Hkv, int D, int nch, int nch_ld,
                       hipStream_t s) {
  if (nch <= 0 || B <= 0) return hipSuccess;
  if (dt) return D == 128 ? attn_prefix_t<bf16_t, 128>(K, V, cu, q, part, B, Hq, Hkv, nch, nch_ld, s)
                          : attn_prefix_t<bf16_t, 64>(K, V, cu, q, part, B, Hq, Hkv, nch, nch_ld, s);
  return D == 128 ? attn_prefix_t<float, 128>(K, V, cu, q, part, B, Hq, Hkv, nch, nch_ld, s)
                  : attn_prefix_t<float, 64>(K, V, cu, q, part, B, Hq, Hkv, nch, nch_ld, s);
}

hipError_t attn_combine(int dt, const float *part, int nch, int nch_ld, const int32_t *cu,
                        const float *q,
                        const float *knew, const float *vnew, int nctx, void *out, int B, int Hq,
                        int Hkv, int D, hipStream_t s) {
  const dim3 grid(Hq, B);
  if (dt) {
    if (D == 128)
      hipLaunchKernelGGL((k_attn_combine<bf16_t, 128>), grid, dim3(128), 0, s, part, nch, nch_ld, cu, q,
                         knew, vnew, nctx, (bf16_t *)out, Hq, Hkv);
    else
      hipLaunchKernelGGL((k_attn_combine<bf16_t, 64>), grid, dim3(64), 0, s, part, nch, nch_ld, cu, q,
                         knew, vnew, nctx, (bf16_t *)out, Hq, Hkv);
  } else {
    if (D == 128)
      hipLaunchKernelGGL((k_attn_combine<float, 128>), grid, dim3(128), 0, s, part, nch, nch_ld, cu, q,
                         knew, vnew, nctx, (float *)out, Hq, Hkv);
    else
      hipLaunchKernelGGL((k_attn_combine<float, 64>), grid, dim3(64), 0, s, part, nch, nch_ld, cu, q,
                         knew, vnew, nctx, (float *)out, Hq, Hkv);
  }
  return hipGetLastError();
}

}  // namespace fe
