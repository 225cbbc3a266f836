// fe_gemm.hip -- weight-streaming MFMA GEMM for gfx950 with fused epilogues.
//
// Every FC of the drafter (feature fusion and input FC of Eq. 1; Q/K/V, O,
// gate/up and down projections of each cascade layer; the shared LM head) is
// Y[M, C] = A[M, K] * W[C, K]^T with a weight matrix that is read exactly once
// per pass and a handful of activation rows (M = batch, or batch x cascade
// rows).  The kernel is built around streaming W from HBM:
//
//  * A wave owns NT tiles of 16 output columns and a K slice.  Lane (r, g)
//    (r = lane % 16, g = lane / 16) loads 16 contiguous bytes of weight row
//    r at K offset g*E of every K step (E = 8 bf16 or 4 fp32 elements), which
//    is exactly the B operand of v_mfma_f32_16x16x32_bf16 (one MFMA per step)
//    or of four v_mfma_f32_16x16x4_f32.  No LDS staging for weights, no
//    re-reads: each weight byte is loaded by one lane once.
//  * Activation rows are the A operand, loaded with the same (g, element) ->
//    k mapping, so the products pair up correctly whatever order the matrix
//    core sums the K elements in.  Rows beyond M are fed as zeros.
//  * Loads are double-buffered in registers: the next U steps of weights and
//    activations are in flight while the current U steps run on the MFMA.
//  * WK waves of a workgroup split K; their partial tiles are summed in LDS in
//    a fixed order (deterministic, no atomics), then an epilogue functor
//    consumes the [M, span] fp32 tile.
//  * Which weight row feeds a "virtual column" is the epilogue's choice:
//    Q/K tiles pair rotary halves (dims m and m + D/2) inside one 16-column
//    tile; gate/up tiles pair gate row c with up row c.
#include "fe_internal.h"

namespace fe {

template <typename T> __device__ __forceinline__ void mma16(f32x4 &acc, u32x4 a, u32x4 b);

template <> __device__ __forceinline__ void mma16<uint16_t>(f32x4 &acc, u32x4 a, u32x4 b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}

// Four K=4 fp32 MFMAs, one per element of the lanes' 16-byte fragments.  The
// elements are named explicitly: a loop over a vector element index here was
// compiled to four uses of element 0.
template <> __device__ __forceinline__ void mma16<float>(f32x4 &acc, u32x4 a, u32x4 b) {
  const f32x4 af = __builtin_bit_cast(f32x4, a), bf = __builtin_bit_cast(f32x4, b);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af.x, bf.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af.y, bf.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af.z, bf.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(af.w, bf.w, acc, 0, 0, 0);
}

__device__ __forceinline__ u32x4 ldg_stream(const u32x4 *p) { return __builtin_nontemporal_load(p); }

// ---------------------------------------------------------------------------
// Accumulation paths.  Both leave, in lane (r, g) of a wave, the 16x16 tiles
// acc[i][f] = rows 16i.. of A times weight rows of virtual columns c0+16f..,
// summed over this wave's share of K.
// ---------------------------------------------------------------------------

// Staged path (M <= 32): weights are read as 512-byte contiguous pieces of
// two rows per load instruction (the access pattern HBM streams best), parked
// in the wave's own padded LDS tile, and read back as MFMA B fragments; the
// next 512-byte chunk of every row is in flight while the current one is
// multiplied.  K is walked in chunks of KC elements, split over WK waves.
constexpr int kStageRowBytes = 512 + 16;  // padded LDS row: 16 rows hit distinct banks

template <typename T, int MT, int NT, class Epi>
__device__ __forceinline__ void accum_staged(const T *__restrict__ A, int lda, const ARows &ar_,
                                             int M, int K, const Epi &epi, int c0, int wk,
                                             int WKn, char *stage, f32x4 (&acc)[MT][NT]) {
  constexpr int E = Elt<T>::kPer16B;
  constexpr int KC = 32 * E;       // elements per chunk: 512 bytes of a row
  constexpr int KS = 4 * E;        // elements per MFMA step
  constexpr int STEPS = KC / KS;   // 8
  constexpr int NLD = NT * 8;      // load instructions per chunk (2 rows each)
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int half = lane >> 5, l32 = lane & 31;
  const int nchunk = (K + KC - 1) / KC;
  const int ch0 = (int)(((long)nchunk * wk) / WKn), ch1 = (int)(((long)nchunk * (wk + 1)) / WKn);
  if (ch0 >= ch1) return;
  const u32x4 *src[NLD];
#pragma unroll
  for (int j = 0; j < NLD; ++j)
    src[j] = reinterpret_cast<const u32x4 *>(epi.wrow(c0 + 2 * j + half)) + l32;
  const u32x4 *ap[MT];
  bool am[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int m = i * 16 + r;
    am[i] = m < M;
    ap[i] = reinterpret_cast<const u32x4 *>(A + (size_t)(am[i] ? ar_.row(m) : 0) * lda) + g;
  }
  const u32x4 zero = {0u, 0u, 0u, 0u};
  u32x4 wr[NLD], ar[STEPS][MT];
  auto load = [&](int ch) {
    const int kb = ch * KC;
    const bool wok = kb + l32 * E < K;
#pragma unroll
    for (int j = 0; j < NLD; ++j) wr[j] = wok ? ldg_stream(src[j] + ch * 32) : zero;
#pragma unroll
    for (int st = 0; st < STEPS; ++st)
#pragma unroll
      for (int i = 0; i < MT; ++i)
        ar[st][i] = (am[i] && kb + st * KS + g * E < K) ? ap[i][ch * 32 + st * 4] : zero;
  };
  load(ch0);
  for (int ch = ch0; ch < ch1; ++ch) {
    // the previous chunk's LDS reads are complete before its rows are overwritten
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int j = 0; j < NLD; ++j)
      *reinterpret_cast<u32x4 *>(stage + (2 * j + half) * kStageRowBytes + l32 * 16) = wr[j];
    u32x4 ac[STEPS][MT];
#pragma unroll
    for (int st = 0; st < STEPS; ++st)
#pragma unroll
      for (int i = 0; i < MT; ++i) ac[st][i] = ar[st][i];
    // this chunk's rows are in LDS before any lane reads them
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (ch + 1 < ch1) load(ch + 1);
    const int nst = min(STEPS, (K - ch * KC) / KS);
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
      if (st < nst) {
#pragma unroll
        for (int f = 0; f < NT; ++f) {
          const u32x4 bfr = *reinterpret_cast<const u32x4 *>(
              stage + (f * 16 + r) * kStageRowBytes + st * 64 + g * 16);
#pragma unroll
          for (int i = 0; i < MT; ++i) mma16<T>(acc[i][f], ac[st][i], bfr);
        }
      }
    }
  }
}

// Direct path (larger M): lane (r, g) loads 16 bytes of weight row r per
// K step straight into the B operand; U steps double-buffered in registers.
template <typename T, int MT, int NT, int U, class Epi>
__device__ __forceinline__ void accum_direct(const T *__restrict__ A, int lda, const ARows &ar_,
                                             int M, int K, const Epi &epi, int c0, int wk,
                                             int WKn, f32x4 (&acc)[MT][NT]) {
  constexpr int E = Elt<T>::kPer16B;
  constexpr int KS = 4 * E;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int nsteps = K / KS;
  const int s0 = (int)(((long)nsteps * wk) / WKn);
  const int s1 = (int)(((long)nsteps * (wk + 1)) / WKn);
  const u32x4 *wp[NT];
#pragma unroll
  for (int f = 0; f < NT; ++f)
    wp[f] = reinterpret_cast<const u32x4 *>(epi.wrow(c0 + f * 16 + r)) + g;
  const u32x4 *ap[MT];
  bool am[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int m = i * 16 + r;
    am[i] = m < M;
    ap[i] = reinterpret_cast<const u32x4 *>(A + (size_t)(am[i] ? ar_.row(m) : 0) * lda) + g;
  }
  const u32x4 zero = {0u, 0u, 0u, 0u};
  u32x4 wc[U][NT], ac[U][MT];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int s = s0 + u;
    const bool ok = s < s1;
#pragma unroll
    for (int f = 0; f < NT; ++f) wc[u][f] = ok ? ldg_stream(wp[f] + 4 * s) : zero;
#pragma unroll
    for (int i = 0; i < MT; ++i) ac[u][i] = (ok && am[i]) ? ap[i][4 * s] : zero;
  }
  for (int sb = s0; sb < s1; sb += U) {
    u32x4 wn_[U][NT], an_[U][MT];
    const int sn = sb + U;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = sn + u;
      const bool ok = s < s1;
#pragma unroll
      for (int f = 0; f < NT; ++f) wn_[u][f] = ok ? ldg_stream(wp[f] + 4 * s) : zero;
#pragma unroll
      for (int i = 0; i < MT; ++i) an_[u][i] = (ok && am[i]) ? ap[i][4 * s] : zero;
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int f = 0; f < NT; ++f) mma16<T>(acc[i][f], ac[u][i], wc[u][f]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int f = 0; f < NT; ++f) wc[u][f] = wn_[u][f];
#pragma unroll
      for (int i = 0; i < MT; ++i) ac[u][i] = an_[u][i];
    }
  }
}

// ---------------------------------------------------------------------------
// The GEMM body: WN x WK waves; wave (wn, wk) owns NT 16-column tiles and the
// wk-th share of K.  Partial tiles are summed over wk in LDS in a fixed order
// (deterministic, no atomics), then the epilogue consumes the [M, span] tile.
// ---------------------------------------------------------------------------
template <int MT> struct Unroll {
  static constexpr int value = MT <= 2 ? 8 : (MT <= 4 ? 4 : (MT <= 8 ? 2 : 1));
};

template <typename T, int MT, int NT, int WK, int WN, bool NORM, class Epi>
__global__ __launch_bounds__(64 * WK * WN) void k_gemm(const T *__restrict__ A, int lda, ARows arows,
                                                       int M, int K, NormA na, Epi epi) {
  constexpr bool kStaged = MT <= 2;
  static_assert(!NORM || MT == 1, "fused RMSNorm is for M <= 16");
  constexpr int NTHR = 64 * WK * WN;
  constexpr int SPAN = WN * NT * 16;
  constexpr int LDT = SPAN + 1;
  constexpr int kStageBytes = kStaged ? WK * WN * NT * 16 * kStageRowBytes : 0;
  constexpr int kRedBytes = WK * MT * 16 * LDT * 4;
  constexpr int kSmem = kStageBytes > kRedBytes ? kStageBytes : kRedBytes;
  __shared__ __attribute__((aligned(16))) char smem[kSmem];
  __shared__ float s_inv[16];
  float(*red)[MT * 16][LDT] = reinterpret_cast<float(*)[MT * 16][LDT]>(smem);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wn = wave % WN, wk = wave / WN;
  const int r = lane & 15, g = lane >> 4;
  const int c0_wg = blockIdx.x * SPAN;
  const int c0 = c0_wg + wn * NT * 16;

  // Fused RMSNorm: A holds gamma * x rows; each row's 1/rms comes from the
  // producer's per-tile sums of squares.  Thread t sums tiles p, p+PARTS, ...
  // of row t / PARTS; the loads are issued here and consumed after the main
  // loop, so their latency hides behind the weight stream.
  constexpr int PARTS = NTHR / 16;
  constexpr int kNormLoads = 16;  // tiles per thread covered by the unrolled loads
  float nv[NORM ? kNormLoads : 1];
  const int nrow = threadIdx.x / PARTS, npart = threadIdx.x % PARTS;
  if constexpr (NORM) {
    const float *sr = na.ssq + (size_t)na.row(min(nrow, M - 1)) * na.ntile;
#pragma unroll
    for (int u = 0; u < kNormLoads; ++u) nv[u] = sr[min(npart + PARTS * u, na.ntile - 1)];
  }

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int f = 0; f < NT; ++f) acc[i][f] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (c0 < epi.nvcols) {
    if constexpr (kStaged)
      accum_staged<T, MT, NT>(A, lda, arows, M, K, epi, c0, wk, WK,
                              smem + wave * NT * 16 * kStageRowBytes, acc);
    else
      accum_direct<T, MT, NT, Unroll<MT>::value>(A, lda, arows, M, K, epi, c0, wk, WK, acc);
  }
  if constexpr (NORM) {
    float ssum = 0.f;
#pragma unroll
    for (int u = 0; u < kNormLoads; ++u) ssum += (npart + PARTS * u < na.ntile) ? nv[u] : 0.f;
    const float *sr = na.ssq + (size_t)na.row(min(nrow, M - 1)) * na.ntile;
    for (int t = npart + PARTS * kNormLoads; t < na.ntile; t += PARTS) ssum += sr[t];
#pragma unroll
    for (int off = PARTS / 2; off >= 1; off >>= 1) ssum += __shfl_xor(ssum, off);
    if (npart == 0 && nrow < M) s_inv[nrow] = 1.0f / sqrtf(ssum / (float)na.d + na.eps);
  }
  __syncthreads();  // staging tiles are dead; the buffer becomes the reduction tile

  // Lane (r, g) holds C[row 4g+v][col r] of each 16x16 tile.
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int f = 0; f < NT; ++f)
#pragma unroll
      for (int v = 0; v < 4; ++v) red[wk][i * 16 + 4 * g + v][wn * NT * 16 + f * 16 + r] = acc[i][f][v];
  __syncthreads();
  if (WK > 1 || NORM) {
    for (int idx = threadIdx.x; idx < MT * 16 * SPAN; idx += NTHR) {
      const int m = idx / SPAN, c = idx % SPAN;
      float sum = red[0][m][c];
#pragma unroll
      for (int w = 1; w < WK; ++w) sum += red[w][m][c];
      if constexpr (NORM) sum *= (m < M ? s_inv[m] : 0.f);
      red[0][m][c] = sum;
    }
    __syncthreads();
  }
  epi.finish(&red[0][0][0], LDT, M, c0_wg, SPAN);
}

// ---------------------------------------------------------------------------
// Epilogues.
// ---------------------------------------------------------------------------
template <typename T> struct EpiStore {
  const T *w;
  int ldw, nvcols;
  T *out;
  int ldo;
  const T *embed;
  const int32_t *tokens;
  int vocab;
  T *gather_out;
  int ld_gather, d, B;
  __device__ const T *wrow(int c) const { return w + (size_t)c * ldw; }
  __device__ void finish(float *tile, int ldt, int M, int c0, int span) const {
    for (int idx = threadIdx.x; idx < M * span; idx += blockDim.x) {
      const int m = idx / span, c = idx % span;
      if (c0 + c < nvcols) out[(size_t)m * ldo + c0 + c] = Elt<T>::from_f(tile[m * ldt + c]);
    }
    if (embed) {  // the embedding row e_{t+1} of every sequence, copied next to g_t
      constexpr int E = Elt<T>::kPer16B;
      for (int b = blockIdx.x; b < B; b += gridDim.x) {
        const int tok = tokens[b];
        T *dst = gather_out + (size_t)b * ld_gather;
        if (tok < 0 || tok >= vocab) {
          for (int e = threadIdx.x; e < d; e += blockDim.x) dst[e] = Elt<T>::from_f(__int_as_float(0x7fc00000));
          continue;
        }
        const u32x4 *src = reinterpret_cast<const u32x4 *>(embed + (size_t)tok * d);
        u32x4 *dv = reinterpret_cast<u32x4 *>(dst);
        for (int e = threadIdx.x; e < d / E; e += blockDim.x) dv[e] = src[e];
      }
    }
  }
};

template <typename T> struct EpiResid {
  const T *w;
  int ldw, nvcols;
  float *out;
  long ldo;
  const float *resid;
  long ldr;
  float *ssq;  // optional per-(row, 16-column tile) sums of squares of the output
  int ssq_rs, ssq_off;
  GainCopies gc;
  __device__ const T *wrow(int c) const { return w + (size_t)c * ldw; }
  __device__ void finish(float *tile, int ldt, int M, int c0, int span) const {
    for (int idx = threadIdx.x; idx < M * span; idx += blockDim.x) {
      const int m = idx / span, c = idx % span;
      if (c0 + c >= nvcols) continue;
      float v = tile[m * ldt + c];
      if (resid) v = resid[(size_t)m * ldr + c0 + c] + v;
      out[(size_t)m * ldo + c0 + c] = v;
      tile[m * ldt + c] = v;
      for (int q = 0; q < gc.n; ++q)
        ((T *)gc.dst[q])[(size_t)m * gc.ld[q] + c0 + c] =
            Elt<T>::from_f(Elt<T>::to_f(((const T *)gc.gamma[q])[c0 + c]) * v);
    }
    if (ssq) {
      __syncthreads();
      const int ntile = nvcols / 16;
      for (int idx = threadIdx.x; idx < M * (span / 16); idx += blockDim.x) {
        const int m = idx / (span / 16), t = idx % (span / 16);
        if (c0 + 16 * t >= nvcols) continue;
        float sq = 0.f;
        for (int c = 16 * t; c < 16 * t + 16; ++c) sq += tile[m * ldt + c] * tile[m * ldt + c];
        ssq[((size_t)m * ssq_rs + ssq_off) * ntile + c0 / 16 + t] = sq;
      }
    }
  }
};

// Within a head, 16-column tile t holds rotary pairs 8t..8t+7: column n < 8 is
// dim 8t+n, column n >= 8 is its partner dim D/2 + 8t + (n-8).
__device__ __forceinline__ int rope_dim(int cc, int D) {
  const int t = cc >> 4, n = cc & 15;
  return ((n & 8) ? (D >> 1) : 0) + 8 * t + (n & 7);
}

template <typename T> struct EpiQkv {
  QkvArgs a;
  int nvcols;
  __device__ const T *wrow(int c) const {
    const int qd = a.Hq * a.D, kvd = a.Hkv * a.D;
    const T *base;
    int row;
    if (c < qd) {
      base = (const T *)a.wq;
      row = (c / a.D) * a.D + rope_dim(c % a.D, a.D);
    } else if (c < qd + kvd) {
      c -= qd;
      base = (const T *)a.wk;
      row = (c / a.D) * a.D + rope_dim(c % a.D, a.D);
    } else {
      base = (const T *)a.wv;
      row = c - qd - kvd;
    }
    return base + (size_t)row * a.d;
  }
  __device__ void finish(float *tile, int ldt, int M, int c0, int span) const {
    const int qd = a.Hq * a.D, kvd = a.Hkv * a.D, D = a.D;
    for (int idx = threadIdx.x; idx < M * span; idx += blockDim.x) {
      const int m = idx / span, c = idx % span;
      int vc = c0 + c;
      if (vc >= nvcols) continue;
      const int b = m / a.nctx, t = m % a.nctx, j = a.j0 + t;
      const float val = tile[m * ldt + c];
      if (vc < qd + kvd) {
        const bool isq = vc < qd;
        if (isq && t != a.nctx - 1) continue;
        const int lc = isq ? vc : vc - qd;
        const int h = lc / D, cc = lc % D, dd = rope_dim(cc, D);
        const float pv = tile[m * ldt + (c ^ 8)];
        const int P = a.cu_prefix[b + 1] - a.cu_prefix[b];
        const int pos = min(a.cascade ? P + j : P, a.rope_npos - 1);
        const int pm = 8 * (cc >> 4) + (cc & 7);
        const float c_ = a.rope[((size_t)pos * (D / 2) + pm) * 2];
        const float s_ = a.rope[((size_t)pos * (D / 2) + pm) * 2 + 1];
        const float o = (cc & 8) ? (val * c_ + pv * s_) : (val * c_ - pv * s_);
        if (isq)
          a.q_out[((size_t)b * a.Hq + h) * D + dd] = o;
        else
          a.k_out[(((size_t)b * a.nctx + t) * a.Hkv + h) * D + dd] = o;
      } else {
        vc -= qd + kvd;
        a.v_out[((size_t)b * a.nctx + t) * kvd + vc] = val;
      }
    }
  }
};

template <typename T> struct EpiSwiglu {
  const T *wg, *wu;
  int ldw, I, nvcols;  // nvcols = 2*I
  T *out;
  int ldo;
  // virtual tile pair (2p, 2p+1) = gate rows and up rows 16p..16p+15
  __device__ const T *wrow(int c) const {
    const int p = c >> 5, f = (c >> 4) & 1, n = c & 15;
    return (f ? wu : wg) + (size_t)(p * 16 + n) * ldw;
  }
  __device__ void finish(float *tile, int ldt, int M, int c0, int span) const {
    const int half = span >> 1;
    for (int idx = threadIdx.x; idx < M * half; idx += blockDim.x) {
      const int m = idx / half, q = idx % half;
      const int c = (q >> 4) * 32 + (q & 15);  // gate column inside the tile
      const int vc = c0 + c;
      if (vc >= nvcols) continue;
      const float gt = tile[m * ldt + c], up = tile[m * ldt + c + 16];
      const float s = gt / (1.f + expf(-gt)) * up;
      const int col = (vc >> 5) * 16 + (vc & 15);
      out[(size_t)m * ldo + col] = Elt<T>::from_f(s);
    }
  }
};

// Shared LM head: per (row, column tile) max, sum of exp(z - max) and the top-k
// (largest logit first, equal logits by lower draft id); logits optionally kept.
template <typename T> struct EpiLm {
  LmArgs a;
  int ldw, nvcols;
  __device__ const T *wrow(int c) const { return (const T *)a.w + (size_t)c * ldw; }
  __device__ void finish(float *tile, int ldt, int M, int c0, int span) const {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const int nvalid = min(span, nvcols - c0);
    const int nwg = gridDim.x, tileid = blockIdx.x;
    for (int m = wave; m < M; m += nw) {
      const float *row = tile + m * ldt;
      constexpr int PER = 4;  // span <= 256
      float v[PER];
      int id[PER];
      float mx = -INFINITY;
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        const int c = lane + 64 * p;
        const bool ok = c < nvalid;
        v[p] = ok ? row[c] : -INFINITY;
        id[p] = ok ? c0 + c : 0x7fffffff;
        mx = fmaxf(mx, v[p]);
      }
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      float se = 0.f;
#pragma unroll
      for (int p = 0; p < PER; ++p) se += (id[p] != 0x7fffffff) ? expf(v[p] - mx) : 0.f;
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) se += __shfl_xor(se, o);
      if (a.logits) {
#pragma unroll
        for (int p = 0; p < PER; ++p)
          if (id[p] != 0x7fffffff) a.logits[(size_t)m * nvcols + id[p]] = v[p];
      }
      const size_t pb = (size_t)m * nwg + tileid;
      if (lane == 0) {
        a.part_max[pb] = mx;
        a.part_sum[pb] = se;
      }
      uint64_t key[PER];
#pragma unroll
      for (int p = 0; p < PER; ++p) key[p] = id[p] != 0x7fffffff ? topk_key(v[p], id[p]) : kNoKey;
      for (int r = 0; r < a.topk; ++r) {
        // lane-local best, then wave max of the ordering keys (lower id wins ties)
        uint64_t best = kNoKey;
#pragma unroll
        for (int p = 0; p < PER; ++p) best = key[p] > best ? key[p] : best;
        best = wave_max_u64(best);
#pragma unroll
        for (int p = 0; p < PER; ++p) key[p] = key[p] == best ? kNoKey : key[p];
        if (lane == 0) {
          const bool got = best != kNoKey;
          a.cand_val[pb * kMaxTopk + r] = got ? topk_key_value(best) : -INFINITY;
          a.cand_idx[pb * kMaxTopk + r] = got ? topk_key_id(best) : 0x7fffffff;
        }
      }
    }
  }
};

// ---------------------------------------------------------------------------
// Dispatch.
// ---------------------------------------------------------------------------
// Unroll depth of the load pipeline and split-K width shrink as the number of
// 16-row tiles grows, to bound registers and the LDS reduction buffer.
template <int WKmax, int MT> struct SplitK {
  static constexpr int cap = MT <= 2 ? 8 : (MT <= 4 ? 2 : 1);
  static constexpr int value = WKmax < cap ? WKmax : cap;
};

template <typename T, int NT, int WKmax, int WN, class Epi>
static hipError_t run_gemm(const T *A, int lda, const ARows &arows, int M, int K, const Epi &epi,
                           const NormA *na, hipStream_t s) {
  constexpr int SPAN = WN * NT * 16;
  const int grid = (epi.nvcols + SPAN - 1) / SPAN;
  const int mt = (M + 15) / 16;
  const NormA n0 = na ? *na : NormA{nullptr, 0, 1, 0, 1, 1, 0.f};
  if (na) {
    if (mt != 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_gemm<T, 1, NT, SplitK<WKmax, 1>::value, WN, true, Epi>), dim3(grid),
                       dim3(64 * SplitK<WKmax, 1>::value * WN), 0, s, A, lda, arows, M, K, n0, epi);
    return hipGetLastError();
  }
#define FE_GEMM_CASE(MTV)                                                              \
  hipLaunchKernelGGL((k_gemm<T, MTV, NT, SplitK<WKmax, MTV>::value, WN, false, Epi>), \
                     dim3(grid), dim3(64 * SplitK<WKmax, MTV>::value * WN), 0, s, A, lda, arows, M, K, n0, epi)
  if (mt <= 1) FE_GEMM_CASE(1);
  else if (mt <= 2) FE_GEMM_CASE(2);
  else if (mt <= 4) FE_GEMM_CASE(4);
  else if (mt <= 8) FE_GEMM_CASE(8);
  else FE_GEMM_CASE(16);
#undef FE_GEMM_CASE
  return hipGetLastError();
}

hipError_t gemm_store(int dt, const void *A, int lda, int M, int K, const void *W, int ncols,
                      void *out, int ldo, const void *embed, const int32_t *tokens, int vocab,
                      void *gather_out, int ld_gather, int d, int B, hipStream_t s) {
  if (dt) {
    EpiStore<bf16_t> e{(const bf16_t *)W, K, ncols, (bf16_t *)out, ldo, (const bf16_t *)embed,
                       tokens, vocab, (bf16_t *)gather_out, ld_gather, d, B};
    return run_gemm<bf16_t, 1, 8, 1>((const bf16_t *)A, lda, kDenseRows, M, K, e, nullptr, s);
  }
  EpiStore<float> e{(const float *)W, K, ncols, (float *)out, ldo, (const float *)embed,
                    tokens, vocab, (float *)gather_out, ld_gather, d, B};
  return run_gemm<float, 1, 8, 1>((const float *)A, lda, kDenseRows, M, K, e, nullptr, s);
}

hipError_t gemm_resid(int dt, const void *A, int lda, int M, int K, const void *W, int ncols,
                      float *out, long ldo, const float *resid, long ldr, float *ssq, int ssq_rs,
                      int ssq_off, const GainCopies *gains, hipStream_t s) {
  GainCopies gc{};
  if (gains) gc = *gains;
  if (dt) {
    EpiResid<bf16_t> e{(const bf16_t *)W, K, ncols, out, ldo, resid, ldr, ssq, ssq_rs, ssq_off, gc};
    return run_gemm<bf16_t, 1, 8, 1>((const bf16_t *)A, lda, kDenseRows, M, K, e, nullptr, s);
  }
  EpiResid<float> e{(const float *)W, K, ncols, out, ldo, resid, ldr, ssq, ssq_rs, ssq_off, gc};
  return run_gemm<float, 1, 8, 1>((const float *)A, lda, kDenseRows, M, K, e, nullptr, s);
}

hipError_t gemm_qkv(int dt, const void *A, int lda, const ARows &arows, int M, const QkvArgs &a,
                    const NormA *na, hipStream_t s) {
  const int nv = (a.Hq + 2 * a.Hkv) * a.D;
  if (dt) {
    EpiQkv<bf16_t> e{a, nv};
    return run_gemm<bf16_t, 1, 8, 1>((const bf16_t *)A, lda, arows, M, a.d, e, na, s);
  }
  EpiQkv<float> e{a, nv};
  return run_gemm<float, 1, 8, 1>((const float *)A, lda, arows, M, a.d, e, na, s);
}

hipError_t gemm_swiglu(int dt, const void *A, int lda, const ARows &arows, int M, int K,
                       const void *w_gate, const void *w_up, int I, void *s_out, int lds,
                       const NormA *na, hipStream_t s) {
  if (dt) {
    EpiSwiglu<bf16_t> e{(const bf16_t *)w_gate, (const bf16_t *)w_up, K, I, 2 * I,
                        (bf16_t *)s_out, lds};
    return run_gemm<bf16_t, 2, 4, 1>((const bf16_t *)A, lda, arows, M, K, e, na, s);
  }
  EpiSwiglu<float> e{(const float *)w_gate, (const float *)w_up, K, I, 2 * I, (float *)s_out, lds};
  return run_gemm<float, 2, 4, 1>((const float *)A, lda, arows, M, K, e, na, s);
}

// LM head: 64-column tiles; 2 x 2 waves, each 32 weight rows x half of K.
constexpr int kLmWN = 2, kLmNT = 2;
int lmhead_tiles(int V) { return (V + kLmWN * kLmNT * 16 - 1) / (kLmWN * kLmNT * 16); }

hipError_t gemm_lmhead(int dt, const void *A, int lda, const ARows &arows, int M, int K,
                       const LmArgs &a, const NormA *na, int *nwg_out, hipStream_t s) {
  *nwg_out = lmhead_tiles(a.V);
  if (dt) {
    EpiLm<bf16_t> e{a, K, a.V};
    return run_gemm<bf16_t, kLmNT, 2, kLmWN>((const bf16_t *)A, lda, arows, M, K, e, na, s);
  }
  EpiLm<float> e{a, K, a.V};
  return run_gemm<float, kLmNT, 2, kLmWN>((const float *)A, lda, arows, M, K, e, na, s);
}

}  // namespace fe
