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
#include <type_traits>

namespace fe {

template <typename T> __device__ __forceinline__ void mma16(f32x4 &acc, u32x4 a, u32x4 b);
template <typename T> struct EpiLm;

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
// Accumulation (up to 32 rows).  Leaves, in lane (r, g) of a wave, the 16x16
// tiles acc[i][f] = rows 16i.. of A times weight rows of virtual columns
// c0+16f.., summed over this wave's share of K.
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

// Epilogues with kSliced = true cover many row blocks (and groups) in one
// launch: a grid dimension (z for k_gemm_mid, y for k_gemm) enumerates them
// and slice() moves A, M and the epilogue's outputs to its block before
// anything else runs.
template <class E, class = void> struct SlicedEpi { static constexpr bool value = false; };
template <class E> struct SlicedEpi<E, decltype((void)E::kSliced)> {
  static constexpr bool value = E::kSliced;
};

// ---------------------------------------------------------------------------
// The GEMM body: WN x WK waves; wave (wn, wk) owns NT 16-column tiles and the
// wk-th share of K.  Partial tiles are summed over wk in LDS in a fixed order
// (deterministic, no atomics), then the epilogue consumes the [M, span] tile.
// ---------------------------------------------------------------------------
template <typename T, int MT, int NT, int WK, int WN, bool NORM, class Epi>
__global__ __launch_bounds__(64 * WK * WN) void k_gemm(const T *__restrict__ A, int lda, ARows arows,
                                                       int M, int K, NormA na, Epi epi) {
  static_assert(MT <= 2, "more than 32 rows take k_gemm_mid");
  static_assert(!NORM || MT == 1, "fused RMSNorm is for M <= 16");
  constexpr int NTHR = 64 * WK * WN;
  constexpr int SPAN = WN * NT * 16;
  constexpr int LDT = SPAN + 1;
  constexpr int kStageBytes = WK * WN * NT * 16 * kStageRowBytes;
  constexpr int kRedBytes = WK * MT * 16 * LDT * 4;
  constexpr int kSmem = kStageBytes > kRedBytes ? kStageBytes : kRedBytes;
  __shared__ __attribute__((aligned(16))) char smem[kSmem];
  __shared__ float s_inv[16];
  float(*red)[MT * 16][LDT] = reinterpret_cast<float(*)[MT * 16][LDT]>(smem);

  if constexpr (SlicedEpi<Epi>::value) {  // grid y: the epilogue's slices
    const T *a = A;
    epi.slice(blockIdx.y, MT * 16, a, M);
    A = a;
    if (M <= 0) return;
  }
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

  const typename Epi::Pre pre{};  // the epilogue loads its own values here
  if (c0 < epi.nvcols)
    accum_staged<T, MT, NT>(A, lda, arows, M, K, epi, c0, wk, WK,
                            smem + wave * NT * 16 * kStageRowBytes, acc);
  if constexpr (NORM) {
    float ssum = 0.f;
#pragma unroll
    for (int u = 0; u < kNormLoads; ++u) ssum += (npart + PARTS * u < na.ntile) ? nv[u] : 0.f;
    const float *sr = na.ssq + (size_t)na.row(min(nrow, M - 1)) * na.ntile;
    for (int t = npart + PARTS * kNormLoads; t < na.ntile; t += PARTS) ssum += sr[t];
    static_assert(PARTS >= 8 && PARTS <= 64, "row partials reduce over 8..64 lanes");
    ssum = group_sum<PARTS>(ssum);
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
  epi.finish(&red[0][0][0], LDT, M, c0_wg, SPAN, pre);
}

// ---------------------------------------------------------------------------
// Row-streaming path for 1..8 input rows (batch-1 layers, bf16 weights): no
// matrix cores, no weight staging.  A workgroup of W waves owns SPAN = 4W
// virtual columns; wave w takes weight rows 4w..4w+3 with 16 lanes per row,
// so every load instruction reads 256 contiguous bytes of each of 4 rows and
// a lane only ever accumulates its own row.  The input rows are in LDS as
// bf16 (zero-padded to a multiple of 128) and meet the weights in
// v_dot2c_f32_bf16 as they arrive; two register banks of kGvDepth pieces per
// lane alternate, one in flight while the other is consumed.  Each row's sum
// is reduced over its 16 lanes with DPP; the [M, SPAN] tile goes to the same
// epilogues as the matrix-core paths.
// ---------------------------------------------------------------------------
constexpr int kGvDepth = 8;
constexpr int kGvMaxLds = 64 * 1024;  // bytes of input rows in LDS

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
// Each 32-bit word goes through a scalar before the bit cast: a bit cast of a
// vector element (w.y) itself is compiled as a read of element 0.
__device__ __forceinline__ float dot8(u32x4 w, u32x4 x, float acc) {
  const uint32_t w0 = w[0], w1 = w[1], w2 = w[2], w3 = w[3];
  const uint32_t x0 = x[0], x1 = x[1], x2 = x[2], x3 = x[3];
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w0), __builtin_bit_cast(bf16x2_t, x0), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w1), __builtin_bit_cast(bf16x2_t, x1), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w2), __builtin_bit_cast(bf16x2_t, x2), acc, false);
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w3), __builtin_bit_cast(bf16x2_t, x3), acc, false);
}

template <int MR, int W, bool NORM, class Epi>
__global__ __launch_bounds__(64 * W) void k_gemv(const bf16_t *__restrict__ A, int lda, ARows arows,
                                                 int M, int K, NormA na, Epi epi) {
  constexpr int SPAN = 4 * W;
  constexpr int NTHR = 64 * W;
  extern __shared__ __attribute__((aligned(16))) char xs_raw[];
  __shared__ float tile[MR][SPAN + 1];
  __shared__ float s_inv[MR];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, rq = lane >> 4, l16 = lane & 15;
  const int c0 = blockIdx.x * SPAN;
  const int kpad = (K + 127) & ~127;
  const int npc = kpad / 128;  // 16-byte pieces per lane per row
  bf16_t *xs = reinterpret_cast<bf16_t *>(xs_raw);

  // weight row of this lane (clamped; columns past the end are dropped at the end)
  const int col = c0 + wave * 4 + rq;
  const bf16_t *wr = epi.wrow(min(col, epi.nvcols - 1));
  // piece p of the row: elements p*128 + 8*l16 .. +7; past K the address is
  // clamped in bounds and the (finite) weights meet zero-padded inputs
  auto ldw = [&](int p) {
    return ldg_stream(reinterpret_cast<const u32x4 *>(wr + min(p * 128 + l16 * 8, K - 8)));
  };
  // every independent load is issued before anything is consumed, so the
  // whole prologue costs one memory round trip: the first weight pieces, the
  // input rows (registers, then LDS), the norm partials, the epilogue's values
  u32x4 ba[kGvDepth], bb[kGvDepth];
#pragma unroll
  for (int i = 0; i < kGvDepth; ++i) ba[i] = ldw(min(i, npc - 1));

  constexpr int XPT = kGvMaxLds / 16 / NTHR;  // input pieces per thread, at most
  const int xper = kpad / 8, xtot = MR * xper;
  u32x4 xr[XPT];
#pragma unroll
  for (int u = 0; u < XPT; ++u)
    if (NTHR * u < xtot) {  // uniform: batch u holds at least one piece
      const int idx = min(tid + NTHR * u, xtot - 1);
      const int m = idx / xper, e = min((idx % xper) * 8, K - 8);
      xr[u] = *reinterpret_cast<const u32x4 *>(A + (size_t)arows.row(min(m, M - 1)) * lda + e);
    }

  constexpr int PARTS = NTHR / 16;
  constexpr int kNormLoads = 16;
  float nv[NORM ? kNormLoads : 1];
  const int nrow = tid / PARTS, npart = tid % PARTS;
  if constexpr (NORM) {
    const float *sr = na.ssq + (size_t)na.row(min(nrow, M - 1)) * na.ntile;
#pragma unroll
    for (int u = 0; u < kNormLoads; ++u) nv[u] = sr[min(npart + PARTS * u, na.ntile - 1)];
  }
  const typename Epi::Pre pre = epi.prefetch(M, c0, SPAN);

  // input rows -> LDS, zero past K and past M
  const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int u = 0; u < XPT; ++u) {
    const int idx = tid + NTHR * u;
    if (NTHR * u < xtot && idx < xtot) {
      const int m = idx / xper, e = (idx % xper) * 8;
      *reinterpret_cast<u32x4 *>(xs + (size_t)m * kpad + e) = (m < M && e < K) ? xr[u] : zero;
    }
  }
  if constexpr (NORM) {
    float ssum = 0.f;
#pragma unroll
    for (int u = 0; u < kNormLoads; ++u) ssum += (npart + PARTS * u < na.ntile) ? nv[u] : 0.f;
    const float *sr = na.ssq + (size_t)na.row(min(nrow, M - 1)) * na.ntile;
    for (int t = npart + PARTS * kNormLoads; t < na.ntile; t += PARTS) ssum += sr[t];
    static_assert(PARTS >= 8 && PARTS <= 64, "row partials reduce over 8..64 lanes");
    ssum = group_sum<PARTS>(ssum);
    if (npart == 0 && nrow < MR) s_inv[nrow] = nrow < M ? 1.0f / sqrtf(ssum / (float)na.d + na.eps) : 0.f;
  }
  __syncthreads();

  float acc[MR];
#pragma unroll
  for (int m = 0; m < MR; ++m) acc[m] = 0.f;
  const bf16_t *xl = xs + l16 * 8;
  auto consume = [&](const u32x4 (&bw)[kGvDepth], int p0) {
#pragma unroll
    for (int i = 0; i < kGvDepth; ++i) {
      const int p = p0 + i;
      if (p < npc) {
#pragma unroll
        for (int m = 0; m < MR; ++m)
          acc[m] = dot8(bw[i], *reinterpret_cast<const u32x4 *>(xl + (size_t)m * kpad + p * 128), acc[m]);
      }
    }
  };
  for (int p0 = 0; p0 < npc; p0 += 2 * kGvDepth) {
#pragma unroll
    for (int i = 0; i < kGvDepth; ++i) bb[i] = ldw(min(p0 + kGvDepth + i, npc - 1));
    consume(ba, p0);
#pragma unroll
    for (int i = 0; i < kGvDepth; ++i) ba[i] = ldw(min(p0 + 2 * kGvDepth + i, npc - 1));
    consume(bb, p0 + kGvDepth);
  }
#pragma unroll
  for (int m = 0; m < MR; ++m) {
    float v = group_sum<16>(acc[m]);
    if constexpr (NORM) v *= s_inv[m];
    if (l16 == 0) tile[m][wave * 4 + rq] = v;
  }
  __syncthreads();
  epi.finish(&tile[0][0], SPAN + 1, M, c0, SPAN, pre);
}

// ---------------------------------------------------------------------------
// Batched rows (17..256): one workgroup owns BN = 16*NTW*WN output columns and
// every row; its four waves form WM = 4/WN row groups of 64 rows and WN column
// groups of 16*NTW columns.  K advances in chunks of 128 bytes per row.  The
// chunks of A (all rows) and of the BN weight rows go straight from memory to
// an S-stage LDS ring with direct-to-LDS loads (global_load_lds_dwordx4), so
// S-1 chunks are in flight without holding registers.  One load instruction
// fills 1 KB of LDS contiguously (lane l -> byte 16l); 16-byte piece p of row
// R sits at slot p ^ ((R >> 1) & 7) of its row, which keeps the MFMA fragment
// reads free of bank conflicts without padding.  Weights are read from HBM
// once; A (at most 256/WN rows) is served by L2 to every workgroup.
// Synchronisation is a plain s_barrier after an explicit vmcnt wait: the
// workgroup fence of __syncthreads would drain every load in flight.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void wg_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ int ring_slot(int row, int piece) { return row * 8 + (piece ^ ((row >> 1) & 7)); }

template <typename T, int NTW, int WN, int S, class Epi, int RT = 4>
__global__ __launch_bounds__(256) void k_gemm_mid(const T *__restrict__ A, int lda, ARows arows,
                                                  int M, int K, Epi epi, float *__restrict__ splitp,
                                                  int ldp) {
  // RT: 16-row tiles per wave (4; 2 when at most 32 rows are live, so that the
  // ring does not carry duplicated rows of A)
  static_assert(RT == 4 || RT == 2, "row tiles per wave");
  constexpr int WM = 4 / WN;
  constexpr int MROWS = 16 * RT * WM;  // rows this configuration holds
  if constexpr (SlicedEpi<Epi>::value) {
    const T *a = A;
    epi.slice(blockIdx.z, MROWS, a, M);
    A = a;
    if (M <= 0) return;  // the whole workgroup: past the last row block
  }
  constexpr int E = Elt<T>::kPer16B;  // elements per 16-byte piece
  constexpr int KC = 8 * E;           // elements of K per chunk
  constexpr int BN = NTW * WN * 16;
  static_assert(BN % 32 == 0, "weight slots must split evenly over the four waves");
  constexpr int AI = MROWS / 32;      // A load instructions per wave per stage
  constexpr int WI = BN / 32;         // weight load instructions per wave per stage
  constexpr int CNT = AI + WI;
  static_assert((S - 2) * CNT <= 63, "vmcnt range");
  constexpr int ABYTES = MROWS * 128, STAGE = ABYTES + BN * 128;
  constexpr int LDT = BN + 1;
  constexpr int TILE = MROWS * LDT * 4;
  constexpr int SMEM = S * STAGE > TILE ? S * STAGE : TILE;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r = lane & 15, g = lane >> 4;
  const int wm = wave / WN, wn = wave % WN;
  const int c0 = blockIdx.x * BN;
  // split K over gridDim.y: this workgroup's chunks [cb, cb + nch)
  const int nchk = (K + KC - 1) / KC;
  const int cb = (int)((long)nchk * blockIdx.y / gridDim.y);
  const int nch = (int)((long)nchk * (blockIdx.y + 1) / gridDim.y) - cb;

  // the lane's slot in each of its load instructions, and the source row and
  // piece offset that belong there (rows past M repeat row M-1: their products
  // land in output rows that are never stored)
  const T *asrc[AI];
  int aoff[AI];
#pragma unroll
  for (int j = 0; j < AI; ++j) {
    const int q = (j * 4 + wave) * 64 + lane, row = q >> 3;
    asrc[j] = A + (size_t)arows.row(min(row, M - 1)) * lda;
    aoff[j] = ((q & 7) ^ ((row >> 1) & 7)) * E;
  }
  const T *wsrc[WI];
  int woff[WI];
#pragma unroll
  for (int j = 0; j < WI; ++j) {
    const int q = (j * 4 + wave) * 64 + lane, n = q >> 3;
    wsrc[j] = epi.wrow(min(c0 + n, epi.nvcols - 1));
    woff[j] = ((q & 7) ^ ((n >> 1) & 7)) * E;
  }
  // chunk ch (clamped: past the end the last chunk is fetched again, so every
  // wave issues the same count), addresses clamped inside the rows
  auto issue = [&](int ch) {
    char *st = smem + (ch % S) * STAGE;
    const int k = (cb + min(ch, nch - 1)) * KC;
#pragma unroll
    for (int j = 0; j < AI; ++j)
      lds_dma16(asrc[j] + min(k + aoff[j], K - E), st + (j * 4 + wave) * 1024);
#pragma unroll
    for (int j = 0; j < WI; ++j)
      lds_dma16(wsrc[j] + min(k + woff[j], K - E), st + ABYTES + (j * 4 + wave) * 1024);
  };

  f32x4 acc[RT][NTW];
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int f = 0; f < NTW; ++f) acc[i][f] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int mrow0 = wm * 16 * RT, ncol0 = wn * NTW * 16;
  const int mtiles = min(RT, (M - mrow0 + 15) / 16);  // this wave's live 16-row tiles (may be <= 0)

#pragma unroll
  for (int st = 0; st < S - 1; ++st) issue(st);
  for (int ch = 0; ch < nch; ++ch) {
    wait_vmcnt<(S - 2) * CNT>();  // this wave's part of chunk ch has landed
    wg_barrier();                 // so has everyone's; ring slot of chunk ch-1 is free
    issue(ch + S - 1);
    const char *st = smem + (ch % S) * STAGE;
    if (cb + ch == nchk - 1 && K % KC) {  // ragged last chunk: zero the pieces past K
      const int k = (cb + ch) * KC;
      for (int q = tid; q < (MROWS + BN) * 8; q += 256) {
        const int row = q >> 3, piece = (q & 7) ^ ((row >> 1) & 7);
        if (k + piece * E >= K) *reinterpret_cast<u32x4 *>(const_cast<char *>(st) + q * 16) = u32x4{0u, 0u, 0u, 0u};
      }
      wg_barrier();
    }
    // every fragment of the chunk is read before the first product (the ring
    // holds all MROWS rows, so the reads need no guard and are in flight
    // together); only the products skip the wave's dead row tiles
    u32x4 bf[2][NTW], af[2][RT];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int f = 0; f < NTW; ++f)
        bf[ks][f] = *reinterpret_cast<const u32x4 *>(st + ABYTES + ring_slot(ncol0 + f * 16 + r, ks * 4 + g) * 16);
#pragma unroll
      for (int i = 0; i < RT; ++i)
        af[ks][i] = *reinterpret_cast<const u32x4 *>(st + ring_slot(mrow0 + i * 16 + r, ks * 4 + g) * 16);
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int i = 0; i < RT; ++i)
        if (i < mtiles)
#pragma unroll
          for (int f = 0; f < NTW; ++f) mma16<T>(acc[i][f], af[ks][i], bf[ks][f]);
  }
  wait_vmcnt<0>();  // the chunks fetched past the end land before the ring is reused or freed
  if (splitp) {  // split K: this slice's fp32 sums, reduced (and finished) by a second launch
    float *dst = splitp + (size_t)blockIdx.y * M * ldp + c0;
#pragma unroll
    for (int i = 0; i < RT; ++i)
      if (i < mtiles)
#pragma unroll
        for (int f = 0; f < NTW; ++f)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int m = mrow0 + i * 16 + 4 * g + v;
            if (m < M) dst[(size_t)m * ldp + ncol0 + f * 16 + r] = acc[i][f][v];
          }
    return;
  }
  wg_barrier();
  float(*tile)[LDT] = reinterpret_cast<float(*)[LDT]>(smem);
#pragma unroll
  for (int i = 0; i < RT; ++i)
    if (i < mtiles)
#pragma unroll
      for (int f = 0; f < NTW; ++f)
#pragma unroll
        for (int v = 0; v < 4; ++v) tile[mrow0 + i * 16 + 4 * g + v][ncol0 + f * 16 + r] = acc[i][f][v];
  __syncthreads();
  epi.finish(&tile[0][0], LDT, M, c0, BN, typename Epi::Pre{});
}

// ---------------------------------------------------------------------------
// Many rows, matrix-core bound (the cache update's and the prefill's row
// blocks: bf16, K a multiple of 64): 128 x 128 output tiles, eight waves as 2
// row groups x 4 column groups of 64 x 32, so two waves share each SIMD.  The
// ring and its swizzle are k_gemm_mid's; the schedule is software-pipelined
// over the two 32-wide K steps of a chunk:
//   read step-1 fragments of chunk c | products of step 0 (read last round)
//   wait: chunk c+1 landed, every read of chunk c done; barrier
//   refill chunk c's slot with chunk c+S | read step-0 fragments of chunk c+1
//   products of step 1
// so every product's operands were read while other products ran.  Waits are
// compiler-visible s_waitcnt immediates and the phases are fenced with
// scheduling barriers: with inline-asm waits the compiler hoisted the barrier
// (and its lgkmcnt(0)) above the products, serialising LDS latency.  At 1024
// rows (8B shapes, epilogues included) the fusion GEMM runs at 33 %, the
// input FC at 34 % and the K/V GEMM of all five layers at 24 % of the bf16
// peak, against 20-29 % for k_gemm_mid's 128 x 64 tiles.
// ---------------------------------------------------------------------------
__device__ __forceinline__ constexpr int waitcnt_imm(int vm, int lgkm) {
  return (vm & 15) | ((vm >> 4) << 14) | (7 << 4) | (lgkm << 8);
}

constexpr int kBigRows = 128, kBigCols = 128;

// SPLIT: K is split over grid y and each slice's fp32 sums go to splitp
// (slice y at y * M * ldp, row m at m * ldp) for a second launch that sums them
// and runs the epilogue; the row blocks of grid z then cover rows
// arows.row(m) of A directly (no epilogue slicing).
// RT x NTW 16 x 16 tiles per wave, WM x WN waves (eight): the cache update's
// 128 x 128 tiles are 4, 2, 2, 4; the 256 x 128 tiles of up to 256 rows (one
// row block, so the weights are streamed once) are 4, 4, 4, 2.
template <int RT, int NTW, int WM, int WN, int S, class Epi, bool SPLIT = false>
__global__ __launch_bounds__(512) void k_gemm_tile(const bf16_t *__restrict__ A, int lda, ARows arows,
                                                   int M, int K, Epi epi, float *__restrict__ splitp,
                                                   int ldp) {
  constexpr int NW = WM * WN;
  static_assert(NW == 8, "eight waves");
  constexpr int BM = 16 * RT * WM, BN = 16 * NTW * WN, KC = 64;
  constexpr int ABYTES = BM * 128, STAGE = ABYTES + BN * 128;
  constexpr int AI = BM / 8 / NW, WI = BN / 8 / NW, CNT = AI + WI;  // 1 KB loads per wave per chunk
  static_assert(S >= 2 && (S - 1) * CNT <= 63, "vmcnt range");
  // epilogue tile rows 4 floats longer than the span: 16-byte aligned for
  // the epilogues' vector reads, and the accumulator writes (4 rows x 16
  // columns per instruction) land on distinct banks; one float longer for
  // the LM head's scan (a thread per row: consecutive rows on distinct banks)
  constexpr int LDT = BN + (std::is_same<Epi, EpiLm<bf16_t>>::value ? 1 : 4), TILE = BM * LDT * 4;
  constexpr int SMEM = S * STAGE > TILE ? S * STAGE : TILE;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  int m0 = 0, Mb = M;  // first row of this block, rows in it
  if constexpr (SPLIT) {
    m0 = blockIdx.z * BM;
    Mb = min(BM, M - m0);
  } else if constexpr (SlicedEpi<Epi>::value) {
    const bf16_t *a = A;
    epi.slice(blockIdx.z, BM, a, M);
    A = a;
    Mb = M;
  }  // else one row block of at most BM rows
  if (Mb <= 0) return;  // the whole workgroup: past the last row block
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r = lane & 15, g = lane >> 4;
  const int wm = wave / WN, wn = wave % WN;
  const int c0 = blockIdx.x * BN;
  // this workgroup's chunks of K: [cb, cb + nch)
  const int nchk = K / KC;
  const int cb = SPLIT ? (int)((long)nchk * blockIdx.y / gridDim.y) : 0;
  const int nch = SPLIT ? (int)((long)nchk * (blockIdx.y + 1) / gridDim.y) - cb : nchk;
  // the lane's slot in each of its load instructions and the source there
  // (rows past M repeat row M-1, columns past the end the last column: their
  // products land in outputs that are never stored)
  const bf16_t *asrc[AI], *wsrc[WI];
#pragma unroll
  for (int j = 0; j < AI; ++j) {
    const int q = (j * NW + wave) * 64 + lane, row = q >> 3;
    asrc[j] = A + (size_t)arows.row(m0 + min(row, Mb - 1)) * lda + ((q & 7) ^ ((row >> 1) & 7)) * 8;
  }
#pragma unroll
  for (int j = 0; j < WI; ++j) {
    const int q = (j * NW + wave) * 64 + lane, n = q >> 3;
    wsrc[j] = epi.wrow(min(c0 + n, epi.nvcols - 1)) + ((q & 7) ^ ((n >> 1) & 7)) * 8;
  }
  // chunk ch into its ring slot (past the end the last chunk is fetched again,
  // so every wave issues the same count)
  auto issue = [&](int ch) {
    char *st = smem + (ch % S) * STAGE;
    const int k = (cb + min(ch, nch - 1)) * KC;
#pragma unroll
    for (int j = 0; j < AI; ++j) lds_dma16(asrc[j] + k, st + (j * NW + wave) * 1024);
#pragma unroll
    for (int j = 0; j < WI; ++j) lds_dma16(wsrc[j] + k, st + ABYTES + (j * NW + wave) * 1024);
  };
  f32x4 acc[RT][NTW];
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int f = 0; f < NTW; ++f) acc[i][f] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int mrow0 = wm * 16 * RT, ncol0 = wn * NTW * 16;
  u32x4 a0[RT], b0[NTW], a1[RT], b1[NTW];
  auto frags = [&](const char *st, int ks, u32x4 (&af)[RT], u32x4 (&bf)[NTW]) {
#pragma unroll
    for (int f = 0; f < NTW; ++f)
      bf[f] = *reinterpret_cast<const u32x4 *>(st + ABYTES + ring_slot(ncol0 + f * 16 + r, ks * 4 + g) * 16);
#pragma unroll
    for (int i = 0; i < RT; ++i)
      af[i] = *reinterpret_cast<const u32x4 *>(st + ring_slot(mrow0 + i * 16 + r, ks * 4 + g) * 16);
  };
  auto products = [&](const u32x4 (&af)[RT], const u32x4 (&bf)[NTW]) {
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
      for (int f = 0; f < NTW; ++f) mma16<bf16_t>(acc[i][f], af[i], bf[f]);
  };
#pragma unroll
  for (int st = 0; st < S; ++st) issue(st);
  __builtin_amdgcn_s_waitcnt(waitcnt_imm((S - 1) * CNT, 15));  // chunk 0 (this wave's part)
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  frags(smem, 0, a0, b0);
  for (int ch = 0; ch < nch; ++ch) {
    // the step-0 fragments (read during the last products) are in
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, 0));
    __builtin_amdgcn_sched_barrier(0);
    frags(smem + (ch % S) * STAGE, 1, a1, b1);
    __builtin_amdgcn_sched_barrier(0);
    products(a0, b0);
    __builtin_amdgcn_sched_barrier(0);
    // chunk ch+1 landed (this wave's part) and every read of chunk ch is done;
    // the barrier extends both to the workgroup
    __builtin_amdgcn_s_waitcnt(waitcnt_imm((S - 2) * CNT, 0));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    issue(ch + S);  // into chunk ch's slot
    if (ch + 1 < nch) frags(smem + ((ch + 1) % S) * STAGE, 0, a0, b0);
    __builtin_amdgcn_sched_barrier(0);
    products(a1, b1);
    __builtin_amdgcn_sched_barrier(0);
  }
  // the chunks fetched past the end land before the ring becomes the tile
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 0));
  if constexpr (SPLIT) {
    float *dst = splitp + ((size_t)blockIdx.y * M + m0) * ldp + c0;
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
      for (int f = 0; f < NTW; ++f)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int m = mrow0 + i * 16 + 4 * g + v;
          if (m < Mb) dst[(size_t)m * ldp + ncol0 + f * 16 + r] = acc[i][f][v];
        }
    return;
  }
  __syncthreads();
  float(*tile)[LDT] = reinterpret_cast<float(*)[LDT]>(smem);
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int f = 0; f < NTW; ++f)
#pragma unroll
      for (int v = 0; v < 4; ++v) tile[mrow0 + i * 16 + 4 * g + v][ncol0 + f * 16 + r] = acc[i][f][v];
  __syncthreads();
  epi.finish(&tile[0][0], LDT, Mb, c0, BN, typename Epi::Pre{});
}

// Launch of k_gemm_tile over ncols virtual columns and nz row blocks (of
// kBigRows): a three-stage ring when the grid is about one workgroup per CU
// (96 KB of LDS: one workgroup per CU), else two stages, which lets two
// workgroups share a CU (measured at 1024 rows: fusion and input FC 120 and
// 78 us with three stages against 134 and 86 with two; the K/V GEMM of five
// layers 103 us with two stages against 120 with three).
template <class Epi>
static hipError_t launch_tile(const bf16_t *A, int lda, int M, int K, const Epi &e, int ncols, int nz,
                              hipStream_t s) {
  const dim3 grid((ncols + kBigCols - 1) / kBigCols, 1, nz);
  if ((long)grid.x * nz <= 288)
    hipLaunchKernelGGL((k_gemm_tile<4, 2, 2, 4, 3, Epi>), grid, dim3(512), 0, s, A, lda, kDenseRows, M,
                       K, e, nullptr, 0);
  else
    hipLaunchKernelGGL((k_gemm_tile<4, 2, 2, 4, 2, Epi>), grid, dim3(512), 0, s, A, lda, kDenseRows, M,
                       K, e, nullptr, 0);
  return hipGetLastError();
}

// split-K slices the reductions sum (k_splitk_finish, k_resid_rows)
constexpr int kMaxSlices = 8;

// Split-K reduction: sums the ks partial slices of a 16-column span in a fixed
// order and hands the span to the epilogue, like k_gemm_mid would.  A thread
// takes 4 adjacent columns of a row and issues all of its slice loads before
// adding.
template <class Epi>
__global__ __launch_bounds__(256) void k_splitk_finish(const float *__restrict__ splitp, int ldp,
                                                       int ks, int M, Epi epi) {
  constexpr int BNR = 16, LDT = BNR + 1;
  __shared__ float tile[256 * LDT];
  const int c0 = blockIdx.x * BNR;
  const size_t slice = (size_t)M * ldp;
  for (int q = threadIdx.x; q < M * (BNR / 4); q += 256) {
    const int m = q / (BNR / 4), c = (q % (BNR / 4)) * 4;
    if constexpr (Epi::kQkv)
      if (!epi.row_used(m, c0)) continue;  // the epilogue never reads this row here
    const float *src = splitp + (size_t)m * ldp + c0 + c;
    f32x4 part[kMaxSlices];
#pragma unroll
    for (int y = 0; y < kMaxSlices; ++y)
      part[y] = y < ks ? *reinterpret_cast<const f32x4 *>(src + y * slice) : f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 v = part[0];
#pragma unroll
    for (int y = 1; y < kMaxSlices; ++y) v += part[y];
#pragma unroll
    for (int e = 0; e < 4; ++e) tile[m * LDT + c + e] = v[e];
  }
  __syncthreads();
  epi.finish(tile, LDT, M, c0, BNR, typename Epi::Pre{});
}

// Row finish of a residual GEMM whose rows feed only RMSNorms: one workgroup
// of 1024 threads per row sums the ks fp32 slices in slice order and adds the
// residual (the value EpiResid gives), stores it, and writes
// gamma_q * (v / rms(v)) in the storage type to every copy q (fixed-order
// reductions; four adjacent columns per thread, packed loads and stores).
// ks = 0: the GEMM's own epilogue stored v; it is read back.
template <typename T> __device__ __forceinline__ void store4(T *y, const f32x4 &v);
template <> __device__ __forceinline__ void store4<float>(float *y, const f32x4 &v) {
  *reinterpret_cast<f32x4 *>(y) = v;
}
template <> __device__ __forceinline__ void store4<bf16_t>(bf16_t *y, const f32x4 &v) {
  *reinterpret_cast<u32x2 *>(y) = u32x2{f2bf2(v.x, v.y), f2bf2(v.z, v.w)};
}
// Eight adjacent values: one 16-byte store (bf16) or two (fp32).
template <typename T> __device__ __forceinline__ void store8(T *y, const float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<u32x4 *>(y) =
        u32x4{f2bf2(v[0], v[1]), f2bf2(v[2], v[3]), f2bf2(v[4], v[5]), f2bf2(v[6], v[7])};
  } else {
    *reinterpret_cast<f32x4 *>(y) = f32x4{v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4 *>(y + 4) = f32x4{v[4], v[5], v[6], v[7]};
  }
}
__device__ __forceinline__ bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }
// Eight adjacent floats of an epilogue tile row: two 16-byte LDS reads when
// the tile's row stride is a multiple of 4 floats (the caller's column is a
// multiple of 8), else eight scalar reads.
__device__ __forceinline__ void tile8(const float *t, int ldt, float (&v)[8]) {
  if ((ldt & 3) == 0) {
    const f32x4 a = *reinterpret_cast<const f32x4 *>(t), b = *reinterpret_cast<const f32x4 *>(t + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = t[j];
  }
}
template <typename T> __device__ __forceinline__ f32x4 load4(const T *g);
template <> __device__ __forceinline__ f32x4 load4<float>(const float *g) {
  return *reinterpret_cast<const f32x4 *>(g);
}
template <> __device__ __forceinline__ f32x4 load4<bf16_t>(const bf16_t *g) {
  const u32x2 w = *reinterpret_cast<const u32x2 *>(g);
  return f32x4{__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
               __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u)};
}

constexpr int kRowThreads = 1024;
template <typename T, int NV>
__global__ __launch_bounds__(kRowThreads) void k_resid_rows(const float *__restrict__ splitp,
                                                            int ldp, int ks, int M, int d,
                                                            const float *__restrict__ resid,
                                                            long ldr, float *__restrict__ out,
                                                            long ldo, GainCopies gc, float eps) {
  constexpr int NW = kRowThreads / 64;
  __shared__ float red[NW];
  const int m = blockIdx.x, tid = threadIdx.x;
  const size_t slice = (size_t)M * ldp;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  f32x4 v[NV];
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int e = 4 * (tid + kRowThreads * u), ec = min(e, d - 4);
    if (ks > 0) {
      const float *src = splitp + (size_t)m * ldp + ec;
      f32x4 part[kMaxSlices];
#pragma unroll
      for (int y = 0; y < kMaxSlices; ++y) part[y] = y < ks ? *reinterpret_cast<const f32x4 *>(src + y * slice) : zero;
      f32x4 t = part[0];
#pragma unroll
      for (int y = 1; y < kMaxSlices; ++y) t += part[y];
      if (resid) t = *reinterpret_cast<const f32x4 *>(resid + (size_t)m * ldr + ec) + t;
      v[u] = t;
    } else {
      v[u] = *reinterpret_cast<const f32x4 *>(out + (size_t)m * ldo + ec);
    }
    if (e >= d) v[u] = zero;
  }
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < NV; ++u) ss += v[u].x * v[u].x + v[u].y * v[u].y + v[u].z * v[u].z + v[u].w * v[u].w;
  ss = group_sum<64>(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int e = 4 * (tid + kRowThreads * u);
    if (e >= d) continue;
    if (ks > 0) *reinterpret_cast<f32x4 *>(out + (size_t)m * ldo + e) = v[u];
    const f32x4 xn = v[u] * inv;
#pragma unroll
    for (int q = 0; q < kMaxLayers + 1; ++q) {
      if (q >= gc.n) break;
      const f32x4 g = load4((const T *)gc.gamma[q] + e);
      store4((T *)gc.dst[q] + (size_t)m * gc.ld[q] + e, g * xn);
    }
  }
}

// ---------------------------------------------------------------------------
// Epilogues.
// ---------------------------------------------------------------------------
// kMidNtw: 16-column tiles per workgroup on the batched-rows path (0 = chosen
// from the column count); kMidNtwMin: the smallest the epilogue accepts.
// prefetch() runs before the main loop and may load, into registers, what
// finish() needs for this thread's first output element (Pre::ok), so those
// loads ride along with the first weight chunk.
struct NoPre {
  bool ok = false;
};
template <typename T> struct EpiStore {
  static constexpr bool kRowStream = true, kSplitK = true, kQkv = false;
  using Pre = NoPre;
  __device__ Pre prefetch(int, int, int) const { return {}; }
  static constexpr int kMidNtw = 0, kMidNtwMin = 1;
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
  // a thread per element when that is one round, else per (row, 8 adjacent
  // columns) with one vector store where aligned
  __device__ void finish(float *tile, int ldt, int M, int c0, int span, const Pre &) const {
    const int gpr = span >> 3;
    if (M * span <= (int)blockDim.x) {
      const int idx = threadIdx.x, m = idx / span, c = idx % span;
      if (idx < M * span && c0 + c < nvcols) out[(size_t)m * ldo + c0 + c] = Elt<T>::from_f(tile[m * ldt + c]);
    }
    for (int idx = threadIdx.x; M * span > (int)blockDim.x && idx < M * gpr; idx += blockDim.x) {
      const int m = idx / gpr, c = (idx % gpr) * 8;
      T *y = out + (size_t)m * ldo + c0 + c;
      const float *t = tile + m * ldt + c;
      if (c0 + c + 8 <= nvcols && aligned16(y)) {
        float v[8];
        tile8(t, ldt, v);
        store8<T>(y, v);
      } else {
        for (int j = 0; j < 8 && c0 + c + j < nvcols; ++j) y[j] = Elt<T>::from_f(t[j]);
      }
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
  static constexpr bool kRowStream = true, kSplitK = true, kQkv = false;
  static constexpr int kMidNtw = 0, kMidNtwMin = 1;
  const T *w;
  int ldw, nvcols;
  float *out;
  long ldo;
  const float *resid;
  long ldr;
  float *ssq;  // optional per-(row, 16-column tile) sums of squares of the output
  int ssq_rs, ssq_off;
  GainCopies gc;
  struct Pre {  // raw values: converted where used, so no load is waited for early
    bool ok = false;
    float r = 0.f;
    T g[kMaxLayers + 1];
  };
  __device__ const T *wrow(int c) const { return w + (size_t)c * ldw; }
  // residual and gains of element idx = threadIdx.x, when every element has
  // its own thread (clamped in-bounds loads)
  __device__ Pre prefetch(int M, int c0, int span) const {
    Pre p;
    const int idx = threadIdx.x;
    if (M * span > (int)blockDim.x || idx >= M * span) return p;
    const int m = idx / span, cc = min(c0 + idx % span, nvcols - 1);
    p.ok = true;
    if (resid) p.r = resid[(size_t)m * ldr + cc];
    if (gc.n > 0) {
#pragma unroll
      for (int q = 0; q < kMaxLayers + 1; ++q)
        p.g[q] = ((const T *)gc.gamma[min(q, gc.n - 1)])[cc];
    }
    return p;
  }
  __device__ void finish(float *tile, int ldt, int M, int c0, int span, const Pre &pre) const {
    for (int idx = threadIdx.x; idx < M * span; idx += blockDim.x) {
      const int m = idx / span, c = idx % span;
      if (c0 + c >= nvcols) continue;
      const bool own = pre.ok && idx == (int)threadIdx.x;
      float v = tile[m * ldt + c];
      if (resid) v = (own ? pre.r : resid[(size_t)m * ldr + c0 + c]) + v;
      out[(size_t)m * ldo + c0 + c] = v;
      tile[m * ldt + c] = v;
      if (own) {
#pragma unroll
        for (int q = 0; q < kMaxLayers + 1; ++q)
          if (q < gc.n)
            ((T *)gc.dst[q])[(size_t)m * gc.ld[q] + c0 + c] = Elt<T>::from_f(Elt<T>::to_f(pre.g[q]) * v);
      } else {
        for (int q = 0; q < gc.n; ++q)
          ((T *)gc.dst[q])[(size_t)m * gc.ld[q] + c0 + c] =
              Elt<T>::from_f(Elt<T>::to_f(((const T *)gc.gamma[q])[c0 + c]) * v);
      }
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
  static constexpr bool kRowStream = true, kSplitK = true, kQkv = true;
  using Pre = NoPre;
  __device__ Pre prefetch(int, int, int) const { return {}; }
  static constexpr int kMidNtw = 0, kMidNtwMin = 1;
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
  // only the last context row of a sequence carries a query
  __device__ bool row_used(int m, int c0) const {
    return c0 >= a.Hq * a.D || m % a.nctx == a.nctx - 1;
  }
  __device__ void finish(float *tile, int ldt, int M, int c0, int span, const Pre &p) const {
    if (M * span > (int)blockDim.x) {
      finish8(tile, ldt, M, c0, span);
      return;
    }
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
        if (!a.rotate) {  // attention rotates
          if (isq)
            a.q_out[((size_t)b * a.Hq + h) * D + dd] = val;
          else
            a.k_out[(((size_t)b * a.nctx + t) * a.Hkv + h) * D + dd] = val;
          continue;
        }
        const float pv = tile[m * ldt + (c ^ 8)];
        const int P = a.seqs.end(b) - a.seqs.start(b);
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
  // Many rows: a thread per (row, 8 adjacent virtual columns), which are 8
  // adjacent dimensions of one head's query or key (one rotary half, paired
  // with the 8 columns 8 away in the same 16-column tile) or of a value row.
  __device__ void finish8(const float *tile, int ldt, int M, int c0, int span) const {
    const int qd = a.Hq * a.D, kvd = a.Hkv * a.D, D = a.D;
    const int gpr = span >> 3;
    for (int idx = threadIdx.x; idx < M * gpr; idx += blockDim.x) {
      const int m = idx / gpr, c = (idx % gpr) * 8, vc = c0 + c;
      if (vc >= nvcols) continue;
      const int b = m / a.nctx, t = m % a.nctx;
      const float *tv = tile + m * ldt + c;
      float o[8];
      float *y;
      if (vc < qd + kvd) {
        const bool isq = vc < qd;
        if (isq && t != a.nctx - 1) continue;
        const int lc = isq ? vc : vc - qd;
        const int h = lc / D, cc = lc % D;
        if (!a.rotate) {  // attention rotates
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = tv[e];
        } else {
          const float *pt = tile + m * ldt + (c ^ 8);
          const int P = a.seqs.end(b) - a.seqs.start(b);
          const int pos = min(a.cascade ? P + a.j0 + t : P, a.rope_npos - 1);
          // rotary pair index 8 (cc >> 4) + e of dims rope_dim(cc, D) + e
          const float *rp = a.rope + ((size_t)pos * (D / 2) + 8 * (cc >> 4)) * 2;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float cs = rp[2 * e], sn = rp[2 * e + 1];
            o[e] = (cc & 8) ? (tv[e] * cs + pt[e] * sn) : (tv[e] * cs - pt[e] * sn);
          }
        }
        y = isq ? a.q_out + ((size_t)b * a.Hq + h) * D + rope_dim(cc, D)
                : a.k_out + (((size_t)b * a.nctx + t) * a.Hkv + h) * D + rope_dim(cc, D);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = tv[e];
        y = a.v_out + ((size_t)b * a.nctx + t) * kvd + (vc - qd - kvd);
      }
      if (aligned16(y)) {
        store8<float>(y, o);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] = o[e];
      }
    }
  }
};

// Cache rows of verified positions: virtual columns [0, kvd) are the key
// rows of W_k (rotary pairs packed per 16-column tile as for EpiQkv), then
// the value rows; row m is rotated at positions[m] and stored in the storage
// type at cache row dst_rows[m].
template <typename T> struct EpiKvCache {
  static constexpr bool kRowStream = true, kSplitK = true, kQkv = false;
  using Pre = NoPre;
  __device__ Pre prefetch(int, int, int) const { return {}; }
  static constexpr int kMidNtw = 0, kMidNtwMin = 1;
  KvCacheArgs a;
  int nvcols;  // 2 * Hkv * D
  __device__ const T *wrow(int c) const {
    const int kvd = a.Hkv * a.D;
    if (c < kvd) return (const T *)a.wk + (size_t)((c / a.D) * a.D + rope_dim(c % a.D, a.D)) * a.d;
    return (const T *)a.wv + (size_t)(c - kvd) * a.d;
  }
  // A thread per (row, 8 adjacent virtual columns): those are 8 adjacent
  // dimensions of one head's key (inside one rotary half, paired with the 8
  // columns 8 away in the same 16-column tile) or of a value row, so each
  // group is one vector store of the cache row piece.
  // With at most one element per thread the thread takes one element.
  __device__ void finish(float *tile, int ldt, int M, int c0, int span, const Pre &) const {
    const int kvd = a.Hkv * a.D, D = a.D;
    const float qnan = __int_as_float(0x7fc00000);
    const bool one = M * span <= (int)blockDim.x;
    const int per = one ? 1 : 8, gpr = span / per;
    for (int idx = threadIdx.x; idx < M * gpr; idx += blockDim.x) {
      const int m = idx / gpr, c = (idx % gpr) * per, vc = c0 + c;
      if (vc >= nvcols) continue;
      const long dst = a.dst_rows[m];
      if (dst < 0 || dst >= a.cache_rows) continue;  // nowhere to write
      const int pos = a.positions[m];
      const bool bad = pos < 0 || pos >= a.pos_limit;
      const float *t = tile + m * ldt + c;
      float o[8];
      T *y;
      if (one) {  // a single element
        if (vc < kvd) {
          const int h = vc / D, cc = vc % D;
          const int pc = min(max(pos, 0), a.pos_limit - 1);
          const float *rp = a.rope + ((size_t)pc * (D / 2) + 8 * (cc >> 4) + (cc & 7)) * 2;
          const float pv = tile[m * ldt + (c ^ 8)];
          const float v = bad ? qnan : ((cc & 8) ? (t[0] * rp[0] + pv * rp[1]) : (t[0] * rp[0] - pv * rp[1]));
          ((T *)a.k_cache)[(size_t)dst * kvd + (size_t)h * D + rope_dim(cc, D)] = Elt<T>::from_f(v);
        } else {
          ((T *)a.v_cache)[(size_t)dst * kvd + (vc - kvd)] = Elt<T>::from_f(bad ? qnan : t[0]);
        }
        continue;
      }
      if (vc < kvd) {
        const int h = vc / D, cc = vc % D;
        const int pc = min(max(pos, 0), a.pos_limit - 1);
        // rotary pair index 8 (cc >> 4) + j of dims rope_dim(cc, D) + j
        const float *rp = a.rope + ((size_t)pc * (D / 2) + 8 * (cc >> 4)) * 2;
        float tv[8], pv[8];
        tile8(t, ldt, tv);
        tile8(tile + m * ldt + (c ^ 8), ldt, pv);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float cs = rp[2 * j], sn = rp[2 * j + 1];
          o[j] = bad ? qnan : ((cc & 8) ? (tv[j] * cs + pv[j] * sn) : (tv[j] * cs - pv[j] * sn));
        }
        y = (T *)a.k_cache + (size_t)dst * kvd + (size_t)h * D + rope_dim(cc, D);
      } else {
        tile8(t, ldt, o);
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = bad ? qnan : o[j];
        y = (T *)a.v_cache + (size_t)dst * kvd + (vc - kvd);
      }
      if (aligned16(y)) {
        store8<T>(y, o);
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = Elt<T>::from_f(o[j]);
      }
    }
  }
};

// Row-block slices of the cache update's GEMMs (bf16, many rows per launch).
// Fusion FC: EpiStore with the embedding gather of the block's own rows.
struct TileStore : EpiStore<bf16_t> {
  static constexpr bool kSliced = true;
  int lda;
  __device__ void slice(int z, int mrows, const bf16_t *&A, int &M) {
    const int m0 = z * mrows;
    A += (size_t)m0 * lda;
    M = min(mrows, M - m0);
    out += (size_t)m0 * ldo;
    if (embed) {
      tokens += m0;
      gather_out += (size_t)m0 * ld_gather;
      B = M;
    }
  }
};
// Input FC into fp32 rows (out = A W^T), or with `resid` a residual FC
// (out = resid + A W^T).
struct TileF32 {
  static constexpr bool kRowStream = true, kSplitK = false, kSliced = true;
  using Pre = NoPre;
  __device__ Pre prefetch(int, int, int) const { return {}; }
  static constexpr int kMidNtw = 0, kMidNtwMin = 1;
  const bf16_t *w;
  int ldw, nvcols;
  float *out;
  long ldo;
  int lda;
  const float *resid = nullptr;
  long ldr = 0;
  __device__ const bf16_t *wrow(int c) const { return w + (size_t)c * ldw; }
  __device__ void slice(int z, int mrows, const bf16_t *&A, int &M) {
    const int m0 = z * mrows;
    A += (size_t)m0 * lda;
    M = min(mrows, M - m0);
    out += (size_t)m0 * ldo;
    if (resid) resid += (size_t)m0 * ldr;
  }
  // a thread per (row, 4 adjacent columns): vector loads and stores where aligned
  __device__ void finish(float *tile, int ldt, int M, int c0, int span, const Pre &) const {
    const int gpr = span >> 2;
    for (int idx = threadIdx.x; idx < M * gpr; idx += blockDim.x) {
      const int m = idx / gpr, c = (idx % gpr) * 4;
      float *y = out + (size_t)m * ldo + c0 + c;
      const float *rr = resid ? resid + (size_t)m * ldr + c0 + c : nullptr;
      const float *t = tile + m * ldt + c;
      if (c0 + c + 4 <= nvcols && aligned16(y) && (!rr || aligned16(rr))) {
        f32x4 v = (ldt & 3) == 0 ? *reinterpret_cast<const f32x4 *>(t) : f32x4{t[0], t[1], t[2], t[3]};
        if (rr) v += *reinterpret_cast<const f32x4 *>(rr);
        *reinterpret_cast<f32x4 *>(y) = v;
      } else {
        for (int j = 0; j < 4 && c0 + c + j < nvcols; ++j) y[j] = t[j] + (rr ? rr[j] : 0.f);
      }
    }
  }
};
// K/V cache rows of every layer: slice z = layer * row blocks + block, A
// holds the layers' normalised rows a_layer_stride elements apart.  The layers
// differ only in their weights and caches; those pointers travel in the kernel
// arguments and a slice picks its layer's with an unrolled select (a uniform
// choice: no indexed copy of the arguments).
struct KvGroup {
  int nblocks, lda;
  long a_layer_stride;
  const void *wk[kMaxLayers], *wv[kMaxLayers];
  void *kc[kMaxLayers], *vc[kMaxLayers];
};
struct TileKv {
  static constexpr bool kRowStream = true, kSplitK = false, kSliced = true;
  using Pre = NoPre;
  __device__ Pre prefetch(int, int, int) const { return {}; }
  static constexpr int kMidNtw = 0, kMidNtwMin = 1;
  EpiKvCache<bf16_t> cur;
  int nvcols;
  KvGroup g;
  __device__ void slice(int z, int mrows, const bf16_t *&A, int &M) {
    const int l = z / g.nblocks, m0 = (z % g.nblocks) * mrows;
#pragma unroll
    for (int q = 0; q < kMaxLayers; ++q)
      if (q == l) {
        cur.a.wk = g.wk[q];
        cur.a.wv = g.wv[q];
        cur.a.k_cache = g.kc[q];
        cur.a.v_cache = g.vc[q];
      }
    cur.a.positions += m0;
    cur.a.dst_rows += m0;
    A += l * g.a_layer_stride + (size_t)m0 * g.lda;
    M = min(mrows, M - m0);
  }
  __device__ const bf16_t *wrow(int c) const { return cur.wrow(c); }
  __device__ void finish(float *tile, int ldt, int M, int c0, int span, const Pre &p) const {
    cur.finish(tile, ldt, M, c0, span, p);
  }
};

template <typename T> struct EpiSwiglu {
  static constexpr bool kRowStream = true, kSplitK = false;
  using Pre = NoPre;
  __device__ Pre prefetch(int, int, int) const { return {}; }
  static constexpr int kMidNtw = 0, kMidNtwMin = 2;  // gate/up tile pairs
  const T *wg, *wu;
  int ldw, I, nvcols;  // nvcols = 2*I
  T *out;
  int ldo;
  // virtual tile pair (2p, 2p+1) = gate rows and up rows 16p..16p+15
  __device__ const T *wrow(int c) const {
    const int p = c >> 5, f = (c >> 4) & 1, n = c & 15;
    return (f ? wu : wg) + (size_t)(p * 16 + n) * ldw;
  }
  // a thread per output when that is one round, else per (row, 8 adjacent
  // gate columns): 8 adjacent outputs, one vector store where aligned
  __device__ void finish(float *tile, int ldt, int M, int c0, int span, const Pre &) const {
    const int half = span >> 1, gpr = span >> 4;
    if (M * half <= (int)blockDim.x) {
      const int idx = threadIdx.x, m = idx / half, q = idx % half;
      const int c = (q >> 4) * 32 + (q & 15);  // gate column inside the tile
      const int vc = c0 + c;
      if (idx < M * half && vc < nvcols) {
        const float gt = tile[m * ldt + c], up = tile[m * ldt + c + 16];
        const float s = gt / (1.f + expf(-gt)) * up;
        out[(size_t)m * ldo + (vc >> 5) * 16 + (vc & 15)] = Elt<T>::from_f(s);
      }
      return;
    }
    for (int idx = threadIdx.x; idx < M * gpr; idx += blockDim.x) {
      const int m = idx / gpr, q = (idx % gpr) * 8;
      const int c = (q >> 4) * 32 + (q & 15);  // first gate column inside the tile
      const int vc = c0 + c;
      if (vc >= nvcols) continue;
      const float *t = tile + m * ldt + c;
      float gt[8], up[8], s[8];
      tile8(t, ldt, gt);
      tile8(t + 16, ldt, up);
#pragma unroll
      for (int j = 0; j < 8; ++j) s[j] = gt[j] / (1.f + expf(-gt[j])) * up[j];
      T *y = out + (size_t)m * ldo + (vc >> 5) * 16 + (vc & 15);
      if (vc + 8 <= nvcols && aligned16(y)) {
        store8<T>(y, s);
      } else {
        for (int j = 0; j < 8 && vc + j < nvcols; ++j) y[j] = Elt<T>::from_f(s[j]);
      }
    }
  }
};

// Gate/up + SwiGLU over row blocks (the multi-position prefill's MLP).
struct TileSwiglu : EpiSwiglu<bf16_t> {
  static constexpr bool kSliced = true;
  int lda;
  __device__ void slice(int z, int mrows, const bf16_t *&A, int &M) {
    const int m0 = z * mrows;
    A += (size_t)m0 * lda;
    M = min(mrows, M - m0);
    out += (size_t)m0 * ldo;
  }
};

// Shared LM head: per (row, column tile) max, sum of exp(z - max) and the top-k
// (largest logit first, equal logits by lower draft id); logits optionally kept.
template <typename T> struct EpiLm {
  static constexpr bool kRowStream = false, kSplitK = false;
  using Pre = NoPre;
  __device__ Pre prefetch(int, int, int) const { return {}; }
  static constexpr int kMidNtw = 4, kMidNtwMin = 4;  // 64-column tiles, as lmhead_tiles counts
  LmArgs a;
  int ldw, nvcols;
  __device__ const T *wrow(int c) const { return (const T *)a.w + (size_t)c * ldw; }

  // Many rows (batched drafting): thread = row.  The tile's columns are
  // scanned in increasing id order into a sorted list of KL (value, id)
  // pairs; an equal value never displaces an earlier entry, so ties go to the
  // lower id without comparing ids.  NaN compares false and is never taken.
  // selection key of tempered logit xt at column col of row m: xt, or
  // xt + Gumbel(u) = xt - log(-log(u)) for sampling without replacement
  __device__ float sel_key(float xt, int m, int col) const {
    if (!a.draws.on()) return xt;
    const float u = a.draws.at((uint64_t)m * nvcols + col);
    return xt - logf(-logf(u));
  }

  template <int KL>
  __device__ void finish_rows(const float *tile, int ldt, int M, int c0, int span) const {
    const int m = threadIdx.x;
    if (m >= M) return;
    const int nvalid = min(span, nvcols - c0);
    const int nwg = gridDim.x, tileid = blockIdx.x;
    const float *row = tile + m * ldt;
    float mx = -INFINITY;
    for (int c = 0; c < nvalid; ++c) mx = fmaxf(mx, row[c] * a.inv_temp);
    float se = 0.f;
    float vs[KL], zs[KL];
    int is[KL];
#pragma unroll
    for (int j = 0; j < KL; ++j) {
      vs[j] = -INFINITY;
      zs[j] = -INFINITY;
      is[j] = 0x7fffffff;
    }
    // counter-based draws: one generator block per four consecutive columns
    const bool gen = a.draws.so != nullptr;
    const uint64_t seed = gen ? a.draws.so[0] : 0, offset = gen ? a.draws.so[1] : 0;
    uint64_t have = ~0ull;
    float ub[4] = {0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < nvalid; ++c) {
      const float x = row[c], xt = x * a.inv_temp;
      float key = xt;
      if (gen) {
        const uint64_t e = (uint64_t)m * nvcols + c0 + c;
        if ((e >> 2) != have) {
          have = e >> 2;
          philox_block(seed, offset, have, ub);
        }
        const int w = (int)(e & 3);
        const float u = w == 0 ? ub[0] : w == 1 ? ub[1] : w == 2 ? ub[2] : ub[3];
        key = xt - logf(-logf(u));
      } else {
        key = sel_key(xt, m, c0 + c);
      }
      se += expf(xt - mx);
      if (a.logits) a.logits[(size_t)m * nvcols + c0 + c] = x;
      if (!(vs[KL - 1] < key)) continue;  // not in the list: nothing below would change
#pragma unroll
      for (int j = KL - 1; j >= 1; --j) {
        const bool prev = vs[j - 1] < key, here = vs[j] < key;
        vs[j] = prev ? vs[j - 1] : (here ? key : vs[j]);
        zs[j] = prev ? zs[j - 1] : (here ? xt : zs[j]);
        is[j] = prev ? is[j - 1] : (here ? c0 + c : is[j]);
      }
      if (vs[0] < key) {
        vs[0] = key;
        zs[0] = xt;
        is[0] = c0 + c;
      }
    }
    const size_t pb = (size_t)m * nwg + tileid;
    a.part_max[pb] = mx;
    a.part_sum[pb] = se;
#pragma unroll
    for (int j = 0; j < KL; ++j)
      if (j < a.topk) {
        a.cand_val[pb * kMaxTopk + j] = is[j] != 0x7fffffff ? vs[j] : -INFINITY;
        a.cand_idx[pb * kMaxTopk + j] = is[j];
        if (a.draws.on()) a.cand_z[pb * kMaxTopk + j] = zs[j];
      }
  }

  __device__ void finish(float *tile, int ldt, int M, int c0, int span, const Pre &) const {
    if (M > 16) {
      if (a.topk <= 2) finish_rows<2>(tile, ldt, M, c0, span);
      else if (a.topk <= 4) finish_rows<4>(tile, ldt, M, c0, span);
      else if (a.topk <= 8) finish_rows<8>(tile, ldt, M, c0, span);
      else finish_rows<16>(tile, ldt, M, c0, span);
      return;
    }
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
        if (a.logits && ok) a.logits[(size_t)m * nvcols + id[p]] = v[p];
        v[p] *= a.inv_temp;   // statistics and candidates at temperature T
        mx = fmaxf(mx, v[p]);
      }
      mx = group_max<64>(mx);
      float se = 0.f;
#pragma unroll
      for (int p = 0; p < PER; ++p) se += (id[p] != 0x7fffffff) ? expf(v[p] - mx) : 0.f;
      se = group_sum<64>(se);
      const size_t pb = (size_t)m * nwg + tileid;
      if (lane == 0) {
        a.part_max[pb] = mx;
        a.part_sum[pb] = se;
      }
      uint64_t key[PER];
      const uint64_t e0 = (uint64_t)m * nvcols + c0;  // uniform of column c0
      if (a.draws.so != nullptr && (e0 & 3) == 0) {
        // counter-based draws, block-aligned tile row: lane q draws block
        // e0/4 + q (columns 4q .. 4q+3), and lane l takes column l + 64p's
        // uniform from lane l/4 + 16p, word l & 3
        float ub[4];
        philox_block(a.draws.so[0], a.draws.so[1], (e0 >> 2) + lane, ub);
        const int w = lane & 3;
#pragma unroll
        for (int p = 0; p < PER; ++p) {
          const int src = (lane >> 2) + 16 * p;
          const float u0 = __shfl(ub[0], src, 64), u1 = __shfl(ub[1], src, 64);
          const float u2 = __shfl(ub[2], src, 64), u3 = __shfl(ub[3], src, 64);
          const float u = w == 0 ? u0 : w == 1 ? u1 : w == 2 ? u2 : u3;
          key[p] = id[p] != 0x7fffffff ? topk_key(v[p] - logf(-logf(u)), id[p]) : kNoKey;
        }
      } else {
#pragma unroll
        for (int p = 0; p < PER; ++p)
          key[p] = id[p] != 0x7fffffff ? topk_key(sel_key(v[p], m, id[p]), id[p]) : kNoKey;
      }
      for (int r = 0; r < a.topk; ++r) {
        // lane-local best, then wave max of the ordering keys (lower id wins ties)
        uint64_t best = kNoKey;
#pragma unroll
        for (int p = 0; p < PER; ++p) best = key[p] > best ? key[p] : best;
        best = wave_max_u64(best);
        float zb = -INFINITY;  // z / T of the winner, from the lane that holds it
#pragma unroll
        for (int p = 0; p < PER; ++p) {
          zb = key[p] == best ? v[p] : zb;
          key[p] = key[p] == best ? kNoKey : key[p];
        }
        if (a.draws.on()) zb = group_max<64>(zb);
        if (lane == 0) {
          const bool got = best != kNoKey;
          a.cand_val[pb * kMaxTopk + r] = got ? topk_key_value(best) : -INFINITY;
          a.cand_idx[pb * kMaxTopk + r] = got ? topk_key_id(best) : 0x7fffffff;
          if (a.draws.on()) a.cand_z[pb * kMaxTopk + r] = got ? zb : -INFINITY;
        }
      }
    }
  }
};

// ---------------------------------------------------------------------------
// Dispatch.
// ---------------------------------------------------------------------------
// Split-K width of the up-to-32-row kernel.
template <int WKmax, int MT> struct SplitK {
  static constexpr int cap = 8;
  static constexpr int value = WKmax < cap ? WKmax : cap;
};

template <class Epi>
static hipError_t run_gemv(const bf16_t *A, int lda, const ARows &arows, int M, int K,
                           const Epi &epi, const NormA *na, int mr, size_t lds, hipStream_t s) {
  constexpr int W = 4 * (Epi::kMidNtwMin > 1 ? Epi::kMidNtwMin : 1);  // SPAN = 16 * kMidNtwMin
  constexpr int SPAN = 4 * W;
  const int grid = (epi.nvcols + SPAN - 1) / SPAN;
  const NormA n0 = na ? *na : NormA{nullptr, 0, 1, 0, 1, 1, 0.f};
#define FE_GEMV(MRV, NORMV)                                                                      \
  hipLaunchKernelGGL((k_gemv<MRV, W, NORMV, Epi>), dim3(grid), dim3(64 * W), lds, s, A, lda, arows, \
                     M, K, n0, epi)
#define FE_GEMV_M(NORMV)              \
  switch (mr) {                       \
    case 1: FE_GEMV(1, NORMV); break; \
    case 2: FE_GEMV(2, NORMV); break; \
    default: FE_GEMV(4, NORMV); break; \
  }
  if (na) FE_GEMV_M(true) else FE_GEMV_M(false)
#undef FE_GEMV_M
#undef FE_GEMV
  return hipGetLastError();
}

// Where a split-K GEMM left its fp32 slices when the caller finishes them
// itself (ks = 0: the GEMM was not split and its epilogue ran).
struct SplitOut {
  const float *p = nullptr;
  int ldp = 0, ks = 0;
};

// batched rows above this go to k_gemm_tile's split-K path when the epilogue
// allows (measured at batch 32: the Q/K/V GEMM from 32 rows, 15.7 us against
// 18.4 on k_gemm_mid; the 32-row residual GEMMs stay on k_gemm_mid, whose
// half-height tiles were 8 % faster there)
constexpr int kTileSplitMinRows = 32, kTileSplitMinRowsQkv = 16;

// split-K slices of the narrow batched-rows GEMMs (at most 128 rows): up to
// kSliceCap32 slices, about kSliceWgs workgroups
constexpr int kSliceCap32 = 8, kSliceWgs = 256;

// ring stages of the at-most-32-row configuration: four keep two workgroups
// per CU (measured at the 8B batch-32 shapes: 1962 us per pass, against 1992
// with six stages and 1996 with 64-row tiles)
constexpr int kHalfStages = 4;

template <typename T, int NT, int WKmax, int WN, class Epi>
static hipError_t run_gemm(const T *A, int lda, const ARows &arows, int M, int K, const Epi &epi,
                           const NormA *na, hipStream_t s, const SplitScratch *ss = nullptr,
                           SplitOut *so = nullptr) {
  if (so) *so = SplitOut{};
  constexpr int SPAN = WN * NT * 16;
  const int grid = (epi.nvcols + SPAN - 1) / SPAN;
  const int mt = (M + 15) / 16;
  const NormA n0 = na ? *na : NormA{nullptr, 0, 1, 0, 1, 1, 0.f};
  if constexpr (sizeof(T) == 2) {
    // up to 4 rows whose padded input rows fit the LDS budget: row streaming
    // (the LM head's per-row top-k is cheaper on the matrix-core tiles)
    if constexpr (Epi::kRowStream) {
      const int mr = M <= 1 ? 1 : M <= 2 ? 2 : 4;
      const size_t lds = (size_t)mr * ((K + 127) & ~127) * 2;
      if (M <= 4 && lds <= (size_t)kGvMaxLds && K >= 8) return run_gemv(A, lda, arows, M, K, epi, na, mr, lds, s);
    }
  }
  if (na) {
    if (mt != 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_gemm<T, 1, NT, SplitK<WKmax, 1>::value, WN, true, Epi>), dim3(grid),
                       dim3(64 * SplitK<WKmax, 1>::value * WN), 0, s, A, lda, arows, M, K, n0, epi);
    return hipGetLastError();
  }
  // 17..32 rows over wide outputs (the batch-32 gate/up): the LDS-ring kernel
  // with column-split waves beats the per-wave staging; narrow outputs take
  // it too when their epilogue can follow a split-K reduction, else they
  // would leave it too few workgroups
  bool splittable = false;
  if constexpr (Epi::kSplitK) splittable = ss != nullptr && ss->p != nullptr;
  const bool ring_wide = mt == 2 && (epi.nvcols >= 64 * 256 || splittable);
  if (mt <= 2 && !ring_wide) {
    if (mt <= 1)
      hipLaunchKernelGGL((k_gemm<T, 1, NT, SplitK<WKmax, 1>::value, WN, false, Epi>), dim3(grid),
                         dim3(64 * SplitK<WKmax, 1>::value * WN), 0, s, A, lda, arows, M, K, n0, epi);
    else
      hipLaunchKernelGGL((k_gemm<T, 2, NT, SplitK<WKmax, 2>::value, WN, false, Epi>), dim3(grid),
                         dim3(64 * SplitK<WKmax, 2>::value * WN), 0, s, A, lda, arows, M, K, n0, epi);
    return hipGetLastError();
  }
  // batched rows: all M rows per workgroup, columns split over the grid; the
  // waves split columns as well when the rows do not fill four row groups
  if (M > 256) return hipErrorInvalidValue;
  if constexpr (sizeof(T) == 2 && Epi::kSplitK) {
    // More than 32 rows (bf16, K a multiple of 64), when the epilogue can
    // follow a split-K reduction: k_gemm_tile's 256 x 128 tiles (128 x 128 up
    // to 128 rows; all rows in one block, so the weights are streamed once), K split so that the grid
    // is about one workgroup per CU (k_gemm_mid has only one column wave
    // here); the slices are summed, in a fixed order, by the finish launch.
    // The Q/K/V GEMM (6144 columns) aims at fewer slices: six cost more to
    // write and sum than they save (layers of 160-224 rows at batch 32: 33.5
    // us per launch with six, 25.3 with four, 30.3 on k_gemm_mid).
    if (M > (Epi::kQkv ? kTileSplitMinRowsQkv : kTileSplitMinRows) && K % 64 == 0 && ss != nullptr &&
        ss->p != nullptr) {
      const int gx = (epi.nvcols + 127) / 128;
      int ksb = ((Epi::kQkv ? 192 : 288) + gx - 1) / gx;
      ksb = min(ksb, kMaxSlices);
      ksb = max(1, min(ksb, (K / 64) / 8));  // at least 8 chunks of K per slice
      const int ldpb = gx * 128;
      if ((size_t)ksb * M * ldpb <= ss->floats) {
        if (M > 128)
          hipLaunchKernelGGL((k_gemm_tile<4, 4, 4, 2, 3, Epi, true>), dim3(gx, ksb, 1), dim3(512), 0, s,
                             A, lda, arows, M, K, epi, ss->p, ldpb);
        else  // 128 x 128 tiles
          hipLaunchKernelGGL((k_gemm_tile<4, 2, 2, 4, 3, Epi, true>), dim3(gx, ksb, 1), dim3(512), 0, s,
                             A, lda, arows, M, K, epi, ss->p, ldpb);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess || so) {  // the caller sums the slices
          if (so) *so = SplitOut{ss->p, ldpb, ksb};
          return e;
        }
        hipLaunchKernelGGL((k_splitk_finish<Epi>), dim3((epi.nvcols + 15) / 16), dim3(256), 0, s,
                           (const float *)ss->p, ldpb, ksb, M, epi);
        return hipGetLastError();
      }
    }
  }
  const int wn = M <= 64 ? 4 : (M <= 128 ? 2 : 1);
  int tt = Epi::kMidNtw;  // 16-column tiles per workgroup
  if (tt == 0) {
    tt = 2;
    while (tt < 4 && (epi.nvcols + 32 * tt - 1) / (32 * tt) >= 192) tt *= 2;
  }
  if (tt < Epi::kMidNtwMin) tt = Epi::kMidNtwMin;
  if (tt < wn) tt = wn;  // a tile per column group at least
  if (tt < 2) tt = 2;    // weight slots split evenly over the waves
  const int ntw = tt / wn;
  // Narrow outputs whose epilogue allows it: 128-column tiles (a quarter of
  // the re-reading of A that 32-column tiles cost) and K split over enough
  // workgroups to cover the CUs; the fp32 slices are summed, in a fixed order,
  // by a second launch that runs the epilogue.
  int ks = 1;
  float *sp = nullptr;
  int ldp = 0;
  if (splittable) {
    constexpr int KC = 8 * Elt<T>::kPer16B;
    const int gx = (epi.nvcols + 127) / 128, nchk = (K + KC - 1) / KC;
    // about one workgroup per CU (k_splitk_finish sums at most 8 slices); many
    // rows make each slice heavier and its partial sums larger: fewer slices
    ks = min(M > 128 ? 4 : kSliceCap32, max(1, (kSliceWgs + gx - 1) / gx));
    ks = min(ks, kMaxSlices);
    ks = min(ks, max(1, nchk / 4));  // a few chunks per slice for the ring
    ldp = gx * 128;
    if ((size_t)ks * M * ldp > ss->floats) ks = 1;
    if (ks > 1) sp = ss->p;
  }
#define FE_GEMM_MID_RT(NTWV, WNV, SV, RTV)                                                           \
  hipLaunchKernelGGL((k_gemm_mid<T, NTWV, WNV, SV, Epi, RTV>),                                      \
                     dim3((epi.nvcols + 16 * NTWV * WNV - 1) / (16 * NTWV * WNV), ks), dim3(256), 0,  \
                     s, A, lda, arows, M, K, epi, sp, ldp)
#define FE_GEMM_MID(NTWV, WNV, SV) FE_GEMM_MID_RT(NTWV, WNV, SV, 4)
  // at most 32 rows: two 16-row tiles per wave, so the ring carries no
  // duplicated rows of A, and the stages it frees go to a deeper ring
  const bool half = wn == 4 && M <= 32;
  if constexpr (Epi::kSplitK) {
    if (sp) {
      if (wn == 4 && half) FE_GEMM_MID_RT(2, 4, kHalfStages, 2);
      else if (wn == 4) FE_GEMM_MID(2, 4, 4);
      else if (wn == 2) FE_GEMM_MID(4, 2, 4);
      else FE_GEMM_MID(8, 1, 3);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess || so) {  // the caller sums the slices
        if (so) *so = SplitOut{sp, ldp, ks};
        return e;
      }
      hipLaunchKernelGGL((k_splitk_finish<Epi>), dim3((epi.nvcols + 15) / 16), dim3(256), 0, s,
                         (const float *)sp, ldp, ks, M, epi);
      return hipGetLastError();
    }
  }
  if (wn == 4 && half) {
    if (ntw >= 2) FE_GEMM_MID_RT(2, 4, kHalfStages, 2);
    else FE_GEMM_MID_RT(1, 4, kHalfStages, 2);
  } else if (wn == 4) {
    if (ntw >= 2) FE_GEMM_MID(2, 4, 4);
    else FE_GEMM_MID(1, 4, 4);
  } else if (wn == 2) {
    if (ntw >= 2) FE_GEMM_MID(2, 2, 4);
    else FE_GEMM_MID(1, 2, 4);
  } else {
    if (ntw >= 4) FE_GEMM_MID(4, 1, 2);  // the LM head's grid is wide: two workgroups per CU
    else FE_GEMM_MID(2, 1, 3);
  }
#undef FE_GEMM_MID
#undef FE_GEMM_MID_RT
  return hipGetLastError();
}

hipError_t gemm_store(int dt, const void *A, int lda, int M, int K, const void *W, int ncols,
                      void *out, int ldo, const void *embed, const int32_t *tokens, int vocab,
                      void *gather_out, int ld_gather, int d, int B, hipStream_t s,
                      const SplitScratch *ss) {
  if (dt) {
    EpiStore<bf16_t> e{(const bf16_t *)W, K, ncols, (bf16_t *)out, ldo, (const bf16_t *)embed,
                       tokens, vocab, (bf16_t *)gather_out, ld_gather, d, B};
    return run_gemm<bf16_t, 1, 8, 1>((const bf16_t *)A, lda, kDenseRows, M, K, e, nullptr, s, ss);
  }
  EpiStore<float> e{(const float *)W, K, ncols, (float *)out, ldo, (const float *)embed,
                    tokens, vocab, (float *)gather_out, ld_gather, d, B};
  return run_gemm<float, 1, 8, 1>((const float *)A, lda, kDenseRows, M, K, e, nullptr, s, ss);
}

template <typename T>
static hipError_t resid_norm_rows(const T *A, int lda, int M, int K, const T *W, int ncols,
                                  float *out, long ldo, const float *resid, long ldr,
                                  const GainCopies &gains, float eps, hipStream_t s,
                                  const SplitScratch *ss) {
  if (M <= 0) return hipSuccess;
  if (ncols > 8192 || ncols % 4) return hipErrorInvalidValue;
  EpiResid<T> e{W, K, ncols, out, ldo, resid, ldr, nullptr, 1, 0, GainCopies{}};
  SplitOut so;
  const hipError_t ge = run_gemm<T, 1, 8, 1>(A, lda, kDenseRows, M, K, e, nullptr, s, ss, &so);
  if (ge != hipSuccess) return ge;
#define FE_RROWS(NVV)                                                                            \
  hipLaunchKernelGGL((k_resid_rows<T, NVV>), dim3(M), dim3(kRowThreads), 0, s, so.p, so.ldp,      \
                     so.ks, M, ncols, resid, ldr, out, ldo, gains, eps)
  if (ncols <= 4 * kRowThreads) FE_RROWS(1);
  else FE_RROWS(2);
#undef FE_RROWS
  return hipGetLastError();
}

hipError_t gemm_resid(int dt, const void *A, int lda, int M, int K, const void *W, int ncols,
                      float *out, long ldo, const float *resid, long ldr, float *ssq, int ssq_rs,
                      int ssq_off, const GainCopies *gains, hipStream_t s, const SplitScratch *ss,
                      float norm_eps) {
  if (norm_eps >= 0.f && gains && gains->n > 0) {
    if (dt)
      return resid_norm_rows<bf16_t>((const bf16_t *)A, lda, M, K, (const bf16_t *)W, ncols, out,
                                     ldo, resid, ldr, *gains, norm_eps, s, ss);
    return resid_norm_rows<float>((const float *)A, lda, M, K, (const float *)W, ncols, out, ldo,
                                  resid, ldr, *gains, norm_eps, s, ss);
  }
  GainCopies gc{};
  if (gains) gc = *gains;
  if (dt) {
    EpiResid<bf16_t> e{(const bf16_t *)W, K, ncols, out, ldo, resid, ldr, ssq, ssq_rs, ssq_off, gc};
    return run_gemm<bf16_t, 1, 8, 1>((const bf16_t *)A, lda, kDenseRows, M, K, e, nullptr, s, ss);
  }
  EpiResid<float> e{(const float *)W, K, ncols, out, ldo, resid, ldr, ssq, ssq_rs, ssq_off, gc};
  return run_gemm<float, 1, 8, 1>((const float *)A, lda, kDenseRows, M, K, e, nullptr, s, ss);
}

hipError_t gemm_qkv(int dt, const void *A, int lda, const ARows &arows, int M, const QkvArgs &a,
                    const NormA *na, hipStream_t s, const SplitScratch *ss) {
  const int nv = (a.Hq + 2 * a.Hkv) * a.D;
  if (dt) {
    EpiQkv<bf16_t> e{a, nv};
    return run_gemm<bf16_t, 1, 4, 1>((const bf16_t *)A, lda, arows, M, a.d, e, na, s, ss);
  }
  EpiQkv<float> e{a, nv};
  return run_gemm<float, 1, 8, 1>((const float *)A, lda, arows, M, a.d, e, na, s, ss);
}

hipError_t gemm_kvcache(int dt, const void *A, int lda, int M, const KvCacheArgs &a,
                        hipStream_t s, const SplitScratch *ss) {
  if (M <= 0) return hipSuccess;
  const int nv = 2 * a.Hkv * a.D;
  if (dt) {
    EpiKvCache<bf16_t> e{a, nv};
    return run_gemm<bf16_t, 1, 4, 1>((const bf16_t *)A, lda, kDenseRows, M, a.d, e, nullptr, s, ss);
  }
  EpiKvCache<float> e{a, nv};
  return run_gemm<float, 1, 8, 1>((const float *)A, lda, kDenseRows, M, a.d, e, nullptr, s, ss);
}

// Many rows at once (bf16): 128 x 128 output tiles of k_gemm_tile (K a
// multiple of 64; else k_gemm_mid's 128 x 64 tiles), grid z over 128-row
// blocks (and layers), no split of K.
constexpr int kTileNtw = 2, kTileWn = 2, kTileStages = 3, kTileRows = 64 * (4 / kTileWn),
              kTileCols = 16 * kTileNtw * kTileWn;
static_assert(kTileRows == kBigRows, "both tiled kernels slice 128-row blocks (TileKv's nblocks)");

hipError_t gemm_store_rows(const void *A, int lda, int M, int K, const void *W, int ncols, void *out,
                           int ldo, const void *embed, const int32_t *tokens, int vocab,
                           void *gather_out, int ld_gather, int d, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  TileStore e;
  static_cast<EpiStore<bf16_t> &>(e) = EpiStore<bf16_t>{(const bf16_t *)W, K, ncols, (bf16_t *)out,
                                                        ldo, (const bf16_t *)embed, tokens, vocab,
                                                        (bf16_t *)gather_out, ld_gather, d, M};
  e.lda = lda;
  if (K % 64 == 0) return launch_tile((const bf16_t *)A, lda, M, K, e, ncols, (M + kBigRows - 1) / kBigRows, s);
  const dim3 grid((ncols + kTileCols - 1) / kTileCols, 1, (M + kTileRows - 1) / kTileRows);
  hipLaunchKernelGGL((k_gemm_mid<bf16_t, kTileNtw, kTileWn, kTileStages, TileStore>), grid, dim3(256),
                     0, s, (const bf16_t *)A, lda, kDenseRows, M, K, e, nullptr, 0);
  return hipGetLastError();
}

hipError_t gemm_swiglu_rows(const void *A, int lda, int M, int K, const void *w_gate,
                            const void *w_up, int I, void *out, int ldo, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  TileSwiglu e;
  static_cast<EpiSwiglu<bf16_t> &>(e) = EpiSwiglu<bf16_t>{(const bf16_t *)w_gate, (const bf16_t *)w_up,
                                                          K, I, 2 * I, (bf16_t *)out, ldo};
  e.lda = lda;
  if (K % 64 == 0) return launch_tile((const bf16_t *)A, lda, M, K, e, 2 * I, (M + kBigRows - 1) / kBigRows, s);
  const dim3 grid((2 * I + kTileCols - 1) / kTileCols, 1, (M + kTileRows - 1) / kTileRows);
  hipLaunchKernelGGL((k_gemm_mid<bf16_t, kTileNtw, kTileWn, kTileStages, TileSwiglu>), grid,
                     dim3(256), 0, s, (const bf16_t *)A, lda, kDenseRows, M, K, e, nullptr, 0);
  return hipGetLastError();
}

hipError_t gemm_resid_rows(const void *A, int lda, int M, int K, const void *W, int ncols, float *out,
                           long ldo, hipStream_t s, const float *resid, long ldr) {
  if (M <= 0) return hipSuccess;
  TileF32 e{(const bf16_t *)W, K, ncols, out, ldo, lda};
  e.resid = resid;
  e.ldr = ldr;
  if (K % 64 == 0) return launch_tile((const bf16_t *)A, lda, M, K, e, ncols, (M + kBigRows - 1) / kBigRows, s);
  const dim3 grid((ncols + kTileCols - 1) / kTileCols, 1, (M + kTileRows - 1) / kTileRows);
  hipLaunchKernelGGL((k_gemm_mid<bf16_t, kTileNtw, kTileWn, kTileStages, TileF32>), grid, dim3(256),
                     0, s, (const bf16_t *)A, lda, kDenseRows, M, K, e, nullptr, 0);
  return hipGetLastError();
}

hipError_t gemm_kv_rows(const void *A, int lda, long a_layer_stride, int M, int nlayers,
                        const KvCacheArgs *layers, const NormA *na, hipStream_t s) {
  if (M <= 0 || nlayers <= 0) return hipSuccess;
  if (nlayers > kMaxLayers || (na && M > 16)) return hipErrorInvalidValue;
  TileKv e{};
  e.cur = EpiKvCache<bf16_t>{layers[0], 2 * layers[0].Hkv * layers[0].D};
  e.nvcols = e.cur.nvcols;
  e.g.lda = lda;
  e.g.a_layer_stride = a_layer_stride;
  for (int l = 0; l < nlayers; ++l) {
    e.g.wk[l] = layers[l].wk;
    e.g.wv[l] = layers[l].wv;
    e.g.kc[l] = layers[l].k_cache;
    e.g.vc[l] = layers[l].v_cache;
  }
  if (na) {
    // up to 16 rows, A = gamma * x per layer and the rows' sums of squares:
    // 16-column workgroups with K split over their four waves, grid y = layer
    e.g.nblocks = 1;
    const dim3 grid((e.nvcols + 15) / 16, nlayers);
    hipLaunchKernelGGL((k_gemm<bf16_t, 1, 1, 4, 1, true, TileKv>), grid, dim3(256), 0, s,
                       (const bf16_t *)A, lda, kDenseRows, M, layers[0].d, *na, e);
    return hipGetLastError();
  }
  e.g.nblocks = (M + kTileRows - 1) / kTileRows;
  if (M < kTileRows) {
    // one row block: the weights are the work, so narrower column tiles give
    // every compute unit a share of them
    constexpr int cols = 16 * 1 * kTileWn;
    const dim3 grid((e.nvcols + cols - 1) / cols, 1, e.g.nblocks * nlayers);
    hipLaunchKernelGGL((k_gemm_mid<bf16_t, 1, kTileWn, kTileStages, TileKv>), grid, dim3(256), 0, s,
                       (const bf16_t *)A, lda, kDenseRows, M, layers[0].d, e, nullptr, 0);
    return hipGetLastError();
  }
  if (layers[0].d % 64 == 0)
    return launch_tile((const bf16_t *)A, lda, M, layers[0].d, e, e.nvcols, e.g.nblocks * nlayers, s);
  const dim3 grid((e.nvcols + kTileCols - 1) / kTileCols, 1, e.g.nblocks * nlayers);
  hipLaunchKernelGGL((k_gemm_mid<bf16_t, kTileNtw, kTileWn, kTileStages, TileKv>), grid, dim3(256), 0,
                     s, (const bf16_t *)A, lda, kDenseRows, M, layers[0].d, e, nullptr, 0);
  return hipGetLastError();
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

// LM head: 64-column tiles, four waves of 16 weight rows each over all of K
// (bf16; 8B batch 1: 49.5 us against 51.7 us for 2 x 2 waves of 32 rows x
// half of K, and 55-88 us for the 8- and 16-wave shapes).
constexpr int kLmWN = 4, kLmNT = 1;
int lmhead_tiles(int V) { return (V + kLmWN * kLmNT * 16 - 1) / (kLmWN * kLmNT * 16); }

hipError_t gemm_lmhead(int dt, const void *A, int lda, const ARows &arows, int M, int K,
                       const LmArgs &a, const NormA *na, int *nwg_out, hipStream_t s) {
  *nwg_out = lmhead_tiles(a.V);
  if (dt && !na && M > 128 && M <= 256 && K % 64 == 0) {
    // many rows (batched drafting, B x N of them): every row in one 256 x 128
    // tile of k_gemm_tile, so the head is streamed once; 128-column tiles
    // (half as many as lmhead_tiles counts)
    EpiLm<bf16_t> e{a, K, a.V};
    const int gx = (a.V + 127) / 128;
    *nwg_out = gx;
    hipLaunchKernelGGL((k_gemm_tile<4, 4, 4, 2, 3, EpiLm<bf16_t>>), dim3(gx), dim3(512), 0, s,
                       (const bf16_t *)A, lda, arows, M, K, e, nullptr, 0);
    return hipGetLastError();
  }
  if (dt) {
    EpiLm<bf16_t> e{a, K, a.V};
    return run_gemm<bf16_t, kLmNT, 1, kLmWN>((const bf16_t *)A, lda, arows, M, K, e, na, s);
  }
  EpiLm<float> e{a, K, a.V};
  return run_gemm<float, kLmNT, 2, kLmWN>((const float *)A, lda, arows, M, K, e, na, s);
}

}  // namespace fe
