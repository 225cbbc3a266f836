// fe_internal.h -- shared device helpers and kernel launchers of libfe.so
// (gfx950 / CDNA4 only).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace fe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

// Storage types: bf16 is carried as its 16-bit pattern.
typedef uint16_t bf16_t;

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float -> bf16, round to nearest even (NaN stays NaN): gfx950's
// v_cvt_pk_bf16_f32, two values per instruction.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f2bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}
__device__ __forceinline__ uint16_t f2bf(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// Top-k ordering key: larger logit first, equal logits by lower id.  The float
// is mapped to an order-preserving 32-bit integer (NaN lowest), the id stored
// inverted below it, so one unsigned 64-bit compare decides.
__device__ __forceinline__ uint64_t topk_key(float v, int id) {
  const uint32_t u = __float_as_uint(v);
  const uint32_t k = (v != v) ? 0u : ((u & 0x80000000u) ? ~u : (u | 0x80000000u));
  return ((uint64_t)k << 32) | (uint64_t)(0xffffffffu - (uint32_t)id);
}
__device__ __forceinline__ float topk_key_value(uint64_t key) {
  const uint32_t k = (uint32_t)(key >> 32);
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}
__device__ __forceinline__ int topk_key_id(uint64_t key) {
  return (int)(0xffffffffu - (uint32_t)key);
}
// 16 bytes per lane from global memory straight into LDS: lane l writes bytes
// 16l..16l+15 after `lds` (wave-uniform).  A plain device function: called
// directly from a kernel template the builtin leaves the kernel without its
// host-side launch stub.
__device__ __forceinline__ void lds_dma16(const void *src, void *lds) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)lds, 16, 0, 0);
}
template <int N> __device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// ---- cross-lane reductions in registers (no LDS traffic) -------------------------
// DPP controls: quad_perm [1,0,3,2] (lane^1), [2,3,0,1] (lane^2), row_half_mirror
// (the other quad of an 8-lane half once quads are uniform), row_ror:8 (lane^8).
template <int CTRL> __device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
// permlane16_swap / permlane32_swap of a register with itself return, in every
// lane, the pair {x[lane], x[lane ^ 16]} (resp. lane ^ 32) in some order.
__device__ __forceinline__ float xor16_sum(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor32_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor16_max(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
// Sum over aligned groups of RL lanes (8, 16, 32), result in every lane of the
// group; each step adds two equal-valued halves in either order, so all lanes
// of a group hold bit-identical sums.
template <int RL> __device__ __forceinline__ float group_sum(float x) {
  x += dpp_f<0xB1>(x);
  x += dpp_f<0x4E>(x);
  x += dpp_f<0x141>(x);
  if constexpr (RL >= 16) x += dpp_f<0x128>(x);
  if constexpr (RL >= 32) x = xor16_sum(x);
  if constexpr (RL >= 64) x = xor32_sum(x);
  return x;
}
template <int RL> __device__ __forceinline__ float group_max(float x) {
  x = fmaxf(x, dpp_f<0xB1>(x));
  x = fmaxf(x, dpp_f<0x4E>(x));
  x = fmaxf(x, dpp_f<0x141>(x));
  if constexpr (RL >= 16) x = fmaxf(x, dpp_f<0x128>(x));
  if constexpr (RL >= 32) x = xor16_max(x);
  if constexpr (RL >= 64) x = xor32_max(x);
  return x;
}
// Max over the row groups of a wave, given values uniform within RL-lane groups.
template <int RL> __device__ __forceinline__ float across_groups_max(float x) {
  if constexpr (RL <= 8) x = fmaxf(x, dpp_f<0x128>(x));
  if constexpr (RL <= 16) x = xor16_max(x);
  if constexpr (RL <= 32) x = xor32_max(x);
  return x;
}

// 64-bit versions: both halves take the same lane permutation.
template <int CTRL> __device__ __forceinline__ uint64_t dpp_u64(uint64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, CTRL, 0xf, 0xf, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(x >> 32), CTRL, 0xf, 0xf, false);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint64_t xor16_max_u64(uint64_t x) {
  const auto l = __builtin_amdgcn_permlane16_swap((uint32_t)x, (uint32_t)x, false, false);
  const auto h = __builtin_amdgcn_permlane16_swap((uint32_t)(x >> 32), (uint32_t)(x >> 32), false, false);
  return umax64(((uint64_t)h[0] << 32) | l[0], ((uint64_t)h[1] << 32) | l[1]);
}
__device__ __forceinline__ uint64_t xor32_max_u64(uint64_t x) {
  const auto l = __builtin_amdgcn_permlane32_swap((uint32_t)x, (uint32_t)x, false, false);
  const auto h = __builtin_amdgcn_permlane32_swap((uint32_t)(x >> 32), (uint32_t)(x >> 32), false, false);
  return umax64(((uint64_t)h[0] << 32) | l[0], ((uint64_t)h[1] << 32) | l[1]);
}
// Maximum over the whole wave, in every lane.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  v = umax64(v, dpp_u64<0xB1>(v));
  v = umax64(v, dpp_u64<0x4E>(v));
  v = umax64(v, dpp_u64<0x141>(v));
  v = umax64(v, dpp_u64<0x128>(v));
  v = xor16_max_u64(v);
  return xor32_max_u64(v);
}
constexpr uint64_t kNoKey = 0ull;  // below every real key (the id 0xffffffff never occurs)

template <typename T> struct Elt;
template <> struct Elt<uint16_t> {
  static constexpr int kPer16B = 8;
  __device__ static __forceinline__ float to_f(uint16_t v) { return bf2f(v); }
  __device__ static __forceinline__ uint16_t from_f(float f) { return f2bf(f); }
};
template <> struct Elt<float> {
  static constexpr int kPer16B = 4;
  __device__ static __forceinline__ float to_f(float v) { return v; }
  __device__ static __forceinline__ float from_f(float f) { return f; }
};

constexpr int kMaxLayers = 16;
// Prefix keys per attention workgroup (4 waves of 32 keys).
constexpr int kAttnChunk = 64;
// Tile candidates the top-k merge holds in registers: 256 threads x 32.
constexpr int kMergeMaxCand = 256 * 32;
// Largest M (rows) one GEMM launch handles; larger M is split on the host.
constexpr int kGemmMaxRows = 256;
constexpr int kMaxTopk = 16;

// Where each query's prefix rows sit in the cache: packed, one sequence after
// the other ([B+1] offsets, rows p[b] .. p[b+1] - 1), or one (start, end) pair
// per query ([2B], rows p[2b] .. p[2b+1] - 1; the ranges may overlap, as the
// queries of a multi-position prefill share their sequence's rows).
struct Seqs {
  const int32_t *p;
  int pairs;
  __host__ __device__ int start(int b) const { return pairs ? p[2 * b] : p[b]; }
  __host__ __device__ int end(int b) const { return pairs ? p[2 * b + 1] : p[b + 1]; }
};

// Counter-based uniforms (Philox4x64-10, Salmon, Moraes, Dror and Shaw, SC
// 2011): uniform e of the stream (seed, offset) is word e mod 4 of the block
// at counter (e / 4, offset, 0, 0) under key (seed, 0), its top 23 bits j
// giving (j + 1/2) / 2^23, exact in float and inside (0, 1).  Ten rounds; a
// round multiplies counter words 0 and 2 by the two round multipliers and
// rebuilds the counter from the products' halves, the other two words and the
// key, which the Weyl constants advance between rounds.
// The four uniforms of block `blk` (uniforms 4 blk .. 4 blk + 3) of the stream.
__device__ inline void philox_block(uint64_t seed, uint64_t offset, uint64_t blk, float u[4]) {
  constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
  uint64_t c0 = blk, c1 = offset, c2 = 0, c3 = 0, k0 = seed, k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += W0;
      k1 += W1;
    }
    const uint64_t hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
    const uint64_t hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
    c0 = hi1 ^ c1 ^ k0;
    c1 = lo1;
    c2 = hi0 ^ c3 ^ k1;
    c3 = lo0;
  }
  u[0] = ((float)(c0 >> 41) + 0.5f) * 0x1p-23f;
  u[1] = ((float)(c1 >> 41) + 0.5f) * 0x1p-23f;
  u[2] = ((float)(c2 >> 41) + 0.5f) * 0x1p-23f;
  u[3] = ((float)(c3 >> 41) + 0.5f) * 0x1p-23f;
}
__device__ inline float philox_uniform(uint64_t seed, uint64_t offset, uint64_t e) {
  float u[4];
  philox_block(seed, offset, e >> 2, u);
  const int w = (int)(e & 3);
  return w == 0 ? u[0] : w == 1 ? u[1] : w == 2 ? u[2] : u[3];
}

// The uniforms of stochastic drafting, uniform e = (row) * V + draft id: a
// stored array (the caller's), or the counter-based stream whose (seed,
// offset) pair sits in device memory (so a captured pass replays with new
// values); neither means greedy selection.
struct Draws {
  const float *u = nullptr;      // [rows, V] or null
  const uint64_t *so = nullptr;  // device (seed, offset) or null
  __host__ __device__ bool on() const { return u != nullptr || so != nullptr; }
  __device__ float at(uint64_t e) const { return u ? u[e] : philox_uniform(so[0], so[1], e); }
};

// Prefix length of query b as the attention kernels use it: P_b from its
// rows, or 0 with bad = true when it lies outside [0, pmax] (the caller's
// bound on every P_b).  A bad query reads no cache row and its attention
// output is NaN.
__host__ __device__ inline int attn_prefix(Seqs cu, int b, int pmax, bool &bad) {
  const int P = cu.end(b) - cu.start(b);
  bad = P < 0 || P > pmax;
  return bad ? 0 : P;
}

// Equal-chunk split of the persistent attention.  The work items of all
// (sequence, column) segments -- each segment's 64-key prefix chunks and, as
// its last item, its cascade keys (about a chunk's work, so that the waves
// that take them do not finish last) -- numbered sequence by sequence and
// column by column (total of them), are cut into W contiguous ranges, range w
// starting at item floor(total * w / W).  A range crossing segments does one piece per
// segment.  The pieces of the segment at [S, S + n) are numbered by the range
// starts they contain: the piece at chunk x takes partial slot
// starts(x) - starts(S), where starts(y) counts the w >= 1 whose range begins
// at or before y.
struct AttnSplit {
  long total, W;
  __host__ __device__ long starts(long y) const {
    const long v = ((y + 1) * W + total - 1) / total - 1;
    return v < W - 1 ? v : W - 1;
  }
  __host__ __device__ int begin(long w) const { return (int)(total * w / W); }
  // The piece of range [.., xe) that starts at chunk x, inside the segment of
  // sequence b whose chunks (all columns) are [first, first + cnt), ncols
  // columns of cnt / ncols chunks each: its column, first chunk, chunk count,
  // partial slot, and (first piece of a column's segment only, else 0) the
  // number of pieces of that segment.
  __host__ __device__ void piece(int x, int xe, int first, int cnt, int ncols, int &col, int &ch0,
                                 int &n, int &slot, int &npieces) const {
    const int nch_b = cnt / ncols, off = x - first;
    col = off / nch_b;
    ch0 = off % nch_b;
    n = nch_b - ch0 < xe - x ? nch_b - ch0 : xe - x;
    const long S = (long)x - ch0;
    slot = (int)(starts(x) - starts(S));
    npieces = ch0 == 0 ? (int)(starts(S + nch_b - 1) - starts(S)) + 1 : 0;
  }
};
// Work items of one (sequence, column) segment in that split: its prefix
// chunks (at most nch_ld - 1, nch_ld being the partial slots per segment)
// followed by one item for its cascade keys, so between 1 and nch_ld.
__host__ __device__ inline int attn_seg_chunks(int P, int nch_ld) {
  const int n = (P + kAttnChunk - 1) / kAttnChunk;
  return (n < 0 ? 0 : (n > nch_ld - 1 ? nch_ld - 1 : n)) + 1;
}

// Row m of a GEMM's A operand is row (m / per) * outer + j0 + m % per of its buffer.
struct ARows {
  int per, j0, outer;
  __host__ __device__ int row(int m) const { return (m / per) * outer + j0 + m % per; }
};
constexpr ARows kDenseRows{1, 0, 1};

// RMSNorm fused into a GEMM (M <= 16): A holds the rows gamma * x in storage
// precision, and output row m is scaled by 1/sqrt(sum(x^2)/d + eps), with
// sum(x^2) the sum of the ntile per-16-column partials in row
// (m / per) * outer + j0 + m % per of ssq, written by the GEMM that produced x.
struct NormA {
  const float *ssq;
  int ntile;
  int per, j0, outer;
  int d;
  float eps;
  __host__ __device__ int row(int m) const { return (m / per) * outer + j0 + m % per; }
};

// Storage-type copies gamma_g * y of an fp32 output row y, written by the
// producing GEMM for later fused-RMSNorm GEMMs: row m of copy g goes to
// dst[g] + m * ld[g] (elements).
struct GainCopies {
  int n;
  const void *gamma[kMaxLayers + 1];
  void *dst[kMaxLayers + 1];
  long ld[kMaxLayers + 1];
};

// ---------------------------------------------------------------------------
// Launchers.  `dt` is 0 for fp32 storage, 1 for bf16.  All return the status
// of hipGetLastError() after the launch.
// ---------------------------------------------------------------------------

// fp32 scratch for split-K partial sums (batched rows over narrow outputs);
// without it those GEMMs run unsplit.
struct SplitScratch {
  float *p = nullptr;
  size_t floats = 0;
};

// out[m, c] = round_T(sum_k A[m,k] W[c,k]) for c < ncols; when `embed` is not
// null, also copies embed[tokens[b]] (d elements) to gather_out + b*ld_gather.
// Token ids outside [0, vocab) get a NaN row, so a bad id poisons that sequence's
// outputs instead of reading outside the table.
hipError_t gemm_store(int dt, const void *A, int lda, int M, int K, const void *W, int ncols,
                      void *out, int ldo, const void *embed, const int32_t *tokens, int vocab,
                      void *gather_out, int ld_gather, int d, int B, hipStream_t s,
                      const SplitScratch *ss = nullptr);

// out[m, c] = (resid ? resid[m, c] : 0) + sum_k A[m,k] W[c,k]   (fp32 out/resid).
// When ssq is not null, also writes the sum of squares of every output row over
// each 16-column tile t to ssq[(m * ssq_rs + ssq_off) * (ncols/16) + t]; when
// gains is not null, also writes its gain copies of every output row.  With
// norm_eps >= 0 the copies are RMS-normalised, gamma * v / sqrt(mean(v^2) +
// norm_eps), written by a row pass that also sums the split-K slices (ssq is
// then ignored; ncols <= 8192, a multiple of 4).
hipError_t gemm_resid(int dt, const void *A, int lda, int M, int K, const void *W, int ncols,
                      float *out, long ldo, const float *resid, long ldr, float *ssq, int ssq_rs,
                      int ssq_off, const GainCopies *gains, hipStream_t s,
                      const SplitScratch *ss = nullptr, float norm_eps = -1.f);

struct QkvArgs {
  const void *wq, *wk, *wv;
  int d, D, Hq, Hkv;
  int nctx, j0, cascade;     // rows are (b, t) with t < nctx, cascade state j = j0 + t
  Seqs seqs;                 // prefix rows of each sequence (P_b, the position)
  const float *rope;         // [rope_npos, D/2, 2]: cos, sin of pos * theta^(-2m/D)
  int rope_npos;
  float *q_out;              // [B, Hq, D]       (row t == nctx-1 only)
  float *k_out, *v_out;      // [B, nctx, Hkv, D]
  int rotate;                // apply the rotary embedding here (else attention does)
};
// Q/K/V projections of the RMS-normed context rows; with a.rotate, rotary embedding of Q and K.
// With `na` (M <= 16) A holds gamma * x rows and the RMSNorm scale is fused.
hipError_t gemm_qkv(int dt, const void *A, int lda, const ARows &arows, int M, const QkvArgs &a,
                    const NormA *na, hipStream_t s, const SplitScratch *ss = nullptr);

struct KvCacheArgs {
  const void *wk, *wv;
  int d, D, Hkv;
  const int32_t *positions;  // [M] rotary position of each row
  const int32_t *dst_rows;   // [M] cache row of each row
  long cache_rows;           // rows outside [0, cache_rows) are not written
  int pos_limit;             // positions outside [0, pos_limit) give NaN rows
  const float *rope;         // rotary table covering [0, pos_limit)
  void *k_cache, *v_cache;   // [cache_rows, Hkv, D] storage type
};
// K/V projections of M RMS-normed rows (A [M, d]), keys rotated; written to
// the cache rows dst_rows[m] in the storage type.
hipError_t gemm_kvcache(int dt, const void *A, int lda, int M, const KvCacheArgs &a,
                        hipStream_t s, const SplitScratch *ss = nullptr);

// Many-row bf16 GEMMs of the cache update: 128 x 64 output tiles over a 2-D
// grid (row blocks in grid z), K unsplit.  gemm_store_rows / gemm_resid_rows
// behave as gemm_store / gemm_resid (no residual, sums of squares or gain
// copies).
hipError_t gemm_store_rows(const void *A, int lda, int M, int K, const void *W, int ncols, void *out,
                           int ldo, const void *embed, const int32_t *tokens, int vocab,
                           void *gather_out, int ld_gather, int d, hipStream_t s);
hipError_t gemm_resid_rows(const void *A, int lda, int M, int K, const void *W, int ncols, float *out,
                           long ldo, hipStream_t s, const float *resid = nullptr, long ldr = 0);
hipError_t gemm_swiglu_rows(const void *A, int lda, int M, int K, const void *w_gate,
                            const void *w_up, int I, void *out, int ldo, hipStream_t s);
// Every layer's K/V projection into its cache in one launch (bf16): layer l's
// normalised rows at A + l * a_layer_stride.  With na (M <= 16) A holds
// gamma * x per layer and the rows' 1/rms come from na's sums of squares;
// otherwise 128-row tiles (32 columns wide below 128 rows, 64 from there on).
hipError_t gemm_kv_rows(const void *A, int lda, long a_layer_stride, int M, int nlayers,
                        const KvCacheArgs *layers, const NormA *na, hipStream_t s);

// s_out[m, c] = silu(A W_gate^T)[m,c] * (A W_up^T)[m,c]
hipError_t gemm_swiglu(int dt, const void *A, int lda, const ARows &arows, int M, int K,
                       const void *w_gate, const void *w_up, int I, void *s_out, int lds,
                       const NormA *na, hipStream_t s);

struct LmArgs {
  const void *w;             // [V, d]
  int V;
  int topk;
  float *logits;             // optional [M, V] (raw logits z)
  float *part_max, *part_sum;// [M, nwg] statistics of z / T
  float *cand_val;           // [M, nwg, kMaxTopk] selection keys
  int32_t *cand_idx;         // [M, nwg, kMaxTopk]
  float inv_temp;            // 1 / T
  Draws draws;               // uniforms u in (0, 1): key = z/T + Gumbel(u); none: z/T
  float *cand_z;             // [M, nwg, kMaxTopk] z / T of each candidate (with draws)
};
// LM head tiles with per-tile max, sum of exponentials and top-k candidates.
// Returns the number of column tiles (nwg) through *nwg_out.
hipError_t gemm_lmhead(int dt, const void *A, int lda, const ARows &arows, int M, int K,
                       const LmArgs &a, const NormA *na, int *nwg_out, hipStream_t s);
int lmhead_tiles(int V);

// The same RMS of each dense fp32 row x (rows r at X + r * d) under several
// gains: copy q = gamma[q] * x / rms(x) at out[q] + r * d, storage type.
struct RmsCopies {
  int n;
  const void *gamma[kMaxLayers];
  void *out[kMaxLayers];
};
hipError_t rmsnorm_copies(int dt, const float *X, int rows, const RmsCopies &c, int d, float eps,
                          hipStream_t s);

// RMSNorm of rows r < rows: source row = X + (r / per)*outer + (j0 + r % per)*inner.
hipError_t rmsnorm_rows(int dt, const float *X, int rows, int per, int j0, long outer,
                        long inner, const void *gamma, void *out, int d, float eps,
                        hipStream_t s);

// Attention of the query rows q [B, Hq, D] over the prefix cache (chunks
// 0..nch-1 of kAttnChunk keys; keys beyond are not read; a sequence whose P_b
// lies outside [0, pmax] reads no cache row and gets NaN rows) and the nctx cascade
// keys/values knew/vnew [B, nctx, Hkv, D] -> out [B, Hq*D] (storage type).
// bf16: q and the cascade keys arrive unrotated and are rotated here with the
// table `rope` (cascade != 0: cascade row j at position P + j, else P); fp32:
// they arrive rotated.  A work unit covers cpw chunks (kAttnChunk keys) of
// one sequence; bf16 launches with more units than resident waves instead
// give every resident wave an equal share of all chunks.  part
// (B*Hq*(nch_ld*(D+2) + 1) floats, nch_ld >= nch = chunks of the longest
// prefix) holds the partials of sequences that span several units (and, for
// the equal shares, the partial count per head), merged by a second launch.
hipError_t attention(int dt, const void *K, const void *V, Seqs seqs,
                     const float *q, const float *knew, const float *vnew, int nctx,
                     float *part, int nch, int nch_ld, int cpw, void *out, int B, int Hq,
                     int Hkv, int D, const float *rope, int cascade, int pmax, hipStream_t s);
// kAttnChunk-key chunks per attention work unit for a launch of B sequences
// over nch = ceil(max_prefix / kAttnChunk) chunks
int attention_cpw(int B, int Hkv, int ngroups, int nch);

// Rotary table: tab[(p * D/2 + m) * 2 + {0,1}] = cos, sin of p * theta^(-2m/D),
// formed in double precision and rounded to fp32, for p < npos.
hipError_t rope_table(float *tab, int npos, int D, double theta, hipStream_t s);

// Multi-position prefill (self context): each new row's prefix rows as Seqs
// pairs, and the rows' K/V written into the cache (see fe_misc.hip).
hipError_t prefill_ranges(const int32_t *positions, const int32_t *dst_rows, int M,
                          long cache_rows, int pos_limit, int pmax, int32_t *ranges, hipStream_t s);
hipError_t kv_scatter(int dt, const float *knew, const float *vnew, int M, int Hkv, int D,
                      const int32_t *positions, const int32_t *dst_rows, long cache_rows,
                      int pos_limit, const float *rope, int rotated, void *kc, void *vc,
                      hipStream_t s);

// Greedy acceptance over the trees of B sequences (N levels, k per level):
// tokens/target_next [B, 1+N*k], retrieve [B, N*(k-1)+1, N+1] -> accept_len [B],
// accept_path [B], accepted [B, N+1] (accepted draft tokens, the target's next
// token, -1 padding).
hipError_t accept_greedy(int B, int N, int k, const int32_t *tokens, const int32_t *retrieve,
                         const int32_t *target_next, int32_t *accept_len, int32_t *accept_path,
                         int32_t *accepted, hipStream_t s);

// Speculative-sampling acceptance at temperature 1/inv_temp of B trees (N
// levels, k per level): topk_draft [B, N, k] draft ids of the children,
// draft_logits [B, N, V], draft_uniforms [B, N, V] or NULL (unsampled
// children), target_probs [B, 1+N*k, Vt], uniforms [B, N*k+1].  Outputs as
// accept_greedy.  V <= kAccSampleMaxV, Vt <= kAccSampleMaxVt (LDS residual).
// img: the bitmask of the target ids that d2t maps to, from accept_img.
constexpr int kAccSampleMaxV = 32768, kAccSampleMaxVt = 131072;
// Workspace of the acceptance's row pre-pass (batches of at most max_batch
// sequences): per (sequence, node) 16 chunk sums and unmapped sums, 16 last
// unmapped ids, and p at the V mapped ids.  Used for a single sequence only:
// measured on the 8B vocabularies, 58 us per call against 64 at batch 1, but
// 121 against 102 at batch 4 (every node's row is read, not just the visited
// ones).
struct AccPre {
  float *p = nullptr;
  int max_batch = 0;
};
constexpr int kAccPreMaxBatch = 1;
inline size_t acc_pre_bytes(int B, int T, int V) { return (size_t)B * T * (16 * 3 + (size_t)V) * 4; }
hipError_t accept_img(const int32_t *d2t, int V, int Vt, uint32_t *img, hipStream_t s);
hipError_t accept_sample(int B, int N, int k, int V, int Vt, const int32_t *tokens,
                         const int32_t *retrieve, const int32_t *topk_draft,
                         const float *draft_logits, float inv_temp, Draws draft_draws,
                         const int32_t *d2t, const float *target_probs, const float *uniforms,
                         const uint32_t *img, int32_t *accept_len, int32_t *accept_path,
                         int32_t *accepted, hipStream_t s, AccPre pre = AccPre{});
// Uniforms first .. first+n-1 of the counter-based stream ((seed, offset) in
// device memory) into out (test export of the generator).
hipError_t philox_fill(const uint64_t *seed_offset, uint64_t first, long n, float *out,
                       hipStream_t s);

// The pass's draft tree, written by the top-k merge itself: rows are
// (sequence, level) pairs, N levels per sequence; the arrays as build_tree
// writes them (tokens == nullptr: no tree).
struct TreeRows {
  int N = 0;
  const int32_t *root = nullptr, *cu_prefix = nullptr;
  int32_t *tokens = nullptr, *parents = nullptr, *depth = nullptr, *positions = nullptr;
  uint8_t *mask = nullptr;
  int32_t *retrieve = nullptr;
};

// ---- persistent batch-1 pass (fe_pass.hip) -----------------------------------
// Between two attention launches the stages of a batch-1 pass run inside one
// launch of resident workgroups (one per compute unit) that hand results to
// each other as tagged 64-bit words (payload + the pass's tag).
constexpr int kSegMaxStages = 4;    // stages per launch
constexpr int kSegMaxRows = 8;      // activation rows of a stage (cascade layers)
constexpr int kSegMaxCopies = 9;    // normalised copies one produced row feeds
constexpr int kSegMaxWg = 256;      // workgroups (compute units) at most
constexpr int kSegRedFloats = 2048; // row partial sums of one stage: rows * 2
constexpr int kSegResRows = 64;     // residual rows a workgroup keeps (d <= 64 * 256)
constexpr int kSegLmMaxCols = 128;  // LM-head rows (vocabulary entries) per workgroup
// sync words in the workspace (uint32, 128 bytes apart)
constexpr int kSegEpochWord = 0, kSegDepartWord = 32, kSegStatusWord = 64, kSegSyncWords = 96;
constexpr uint32_t kSegStatusTimeout = 1u;  // a poll gave up (results unspecified)
constexpr uint32_t kSegStatusPersistent = 1u << 16;  // the last pass ran as persistent launches
// The persistent launches can be switched off here (fe_set_pass_mode(0) is then
// refused and every pass runs one launch per stage).
constexpr bool kSegEnabled = true;
enum SegKind : int { kSegFuse = 0, kSegInput, kSegQkv, kSegO, kSegGu, kSegDown, kSegLm };
enum SegSrcKind : int { kSrcPlain = 0, kSrcTagged = 1, kSrcEmbed = 2 };
// elements [e0, e0 + n) of input row m: plain bf16 at p (element 0 of the
// part), tagged words at p (two bf16 each), or the embedding-table row of
// token tok[0] (NaN when it lies outside [0, vocab))
struct SegSrc {
  const void *p;
  const int32_t *tok;
  int kind, m, e0, n, vocab;
};
struct SegStage {
  int kind, C, K, mr, gran;
  const bf16_t *w0, *w1, *w2;  // Q/K/V: rows split at split1, split2; gate/up: even/odd rows
  int split1, split2, qrow;
  int nsrc;
  SegSrc src[kSegMaxRows + 1];
  const uint64_t *ssq[kSegMaxRows];  // tagged per-workgroup sums of squares of input row m, or null
  uint64_t *out_t;                   // tagged outputs (fusion: g_t; gate/up: SwiGLU; LM: candidates)
  float *x_out;                      // plain fp32 output row (input FC, down; Q/K/V: q)
  float *k_out, *v_out;              // Q/K/V: k, v rows [mr, H_kv * D]
  const float *resid;                // O projection: the residual row
  uint64_t *ssq_out;                 // tagged sums of squares of the output row
  int ncopy;                         // gamma_q * row copies for later normalised GEMVs
  const bf16_t *gamma[kSegMaxCopies];
  uint64_t *copy_t[kSegMaxCopies];
};
struct SegArgs {
  SegStage st[kSegMaxStages];
  int nst, nwg, d, V, topk, last;
  float eps;
  uint32_t *sync;
  const uint64_t *cand_t;  // LM-head candidates (the last stage's out_t), merged when last
  const int32_t *d2t;
  int32_t *ids, *draft_ids;
  float *probs, *logits;
  TreeRows tree;
};
int seg_variant(int xbytes);  // workgroup shape for the largest activation block (-1: none)
hipError_t seg_occupancy(int variant, int *blocks_per_cu);
hipError_t seg_launch(int variant, const SegArgs &a, hipStream_t s);
hipError_t seg_zero(uint64_t *words, size_t n, hipStream_t s);


// Global top-k of every row from the tile candidates (by key); softmax
// statistics merge.  With cand_z (sampled candidates) the k winners are
// listed by z / T (larger first, lower id on ties), else in key order.  With
// tree, also the Backbone Expansion tree of the rows' sequences.
hipError_t topk_merge(const float *part_max, const float *part_sum, const float *cand_val,
                      const int32_t *cand_idx, const float *cand_z, int rows, int nwg, int topk,
                      int V, const int32_t *d2t, int32_t *ids, int32_t *draft_ids, float *probs,
                      hipStream_t s, const TreeRows *tree = nullptr);

// Backbone Expansion tree of every sequence; P_b from prefix_lens, or from
// cu_prefix when prefix_lens is NULL.
hipError_t build_tree(int B, int N, int k, const int32_t *root_tokens, const int32_t *topk_ids,
                      const int32_t *prefix_lens, const int32_t *cu_prefix, int32_t *tokens,
                      int32_t *parents, int32_t *depth, int32_t *positions, uint8_t *mask,
                      int32_t *retrieve, hipStream_t s);

}  // namespace fe
