// fe_attn_unit.h -- one piece of GQA decode attention on the matrix cores
// (gfx950), shared by the attention kernel and the persistent batch-1 pass.
// Not part of the public ABI.
#pragma once

#include "fe_internal.h"

namespace fe {

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
// it); the kernels that use this have no other M0 users.
__device__ __forceinline__ void ring_dma16(const void *src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds) : "memory");
}

// LDS one unit works in: the K/V ring of DEPTH stages of 16 keys and the
// cascade keys' partial (o, max, sum per head).
template <int D, int GH, int DEPTH> struct AttnLds {
  static constexpr int kStage = 2 * 16 * 2 * D;
  unsigned char ring[DEPTH][kStage];
  float oc[GH][D];
  float mc[GH], lc[GH];
};

// One piece of work for one wave (any wave of a workgroup): prefix keys
// [64 ch0, 64 (ch0 + nchunk)) of one sequence (P cached keys at kb / vb, rows
// rs elements apart, keys already rotated) for the GH query heads at qin (D
// floats apart, unrotated), plus the (at most NCX) cascade keys/values kn / vn
// (rows kvs floats apart, unrotated) when casc.  Rotary positions: the query at
// P + nctx - 1 and cascade key j at P + j (cascade != 0), else all at P.  bad
// (a prefix outside its bound) gives NaN results.  The result goes to outp
// (bf16, head r at r * D) when `whole`, else as a partial (o scaled to its max
// at po + r * po_hs, (max, sum) at pml + r * pml_hs); npieces > 0 is stored at
// pcount[r].
template <int D, int GH, int DEPTH, int NCX>
__device__ __forceinline__ void attn_unit(const bf16_t *__restrict__ kb,
                                          const bf16_t *__restrict__ vb, size_t rs, int P,
                                          bool bad, const float *qin, const float *kn,
                                          const float *vn, size_t kvs, int nctx,
                                          const float *__restrict__ rope, int cascade, int ch0,
                                          int nchunk, bool whole, bool casc, float *po, int po_hs,
                                          float *pml, int pml_hs, bf16_t *outp, float *pcount,
                                          int npieces, AttnLds<D, GH, DEPTH> &lds) {
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
  static_assert(STAGE == AttnLds<D, GH, DEPTH>::kStage, "ring stage size");
  constexpr int HD = D / 2;            // rotary pairs (m, m + D/2)
  auto &s_ring = lds.ring;
  auto &s_oc = lds.oc;
  float *s_mc = lds.mc, *s_lc = lds.lc;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const float qscale = 1.4426950408889634f * rsqrtf((float)D);

  // Loads that do not depend on the prefix bounds go first, so their latency
  // overlaps the read of cu: q (B-operand layout), and in chunk 0 the cascade
  // rows.
  f32x4 qraw[NKC][2];
  {
    const float *qp = qin + (size_t)min(r, GH - 1) * D;
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
      for (int e = 0; e < 2; ++e) qc[gh][e] = qin[(size_t)gh * D + m2 + e * HD];
#pragma unroll
    for (int j = 0; j < NCX; ++j) {
      const size_t off = (size_t)min(j, nctx - 1) * kvs + m2;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        kj[j][e] = kn[off + e * HD];
        vj[j][e] = vn[off + e * HD];
      }
    }
  }

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

  // Stage st: keys base + SK st + R, R < SK, K rows then V rows, loaded straight
  // into ring slot `slot`.  Load i moves 1 KB: lane l the 16 bytes at 16 l of
  // it, i.e. row R, position sl of that row, which holds 16-byte piece
  // sl ^ swz(R).  The swizzle spreads the pieces that one MFMA operand read
  // gathers from 16 rows (K: one piece of rows 0..15; V: two pieces of rows
  // 4g + e) over distinct banks.
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
  if (npieces > 0 && g == 0 && r < GH) pcount[r] = (float)npieces;
  if (r >= GH) return;  // padding columns of the MFMA tiles
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
      *reinterpret_cast<u32x2 *>(outp + (size_t)r * D + d0) = w;
    } else {
      *reinterpret_cast<f32x4 *>(po + (size_t)r * po_hs + d0) = o;
    }
  }
  if (!whole && g == 0) {
    float *ml = pml + (size_t)r * pml_hs;
    ml[0] = M;
    ml[1] = L;
  }
}

}  // namespace fe
