// fe_tree.h -- the Backbone Expansion tree's value-independent structure
// (Section 2.2), shared by the top-k merge kernels.  Not part of the public ABI.
#pragma once

#include "fe_internal.h"

namespace fe {

// Everything of sequence b's tree except the tokens (closed form in N, k and
// the prefix length P), spread over the calling workgroup's threads.
__device__ inline void tree_structure(int b, int N, int k, int P, int32_t *parents, int32_t *depth,
                                  int32_t *positions, uint8_t *mask, int32_t *retrieve) {
  const int T = 1 + N * k, NL = N * (k - 1) + 1;
  for (int n = threadIdx.x; n < T; n += blockDim.x) {
    int lvl = 0, par = -1;
    if (n > 0) {
      lvl = 1 + (n - 1) / k;
      par = (lvl == 1) ? 0 : 1 + (lvl - 2) * k;
    }
    const size_t o = (size_t)b * T + n;
    parents[o] = par;
    depth[o] = lvl;
    positions[o] = P + lvl;
  }
  uint8_t *mb = mask + (size_t)b * T * T;
  for (int idx = threadIdx.x; idx < T * T; idx += blockDim.x) {
    const int a = idx / T, c = idx % T;
    const int la = a == 0 ? 0 : 1 + (a - 1) / k;
    const int lc = c == 0 ? 0 : 1 + (c - 1) / k;
    const bool backbone_c = c > 0 && (c - 1) % k == 0;
    mb[idx] = (c == a) || (c == 0) || (backbone_c && lc < la);
  }
  int32_t *rb = retrieve + (size_t)b * NL * (N + 1);
  for (int leaf = threadIdx.x; leaf < NL; leaf += blockDim.x) {
    // leaves in node order: levels 1..N-1 contribute ranks 1..k-1; level N
    // contributes its backbone node and then ranks 1..k-1
    int lvl, rho;
    if (leaf < (N - 1) * (k - 1)) {
      lvl = 1 + leaf / (k - 1);
      rho = 1 + leaf % (k - 1);
    } else {
      lvl = N;
      rho = leaf - (N - 1) * (k - 1);
    }
    int32_t *row = rb + (size_t)leaf * (N + 1);
    row[0] = 0;
    for (int l = 1; l < lvl; ++l) row[l] = 1 + (l - 1) * k;
    row[lvl] = 1 + (lvl - 1) * k + rho;
    for (int t = lvl + 1; t <= N; ++t) row[t] = -1;
  }
}

}  // namespace fe
