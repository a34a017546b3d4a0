// Split-table lookup shared by the epilogues that relax ReLU coefficients on branch-and-bound
// subdomains (paper, Sec. 2.1: a split fixes a neuron active or inactive; Sec. 2.2: each split
// enters the bound with a multiplier).  Device code only.
#pragma once

#include "kernels.h"

namespace vcr {

// The split entry of (the row's domain, relu, neuron n), if any: its relaxation replaces
// (lam, s, t); *ent receives the entry index and *sterm its Lagrangian sign.
__device__ __forceinline__ float4 split_override(const SplitTable &st, int row, int relu, int n, float4 prm,
                                                 int *ent = nullptr, float *sterm = nullptr) {
  int d = row / st.rows_per_domain;
  d = d < st.D ? d : st.D - 1;
  const int e0 = st.off[d * (st.R + 1) + relu];
  const int e1 = st.off[d * (st.R + 1) + relu + 1];
  for (int e = e0; e < e1; ++e) {
    if (st.ent_n[d * st.S + e] == n) {
      const float4 q = st.ent_p[d * st.S + e];
      prm.x = q.x;
      prm.y = q.y;
      prm.z = q.z;
      if (ent) {
        *ent = e;
        *sterm = q.w;
      }
    }
  }
  return prm;
}

}  // namespace vcr
