// Row statistics and the fused epilogues of the deferred norm-then-project kernels.
//
// After the K loop a lane holds, for one activation row m, the row's sum of
// squares ss (and, for LayerNorm, its sum sa) and four accumulators of
// consecutive packed columns p..p+3 (for a GLU: the gate block's four and the
// matching up block's four).  The epilogue applies the single per-row scalar
// that FlashNorm defers past the matrix multiply (Prop. 2, Cor. 1), then the
// bias / GLU / LayerNorm mean correction, and rounds once to bf16 on the store.
#pragma once

#include "fn_device.h"

namespace fn {

struct RowStat {
  float s;   // 1/RMSe(a) (RMSNorm) or 1/sigma (LayerNorm); 1 for the baselines
  float mu;  // LayerNorm mean (0 otherwise)
};

template <int EPI>
__device__ __forceinline__ RowStat row_stat(float ss, float sa, const EpiArgs& ep) {
  RowStat st{1.0f, 0.0f};
  if constexpr (EPI == EPI_RMS || EPI == EPI_GLU) {
    // RMSe(a) = sqrt(eps + ss/K)  (App. "RMS with epsilon")
    st.s = rsqrtf(fmaf(ss, ep.inv_k, ep.eps));
  } else if constexpr (EPI == EPI_LN) {
    float mu = sa * ep.inv_k;
    float var = fmaxf(fmaf(ss, ep.inv_k, -mu * mu), 0.0f);
    st.mu = mu;
    st.s = rsqrtf(var + ep.eps);
  }
  (void)ss;
  (void)sa;
  (void)ep;
  return st;
}

// Store 4 consecutive outputs of row m starting at logical column n (a multiple
// of 4).  v: accumulators of the 4 columns (GLU: gate); u: the up accumulators.
// ncols: number of logical output columns (N, or F for a GLU).
template <int EPI>
__device__ __forceinline__ void store4_bf16(__bf16* __restrict__ y, int64_t ldy, int ncols, int m,
                                            int n, f32x4 v, f32x4 u, RowStat st,
                                            const EpiArgs& ep) {
  float o[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int c = n + r;
    float val;
    if constexpr (EPI == EPI_RMS) {
      val = v[r] * st.s;
      if (ep.bias && c < ncols) val += ep.bias[c];
    } else if constexpr (EPI == EPI_GLU) {
      val = silu(v[r] * st.s) * (u[r] * st.s);
    } else if constexpr (EPI == EPI_LN) {
      float cs = c < ncols ? ep.colsum[c] : 0.0f;
      float cb = (ep.cstar && c < ncols) ? ep.cstar[c] : 0.0f;
      val = fmaf(fmaf(-st.mu, cs, v[r]), st.s, cb);
    } else if constexpr (EPI == EPI_NONE) {
      val = v[r];
    } else {  // EPI_GLU_NOSCALE
      val = silu(v[r]) * u[r];
    }
    o[r] = val;
  }
  __bf16* dst = y + (int64_t)m * ldy + n;
  if (n + 3 < ncols) {
    u32x2 w = {pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
    *reinterpret_cast<u32x2*>(dst) = w;
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (n + r < ncols) reinterpret_cast<unsigned short*>(dst)[r] = (unsigned short)f32_to_bf16_bits(o[r]);
  }
}

}  // namespace fn
