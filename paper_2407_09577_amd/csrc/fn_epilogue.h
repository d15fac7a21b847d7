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
  float s;   // 1/RMSe(a) (RMSNorm kinds), 1/MSe(a) (ReGLU, bilinear), 1/sigma (LayerNorm),
             // the given row scale (EPI_ROWSCALE); 1 for the baselines
  float mu;  // LayerNorm mean (0 otherwise)
};

template <int EPI>
__device__ __forceinline__ RowStat row_stat(float ss, float sa, const EpiArgs& ep) {
  RowStat st{1.0f, 0.0f};
  if constexpr (EPI == EPI_RMS || EPI == EPI_GLU || EPI == EPI_GLU_DEFER || EPI == EPI_RELU_DEFER) {
    // RMSe(a) = sqrt(eps + ss/K)  (App. "RMS with epsilon")
    st.s = rsqrtf(fmaf(ss, ep.inv_k, ep.eps));
  } else if constexpr (EPI == EPI_REGLU || EPI == EPI_BILINEAR) {
    // both branch scales merged: 1/RMSe^2 = 1/MSe = 1/(eps + ss/K)  (App. "FFN with ReGLU
    // and Bilinear GLU"; ReLU(s t) = s ReLU(t) for s >= 0)
    st.s = 1.0f / fmaf(ss, ep.inv_k, ep.eps);
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

// Row statistics of output row m (< M for the rows that are stored): the kinds
// that apply a scale computed elsewhere read it here.
template <int EPI>
__device__ __forceinline__ RowStat row_stat_at(float ss, float sa, const EpiArgs& ep, int m, int M) {
  RowStat st = row_stat<EPI>(ss, sa, ep);
  if constexpr (EPI == EPI_ROWSCALE) st.s = m < M ? ep.row_scale[m] : 0.0f;
  return st;
}

// Four fp32 values -> four bf16 (hardware round to nearest even), as 8 bytes.
__device__ __forceinline__ u32x2 pack4_bf16(const float (&o)[4]) {
  typedef __attribute__((ext_vector_type(2))) float f32x2;
  const bf16x2 lo = __builtin_convertvector((f32x2{o[0], o[1]}), bf16x2);
  const bf16x2 hi = __builtin_convertvector((f32x2{o[2], o[3]}), bf16x2);
  return u32x2{__builtin_bit_cast(unsigned, lo), __builtin_bit_cast(unsigned, hi)};
}

// Epilogue value of one output.  vec: the optional per-column vector (RMS: the
// bias, added after the scaling; LN: c*), 0 when absent; cs: colsum (LN).
template <int EPI>
__device__ __forceinline__ float epi_value(float v, float u, RowStat st, float vec, float cs) {
  if constexpr (EPI == EPI_RMS) return fmaf(v, st.s, vec);
  else if constexpr (EPI == EPI_GLU) return silu(v * st.s) * (u * st.s);
  else if constexpr (EPI == EPI_LN) return fmaf(fmaf(-st.mu, cs, v), st.s, vec);
  else if constexpr (EPI == EPI_NONE) return v;
  else if constexpr (EPI == EPI_GLU_NOSCALE) return silu(v) * u;
  else if constexpr (EPI == EPI_REGLU) return (v > 0.0f ? v : 0.0f) * u * st.s;
  else if constexpr (EPI == EPI_BILINEAR) return v * u * st.s;
  else if constexpr (EPI == EPI_GLU_DEFER) return silu(v * st.s) * u;
  else if constexpr (EPI == EPI_RELU_DEFER) return v > 0.0f ? v : 0.0f;
  else return v * st.s;  // EPI_ROWSCALE
}

// The optional per-column vector of an epilogue (bias or c*), or nullptr.
template <int EPI>
__device__ __forceinline__ const float* epi_vec(const EpiArgs& ep) {
  if constexpr (EPI == EPI_RMS) return ep.bias;
  else if constexpr (EPI == EPI_LN) return ep.cstar;
  else return nullptr;
}

// The 4 outputs of one lane (logical columns n .. n+3, n % 4 == 0, all inside
// the output) as bf16: 16-byte vector loads of the per-column vectors.
template <int EPI, bool VEC>
__device__ __forceinline__ u32x2 epi4_bf16(int n, f32x4 v, f32x4 u, RowStat st, const EpiArgs& ep) {
  f32x4 vec = {0.f, 0.f, 0.f, 0.f}, cs = {0.f, 0.f, 0.f, 0.f};
  if constexpr (VEC) vec = *reinterpret_cast<const f32x4*>(epi_vec<EPI>(ep) + n);
  if constexpr (EPI == EPI_LN) cs = *reinterpret_cast<const f32x4*>(ep.colsum + n);
  float o[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) o[r] = epi_value<EPI>(v[r], u[r], st, vec[r], cs[r]);
  return pack4_bf16(o);
}

// Output tiles staged through LDS, so that the global stores are whole rows
// written 16 bytes per lane instead of 8-byte pieces of 16 rows per store
// instruction.  Row r of a staged tile holds UPR 16-byte units.  With UPR a
// multiple of 8, unit u sits at position u ^ (r % 8) of the row; otherwise rows
// are padded by one unit.  Either way the 8-byte writes of 16 lanes on 16 rows
// spread over the LDS banks, and a row reads back as consecutive units.
template <int UPR>
__device__ __forceinline__ constexpr int stage_pos(int r, int u) {
  if constexpr (UPR % 8 == 0) return r * UPR + (u ^ (r & 7));
  else return r * (UPR + 1) + u;
}
template <int ROWS, int UPR>
constexpr int stage_bytes() { return ROWS * (UPR % 8 == 0 ? UPR : UPR + 1) * 16; }

template <int UPR>
__device__ __forceinline__ void stage4(char* tile, int r, int c, u32x2 val) {
  const int byte = c * 2;  // c % 4 == 0: an 8-byte half of a 16-byte unit
  *reinterpret_cast<u32x2*>(tile + stage_pos<UPR>(r, byte >> 4) * 16 + (byte & 8)) = val;
}

// Copy a staged ROWS x (UPR*8) bf16 tile to y[m0.., n0..]: thread tid of NT
// moves 16-byte units in row-major order.  y + n0 and ldy keep 16-byte alignment.
template <int ROWS, int UPR, int NT>
__device__ __forceinline__ void copy_tile_out(const char* tile, __bf16* __restrict__ y, int64_t ldy, int m0, int n0,
                                              int tid) {
#pragma unroll
  for (int q = tid; q < ROWS * UPR; q += NT) {
    const int r = q / UPR, u = q % UPR;
    const u32x4 v = *reinterpret_cast<const u32x4*>(tile + stage_pos<UPR>(r, u) * 16);
    *reinterpret_cast<u32x4*>(y + (int64_t)(m0 + r) * ldy + n0 + u * 8) = v;
  }
}

// Store 4 consecutive outputs of row m starting at logical column n (n % 4 == 0)
// when all four lie inside the output: one 8-byte store, 16-byte vector loads of
// the per-column vectors.  VEC: the optional per-column vector is present.
// v: accumulators of the 4 columns (GLU: gate); u: the up accumulators.
template <int EPI, bool VEC>
__device__ __forceinline__ void store4_bf16_full(__bf16* __restrict__ y, int64_t ldy, int m, int n,
                                                 f32x4 v, f32x4 u, RowStat st, const EpiArgs& ep) {
  *reinterpret_cast<u32x2*>(y + (int64_t)m * ldy + n) = epi4_bf16<EPI, VEC>(n, v, u, st, ep);
}

// The same for the ragged edge: row m may lie past M and columns past ncols
// (number of logical output columns: N, or F for a GLU).
template <int EPI, bool VEC>
__device__ __forceinline__ void store4_bf16_edge(__bf16* __restrict__ y, int64_t ldy, int M, int ncols,
                                                 int m, int n, f32x4 v, f32x4 u, RowStat st,
                                                 const EpiArgs& ep) {
  if (m >= M) return;
  const float* vp = epi_vec<EPI>(ep);
  unsigned short* dst = reinterpret_cast<unsigned short*>(y + (int64_t)m * ldy + n);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int c = n + r;
    if (c < ncols) {
      const float vec = VEC ? vp[c] : 0.f;
      const float cs = EPI == EPI_LN ? ep.colsum[c] : 0.f;
      dst[r] = __builtin_bit_cast(unsigned short, (__bf16)epi_value<EPI>(v[r], u[r], st, vec, cs));
    }
  }
}

}  // namespace fn
