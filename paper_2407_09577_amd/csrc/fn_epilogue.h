// Row statistics and the fused epilogues of the deferred norm-then-project kernels.
//
// After the K loop a lane holds, for one activation row m, the row's sum of
// squares ss (and, for LayerNorm, its sum sa) and four accumulators of
// consecutive packed columns p..p+3 (for a GLU: the gate block's four and the
// matching up block's four).  The epilogue applies the single per-row scalar
// that FlashNorm defers past the matrix multiply (Prop. 2, Cor. 1), then the
// bias / GLU / LayerNorm mean correction, and rounds once to bf16 on the store.
#pragma once

#include <type_traits>

#include "fn_device.h"

namespace fn {

// Accumulator type of a kind's row sums.  LayerNorm takes its variance in one pass as
// E[a^2] - mu^2, which cancels when |mu| >> sigma (the two terms agree in their leading
// digits): its sums are kept in fp64.  The kernels add exact-or-nearly-exact fp32
// partials of a few elements (the squares of bf16 values are exact in fp32) into the
// fp64 totals, so the sums and the variance carry no fp32 accumulation error.
template <int EPI>
using StatT = std::conditional_t<EPI == EPI_LN, double, float>;

struct RowStat {
  float s;   // 1/RMSe(a) (RMSNorm kinds), 1/MSe(a) (ReGLU, bilinear), 1/sigma (LayerNorm),
             // the given row scale (EPI_ROWSCALE); 1 for the baselines
  float mu;  // LayerNorm mean of the values the product consumed (of a - p where the
             // kernel shifts the activations by a pivot p; 0 for the other kinds)
  int pos;   // EPI_ROPE: the token's position (0 otherwise)
};

template <int EPI>
__device__ __forceinline__ RowStat row_stat(StatT<EPI> ss, StatT<EPI> sa, const EpiArgs& ep) {
  RowStat st{1.0f, 0.0f, 0};
  if constexpr (EPI == EPI_RMS || EPI == EPI_GLU || EPI == EPI_GLU_DEFER || EPI == EPI_RELU_DEFER ||
                EPI == EPI_ROPE || EPI == EPI_HEADNORM) {
    // RMSe(a) = sqrt(eps + ss/K)  (App. "RMS with epsilon")
    st.s = rsqrtf(fmaf(ss, ep.inv_k, ep.eps));
  } else if constexpr (EPI == EPI_REGLU || EPI == EPI_BILINEAR) {
    // both branch scales merged: 1/RMSe^2 = 1/MSe = 1/(eps + ss/K)  (App. "FFN with ReGLU
    // and Bilinear GLU"; ReLU(s t) = s ReLU(t) for s >= 0)
    st.s = 1.0f / fmaf(ss, ep.inv_k, ep.eps);
  } else if constexpr (EPI == EPI_LN) {
    // mu = sa/K, var = ss/K - mu^2 in fp64, clamped at 0; a NaN (a row holding NaN or
    // Inf) stays NaN, so that row's outputs are NaN as in the standard form
    const double mu = sa * ep.inv_kd;
    double var = fma(ss, ep.inv_kd, -mu * mu);
    var = var < 0.0 ? 0.0 : var;
    st.mu = (float)mu;
    st.s = rsqrtf((float)(var + (double)ep.eps));
  }
  (void)ss;
  (void)sa;
  (void)ep;
  return st;
}

// Row statistics of output row m (< M for the rows that are stored): the kinds
// that apply a scale computed elsewhere read it here.
template <int EPI>
__device__ __forceinline__ RowStat row_stat_at(StatT<EPI> ss, StatT<EPI> sa, const EpiArgs& ep, int m, int M) {
  RowStat st = row_stat<EPI>(ss, sa, ep);
  if constexpr (EPI == EPI_ROWSCALE) st.s = m < M ? ep.row_scale[m] : 0.0f;
  if constexpr (EPI == EPI_ROPE) st.pos = m < M ? ep.rope_pos[m] : 0;
  if constexpr (EPI == EPI_HEADNORM) st.pos = (m < M && ep.rope_pos) ? ep.rope_pos[m] : 0;
  return st;
}

// Four fp32 values -> four bf16 (hardware round to nearest even), as 8 bytes.
__device__ __forceinline__ u32x2 pack4_bf16(const float (&o)[4]) {
  const bf16x2 lo = __builtin_convertvector((f32x2{o[0], o[1]}), bf16x2);
  const bf16x2 hi = __builtin_convertvector((f32x2{o[2], o[3]}), bf16x2);
  return u32x2{__builtin_bit_cast(unsigned, lo), __builtin_bit_cast(unsigned, hi)};
}

// Epilogue value of one output.  vec: the optional per-column vector (RMS: the
// bias, added after the scaling; LN: c*), 0 when absent; cs: colsum (LN).
template <int EPI>
__device__ __forceinline__ float epi_value(float v, float u, RowStat st, float vec, float cs) {
  static_assert(EPI != EPI_ROPE && EPI != EPI_HEADNORM, "per-pair / per-head kinds: rope4, rope1, headnorm8");
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
  if constexpr (EPI == EPI_RMS || EPI == EPI_ROPE) return ep.bias;
  else if constexpr (EPI == EPI_LN) return ep.cstar;
  else return nullptr;
}

// RoPE after the fused QKV projection (Sec. 4.2, Fig. 5): the four columns n .. n+3
// of one row (n % 4 == 0; heads are a multiple of 4 wide, so these are two whole
// pairs of one head).  Q and K pairs turn by the token's angles; without a bias the
// token's scale s (times the score scale for Q) is folded into the table values,
// cos*s and sin*s, as in Fig. 5(b), so the per-head scaling disappears.  A bias is
// added before the rotation (t = acc*s + c).  V columns take the scale only.  A
// position outside the table makes the Q and K values NaN.
// n % h without an integer division: the quotient from fp32 (exact for a power of
// two; otherwise off by at most one for the column counts allowed, n < 2^24), then
// one correction each way.
__device__ __forceinline__ int rope_col_in_head(int n, const EpiArgs& ep) {
  const int q = (int)((float)n * ep.head_inv_h);
  int r = n - q * ep.head_h;
  r += r < 0 ? ep.head_h : 0;
  r -= r >= ep.head_h ? ep.head_h : 0;
  return r;
}

// The token's angles for the two pairs of columns n .. n+3.  The loads are
// unconditional (a clamped position; V columns load and ignore their values) and
// the choices are selects, so the loads of many column groups and rows can be in
// flight together instead of each waiting inside a branch.
struct RopeTab {
  float c0, c1, s0, s1;
};
__device__ __forceinline__ RopeTab rope_tab(int n, RowStat st, const EpiArgs& ep) {
  const bool valid = (unsigned)st.pos < (unsigned)ep.rope_P;
  const int j = rope_col_in_head(n, ep) >> 1;  // pair of column n (a valid index for V too)
  const int64_t off = (int64_t)(valid ? st.pos : 0) * (ep.head_h >> 1) + j;
  const f32x2 c = *reinterpret_cast<const f32x2*>(ep.rope_cos + off);
  const f32x2 sn = *reinterpret_cast<const f32x2*>(ep.rope_sin + off);
  const float nan = __builtin_nanf("");
  return RopeTab{valid ? c[0] : nan, valid ? c[1] : nan, valid ? sn[0] : nan, valid ? sn[1] : nan};
}

template <bool VEC>
__device__ __forceinline__ void rope_apply(int n, f32x4 v, f32x4 vec, RowStat st, RopeTab tb, const EpiArgs& ep,
                                           float (&o)[4]) {
  const bool is_v = n >= ep.k_end;
  const float qs = n < ep.q_end ? ep.q_scale : 1.0f;
  float r[4];
  if constexpr (VEC) {
    float t[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) t[q] = fmaf(v[q], st.s, vec[q]);
    r[0] = (t[0] * tb.c0 - t[1] * tb.s0) * qs;
    r[1] = (t[0] * tb.s0 + t[1] * tb.c0) * qs;
    r[2] = (t[2] * tb.c1 - t[3] * tb.s1) * qs;
    r[3] = (t[2] * tb.s1 + t[3] * tb.c1) * qs;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = is_v ? t[q] : r[q];
  } else {
    // Fig. 5(b): the token's scale (and the score scale) folded into the angles
    const float f = st.s * qs;
    const float c0 = tb.c0 * f, s0 = tb.s0 * f, c1 = tb.c1 * f, s1 = tb.s1 * f;
    r[0] = v[0] * c0 - v[1] * s0;
    r[1] = v[0] * s0 + v[1] * c0;
    r[2] = v[2] * c1 - v[3] * s1;
    r[3] = v[2] * s1 + v[3] * c1;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = is_v ? v[q] * st.s : r[q];
  }
}

template <bool VEC>
__device__ __forceinline__ void rope4(int n, f32x4 v, f32x4 vec, RowStat st, const EpiArgs& ep, float (&o)[4]) {
  rope_apply<VEC>(n, v, vec, st, rope_tab(n, st, ep), ep, o);
}

// One output of EPI_ROPE at column c from its own accumulator v and that of its
// pair partner w (column c ^ 1), with the per-column bias of each (0 without).
__device__ __forceinline__ float rope1(int c, float v, float w, float bv, float bw, RowStat st, const EpiArgs& ep) {
  const float tv = fmaf(v, st.s, bv);
  if (c >= ep.k_end) return tv;
  if ((unsigned)st.pos >= (unsigned)ep.rope_P) return __builtin_nanf("");
  const float tw = fmaf(w, st.s, bw);
  const float qs = c < ep.q_end ? ep.q_scale : 1.0f;
  const int64_t off = (int64_t)st.pos * (ep.head_h >> 1) + (rope_col_in_head(c, ep) >> 1);
  const float cs = ep.rope_cos[off], sn = ep.rope_sin[off];
  return ((c & 1) ? tw * sn + tv * cs : tv * cs - tw * sn) * qs;
}

// The 4 outputs of one lane (logical columns n .. n+3, n % 4 == 0, all inside
// the output) in fp32: 16-byte vector loads of the per-column vectors.
template <int EPI, bool VEC>
__device__ __forceinline__ void epi4_values(int n, f32x4 v, f32x4 u, RowStat st, const EpiArgs& ep,
                                            float (&o)[4]) {
  f32x4 vec = {0.f, 0.f, 0.f, 0.f}, cs = {0.f, 0.f, 0.f, 0.f};
  if constexpr (VEC) vec = *reinterpret_cast<const f32x4*>(epi_vec<EPI>(ep) + n);
  if constexpr (EPI == EPI_LN) cs = *reinterpret_cast<const f32x4*>(ep.colsum + n);
  if constexpr (EPI == EPI_ROPE) {
    rope4<VEC>(n, v, vec, st, ep, o);
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = epi_value<EPI>(v[r], u[r], st, vec[r], cs[r]);
  }
}

// The same as bf16, 8 bytes.
template <int EPI, bool VEC>
__device__ __forceinline__ u32x2 epi4_bf16(int n, f32x4 v, f32x4 u, RowStat st, const EpiArgs& ep) {
  float o[4];
  epi4_values<EPI, VEC>(n, v, u, st, ep, o);
  return pack4_bf16(o);
}

// EPI_HEADNORM: the 8 columns n .. n+7 of one row, held by one lane; a head's h/8
// such units sit in h/8 consecutive lanes of the wave, which sum their squares by
// butterfly exchange (every lane of the wave takes part).  By Prop. 3 the input
// norm's scale cancels in a normalised head, so Q and K heads (and V heads when gv
// is given: QKV-normalization) are normalised straight from a W*: t / sqrt(eps_h +
// mean(t^2)) * w, then RoPE on Q and K when positions are given, and Q times the
// score scale.  V heads without gv take the input scale s.
__device__ __forceinline__ void headnorm8(int n, f32x4 a0, f32x4 a1, RowStat st, const EpiArgs& ep,
                                          float (&o)[8]) {
  float ss = ((a0[0] * a0[0] + a0[1] * a0[1]) + (a0[2] * a0[2] + a0[3] * a0[3])) +
             ((a1[0] * a1[0] + a1[1] * a1[1]) + (a1[2] * a1[2] + a1[3] * a1[3]));
  for (int off = 1; off < (ep.head_h >> 3); off <<= 1) ss += __shfl_xor(ss, off);
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = a0[e], o[4 + e] = a1[e];
  const bool is_q = n < ep.q_end, is_k = !is_q && n < ep.k_end;
  const float* w = is_q ? ep.hn_gq : is_k ? ep.hn_gk : ep.hn_gv;
  const int c = rope_col_in_head(n, ep);
  if (w) {
    const float sc = rsqrtf(fmaf(ss, ep.head_inv_h, ep.hn_eps));
    const f32x4 w0 = *reinterpret_cast<const f32x4*>(w + c), w1 = *reinterpret_cast<const f32x4*>(w + c + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] *= sc * w0[e], o[4 + e] *= sc * w1[e];
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] *= st.s;
  }
  if ((is_q || is_k) && ep.rope_pos) {
    const bool valid = (unsigned)st.pos < (unsigned)ep.rope_P;
    const int64_t off = (int64_t)(valid ? st.pos : 0) * (ep.head_h >> 1) + (c >> 1);
    const f32x4 cs = *reinterpret_cast<const f32x4*>(ep.rope_cos + off);
    const f32x4 sn = *reinterpret_cast<const f32x4*>(ep.rope_sin + off);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float x0 = o[2 * q], x1 = o[2 * q + 1];
      o[2 * q] = valid ? x0 * cs[q] - x1 * sn[q] : __builtin_nanf("");
      o[2 * q + 1] = valid ? x0 * sn[q] + x1 * cs[q] : __builtin_nanf("");
    }
  }
  if (is_q) {
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] *= ep.q_scale;
  }
}

// EPI_ROPE with the angles (rope_tab) and the bias of the four columns (zeros
// without) already loaded.
template <bool VEC>
__device__ __forceinline__ u32x2 rope4_bf16(int n, f32x4 v, f32x4 vec, RowStat st, RopeTab tb, const EpiArgs& ep) {
  float o[4];
  rope_apply<VEC>(n, v, vec, st, tb, ep, o);
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

// Output stores of whole 16-byte units carry the non-temporal hint: the kernel never
// reads its output back, and on MI355X the hint shortened the SmolLM2-width prefill by
// ~18% (no L2 allocation for 6.3 MB of output) and the Llama-7B shapes by ~1%.
__device__ __forceinline__ void store_out16(__bf16* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
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
    store_out16(y + (int64_t)(m0 + r) * ldy + n0 + u * 8, v);
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
  unsigned short* dst = reinterpret_cast<unsigned short*>(y + (int64_t)m * ldy + n);
  if constexpr (EPI == EPI_ROPE) {
    // the output width is a multiple of the head width: the 4 columns lie wholly
    // inside or wholly outside
    if (n >= ncols) return;
    float o[4];
    epi4_values<EPI, VEC>(n, v, u, st, ep, o);
#pragma unroll
    for (int r = 0; r < 4; ++r) dst[r] = __builtin_bit_cast(unsigned short, (__bf16)o[r]);
  } else {
    const float* vp = epi_vec<EPI>(ep);
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
}

}  // namespace fn
