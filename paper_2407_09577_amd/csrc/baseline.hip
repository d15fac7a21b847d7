// Normalisation kernels of the unfused baseline (Fig. 1(a), the sequential
// RMSNorm -> GEMM that FlashNorm replaces): one wave per activation row writes
// x = RMSNorm(a; g) = a / RMSe(a) * g, or the LayerNorm
// x = (a - mu) / sqrt(var + eps) * g + beta (mean first, then the centred sum of
// squares: two passes over the row), rounded once to the activation type.  The
// matrix multiply then runs on x with the same kernels as the fused path, minus
// the epilogue scale.  Memory-bound: 16-byte accesses, the row re-reads hit L2.
#include "fn_device.h"
#include "fn_launch.h"
#include "fn_epilogue.h"

namespace fn {

constexpr int kRowsPerBlock = 4;

template <typename T>
struct Vec16 {
  static constexpr int N = 16 / sizeof(T);
  float v[N];
  __device__ __forceinline__ void load(const T* p) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(p);
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[2 * i] = bf16_lo(w[i]);
        v[2 * i + 1] = bf16_hi(w[i]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = __uint_as_float(w[i]);
    }
  }
  __device__ __forceinline__ void store(T* p) const {
    u32x4 w;
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = __float_as_uint(v[i]);
    }
    __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(p));  // as the fused kernels' output stores
  }
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

template <typename T, bool LN>
__global__ __launch_bounds__(64 * kRowsPerBlock) void norm_rows_kernel(
    const T* __restrict__ a, int M, int K, int lda, const float* __restrict__ g,
    const float* __restrict__ beta, float eps, T* __restrict__ x, int ldx) {
  constexpr int V = Vec16<T>::N;
  const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= M) return;
  const int lane = threadIdx.x & 63;
  const T* ar = a + (int64_t)row * lda;
  T* xr = x + (int64_t)row * ldx;
  float s = 0.f;
  for (int k = lane * V; k < K; k += 64 * V) {
    Vec16<T> c;
    c.load(ar + k);
#pragma unroll
    for (int i = 0; i < V; ++i) s += LN ? c.v[i] : c.v[i] * c.v[i];
  }
  s = wave_sum(s);
  float mu = 0.f, scale;
  if constexpr (LN) {
    mu = s / K;
    float d2 = 0.f;
    for (int k = lane * V; k < K; k += 64 * V) {
      Vec16<T> c;
      c.load(ar + k);
#pragma unroll
      for (int i = 0; i < V; ++i) d2 += (c.v[i] - mu) * (c.v[i] - mu);
    }
    scale = rsqrtf(wave_sum(d2) / K + eps);
  } else {
    scale = rsqrtf(s / K + eps);
  }
  for (int k = lane * V; k < K; k += 64 * V) {
    Vec16<T> c;
    c.load(ar + k);
#pragma unroll
    for (int i = 0; i < V; ++i) {
      float o = (c.v[i] - mu) * scale * g[k + i];
      if constexpr (LN) o += beta[k + i];
      c.v[i] = o;
    }
    c.store(xr + k);
  }
}

template <bool LN>
static hipError_t launch_norm_t(const void* a, int M, int K, int lda, int dtype, const float* g,
                                const float* beta, float eps, void* x, int ldx, hipStream_t s) {
  const dim3 grid((M + kRowsPerBlock - 1) / kRowsPerBlock), block(64 * kRowsPerBlock);
  if (dtype == kDtypeBf16)
    hipLaunchKernelGGL((norm_rows_kernel<__bf16, LN>), grid, block, 0, s, (const __bf16*)a, M, K, lda, g,
                       beta, eps, (__bf16*)x, ldx);
  else
    hipLaunchKernelGGL((norm_rows_kernel<float, LN>), grid, block, 0, s, (const float*)a, M, K, lda, g, beta,
                       eps, (float*)x, ldx);
  return hipGetLastError();
}

hipError_t launch_norm_rows(const void* a, int M, int K, int lda, int dtype, const float* g,
                            const float* beta, float eps, void* x, int ldx, hipStream_t stream) {
  return beta ? launch_norm_t<true>(a, M, K, lda, dtype, g, beta, eps, x, ldx, stream)
              : launch_norm_t<false>(a, M, K, lda, dtype, g, beta, eps, x, ldx, stream);
}

// Stand-alone RoPE over the Q and K heads of y, in place: the separate rotation
// of the unfused chain (Fig. 5(a)).  One thread per 4 columns (two pairs of one
// head) of one row; Q columns also take q_scale.  Memory-bound.
template <typename T>
__global__ __launch_bounds__(256) void rope_rows_kernel(T* __restrict__ y, int M, int ldy, int qk, int q_end,
                                                        int h, const int* __restrict__ pos,
                                                        const float* __restrict__ cos_tab,
                                                        const float* __restrict__ sin_tab, int P, float q_scale) {
  const int groups = qk / 4;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)M * groups) return;
  const int m = (int)(idx / groups), n = (int)(idx % groups) * 4;
  T* p = y + (int64_t)m * ldy + n;
  float t[4];
  if constexpr (sizeof(T) == 2) {
    const u32x2 w = *reinterpret_cast<const u32x2*>(p);
    t[0] = bf16_lo(w[0]), t[1] = bf16_hi(w[0]), t[2] = bf16_lo(w[1]), t[3] = bf16_hi(w[1]);
  } else {
    const f32x4 w = *reinterpret_cast<const f32x4*>(p);
    t[0] = w[0], t[1] = w[1], t[2] = w[2], t[3] = w[3];
  }
  const int ps = pos[m];
  const float qs = n < q_end ? q_scale : 1.0f;
  float o[4];
  if ((unsigned)ps < (unsigned)P) {
    const int64_t off = (int64_t)ps * (h / 2) + (n % h) / 2;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const float c = cos_tab[off + q], sn = sin_tab[off + q];
      o[2 * q] = (t[2 * q] * c - t[2 * q + 1] * sn) * qs;
      o[2 * q + 1] = (t[2 * q] * sn + t[2 * q + 1] * c) * qs;
    }
  } else {
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = __builtin_nanf("");
  }
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<u32x2*>(p) = u32x2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
  } else {
    *reinterpret_cast<f32x4*>(p) = f32x4{o[0], o[1], o[2], o[3]};
  }
}

hipError_t launch_rope_rows(void* y, int M, int ldy, int dtype, int qk, int q_end, int h, const int* pos,
                            const float* cos_tab, const float* sin_tab, int P, float q_scale, hipStream_t stream) {
  const int64_t threads = (int64_t)M * (qk / 4);
  const dim3 grid((unsigned)((threads + 255) / 256)), block(256);
  if (dtype == kDtypeBf16)
    hipLaunchKernelGGL(rope_rows_kernel<__bf16>, grid, block, 0, stream, (__bf16*)y, M, ldy, qk, q_end, h, pos,
                       cos_tab, sin_tab, P, q_scale);
  else
    hipLaunchKernelGGL(rope_rows_kernel<float>, grid, block, 0, stream, (float*)y, M, ldy, qk, q_end, h, pos,
                       cos_tab, sin_tab, P, q_scale);
  return hipGetLastError();
}

// Stand-alone per-head RMSNorm (QK-norm / QKV-normalization) with RoPE over the
// normalised output of the unfused chain, in place: one thread per 8 columns of a
// row; a head's h/8 threads are consecutive lanes (rows hold whole heads), so the
// head's squares are summed by butterfly exchange.  The same per-unit arithmetic
// as the fused epilogue, with the input scale already applied (s = 1).
__global__ __launch_bounds__(256) void headnorm_rows_kernel(__bf16* __restrict__ y, int M, int ldy, int ncols,
                                                            EpiArgs ep) {
  const int U = ncols / 8;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)M * U) return;  // whole heads leave together
  const int m = (int)(idx / U), v = (int)(idx % U);
  __bf16* p = y + (int64_t)m * ldy + v * 8;
  const u32x4 w = *reinterpret_cast<const u32x4*>(p);
  const f32x4 a0 = {bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])};
  const f32x4 a1 = {bf16_lo(w[2]), bf16_hi(w[2]), bf16_lo(w[3]), bf16_hi(w[3])};
  const RowStat st{1.0f, 0.0f, ep.rope_pos ? ep.rope_pos[m] : 0};
  float o[8];
  headnorm8(v * 8, a0, a1, st, ep, o);
  *reinterpret_cast<u32x4*>(p) = u32x4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]),
                                       pack_bf16x2(o[4], o[5]), pack_bf16x2(o[6], o[7])};
}

hipError_t launch_headnorm_rows(void* y, int M, int ldy, int ncols, const EpiArgs& ep, hipStream_t stream) {
  const int64_t threads = (int64_t)M * (ncols / 8);
  const dim3 grid((unsigned)((threads + 255) / 256)), block(256);
  hipLaunchKernelGGL(headnorm_rows_kernel, grid, block, 0, stream, (__bf16*)y, M, ldy, ncols, ep);
  return hipGetLastError();
}

}  // namespace fn
