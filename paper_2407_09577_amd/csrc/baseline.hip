// Normalisation kernels of the unfused baseline (Fig. 1(a), the sequential
// RMSNorm -> GEMM that FlashNorm replaces): one wave per activation row writes
// x = RMSNorm(a; g) = a / RMSe(a) * g, or the LayerNorm
// x = (a - mu) / sqrt(var + eps) * g + beta (mean first, then the centred sum of
// squares: two passes over the row), rounded once to the activation type.  The
// matrix multiply then runs on x with the same kernels as the fused path, minus
// the epilogue scale.  Memory-bound: 16-byte accesses, the row re-reads hit L2.
#include "fn_device.h"
#include "fn_launch.h"

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
    *reinterpret_cast<u32x4*>(p) = w;
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

}  // namespace fn
