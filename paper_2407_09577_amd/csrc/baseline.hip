// Normalisation kernels of the unfused baseline (Fig. 1(a), the sequential
// RMSNorm -> GEMM that FlashNorm replaces): one workgroup per activation row
// writes x = RMSNorm(a; g) = a / RMSe(a) * g, or the LayerNorm
// x = (a - mu) / sqrt(var + eps) * g + beta (two passes over the row held in
// registers), rounded once to the activation type.  The matrix multiply then
// runs on x with the same kernels as the fused path, minus the epilogue scale.
#include "fn_device.h"
#include "fn_launch.h"

namespace fn {

constexpr int kNormThreads = 256;
constexpr int kNormMaxPerThread = 64;  // K <= 16384 elements per row

__device__ __forceinline__ float block_sum(float v, float* sh) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int w = 0; w < kNormThreads / 64; ++w) t += sh[w];
  return t;
}

template <typename T, bool LN>
__global__ __launch_bounds__(kNormThreads) void norm_rows_kernel(const T* __restrict__ a, int K, int lda,
                                                                 const float* __restrict__ g,
                                                                 const float* __restrict__ beta, float eps,
                                                                 T* __restrict__ x, int ldx) {
  __shared__ float sh[kNormThreads / 64];
  const T* ar = a + (int64_t)blockIdx.x * lda;
  T* xr = x + (int64_t)blockIdx.x * ldx;
  float v[kNormMaxPerThread];
  float s1 = 0.f;
#pragma unroll
  for (int i = 0; i < kNormMaxPerThread; ++i) {
    const int k = threadIdx.x + i * kNormThreads;
    v[i] = k < K ? (float)ar[k] : 0.f;
    s1 += LN ? v[i] : v[i] * v[i];
  }
  s1 = block_sum(s1, sh);
  float mu = 0.f, scale;
  if constexpr (LN) {
    mu = s1 / K;
    float s2 = 0.f;
#pragma unroll
    for (int i = 0; i < kNormMaxPerThread; ++i) {
      const int k = threadIdx.x + i * kNormThreads;
      const float d = k < K ? v[i] - mu : 0.f;
      s2 += d * d;
    }
    s2 = block_sum(s2, sh);
    scale = rsqrtf(s2 / K + eps);
  } else {
    scale = rsqrtf(s1 / K + eps);
  }
#pragma unroll
  for (int i = 0; i < kNormMaxPerThread; ++i) {
    const int k = threadIdx.x + i * kNormThreads;
    if (k < K) {
      float o = (v[i] - mu) * scale * g[k];
      if constexpr (LN) o += beta[k];
      xr[k] = (T)o;
    }
  }
}

template <bool LN>
static hipError_t launch_norm_t(const void* a, int M, int K, int lda, int dtype, const float* g,
                                const float* beta, float eps, void* x, int ldx, hipStream_t s) {
  if (dtype == kDtypeBf16)
    hipLaunchKernelGGL((norm_rows_kernel<__bf16, LN>), dim3(M), dim3(kNormThreads), 0, s,
                       (const __bf16*)a, K, lda, g, beta, eps, (__bf16*)x, ldx);
  else
    hipLaunchKernelGGL((norm_rows_kernel<float, LN>), dim3(M), dim3(kNormThreads), 0, s, (const float*)a,
                       K, lda, g, beta, eps, (float*)x, ldx);
  return hipGetLastError();
}

hipError_t launch_norm_rows(const void* a, int M, int K, int lda, int dtype, const float* g,
                            const float* beta, float eps, void* x, int ldx, hipStream_t stream) {
  if (K > kNormThreads * kNormMaxPerThread) return hipErrorInvalidValue;
  return beta ? launch_norm_t<true>(a, M, K, lda, dtype, g, beta, eps, x, ldx, stream)
              : launch_norm_t<false>(a, M, K, lda, dtype, g, beta, eps, x, ldx, stream);
}

}  // namespace fn
