// Offline weight fold (Prop. 1: W*[k,n] = g_k W[k,n]; Sec. 3.4: c* = beta W) and
// the packing into the kernels' layout.  Runs once per weight, off the hot path.
//
// Each stored element is the exact product g_k * W[k,n] (a bf16 or fp32 weight
// times an fp32 g is exact in fp64) rounded once, to nearest with ties to even,
// into the storage type.  colsum sums the stored values and c* the products of
// beta with the unfolded W, both in fp64, rounded once to fp32.
#include "fn_device.h"
#include "fn_launch.h"

namespace fn {

// Packed column -> logical column, or -1 for padding.
__device__ __forceinline__ int64_t logical_col(int64_t p, int64_t N, int glu) {
  if (!glu) return p < N ? p : -1;
  const int64_t F = N / 2;
  const int64_t pair = p / 32, within = p % 32;
  const int64_t f = pair * 16 + (within & 15);
  if (f >= F) return -1;
  return within < 16 ? f : F + f;
}

// Round a double to the nearest bf16 (ties to even), returning the bit pattern.
// Normal range: add the rounding bias below bit 45 of the binary64 pattern (the
// 45 bits that bf16's 7-bit significand drops) and truncate, letting a carry
// ripple into the exponent.  Below 2^-126 bf16 is subnormal with fixed spacing
// 2^-133: scale, round to an integer (rint rounds ties to even), scale back.
__device__ __forceinline__ unsigned short dbl_to_bf16_rne(double x) {
  if (x != x) return 0x7fc0;
  if (fabs(x) < 0x1p-126) {
    const double r = rint(x * 0x1p133) * 0x1p-133;
    return (unsigned short)(__float_as_uint((float)r) >> 16);
  }
  unsigned long long u = (unsigned long long)__double_as_longlong(x);
  u += 0xfffffffffffull + ((u >> 45) & 1ull);
  u &= ~((1ull << 45) - 1ull);
  const float f = (float)__longlong_as_double((long long)u);  // exact, or overflow -> inf
  return (unsigned short)(__float_as_uint(f) >> 16);
}

__device__ __forceinline__ double load_w(const void* W, int64_t idx, int w_dtype) {
  if (w_dtype == kDtypeBf16) {
    const unsigned short b = reinterpret_cast<const unsigned short*>(W)[idx];
    return (double)__uint_as_float((unsigned)b << 16);
  }
  return (double)reinterpret_cast<const float*>(W)[idx];
}

// One thread per 16-byte chunk (8 consecutive k of one packed column) of the
// fragment-major bf16 layout.
__global__ void fold_pack_bf16_kernel(const void* __restrict__ W, int64_t sk, int64_t sn, int w_dtype,
                                      const float* __restrict__ g, int64_t K, int64_t N, int glu,
                                      int64_t NPB, int64_t nchunks, u32x4* __restrict__ out) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nchunks) return;
  const int64_t frag = c / 64;
  const int lane = (int)(c % 64);
  const int64_t kb = frag / NPB, cb = frag % NPB;
  const int64_t p = cb * 16 + (lane & 15);
  const int64_t k0 = kb * kKB + (lane >> 4) * 8;
  const int64_t n = logical_col(p, N, glu);
  unsigned short h[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int64_t k = k0 + e;
    double v = 0.0;
    if (n >= 0 && k < K) v = (g ? (double)g[k] : 1.0) * load_w(W, k * sk + n * sn, w_dtype);
    h[e] = dbl_to_bf16_rne(v);
  }
  out[c] = u32x4{h[0] | ((unsigned)h[1] << 16), h[2] | ((unsigned)h[3] << 16),
                 h[4] | ((unsigned)h[5] << 16), h[6] | ((unsigned)h[7] << 16)};
}

// fp32 storage: row-major [KP][NP] with columns in packed order.
__global__ void fold_pack_f32_kernel(const void* __restrict__ W, int64_t sk, int64_t sn, int w_dtype,
                                     const float* __restrict__ g, int64_t K, int64_t N, int glu,
                                     int64_t KP, int64_t NP, float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= KP * NP) return;
  const int64_t k = i / NP, p = i % NP;
  const int64_t n = logical_col(p, N, glu);
  double v = 0.0;
  if (n >= 0 && k < K) v = (g ? (double)g[k] : 1.0) * load_w(W, k * sk + n * sn, w_dtype);
  out[i] = (float)v;  // one round to nearest even
}

// Stored element (k, p) of a packed buffer, as fp64.
__device__ __forceinline__ double packed_at(const void* ws, int ws_dtype, int64_t k, int64_t p,
                                            int64_t KP, int64_t NP) {
  if (ws_dtype == kDtypeBf16) {
    const int64_t off = ((k / kKB) * (NP / 16) + p / 16) * 512 + (((k % kKB) / 8) * 16 + p % 16) * 8 + k % 8;
    const unsigned short b = reinterpret_cast<const unsigned short*>(ws)[off];
    return (double)__uint_as_float((unsigned)b << 16);
  }
  return (double)reinterpret_cast<const float*>(ws)[k * NP + p];
}

// LayerNorm extras for a linear layout (packed column == logical column).
__global__ void fold_colsum_kernel(const void* __restrict__ ws, int ws_dtype, const void* __restrict__ W,
                                   int64_t sk, int64_t sn, int w_dtype, const float* __restrict__ beta, int64_t K,
                                   int64_t N, int64_t KP, int64_t NP, float* __restrict__ colsum,
                                   float* __restrict__ cstar) {
  const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  double cs = 0.0, cb = 0.0;
  for (int64_t k = 0; k < K; ++k) {
    if (colsum) cs += packed_at(ws, ws_dtype, k, n, KP, NP);
    if (cstar) cb += (double)beta[k] * load_w(W, k * sk + n * sn, w_dtype);
  }
  if (colsum) colsum[n] = (float)cs;
  if (cstar) cstar[n] = (float)cb;
}

__global__ void unpack_kernel(const void* __restrict__ ws, int ws_dtype, int64_t K, int64_t N, int glu,
                              int64_t KP, int64_t NP, void* __restrict__ out, int64_t ldo) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= K * NP) return;
  const int64_t k = i / NP, p = i % NP;
  const int64_t n = logical_col(p, N, glu);
  if (n < 0) return;
  if (ws_dtype == kDtypeBf16) {
    const int64_t off = ((k / kKB) * (NP / 16) + p / 16) * 512 + (((k % kKB) / 8) * 16 + p % 16) * 8 + k % 8;
    reinterpret_cast<unsigned short*>(out)[k * ldo + n] = reinterpret_cast<const unsigned short*>(ws)[off];
  } else {
    reinterpret_cast<float*>(out)[k * ldo + n] = reinterpret_cast<const float*>(ws)[k * NP + p];
  }
}

static unsigned blocks_for(int64_t n, int threads) { return (unsigned)((n + threads - 1) / threads); }

hipError_t launch_fold(const FoldArgs& p) {
  const int64_t KP = packed_rows(p.K), NP = packed_cols(p.N, p.glu);
  if (p.ws_dtype == kDtypeBf16) {
    const int64_t nchunks = KP * NP / 8;
    hipLaunchKernelGGL(fold_pack_bf16_kernel, dim3(blocks_for(nchunks, 256)), dim3(256), 0, p.stream, p.W,
                       p.sk, p.sn, p.w_dtype, p.g, p.K, p.N, p.glu, NP / 16, nchunks,
                       reinterpret_cast<u32x4*>(p.ws));
  } else {
    hipLaunchKernelGGL(fold_pack_f32_kernel, dim3(blocks_for(KP * NP, 256)), dim3(256), 0, p.stream, p.W,
                       p.sk, p.sn, p.w_dtype, p.g, p.K, p.N, p.glu, KP, NP, reinterpret_cast<float*>(p.ws));
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.colsum || p.cstar) {
    hipLaunchKernelGGL(fold_colsum_kernel, dim3(blocks_for(p.N, 128)), dim3(128), 0, p.stream, p.ws,
                       p.ws_dtype, p.W, p.sk, p.sn, p.w_dtype, p.beta, p.K, p.N, KP, NP, p.colsum, p.cstar);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_unpack(const void* ws, int64_t K, int64_t N, int glu, int ws_dtype, void* out,
                         int64_t ldo, hipStream_t stream) {
  const int64_t KP = packed_rows(K), NP = packed_cols(N, glu);
  hipLaunchKernelGGL(unpack_kernel, dim3(blocks_for(K * NP, 256)), dim3(256), 0, stream, ws, ws_dtype, K,
                     N, glu, KP, NP, out, ldo);
  return hipGetLastError();
}

}  // namespace fn
