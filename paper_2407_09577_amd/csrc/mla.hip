// Latent RMSNorm and rotary key of the MLA down-projection (Sec. 3.3, the
// paragraph on multi-head latent attention): the row pass that follows the
// projection y = a W* of the fused kernels.
//
// The projection leaves u = t * s in y, with t = a W* and s the input row's
// deferred scale 1/RMSe(a) (or s = 1 when the caller takes no statistics of a).
// For the first L columns (the latent) this pass writes the cancelled form of
// Prop. 3, t / sqrt(eps_lat + mean(t^2)) * g_lat, computed from u as
// u * rsqrt(mean(u^2) + eps_lat s^2), which is the same quantity: the input
// norm's scale drops out of a normalised latent.  The R columns after it (the
// rotary key shared by all heads, one head of width R; no norm follows it) keep
// u and are turned by RoPE at the row's position, consecutive pairs as in the
// fused QKV epilogues.  A position outside the table makes them NaN.
//
// One wave per row: lane l holds the 8-column units l, l + 64, ... of the latent
// (L <= 2048: at most four units), sums their squares, and the wave's butterfly
// exchange gives every lane the row total (a fixed order: deterministic).  The
// rotary units go to lanes 0 .. R/8 - 1.  Memory-bound: 16-byte accesses.
#include "fn_device.h"
#include "fn_launch.h"

namespace fn {

namespace {

constexpr int kMlaRowsPerBlock = 4;
constexpr int kMlaMaxUnits = 4;  // 8-column latent units per lane: L <= 2048

template <typename T>
__device__ __forceinline__ void load8(const T* p, float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = bf16_lo(w[i]);
      v[2 * i + 1] = bf16_hi(w[i]);
    }
  } else {
    const f32x4 w0 = *reinterpret_cast<const f32x4*>(p), w1 = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = w0[i], v[4 + i] = w1[i];
  }
}

template <typename T>
__device__ __forceinline__ void store8(T* p, const float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<u32x4*>(p) = u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                         pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
  } else {
    *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4*>(p + 4) = f32x4{v[4], v[5], v[6], v[7]};
  }
}

template <typename T>
__global__ __launch_bounds__(64 * kMlaRowsPerBlock) void mla_latent_rows_kernel(
    T* __restrict__ y, int M, int ldy, int L, int R, float inv_l, const float* __restrict__ g_lat, float eps_lat,
    const float* __restrict__ s_row, const int* __restrict__ pos, const float* __restrict__ cos_tab,
    const float* __restrict__ sin_tab, int P) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * kMlaRowsPerBlock + (threadIdx.x >> 6);
  if (m >= M) return;  // wave-uniform: whole waves leave together
  T* row = y + (int64_t)m * ldy;
  const int UL = L >> 3;
  const bool key = lane < (R >> 3);

  // Every load that does not depend on another goes out first (the latent units,
  // their weights, the row's scale and position, the key unit), so the pass waits
  // for about two memory latencies, not one per step.
  float v[kMlaMaxUnits][8];
  f32x4 gw[kMlaMaxUnits][2];
#pragma unroll
  for (int i = 0; i < kMlaMaxUnits; ++i) {
    const int u = lane + 64 * i;
    if (u < UL) {
      load8(row + u * 8, v[i]);
      gw[i][0] = *reinterpret_cast<const f32x4*>(g_lat + u * 8);
      gw[i][1] = *reinterpret_cast<const f32x4*>(g_lat + u * 8 + 4);
    }
  }
  const float s = s_row ? s_row[m] : 1.0f;
  float t[8];
  int ps = 0;
  if (key) {
    load8(row + L + lane * 8, t);
    ps = pos[m];
  }

  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < kMlaMaxUnits; ++i)
    if (lane + 64 * i < UL) {
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(v[i][e], v[i][e], ss);
    }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
  const float r = rsqrtf(fmaf(ss, inv_l, eps_lat * s * s));
#pragma unroll
  for (int i = 0; i < kMlaMaxUnits; ++i) {
    const int u = lane + 64 * i;
    if (u < UL) {
      float o[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o[e] = v[i][e] * r * gw[i][0][e];
        o[4 + e] = v[i][4 + e] * r * gw[i][1][e];
      }
      store8(row + u * 8, o);
    }
  }

  if (key) {
    const bool valid = (unsigned)ps < (unsigned)P;
    const int64_t off = (int64_t)(valid ? ps : 0) * (R >> 1) + lane * 4;  // pairs 4 lane .. 4 lane + 3
    const f32x4 cs = *reinterpret_cast<const f32x4*>(cos_tab + off);
    const f32x4 sn = *reinterpret_cast<const f32x4*>(sin_tab + off);
    float o[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      o[2 * q] = valid ? t[2 * q] * cs[q] - t[2 * q + 1] * sn[q] : __builtin_nanf("");
      o[2 * q + 1] = valid ? t[2 * q] * sn[q] + t[2 * q + 1] * cs[q] : __builtin_nanf("");
    }
    store8(row + L + lane * 8, o);
  }
}

}  // namespace

hipError_t launch_mla_latent_rows(void* y, int M, int ldy, int dtype, int L, int R, const float* g_lat,
                                  float eps_lat, const float* s_row, const int* pos, const float* cos_tab,
                                  const float* sin_tab, int P, hipStream_t stream) {
  const dim3 grid((unsigned)((M + kMlaRowsPerBlock - 1) / kMlaRowsPerBlock)), block(64 * kMlaRowsPerBlock);
  const float inv_l = 1.0f / (float)L;
  if (dtype == kDtypeBf16)
    hipLaunchKernelGGL(mla_latent_rows_kernel<__bf16>, grid, block, 0, stream, (__bf16*)y, M, ldy, L, R, inv_l,
                       g_lat, eps_lat, s_row, pos, cos_tab, sin_tab, P);
  else
    hipLaunchKernelGGL(mla_latent_rows_kernel<float>, grid, block, 0, stream, (float*)y, M, ldy, L, R, inv_l,
                       g_lat, eps_lat, s_row, pos, cos_tab, sin_tab, P);
  return hipGetLastError();
}

}  // namespace fn
