// Few-row (decode) fused norm-then-project kernel for gfx950.
//
// With M <= 16 activation rows the product is bound by streaming W* from HBM
// once (Sec. 6 and App. "End-to-end validation": decode is memory-bound and
// wants its own kernel instead of a padded prefill tile).  A workgroup owns NCB
// packed column blocks of 16 columns (for a GLU, whole gate/up block pairs) and
// its KSPLIT waves split K: wave w takes the 32-row fragments w, w + KSPLIT, ...
// so the waves of one workgroup read adjacent 1 KiB fragments.  Each fragment is
// one 16-byte load per lane, fed directly to a 16x16x32 bf16 matrix-core op
// together with the matching 16-row activation fragment (rows >= M read as
// zero), so the arithmetic costs nothing next to the stream.  The squares of
// the activation fragments are summed on the way (Cor. 1), the per-wave
// partial products and sums are combined in LDS in a fixed order
// (deterministic), and one wave per output block applies the deferred scale and
// the epilogue.
#include <type_traits>

#include "fn_device.h"
#include "fn_epilogue.h"
#include "fn_launch.h"

namespace fn {

template <int NCB, int KSPLIT, int U, int EPI>
__global__ __launch_bounds__(KSPLIT * 64) void decode_bf16_kernel(
    const __bf16* __restrict__ a, int M, int K, int lda, const __bf16* __restrict__ ws, int NP,
    int KP, int ncols, __bf16* __restrict__ y, int ldy, EpiArgs ep) {
  constexpr bool kSS = epi_needs_ss(EPI);
  constexpr bool kSA = EPI == EPI_LN;
  constexpr int NOUT = epi_is_glu(EPI) ? NCB / 2 : NCB;  // output blocks per workgroup
  static_assert(!epi_is_glu(EPI) || NCB % 2 == 0, "GLU needs gate/up block pairs");

  __shared__ f32x4 red[KSPLIT][NCB][64];
  __shared__ float red_ss[KSPLIT][16];
  __shared__ float red_sa[KSPLIT][16];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int cb0 = blockIdx.x * NCB;
  const int KB = KP / kKB;

  const __amdgpu_buffer_rsrc_t rs_a = make_rsrc(a, (uint32_t)(((int64_t)(M - 1) * lda + K) * 2));
  // Column blocks past the packed width (last workgroup only) read the next k
  // block's fragments, or zeros past the end; their outputs are never stored.
  const int npb = NP / 16;
  const __amdgpu_buffer_rsrc_t rs_w =
      make_rsrc(ws + (int64_t)cb0 * (kFragBytes / 2), (uint32_t)(((int64_t)KB * npb - cb0) * kFragBytes));

  const int lrow = lane & 15;
  const int lk = (lane >> 4) * 8;
  const bool row_ok = lrow < M;
  const unsigned a_row_off = (unsigned)(lrow * lda * 2);

  f32x4 acc[NCB];
#pragma unroll
  for (int c = 0; c < NCB; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  float ss = 0.f, sa = 0.f;

  for (int kb0 = wave; kb0 < KB; kb0 += KSPLIT * U) {
    u32x4 af[U], wf[U][NCB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb0 + KSPLIT * u;
      const int k = kb * kKB + lk;
      const bool kb_ok = kb < KB;
      af[u] = load_buf16(rs_a, (kb_ok && row_ok && k < K) ? a_row_off + (unsigned)k * 2 : kOobOffset);
#pragma unroll
      for (int c = 0; c < NCB; ++c)
        wf[u][c] = load_buf16(rs_w, kb_ok ? (unsigned)((kb * npb + c) * kFragBytes + lane * 16) : kOobOffset);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bf16x8 av = __builtin_bit_cast(bf16x8, af[u]);
      if constexpr (kSS) ss = sumsq8(av, ss);
      if constexpr (kSA) sa = sum8(av, sa);
#pragma unroll
      for (int c = 0; c < NCB; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf[u][c]), av,
                                                          acc[c], 0, 0, 0);
    }
  }

  if constexpr (kSS) {
    ss += __shfl_xor(ss, 16);
    ss += __shfl_xor(ss, 32);
  }
  if constexpr (kSA) {
    sa += __shfl_xor(sa, 16);
    sa += __shfl_xor(sa, 32);
  }
#pragma unroll
  for (int c = 0; c < NCB; ++c) red[wave][c][lane] = acc[c];
  if (lane < 16) {
    red_ss[wave][lane] = ss;
    red_sa[wave][lane] = sa;
  }
  __syncthreads();

  const int m = lrow;
  if (m >= M) return;
  float ss_t = 0.f, sa_t = 0.f;
#pragma unroll
  for (int w = 0; w < KSPLIT; ++w) {
    ss_t += red_ss[w][m];
    sa_t += red_sa[w][m];
  }
  const RowStat st = row_stat<EPI>(ss_t, sa_t, ep);
  if constexpr (EPI == EPI_RMS) {
    if (ep.inv_rms && blockIdx.x == 0 && wave == 0 && lane < 16) ep.inv_rms[m] = st.s;
  }
  const int n_lane = (lane >> 4) * 4;
  auto epilogue = [&](auto vec_tag) {
    constexpr bool VEC = decltype(vec_tag)::value;
    for (int o = wave; o < NOUT; o += KSPLIT) {
      if constexpr (epi_is_glu(EPI)) {
        f32x4 g = red[0][2 * o][lane], u = red[0][2 * o + 1][lane];
#pragma unroll
        for (int w = 1; w < KSPLIT; ++w) {
          g += red[w][2 * o][lane];
          u += red[w][2 * o + 1][lane];
        }
        const int fb = (cb0 / 2 + o) * 16;
        if (fb + 16 <= ncols)
          store4_bf16_full<EPI, VEC>(y, ldy, m, fb + n_lane, g, u, st, ep);
        else
          store4_bf16_edge<EPI, VEC>(y, ldy, M, ncols, m, fb + n_lane, g, u, st, ep);
      } else {
        f32x4 v = red[0][o][lane];
#pragma unroll
        for (int w = 1; w < KSPLIT; ++w) v += red[w][o][lane];
        const int pb = (cb0 + o) * 16;
        if (pb + 16 <= ncols)
          store4_bf16_full<EPI, VEC>(y, ldy, m, pb + n_lane, v, v, st, ep);
        else
          store4_bf16_edge<EPI, VEC>(y, ldy, M, ncols, m, pb + n_lane, v, v, st, ep);
      }
    }
  };
  if (epi_vec<EPI>(ep) != nullptr)
    epilogue(std::true_type{});
  else
    epilogue(std::false_type{});
}

template <int NCB, int KSPLIT, int U, int EPI>
static hipError_t launch_decode_cfg(const DecodeArgs& p) {
  const int nblocks = (p.NP / 16 + NCB - 1) / NCB;
  hipLaunchKernelGGL((decode_bf16_kernel<NCB, KSPLIT, U, EPI>), dim3(nblocks), dim3(KSPLIT * 64), 0,
                     p.stream, p.a, p.M, p.K, p.lda, p.ws, p.NP, p.KP, p.ncols, p.y, p.ldy, p.ep);
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_decode_epi(const DecodeArgs& p) {
  switch (p.cfg) {
    case 0:
    case 3: return launch_decode_cfg<2, 2, 8, EPI>(p);
    case 1: return launch_decode_cfg<2, 8, 8, EPI>(p);
    case 2: return launch_decode_cfg<2, 4, 8, EPI>(p);
    case 4: return launch_decode_cfg<2, 2, 4, EPI>(p);
    case 5: return launch_decode_cfg<2, 2, 16, EPI>(p);
    case 6: return launch_decode_cfg<2, 1, 8, EPI>(p);
    case 7: return launch_decode_cfg<2, 1, 16, EPI>(p);
    case 8: return launch_decode_cfg<4, 2, 8, EPI>(p);
    case 9: return launch_decode_cfg<4, 1, 8, EPI>(p);
    case 10: return launch_decode_cfg<2, 4, 2, EPI>(p);
    case 11: return launch_decode_cfg<4, 4, 4, EPI>(p);
    case 12: return launch_decode_cfg<2, 1, 4, EPI>(p);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_decode_bf16(const DecodeArgs& p) {
  switch (p.epi) {
    case EPI_RMS: return launch_decode_epi<EPI_RMS>(p);
    case EPI_GLU: return launch_decode_epi<EPI_GLU>(p);
    case EPI_LN: return launch_decode_epi<EPI_LN>(p);
    case EPI_NONE: return launch_decode_epi<EPI_NONE>(p);
    case EPI_GLU_NOSCALE: return launch_decode_epi<EPI_GLU_NOSCALE>(p);
  }
  return hipErrorInvalidValue;
}

}  // namespace fn
