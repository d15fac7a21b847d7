// fp32 fused norm-then-project kernel (small fp32 problems; exact fp32 products,
// no reduced-precision matrix-core modes).
//
// A 256-thread workgroup owns a 64 x 64 output tile and walks K in steps of 64,
// staging the activation and weight tiles in LDS.  The threads that stage an
// activation row also accumulate its sum of squares (and sum, for LayerNorm)
// from the values they just loaded, alongside the products (Cor. 1); the
// deferred per-row scale (Prop. 2) is applied in the epilogue.  Thread (tx, ty)
// computes rows ty + 16 i and packed columns tx + 16 j, so columns j = 0, 1 (and
// 2, 3) are a GLU gate block and its up block.
#include "fn_device.h"
#include "fn_epilogue.h"
#include "fn_launch.h"

namespace fn {

template <int EPI, bool GS = false>
__global__ __launch_bounds__(256) void f32_kernel(const float* __restrict__ a, int M, int K, int lda,
                                                  const float* __restrict__ ws, int NP, int KP,
                                                  int ncols, float* __restrict__ y, int ldy,
                                                  EpiArgs ep) {
  constexpr int BM = 64, BN = 64, BK = 64, Q = BK / 16;  // Q quads of each operand per thread and step
  __shared__ float As[BK][BM + 4];
  __shared__ float Wsh[BK][BN];
  __shared__ float row_ss[BM], row_sa[BM];

  const int t = threadIdx.x;
  const int tx = t & 15, ty = t >> 4;
  const int m0 = blockIdx.y * BM, p0 = blockIdx.x * BN;

  const int lr = t >> 2, lkq = (t & 3) * 4;       // activation staging: row, k quads lkq + 16 q
  const int wk = t >> 4, wc = (t & 15) * 4;        // weight staging: k rows wk + 16 q, column quad
  const bool lr_ok = m0 + lr < M;
  const bool wc_ok = p0 + wc < NP;

  float acc[4][4] = {};
  float ss = 0.f, sa = 0.f;
  for (int k0 = 0; k0 < K; k0 += BK) {
    // All of the step's loads first (K is a multiple of 4: a quad is wholly inside
    // or outside; the packed weight has KP >= k0 + BK rows, zero past K).
    float4 av[Q], wv[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int k = k0 + lkq + 16 * q;
      av[q] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (lr_ok && k < K) av[q] = *reinterpret_cast<const float4*>(a + (int64_t)(m0 + lr) * lda + k);
      wv[q] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (wc_ok) wv[q] = *reinterpret_cast<const float4*>(ws + (int64_t)(k0 + wk + 16 * q) * NP + p0 + wc);
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      ss = fmaf(av[q].x, av[q].x, ss);
      ss = fmaf(av[q].y, av[q].y, ss);
      ss = fmaf(av[q].z, av[q].z, ss);
      ss = fmaf(av[q].w, av[q].w, ss);
      sa += (av[q].x + av[q].y) + (av[q].z + av[q].w);
      if constexpr (GS) {  // run-time g (unfolded W): a_k g_k in fp32
        const int k = k0 + lkq + 16 * q;
        if (lr_ok && k < K) {
          const float4 gv = *reinterpret_cast<const float4*>(ep.g_rt + k);
          av[q].x *= gv.x;
          av[q].y *= gv.y;
          av[q].z *= gv.z;
          av[q].w *= gv.w;
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      As[lkq + 16 * q + 0][lr] = av[q].x;
      As[lkq + 16 * q + 1][lr] = av[q].y;
      As[lkq + 16 * q + 2][lr] = av[q].z;
      As[lkq + 16 * q + 3][lr] = av[q].w;
      *reinterpret_cast<float4*>(&Wsh[wk + 16 * q][wc]) = wv[q];
    }
    __syncthreads();
#pragma unroll 16
    for (int kk = 0; kk < BK; ++kk) {
      float ar[4], wr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) ar[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) wr[j] = Wsh[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(ar[i], wr[j], acc[i][j]);
    }
  }
  ss += __shfl_xor(ss, 1);
  ss += __shfl_xor(ss, 2);
  sa += __shfl_xor(sa, 1);
  sa += __shfl_xor(sa, 2);
  if ((t & 3) == 0) {
    row_ss[lr] = ss;
    row_sa[lr] = sa;
  }
  __syncthreads();

  if constexpr (EPI == EPI_ROPE) {
    // Pair partners (column c ^ 1) sit in the neighbouring lane (tx ^ 1, same rows);
    // every lane takes part in the exchange before any guard.
    float part[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) part[i][j] = __shfl_xor(acc[i][j], 1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = ty + 16 * i;
      const int m = m0 + r;
      if (m >= M) continue;
      const RowStat st = row_stat_at<EPI>(row_ss[r], row_sa[r], ep, m, M);
      if (ep.inv_rms && blockIdx.x == 0 && tx == 0) ep.inv_rms[m] = st.s;
      float* yr = y + (int64_t)m * ldy;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c = p0 + tx + 16 * j;
        if (c >= ncols) continue;
        const float bv = ep.bias ? ep.bias[c] : 0.f, bw = ep.bias ? ep.bias[c ^ 1] : 0.f;
        yr[c] = rope1(c, acc[i][j], part[i][j], bv, bw, st, ep);
      }
    }
  } else if constexpr (EPI == EPI_HEADNORM) {
    // Heads of h | 64 columns: a lane holds columns tx + 16 j of its rows.  A head's
    // squares are summed over its lanes (xor 1 .. min(h, 16) / 2) and, for h > 16, over
    // the lane's h / 16 column groups of the head; pair partners sit in lane tx ^ 1.
    // Every lane takes part in the exchanges before any guard.
    const int h = ep.head_h;
    float hs[4][4], part[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v = acc[i][j] * acc[i][j];
        for (int off = 1; off < (h < 16 ? h : 16); off <<= 1) v += __shfl_xor(v, off);
        hs[i][j] = v;
      }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (h >= 32) {  // combine the column groups of one head: j and j ^ 1 (h = 32), all four (h = 64)
        const float s01 = hs[i][0] + hs[i][1], s23 = hs[i][2] + hs[i][3];
        hs[i][0] = hs[i][1] = h == 64 ? s01 + s23 : s01;
        hs[i][2] = hs[i][3] = h == 64 ? s01 + s23 : s23;
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + ty + 16 * i;
      const RowStat st = row_stat_at<EPI>(row_ss[ty + 16 * i], row_sa[ty + 16 * i], ep, m, M);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c = p0 + tx + 16 * j;
        const int ch = c & (h - 1);
        const bool is_q = c < ep.q_end, is_k = !is_q && c < ep.k_end;
        const float* w = is_q ? ep.hn_gq : is_k ? ep.hn_gk : ep.hn_gv;
        float v = acc[i][j];
        if (w && c < ncols) v *= rsqrtf(fmaf(hs[i][j], ep.head_inv_h, ep.hn_eps)) * w[ch];
        else v *= st.s;
        part[i][j] = v;  // the normalised value, also the partner of lane tx ^ 1
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) hs[i][j] = __shfl_xor(part[i][j], 1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = ty + 16 * i;
      const int m = m0 + r;
      if (m >= M) continue;
      const RowStat st = row_stat_at<EPI>(row_ss[r], row_sa[r], ep, m, M);
      if (ep.inv_rms && blockIdx.x == 0 && tx == 0) ep.inv_rms[m] = st.s;
      float* yr = y + (int64_t)m * ldy;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c = p0 + tx + 16 * j;
        if (c >= ncols) continue;
        const bool is_q = c < ep.q_end, is_k = !is_q && c < ep.k_end;
        float v = part[i][j];
        if ((is_q || is_k) && ep.rope_pos) {
          if ((unsigned)st.pos < (unsigned)ep.rope_P) {
            const int64_t off = (int64_t)st.pos * (ep.head_h >> 1) + ((c & (ep.head_h - 1)) >> 1);
            const float cs = ep.rope_cos[off], sn = ep.rope_sin[off], w2 = hs[i][j];
            v = (c & 1) ? w2 * sn + v * cs : v * cs - w2 * sn;
          } else {
            v = __builtin_nanf("");
          }
        }
        yr[c] = is_q ? v * ep.q_scale : v;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = ty + 16 * i;
      const int m = m0 + r;
      if (m >= M) continue;
      const RowStat st = row_stat_at<EPI>(row_ss[r], row_sa[r], ep, m, M);
      if constexpr (epi_exports_s(EPI)) {
        if (ep.inv_rms && blockIdx.x == 0 && tx == 0) ep.inv_rms[m] = st.s;
      }
      float* yr = y + (int64_t)m * ldy;
      if constexpr (epi_is_glu(EPI)) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int f = p0 / 2 + 16 * q + tx;
          if (f < ncols) yr[f] = epi_value<EPI>(acc[i][2 * q], acc[i][2 * q + 1], st, 0.f, 0.f);
        }
      } else {
        const float* vp = epi_vec<EPI>(ep);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int c = p0 + tx + 16 * j;
          if (c >= ncols) continue;
          const float vec = vp ? vp[c] : 0.f;
          const float cs = EPI == EPI_LN ? ep.colsum[c] : 0.f;
          yr[c] = epi_value<EPI>(acc[i][j], acc[i][j], st, vec, cs);
        }
      }
    }
  }
}

template <int EPI, bool GS = false>
static hipError_t launch_f32_epi(const F32Args& p) {
  dim3 grid((p.NP + 63) / 64, (p.M + 63) / 64);
  hipLaunchKernelGGL((f32_kernel<EPI, GS>), grid, dim3(256), 0, p.stream, p.a, p.M, p.K, p.lda, p.ws, p.NP,
                     p.KP, p.ncols, p.y, p.ldy, p.ep);
  return hipGetLastError();
}

hipError_t launch_f32(const F32Args& p) {
  if (p.gs) {  // run-time g: RMS kinds
    if (p.epi == EPI_RMS) return launch_f32_epi<EPI_RMS, true>(p);
    if (p.epi == EPI_GLU) return launch_f32_epi<EPI_GLU, true>(p);
    return hipErrorInvalidValue;
  }
  switch (p.epi) {
    case EPI_RMS: return launch_f32_epi<EPI_RMS>(p);
    case EPI_GLU: return launch_f32_epi<EPI_GLU>(p);
    case EPI_LN: return launch_f32_epi<EPI_LN>(p);
    case EPI_NONE: return launch_f32_epi<EPI_NONE>(p);
    case EPI_GLU_NOSCALE: return launch_f32_epi<EPI_GLU_NOSCALE>(p);
    case EPI_REGLU: return launch_f32_epi<EPI_REGLU>(p);
    case EPI_BILINEAR: return launch_f32_epi<EPI_BILINEAR>(p);
    case EPI_GLU_DEFER: return launch_f32_epi<EPI_GLU_DEFER>(p);
    case EPI_RELU_DEFER: return launch_f32_epi<EPI_RELU_DEFER>(p);
    case EPI_ROWSCALE: return launch_f32_epi<EPI_ROWSCALE>(p);
    case EPI_ROPE: return launch_f32_epi<EPI_ROPE>(p);
    case EPI_HEADNORM: return launch_f32_epi<EPI_HEADNORM>(p);
  }
  return hipErrorInvalidValue;
}

}  // namespace fn
