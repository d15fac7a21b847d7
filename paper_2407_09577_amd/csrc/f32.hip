// fp32 fused norm-then-project kernel (small fp32 problems; exact fp32 products,
// no reduced-precision matrix-core modes).
//
// A workgroup owns a BM x 64 output tile (BM = 16 RI rows) and KS groups of 256
// threads split K between them: group g takes the 64-deep k steps g, g + KS, ...,
// staging its activation and weight tiles in its own LDS buffers.  The threads
// that stage an activation row also accumulate its sum of squares (and sum, for
// LayerNorm) from the values they just loaded, alongside the products (Cor. 1).
// The groups' partial products and sums are added in LDS in a fixed order
// (deterministic; no split across workgroups), and group 0 applies the deferred
// per-row scale (Prop. 2) in the epilogue.  LayerNorm runs on activations shifted
// by a per-row pivot p (the row's first element): the sum exchange of Sec. 3.5 holds
// for any shift, sum_k (a_k - mu) W*_kn = sum_k (a_k - p) W*_kn - (mu - p) colsum_n,
// and with |mu - p| ~ sigma neither the fp32 products nor the statistics cancel when
// |mu| >> sigma (sums of the shifted values in fp64).  Thread (tx, ty) of group 0 finishes
// rows ty + 16 i and packed columns tx + 16 j, so columns j = 0, 1 (and 2, 3) are a
// GLU gate block and its up block.  Few-row problems (the tiny workload has 16
// rows) take RI = 1 with four k groups, so each thread's chain of products is a
// quarter of K long instead of 4 x 4 outputs over all of K.
#include "fn_device.h"
#include "fn_epilogue.h"
#include "fn_launch.h"

namespace fn {

template <int EPI, bool GS, int RI, int KS>
__global__ __launch_bounds__(256 * KS) void f32_kernel(const float* __restrict__ a, int M, int K, int lda,
                                                       const float* __restrict__ ws, int NP, int KP,
                                                       int ncols, float* __restrict__ y, int ldy,
                                                       EpiArgs ep) {
  constexpr int BM = 16 * RI, BN = 64, BK = 64;
  constexpr int TPR = 256 / BM;            // staging threads per activation row
  constexpr int QA = BK / (4 * TPR);       // activation quads per staging thread and step (= RI)
  constexpr int QW = BK * BN / (4 * 256);  // weight quads per thread and step
  using ST = StatT<EPI>;
  struct Stage {
    float As[BK][BM + 4];
    float Wsh[BK][BN];
  };
  __shared__ Stage stg[KS];
  __shared__ ST row_ss[KS][BM], row_sa[KS][BM];

  const int grp = threadIdx.x >> 8;  // k group (wave-uniform)
  const int t = threadIdx.x & 255;
  const int tx = t & 15, ty = t >> 4;
  const int m0 = blockIdx.y * BM, p0 = blockIdx.x * BN;

  const int lr = t / TPR, lkq = (t % TPR) * 4;  // activation staging: row lr, k quads lkq + 4 TPR q
  const int wk = t >> 4, wc = (t & 15) * 4;      // weight staging: k rows wk + 16 q, column quad
  const bool lr_ok = m0 + lr < M;
  const bool wc_ok = p0 + wc < NP;
  float(&As)[BK][BM + 4] = stg[grp].As;
  float(&Wsh)[BK][BN] = stg[grp].Wsh;
  // LayerNorm pivot of the staged row (rows past M stage zeros).
  const float piv = (EPI == EPI_LN && lr_ok) ? a[(int64_t)(m0 + lr) * lda] : 0.0f;

  float acc[RI][4] = {};
  ST ss = ST(0), sa = ST(0);
  // Every group runs the same number of rounds (the barriers need it); a group whose
  // step lies past K stages zeros and skips the products.
  const int rounds = ((K + BK - 1) / BK + KS - 1) / KS;
  for (int rd = 0; rd < rounds; ++rd) {
    const int k0 = (rd * KS + grp) * BK;
    const bool live = k0 < K;  // uniform in the group
    // All of the step's loads first (K is a multiple of 4: a quad is wholly inside
    // or outside; the packed weight has KP >= k0 + BK rows when k0 < K, zero past K).
    float4 av[QA], wv[QW];
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      const int k = k0 + lkq + 4 * TPR * q;
      av[q] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (lr_ok && k < K) {
        av[q] = *reinterpret_cast<const float4*>(a + (int64_t)(m0 + lr) * lda + k);
        if constexpr (EPI == EPI_LN) {
          av[q].x -= piv;
          av[q].y -= piv;
          av[q].z -= piv;
          av[q].w -= piv;
        }
      }
    }
#pragma unroll
    for (int q = 0; q < QW; ++q) {
      wv[q] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (wc_ok && live) wv[q] = *reinterpret_cast<const float4*>(ws + (int64_t)(k0 + wk + 16 * q) * NP + p0 + wc);
    }
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      if constexpr (EPI == EPI_LN) {  // fp64 sums: the squares of fp32 values are exact in fp64
        const double x = av[q].x, yv = av[q].y, z = av[q].z, w = av[q].w;
        ss += (x * x + yv * yv) + (z * z + w * w);
        sa += (x + yv) + (z + w);
      } else {
        ss = fmaf(av[q].x, av[q].x, ss);
        ss = fmaf(av[q].y, av[q].y, ss);
        ss = fmaf(av[q].z, av[q].z, ss);
        ss = fmaf(av[q].w, av[q].w, ss);
      }
      if constexpr (GS) {  // run-time g (unfolded W): a_k g_k in fp32
        const int k = k0 + lkq + 4 * TPR * q;
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
    for (int q = 0; q < QA; ++q) {
      const int kq = lkq + 4 * TPR * q;
      As[kq + 0][lr] = av[q].x;
      As[kq + 1][lr] = av[q].y;
      As[kq + 2][lr] = av[q].z;
      As[kq + 3][lr] = av[q].w;
    }
#pragma unroll
    for (int q = 0; q < QW; ++q) *reinterpret_cast<float4*>(&Wsh[wk + 16 * q][wc]) = wv[q];
    __syncthreads();
    if (live) {
#pragma unroll 16
      for (int kk = 0; kk < BK; ++kk) {
        float ar[RI], wr[4];
#pragma unroll
        for (int i = 0; i < RI; ++i) ar[i] = As[kk][ty + 16 * i];
#pragma unroll
        for (int j = 0; j < 4; ++j) wr[j] = Wsh[kk][tx + 16 * j];
#pragma unroll
        for (int i = 0; i < RI; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(ar[i], wr[j], acc[i][j]);
      }
    }
  }
  // A row's staging threads are TPR consecutive lanes of one wave.
#pragma unroll
  for (int off = 1; off < TPR; off <<= 1) {
    ss += __shfl_xor(ss, off);
    if constexpr (EPI == EPI_LN) sa += __shfl_xor(sa, off);
  }
  if (t % TPR == 0) {
    row_ss[grp][lr] = ss;
    row_sa[grp][lr] = sa;
  }
  __syncthreads();  // every group's products done: the stage buffers are free
  if constexpr (KS > 1) {
    // Groups 1.. hand their partial products to group 0, which adds them in group
    // order; thread t < BM of group 0 adds its row's sums the same way.
    static_assert((KS - 1) * RI * 4 * 256 * sizeof(float) <= sizeof(stg), "reduction buffer");
    float* red = reinterpret_cast<float*>(&stg[0]);
    if (grp > 0) {
#pragma unroll
      for (int i = 0; i < RI; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) red[(((grp - 1) * RI + i) * 4 + j) * 256 + t] = acc[i][j];
    } else if (t < BM) {
      ST s1 = row_ss[0][t], s2 = row_sa[0][t];
#pragma unroll
      for (int g = 1; g < KS; ++g) {
        s1 += row_ss[g][t];
        s2 += row_sa[g][t];
      }
      row_ss[0][t] = s1;
      row_sa[0][t] = s2;
    }
    __syncthreads();
    if (grp > 0) return;
#pragma unroll
    for (int g = 1; g < KS; ++g)
#pragma unroll
      for (int i = 0; i < RI; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += red[(((g - 1) * RI + i) * 4 + j) * 256 + t];
  }

  if constexpr (EPI == EPI_ROPE) {
    // Pair partners (column c ^ 1) sit in the neighbouring lane (tx ^ 1, same rows);
    // every lane takes part in the exchange before any guard.
    float part[RI][4];
#pragma unroll
    for (int i = 0; i < RI; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) part[i][j] = __shfl_xor(acc[i][j], 1);
#pragma unroll
    for (int i = 0; i < RI; ++i) {
      const int r = ty + 16 * i;
      const int m = m0 + r;
      if (m >= M) continue;
      const RowStat st = row_stat_at<EPI>(row_ss[0][r], row_sa[0][r], ep, m, M);
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
    float hs[RI][4], part[RI][4];
#pragma unroll
    for (int i = 0; i < RI; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v = acc[i][j] * acc[i][j];
        for (int off = 1; off < (h < 16 ? h : 16); off <<= 1) v += __shfl_xor(v, off);
        hs[i][j] = v;
      }
#pragma unroll
    for (int i = 0; i < RI; ++i) {
      if (h >= 32) {  // combine the column groups of one head: j and j ^ 1 (h = 32), all four (h = 64)
        const float s01 = hs[i][0] + hs[i][1], s23 = hs[i][2] + hs[i][3];
        hs[i][0] = hs[i][1] = h == 64 ? s01 + s23 : s01;
        hs[i][2] = hs[i][3] = h == 64 ? s01 + s23 : s23;
      }
    }
#pragma unroll
    for (int i = 0; i < RI; ++i) {
      const int m = m0 + ty + 16 * i;
      const RowStat st = row_stat_at<EPI>(row_ss[0][ty + 16 * i], row_sa[0][ty + 16 * i], ep, m, M);
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
    for (int i = 0; i < RI; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) hs[i][j] = __shfl_xor(part[i][j], 1);
#pragma unroll
    for (int i = 0; i < RI; ++i) {
      const int r = ty + 16 * i;
      const int m = m0 + r;
      if (m >= M) continue;
      const RowStat st = row_stat_at<EPI>(row_ss[0][r], row_sa[0][r], ep, m, M);
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
    for (int i = 0; i < RI; ++i) {
      const int r = ty + 16 * i;
      const int m = m0 + r;
      if (m >= M) continue;
      const RowStat st = row_stat_at<EPI>(row_ss[0][r], row_sa[0][r], ep, m, M);
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

// Tile configurations (kF32CfgCount): 0 automatic, 1 = 64-row tiles with one k group,
// 2 = 16-row tiles with four k groups.  Automatic: the 64-row tiles when they make at
// least 128 workgroups, else the short tiles with four k groups (latency: up to four
// times more workgroups for few rows, chains a quarter of K long).

template <int EPI, bool GS = false>
static hipError_t launch_f32_epi(const F32Args& p) {
  int cfg = p.cfg;
  if (cfg == 0) cfg = ((int64_t)(p.M + 63) / 64) * ((p.NP + 63) / 64) >= 128 ? 1 : 2;
  if (cfg == 1) {
    dim3 grid((p.NP + 63) / 64, (p.M + 63) / 64);
    hipLaunchKernelGGL((f32_kernel<EPI, GS, 4, 1>), grid, dim3(256), 0, p.stream, p.a, p.M, p.K, p.lda, p.ws,
                       p.NP, p.KP, p.ncols, p.y, p.ldy, p.ep);
  } else {
    dim3 grid((p.NP + 63) / 64, (p.M + 15) / 16);
    hipLaunchKernelGGL((f32_kernel<EPI, GS, 1, 4>), grid, dim3(1024), 0, p.stream, p.a, p.M, p.K, p.lda, p.ws,
                       p.NP, p.KP, p.ncols, p.y, p.ldy, p.ep);
  }
  return hipGetLastError();
}

hipError_t launch_f32(const F32Args& p) {
  if (p.cfg < 0 || p.cfg >= kF32CfgCount) return hipErrorInvalidValue;
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
