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
// GLU gate block and its up block.  RI = 1 with four k groups makes each thread's
// chain of products a quarter of K long for problems with few 64-row tiles; the
// few-row kernel below goes further for problems with few 16 x 64 tiles.
#include "fn_device.h"
#include "fn_epilogue.h"
#include "fn_launch.h"
#include "fn_tile.h"

#ifndef FEW_MIN_WG
#define FEW_MIN_WG 256
#endif

namespace fn {

// Epilogue of the fp32 kernels.  Thread (tx, ty) holds the accumulators of rows
// ty + 16 i (i < RI) and packed columns tx + 16 j (j < NJ) of the tile at (m0, p0), and
// rss / rsa the sums of its rows; first_tile marks the tile column that writes inv_rms.
template <int EPI, int RI, int NJ>
__device__ __forceinline__ void f32_epilogue(float (&acc)[RI][NJ], const StatT<EPI> (&rss)[RI],
                                             const StatT<EPI> (&rsa)[RI], int tx, int ty, int m0, int p0, int M,
                                             int ncols, float* __restrict__ y, int ldy, const EpiArgs& ep,
                                             bool first_tile) {
  static_assert(!epi_is_glu(EPI) || NJ % 2 == 0, "GLU: gate/up column block pairs");
  static_assert(EPI != EPI_HEADNORM || NJ == 4, "per-head norms: heads up to 64 wide in one tile");
  if constexpr (EPI == EPI_ROPE) {
    // Pair partners (column c ^ 1) sit in the neighbouring lane (tx ^ 1, same rows);
    // every lane takes part in the exchange before any guard.
    float part[RI][NJ];
#pragma unroll
    for (int i = 0; i < RI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) part[i][j] = __shfl_xor(acc[i][j], 1);
#pragma unroll
    for (int i = 0; i < RI; ++i) {
      const int r = ty + 16 * i;
      const int m = m0 + r;
      if (m >= M) continue;
      const RowStat st = row_stat_at<EPI>(rss[i], rsa[i], ep, m, M);
      if (ep.inv_rms && first_tile && tx == 0) ep.inv_rms[m] = st.s;
      float* yr = y + (int64_t)m * ldy;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
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
    float hs[RI][NJ], part[RI][NJ];
#pragma unroll
    for (int i = 0; i < RI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
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
      const RowStat st = row_stat_at<EPI>(rss[i], rsa[i], ep, m, M);
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
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
      for (int j = 0; j < NJ; ++j) hs[i][j] = __shfl_xor(part[i][j], 1);
#pragma unroll
    for (int i = 0; i < RI; ++i) {
      const int r = ty + 16 * i;
      const int m = m0 + r;
      if (m >= M) continue;
      const RowStat st = row_stat_at<EPI>(rss[i], rsa[i], ep, m, M);
      if (ep.inv_rms && first_tile && tx == 0) ep.inv_rms[m] = st.s;
      float* yr = y + (int64_t)m * ldy;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
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
      const RowStat st = row_stat_at<EPI>(rss[i], rsa[i], ep, m, M);
      if constexpr (epi_exports_s(EPI)) {
        if (ep.inv_rms && first_tile && tx == 0) ep.inv_rms[m] = st.s;
      }
      float* yr = y + (int64_t)m * ldy;
      if constexpr (epi_is_glu(EPI)) {
#pragma unroll
        for (int q = 0; q < NJ / 2; ++q) {
          const int f = p0 / 2 + 16 * q + tx;
          if (f < ncols) yr[f] = epi_value<EPI>(acc[i][2 * q], acc[i][2 * q + 1], st, 0.f, 0.f);
        }
      } else {
        const float* vp = epi_vec<EPI>(ep);
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
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

  using STE = StatT<EPI>;
  STE rss[RI], rsa[RI];
#pragma unroll
  for (int i = 0; i < RI; ++i) {
    rss[i] = row_ss[0][ty + 16 * i];
    rsa[i] = row_sa[0][ty + 16 * i];
  }
  f32_epilogue<EPI, RI, 4>(acc, rss, rsa, tx, ty, m0, p0, M, ncols, y, ldy, ep, blockIdx.x == 0);
}

// Few-row kernel.  A workgroup of 256 threads owns a 16-row tile of 4 CQ packed columns
// (CQ column quads) and splits K over KG = 64 / CQ groups of 4 CQ threads.  Group g takes
// the k quads g, g + KG, ...; its thread (rb, cb) keeps a 4 x 4 block of products (four
// rows of 4 rb.., column quad cb) and loads its operands straight from global memory as
// float4 (no LDS staging), PF quads ahead in registers.  The loads are range-checked
// buffer loads: a quad past K, a row past M or a column past NP reads zeros without
// touching memory, so no load sits behind a branch and the quads in flight stay in
// flight.  The thread also sums RS of its four rows (Cor. 1; LayerNorm on pivot-shifted
// values as in f32_kernel): its slots are rotated so that those rows are slots 0..RS-1.
// The groups' partials are added in LDS in a fixed order (deterministic).  CQ = 1, 2 or 4
// for the plain kinds (narrow tiles spread few rows over many workgroups: the 16-row
// tiny workload runs in 144 of them), 2 or 4 for a GLU (gate quads and the matching up
// quads, 16 columns apart in the packed layout), 16 for per-head norms (whole heads of
// up to 64 columns in one tile).
template <int EPI, bool GS, int CQ>
__global__ __launch_bounds__(256) void f32_few_rows_kernel(const float* __restrict__ a, int M, int K, int lda,
                                                           const float* __restrict__ ws, int NP, int ncols,
                                                           float* __restrict__ y, int ldy, EpiArgs ep) {
  constexpr bool kGlu = epi_is_glu(EPI);
  static_assert(EPI == EPI_HEADNORM ? CQ == 16 : kGlu ? (CQ == 2 || CQ == 4) : (CQ == 1 || CQ == 2 || CQ == 4),
                "tile width");
  constexpr int TG = 4 * CQ;                   // threads per k group
  constexpr int KG = 256 / TG;                 // k groups
  constexpr int NV = 4 * CQ;                   // values per tile row
  constexpr int RS = CQ >= 4 ? 1 : 4 / CQ;     // rows a thread sums
  constexpr int PF = 3;                        // k quads in flight per thread
  using ST = StatT<EPI>;
  __shared__ float red[KG][16][NV];
  __shared__ ST red_ss[KG][16], red_sa[KG][16];

  const int t = threadIdx.x;
  const int g = t / TG, u = t % TG;
  const int rb = u & 3, cb = u >> 2;
  // XCD-aware tile order: the workgroups of one XCD take neighbouring column tiles, so
  // the 128-byte weight lines that several narrow tiles share are fetched into one L2.
  int tm, tn;
  tile_of_block(blockIdx.x + gridDim.x * blockIdx.y, gridDim.x * gridDim.y, gridDim.y, gridDim.x, tm, tn);
  const int m0 = tm * 16;
  // Packed columns: plain tiles are 4 CQ consecutive columns; a GLU tile takes FQ = CQ / 2
  // gate quads of a 32-column block and the up quads 16 columns on.  p0e is the epilogue's
  // column origin (twice the first feature for a GLU).
  int colq, p0e;
  if constexpr (kGlu) {
    constexpr int FQ = CQ / 2, TPB = 4 / FQ;  // tiles per 32-column block
    const int blk = tn / TPB, sub = tn % TPB;
    const int fbase = 16 * blk + 4 * FQ * sub;
    colq = 32 * blk + 4 * FQ * sub + (cb < FQ ? 4 * cb : 16 + 4 * (cb - FQ));
    p0e = 2 * fbase;
  } else {
    p0e = tn * NV;
    colq = p0e + 4 * cb;
  }
  const int KQ = K >> 2;                                          // K is a multiple of 4
  const int rounds = ((KQ + KG - 1) / KG + PF - 1) / PF * PF;     // per group, whole batches of PF
  const int arows = M - m0 < 16 ? M - m0 : 16;
  // Extents end at the last valid element (lda >= K: a row past M starts beyond them).
  const __amdgpu_buffer_rsrc_t ars =
      make_rsrc(a + (int64_t)m0 * lda, (uint32_t)(((int64_t)(arows - 1) * lda + K) * 4));
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(ws, (uint32_t)((int64_t)K * NP * 4));
  const __amdgpu_buffer_rsrc_t grs = make_rsrc(GS ? ep.g_rt : nullptr, GS ? (uint32_t)K * 4 : 0u);
  const bool col_ok = colq < NP;
  // Slot i of the thread's four rows is row 4 rb + ((i + RS cb) & 3).
  int rrow[4];
  float piv[4];
  unsigned aoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    rrow[i] = 4 * rb + ((i + RS * cb) & 3);
    const int m = m0 + rrow[i];
    piv[i] = (EPI == EPI_LN && m < M) ? a[(int64_t)m * lda] : 0.f;
    aoff[i] = (unsigned)(rrow[i] * lda) * 4u;
  }
  const bool writes_stats = RS * cb < 4;

  // The load offsets pass through an empty asm so that the compiler keeps one load of a
  // selected offset (not two loads behind a branch).
  auto opaque = [](unsigned v) {
    asm volatile("" : "+v"(v));
    return v;
  };
  const unsigned woff = (unsigned)colq * 4u, wrow = (unsigned)NP * 4u;
  f32x4 A[PF][4], W[PF][4], G[PF];
  auto load = [&](int s, int r) {
    const int q = r * KG + g;
    const bool live = q < KQ, wlive = live & col_ok;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      A[s][i] = __builtin_bit_cast(f32x4, load_buf16(ars, opaque(live ? aoff[i] + (unsigned)q * 16u : kOobOffset)));
#pragma unroll
    for (int i = 0; i < 4; ++i)
      W[s][i] = __builtin_bit_cast(
          f32x4, load_buf16(wrs, opaque(wlive ? (unsigned)(4 * q + i) * wrow + woff : kOobOffset)));
    if constexpr (GS) G[s] = __builtin_bit_cast(f32x4, load_buf16(grs, opaque(live ? (unsigned)q * 16u : kOobOffset)));
  };

  float acc[4][4] = {};
  ST ss[RS] = {}, sa[RS] = {};
  auto compute = [&](int s, int r) {
    f32x4 av[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) av[i] = A[s][i];
    if constexpr (EPI == EPI_LN) {  // shift by the pivot; a quad past K stays zero
      const bool live = r * KG + g < KQ;
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = live ? av[i] - piv[i] : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int j = 0; j < RS; ++j) {
      if constexpr (EPI == EPI_LN) {  // fp64 sums: the squares of fp32 values are exact in fp64
        const double x = av[j].x, yv = av[j].y, z = av[j].z, w = av[j].w;
        ss[j] += (x * x + yv * yv) + (z * z + w * w);
        sa[j] += (x + yv) + (z + w);
      } else {
        ss[j] = fmaf(av[j].x, av[j].x, ss[j]);
        ss[j] = fmaf(av[j].y, av[j].y, ss[j]);
        ss[j] = fmaf(av[j].z, av[j].z, ss[j]);
        ss[j] = fmaf(av[j].w, av[j].w, ss[j]);
      }
    }
    if constexpr (GS) {  // run-time g (unfolded W): a_k g_k in fp32
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] *= G[s];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        acc[i][c] = fmaf(av[i].x, W[s][0][c], acc[i][c]);
        acc[i][c] = fmaf(av[i].y, W[s][1][c], acc[i][c]);
        acc[i][c] = fmaf(av[i].z, W[s][2][c], acc[i][c]);
        acc[i][c] = fmaf(av[i].w, W[s][3][c], acc[i][c]);
      }
  };

#pragma unroll
  for (int s = 0; s < PF; ++s) load(s, s);
  for (int r0 = 0; r0 < rounds; r0 += PF) {
#pragma unroll
    for (int s = 0; s < PF; ++s) {
      compute(s, r0 + s);
      load(s, r0 + s + PF);
    }
  }

#pragma unroll
  for (int i = 0; i < 4; ++i)
    *reinterpret_cast<f32x4*>(&red[g][rrow[i]][4 * cb]) = f32x4{acc[i][0], acc[i][1], acc[i][2], acc[i][3]};
  if (writes_stats) {
#pragma unroll
    for (int j = 0; j < RS; ++j) {
      red_ss[g][rrow[j]] = ss[j];
      red_sa[g][rrow[j]] = sa[j];
    }
  }
  __syncthreads();

  if constexpr (CQ == 16) {
    // 1024 values: thread (tx, ty) adds the KG partials of row ty, columns tx + 16 j.
    const int tx = t & 15, ty = t >> 4;
    float out[1][4];
    ST rss[1] = {ST(0)}, rsa[1] = {ST(0)};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float v = red[0][ty][tx + 16 * j];
#pragma unroll
      for (int k = 1; k < KG; ++k) v += red[k][ty][tx + 16 * j];
      out[0][j] = v;
    }
#pragma unroll
    for (int k = 0; k < KG; ++k) {
      rss[0] += red_ss[k][ty];
      rsa[0] += red_sa[k][ty];
    }
    f32_epilogue<EPI, 1, 4>(out, rss, rsa, tx, ty, m0, p0e, M, ncols, y, ldy, ep, tn == 0);
  } else {
    // 16 NV values, TPV = 4 / CQ threads each adding a contiguous run of KG / TPV
    // partials; then one thread per value adds the TPV runs in order.
    constexpr int V = 16 * NV, TPV = 256 / V, RUN = KG / TPV;
    __shared__ float part[TPV][V];
    __shared__ ST row_ss[16], row_sa[16];
    {
      const int v = t % V, pr = t / V;
      const int row = v / NV, col = v % NV;
      float sum = red[pr * RUN][row][col];
#pragma unroll 8
      for (int k = 1; k < RUN; ++k) sum += red[pr * RUN + k][row][col];
      part[pr][v] = sum;
    }
    if (t < 16) {
      ST s1 = ST(0), s2 = ST(0);
#pragma unroll 8
      for (int k = 0; k < KG; ++k) {
        s1 += red_ss[k][t];
        s2 += red_sa[k][t];
      }
      row_ss[t] = s1;
      row_sa[t] = s2;
    }
    __syncthreads();
    auto value = [&](int v) {
      float sum = part[0][v];
#pragma unroll
      for (int p = 1; p < TPV; ++p) sum += part[p][v];
      return sum;
    };
    if constexpr (kGlu) {
      constexpr int FW = NV / 2;  // features per tile row
      if (t >= 16 * FW) return;   // whole waves
      const int tx = t % FW, ty = t / FW;
      float out[1][2] = {{value(ty * NV + tx), value(ty * NV + FW + tx)}};
      const ST rss[1] = {row_ss[ty]}, rsa[1] = {row_sa[ty]};
      f32_epilogue<EPI, 1, 2>(out, rss, rsa, tx, ty, m0, p0e, M, ncols, y, ldy, ep, tn == 0);
    } else {
      if (t >= V) return;  // whole waves
      const int tx = t % NV, ty = t / NV;
      float out[1][1] = {{value(t)}};
      const ST rss[1] = {row_ss[ty]}, rsa[1] = {row_sa[ty]};
      f32_epilogue<EPI, 1, 1>(out, rss, rsa, tx, ty, m0, p0e, M, ncols, y, ldy, ep, tn == 0);
    }
  }
}

// Tile configurations (kF32CfgCount): 0 automatic, 1 = 64-row tiles with one k group,
// 2 = 16-row tiles of 64 columns with four k groups, 3 = the few-row kernel.  Automatic:
// the 64-row tiles when they make at least 128 workgroups, else the 16 x 64 tiles when
// they make at least 256 (their LDS staging reads each operand once per tile), else the
// few-row kernel (its narrow tiles spread few rows over many workgroups; its operands go
// through the vector memory path four times, which costs more than it gains once the
// 16 x 64 tiles fill the chip).

template <int EPI, bool GS = false>
static hipError_t launch_f32_epi(const F32Args& p) {
  int cfg = p.cfg;
  if (cfg == 0) {
    const int64_t nt = (p.NP + 63) / 64;
    cfg = (int64_t)((p.M + 63) / 64) * nt >= 128 ? 1 : (int64_t)((p.M + 15) / 16) * nt >= 256 ? 2 : 3;
  }
  if (cfg == 1) {
    dim3 grid((p.NP + 63) / 64, (p.M + 63) / 64);
    hipLaunchKernelGGL((f32_kernel<EPI, GS, 4, 1>), grid, dim3(256), 0, p.stream, p.a, p.M, p.K, p.lda, p.ws,
                       p.NP, p.KP, p.ncols, p.y, p.ldy, p.ep);
  } else if (cfg == 2) {
    dim3 grid((p.NP + 63) / 64, (p.M + 15) / 16);
    hipLaunchKernelGGL((f32_kernel<EPI, GS, 1, 4>), grid, dim3(1024), 0, p.stream, p.a, p.M, p.K, p.lda, p.ws,
                       p.NP, p.KP, p.ncols, p.y, p.ldy, p.ep);
  } else {
    // Column quads per tile: the widest of 4, 2, 1 that still makes FEW_MIN_WG workgroups.
    const int64_t mt = (p.M + 15) / 16;
    auto wgs = [&](int cq) { return (int64_t)((p.NP + 4 * cq - 1) / (4 * cq)) * mt; };
    const int cq = EPI == EPI_HEADNORM ? 16
                   : wgs(4) >= FEW_MIN_WG ? 4
                   : (wgs(2) >= FEW_MIN_WG || epi_is_glu(EPI)) ? 2
                                                                : 1;
    auto go = [&](auto kern, int cqv) {
      dim3 grid((p.NP + 4 * cqv - 1) / (4 * cqv), mt);
      hipLaunchKernelGGL(kern, grid, dim3(256), 0, p.stream, p.a, p.M, p.K, p.lda, p.ws, p.NP, p.ncols, p.y,
                         p.ldy, p.ep);
    };
    if constexpr (EPI == EPI_HEADNORM) {
      go(f32_few_rows_kernel<EPI, GS, 16>, 16);
    } else {
      if (cq == 4) go(f32_few_rows_kernel<EPI, GS, 4>, 4);
      else if (cq == 2) go(f32_few_rows_kernel<EPI, GS, 2>, 2);
      else if constexpr (!epi_is_glu(EPI)) go(f32_few_rows_kernel<EPI, GS, 1>, 1);
    }
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
