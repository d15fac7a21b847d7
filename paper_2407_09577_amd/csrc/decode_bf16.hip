// Few-row (decode) fused norm-then-project kernel for gfx950.
//
// With M <= 16 activation rows the product is bound by streaming W* from HBM
// once (Sec. 6 and App. "End-to-end validation": decode is memory-bound and
// wants its own kernel instead of a padded prefill tile).  A workgroup owns NCB
// packed column blocks of 16 columns (for a GLU, whole gate/up block pairs) and
// its KSPLIT waves split K: wave w takes the 32-row k blocks w, w + KSPLIT, ...
// (or, with CW column waves, each of CW waves owns NCB blocks over all of K and
// the waves share the activation fragments through LDS).
// Each weight fragment is one 16-byte load per lane (non-temporal: it is read
// exactly once), fed directly to a 16x16x32 bf16 matrix-core op together with
// the matching 16-row activation fragment (rows >= M read as zero), so the
// arithmetic costs nothing next to the stream.  Loads go in sets of U k blocks,
// optionally double buffered so the next set is in flight while the current
// one is consumed.  The squares of the activation fragments are summed on the
// way (Cor. 1); with several waves the partial products and sums are combined
// in LDS in a fixed order (deterministic), and the lanes holding a row's
// totals apply the deferred scale and the epilogue.
#include <type_traits>

#include "fn_device.h"
#include "fn_epilogue.h"
#include "fn_launch.h"

namespace fn {

template <int NCB, int KSPLIT, int U, bool DB, int CPOL, int EPI, bool GS = false, int CW = 1>
__global__ __launch_bounds__(KSPLIT * CW * 64) void decode_bf16_kernel(
    const __bf16* __restrict__ a, int M, int K, int lda, const __bf16* __restrict__ ws, int NP,
    int KP, int ncols, __bf16* __restrict__ y, int ldy, EpiArgs ep) {
  constexpr bool kSS = epi_needs_ss(EPI);
  constexpr bool kSA = EPI == EPI_LN;
  constexpr int NOUT = epi_is_glu(EPI) ? NCB / 2 : NCB;  // output blocks per workgroup
  static_assert(!epi_is_glu(EPI) || NCB % 2 == 0, "GLU needs gate/up block pairs");
  // CW > 1: the workgroup's CW waves own NCB column blocks each over all of K and share
  // the activation fragments: wave w loads fragments w, w + CW, ... of each set of U k
  // blocks into LDS, and every wave reads all U of them (the activation is read from
  // L2 by the workgroup once, not CW times).
  static_assert(CW == 1 || (KSPLIT == 1 && DB && !GS && U % CW == 0), "shared activations: column waves");
  constexpr int UA = U / CW;  // activation fragments each wave loads per set

  // Per-wave partials for the cross-wave combine (unused with one wave).
  __shared__ f32x4 red[KSPLIT > 1 ? KSPLIT : 1][NCB][64];
  using ST = StatT<EPI>;
  __shared__ ST red_ss[KSPLIT > 1 ? KSPLIT : 1][16];
  __shared__ ST red_sa[KSPLIT > 1 ? KSPLIT : 1][16];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int cb0 = (blockIdx.x * CW + (CW > 1 ? wave : 0)) * NCB;
  const int KB = KP / kKB;

  const __amdgpu_buffer_rsrc_t rs_a = make_rsrc(a, (uint32_t)(((int64_t)(M - 1) * lda + K) * 2));
  // Column blocks past the packed width (last workgroup only) read the next k
  // block's fragments, or zeros past the end; their outputs are never stored.
  const int npb = NP / 16;
  // (CW > 1: a wave wholly past the packed width gets an empty range and reads zeros.)
  const int64_t w_extent = ((int64_t)KB * npb - cb0) * kFragBytes;
  const __amdgpu_buffer_rsrc_t rs_w =
      make_rsrc(ws + (int64_t)cb0 * (kFragBytes / 2), (uint32_t)(w_extent > 0 ? w_extent : 0));

  const int lrow = lane & 15;
  const int lk = (lane >> 4) * 8;
  // Activation fragments are loaded row-contiguously: lane i takes row i / 4, k chunk
  // i % 4, so each group of four lanes reads one 64-byte row segment (one cache line),
  // and are then put into the matrix-core order (lane L: row L % 16, chunk L / 16) by
  // a round trip through this wave's own 1 KiB LDS slot.  Loaded directly in the
  // matrix-core order, four lanes touch four rows, and at M = 16 the address unit
  // work of those loads slowed the weight stream by ~6% (measured on MI355X).
  const int t_row = lane >> 2, t_k = (lane & 3) * 8;
  const bool row_ok = t_row < M;
  const unsigned a_row_off = (unsigned)(t_row * lda * 2);
  __shared__ u32x4 a_slot[CW > 1 ? 2 : KSPLIT][U][64];
  const unsigned a_rd = (unsigned)(4 * lrow + (lane >> 4));  // unit of (row lrow, chunk lane / 16)

  f32x4 acc[NCB];
#pragma unroll
  for (int c = 0; c < NCB; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  ST ss = ST(0), sa = ST(0);

  // One set = U k blocks of this wave (kb, kb + KSPLIT, ...): U activation
  // fragments and U x NCB weight fragments, one 16-byte load per lane each.
  // Blocks past K read as zeros.
  // GS: run-time g (unfolded W): the 8 values of g at this lane's k chunk come
  // with each activation fragment (zeros past K).
  const __amdgpu_buffer_rsrc_t rs_g = make_rsrc(ep.g_rt, GS ? (uint32_t)K * 4u : 0u);
  f32x4 gv0[GS ? U : 1][2], gv1[GS ? U : 1][2];
  auto load_set = [&](int kb0, u32x4 (&af)[U], u32x4 (&wf)[U][NCB], f32x4 (&gv)[GS ? U : 1][2])
                      __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb0 + KSPLIT * u;
      const int k = kb * kKB + lk;
      const int kt = kb * kKB + t_k;
      const bool kb_ok = kb < KB;
      af[u] = load_buf16(rs_a, (kb_ok && row_ok && kt < K) ? a_row_off + (unsigned)kt * 2 : kOobOffset);
      if constexpr (GS) {
        // k >= K lies past the range of rs_g (K * 4 bytes) and reads zeros; the
        // offsets stay unconditional, which keeps the loop free of branches.
        gv[u][0] = __builtin_bit_cast(f32x4, load_buf16(rs_g, (unsigned)k * 4));
        gv[u][1] = __builtin_bit_cast(f32x4, load_buf16(rs_g, (unsigned)k * 4 + 16));
      }
#pragma unroll
      for (int c = 0; c < NCB; ++c)
        wf[u][c] = load_buf16<CPOL>(rs_w, kb_ok ? (unsigned)((kb * npb + c) * kFragBytes + lane * 16) : kOobOffset);
    }
  };
  auto compute_set = [&](const u32x4 (&af)[U], const u32x4 (&wf)[U][NCB], const f32x4 (&gv)[GS ? U : 1][2])
                         __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) a_slot[wave][u][lane] = af[u];  // row-contiguous units
#pragma unroll
    for (int u = 0; u < U; ++u) {
      bf16x8 av = __builtin_bit_cast(bf16x8, a_slot[wave][u][a_rd]);  // matrix-core order
      if constexpr (kSA) {  // LayerNorm: the fragment's fp32 partials, added in fp64
        ss += (double)sumsq8(av, 0.0f);
        sa += (double)sum8(av, 0.0f);
      } else if constexpr (kSS) {
        ss = sumsq8(av, ss);
      }
      if constexpr (GS) {  // a_k g_k, rounded once to bf16
        float o[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[e] = (float)av[e] * gv[u][0][e];
          o[4 + e] = (float)av[4 + e] * gv[u][1][e];
        }
        const u32x2 lo = pack4_bf16(*reinterpret_cast<const float(*)[4]>(o));
        const u32x2 hi = pack4_bf16(*reinterpret_cast<const float(*)[4]>(o + 4));
        av = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
      }
#pragma unroll
      for (int c = 0; c < NCB; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf[u][c]), av,
                                                          acc[c], 0, 0, 0);
    }
  };

  // CW > 1: activation fragments through a double-buffered LDS stage, loaded one set
  // ahead of the weights.  Set s: its weights W(s) were issued during set s-1 and its
  // activations act(s) during set s-2 and written to LDS slot s % 2 during set s-1.
  // Waiting for W(s) therefore also covers act(s+1) (issued before it; loads return in
  // order), so the activations' L2 latency never holds up the weight stream.
  // A set's activations are 16 rows x U 64-byte k-block segments, i.e. U KiB: load
  // ι = i CW + wave (i < UA) takes units 64 ι .. 64 ι + 63 of them in row-major order, so
  // each load covers whole 4 U x 16-byte row runs (full 128-byte lines for U >= 2, half
  // the L2 requests of one 16-row fragment per load), and the unit lands in LDS at
  // k block u, row r, chunk c, where the matrix-core order reads it.
  auto act_unit = [&](int i, int& r, int& u, int& c) __attribute__((always_inline)) {
    const int n = (i * CW + wave) * 64 + lane;
    r = n / (4 * U);
    u = (n % (4 * U)) / 4;
    c = n % 4;
  };
  auto load_act = [&](int kb0, u32x4 (&af)[UA]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      int r, u, c;
      act_unit(i, r, u, c);
      const int kb = kb0 + u;
      const int kt = kb * kKB + c * 8;
      af[i] = load_buf16(rs_a, (kb < KB && r < M && kt < K) ? (unsigned)(r * lda + kt) * 2 : kOobOffset);
    }
  };
  auto load_w = [&](int kb0, u32x4 (&wf)[U][NCB]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb0 + u;
#pragma unroll
      for (int c = 0; c < NCB; ++c)
        wf[u][c] = load_buf16<CPOL>(rs_w, kb < KB ? (unsigned)((kb * npb + c) * kFragBytes + lane * 16) : kOobOffset);
    }
  };
  auto put_act = [&](int buf, const u32x4 (&af)[UA]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      int r, u, c;
      act_unit(i, r, u, c);
      a_slot[buf][u][4 * r + c] = af[i];
    }
  };
  auto compute_shared = [&](int buf, const u32x4 (&wf)[U][NCB]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bf16x8 av = __builtin_bit_cast(bf16x8, a_slot[buf][u][a_rd]);  // matrix-core order
      if constexpr (kSA) {
        ss += (double)sumsq8(av, 0.0f);
        sa += (double)sum8(av, 0.0f);
      } else if constexpr (kSS) {
        ss = sumsq8(av, ss);
      }
#pragma unroll
      for (int c = 0; c < NCB; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf[u][c]), av, acc[c], 0, 0, 0);
    }
  };

  constexpr int STEP = KSPLIT * U;  // k blocks per set across the workgroup
  if constexpr (CW > 1) {
    // Every wave of the workgroup walks the same sets (one barrier per set).  The
    // barrier of set s orders the slot writes of set s-1 (act(s)) before this set's
    // reads, and every wave's reads of slot (s+1) % 2 during set s-1 before its
    // rewrite with act(s+1) here.
    u32x4 a0[UA], a1[UA], w0[U][NCB], w1[U][NCB];
    load_act(0, a0);
    load_act(STEP, a1);
    load_w(0, w0);
    put_act(0, a0);
    for (int kb0 = 0; kb0 < KB; kb0 += 2 * STEP) {
      load_act(kb0 + 2 * STEP, a0);
      load_w(kb0 + STEP, w1);
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      put_act(1, a1);
      compute_shared(0, w0);
      __builtin_amdgcn_sched_barrier(0);
      load_act(kb0 + 3 * STEP, a1);
      load_w(kb0 + 2 * STEP, w0);
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      put_act(0, a0);
      compute_shared(1, w1);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else if constexpr (DB) {
    // Double-buffered register sets: the next set's loads are issued before the
    // current set is consumed, so every wave keeps a full set in flight.  Sets
    // past K are issued as zero-returning loads, which keeps the loop uniform.
    u32x4 af0[U], wf0[U][NCB], af1[U], wf1[U][NCB];
    load_set(wave, af0, wf0, gv0);
    for (int kb0 = wave; kb0 < KB; kb0 += 2 * STEP) {
      load_set(kb0 + STEP, af1, wf1, gv1);
      __builtin_amdgcn_sched_barrier(0);
      compute_set(af0, wf0, gv0);
      __builtin_amdgcn_sched_barrier(0);
      load_set(kb0 + 2 * STEP, af0, wf0, gv0);
      __builtin_amdgcn_sched_barrier(0);
      compute_set(af1, wf1, gv1);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
    for (int kb0 = wave; kb0 < KB; kb0 += STEP) {
      u32x4 af[U], wf[U][NCB];
      load_set(kb0, af, wf, gv0);
      compute_set(af, wf, gv0);
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
  // Combine the waves' partial products and row sums (a fixed order).  With a
  // single wave per workgroup every lane already holds its row's totals.
  if constexpr (KSPLIT > 1) {
#pragma unroll
    for (int c = 0; c < NCB; ++c) red[wave][c][lane] = acc[c];
    if (lane < 16) {
      red_ss[wave][lane] = ss;
      red_sa[wave][lane] = sa;
    }
    __syncthreads();
  }
  auto total = [&](int c) __attribute__((always_inline)) {
    if constexpr (KSPLIT == 1) return acc[c];
    f32x4 v = red[0][c][lane];
#pragma unroll
    for (int w = 1; w < KSPLIT; ++w) v += red[w][c][lane];
    return v;
  };

  const int m = lrow;
  if (m >= M) return;
  ST ss_t = ss, sa_t = sa;
  if constexpr (KSPLIT > 1) {
    ss_t = sa_t = ST(0);
#pragma unroll
    for (int w = 0; w < KSPLIT; ++w) {
      ss_t += red_ss[w][m];
      sa_t += red_sa[w][m];
    }
  }
  const RowStat st = row_stat_at<EPI>(ss_t, sa_t, ep, m, M);
  if constexpr (epi_exports_s(EPI)) {
    if (ep.inv_rms && blockIdx.x == 0 && wave == 0 && lane < 16) ep.inv_rms[m] = st.s;
  }
  const int n_lane = (lane >> 4) * 4;
  auto epilogue = [&](auto vec_tag) __attribute__((always_inline)) {
    constexpr bool VEC = decltype(vec_tag)::value;
    // With one wave per workgroup the output blocks are compile-time indices (the
    // accumulators stay in registers); with several, the totals come from LDS.
#pragma unroll
    for (int oo = 0; oo < NOUT; oo += KSPLIT) {
      const int o = oo + (KSPLIT > 1 ? wave : 0);
      if (KSPLIT > 1 && o >= NOUT) break;
      if constexpr (epi_is_glu(EPI)) {
        const f32x4 g = total(2 * o), u = total(2 * o + 1);
        const int fb = (cb0 / 2 + o) * 16;
        if (fb + 16 <= ncols)
          store4_bf16_full<EPI, VEC>(y, ldy, m, fb + n_lane, g, u, st, ep);
        else
          store4_bf16_edge<EPI, VEC>(y, ldy, M, ncols, m, fb + n_lane, g, u, st, ep);
      } else {
        const f32x4 v = total(o);
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

template <int NCB, int KSPLIT, int U, int EPI, bool DB = false, int CPOL = 0, bool GS = false, int CW = 1>
static hipError_t launch_decode_cfg(const DecodeArgs& p) {
  const int nblocks = (p.NP / 16 + NCB * CW - 1) / (NCB * CW);
  hipLaunchKernelGGL((decode_bf16_kernel<NCB, KSPLIT, U, DB, CPOL, EPI, GS, CW>), dim3(nblocks),
                     dim3(KSPLIT * CW * 64), 0, p.stream, p.a, p.M, p.K, p.lda, p.ws, p.NP, p.KP, p.ncols, p.y,
                     p.ldy, p.ep);
  return hipGetLastError();
}

// Automatic work split, from the number of packed 16-column blocks (npb) and
// the row count.  Measured on MI355X (bf16, K = 576 .. 8192): about 600-1000
// waves in flight over the chip stream the weights fastest, so narrow outputs
// split K over more waves of one workgroup (combined in LDS in a fixed order)
// instead of leaving most compute units idle:
//   npb >= 1088          4 column waves x 2 blocks each, 4 per set, sharing the
//                        activation fragments (1-2% faster than one wave per
//                        workgroup at M = 1..16 on the Llama-7B SwiGLU shape)
//   544 <= npb < 1088    4 blocks x 4 waves x 1
//   272 <= npb < 544     2 blocks x 4 waves x 2
//   npb < 272            2 blocks x 8 waves x 1
// With run-time g the wide case takes 8 x 2 x 2 (M <= 8) or 2 x 1 x 4 (the g
// loads want four blocks per set).
template <int EPI, bool GS>
static hipError_t launch_decode_auto(const DecodeArgs& p) {
  const int npb = p.NP / 16;
  if (npb >= 1088) {
    if constexpr (GS) {
      if (p.M <= 8) return launch_decode_cfg<8, 2, 2, EPI, true, kCachePolicyNT, GS>(p);
      return launch_decode_cfg<2, 1, 4, EPI, true, kCachePolicyNT, GS>(p);
    } else {
      return launch_decode_cfg<2, 1, 4, EPI, true, kCachePolicyNT, false, 4>(p);
    }
  }
  if (npb >= 544) return launch_decode_cfg<4, 4, 1, EPI, true, kCachePolicyNT, GS>(p);
  if (npb >= 272) return launch_decode_cfg<2, 4, 2, EPI, true, kCachePolicyNT, GS>(p);
  return launch_decode_cfg<2, 8, 1, EPI, true, kCachePolicyNT, GS>(p);
}

template <int EPI>
static hipError_t launch_decode_epi(const DecodeArgs& p) {
  if (p.gs) {  // run-time g: RMS kinds, the automatic configuration only
    if constexpr (EPI == EPI_RMS || EPI == EPI_GLU)
      if (p.cfg == 0) return launch_decode_auto<EPI, true>(p);
    return hipErrorInvalidValue;
  }
  if (p.cfg == 0) return launch_decode_auto<EPI, false>(p);
  if constexpr (EPI >= EPI_REGLU) {
    // The epilogue family beyond the core kinds: the automatic configuration only.
    return hipErrorInvalidValue;
  } else {
  // Forced configurations (NCB column blocks per workgroup, KSPLIT waves, U k
  // blocks per load set, double-buffered sets, non-temporal weight loads), for
  // tuning and tests.
  switch (p.cfg) {
    case 1: return launch_decode_cfg<2, 1, 2, EPI, true, kCachePolicyNT>(p);
    case 2: return launch_decode_cfg<2, 1, 4, EPI, true, kCachePolicyNT>(p);
    case 3: return launch_decode_cfg<2, 2, 2, EPI, true, kCachePolicyNT>(p);
    case 4: return launch_decode_cfg<2, 2, 4, EPI, true, kCachePolicyNT>(p);
    case 5: return launch_decode_cfg<2, 1, 8, EPI, true, kCachePolicyNT>(p);
    case 6: return launch_decode_cfg<4, 1, 2, EPI, true, kCachePolicyNT>(p);
    case 7: return launch_decode_cfg<4, 1, 4, EPI, true, kCachePolicyNT>(p);
    case 8: return launch_decode_cfg<2, 2, 8, EPI, false, kCachePolicyNT>(p);
    case 9: return launch_decode_cfg<2, 2, 8, EPI>(p);
    case 10: return launch_decode_cfg<2, 4, 4, EPI, true, kCachePolicyNT>(p);
    case 11: return launch_decode_cfg<8, 1, 2, EPI, true, kCachePolicyNT>(p);
    case 12: return launch_decode_cfg<2, 1, 1, EPI, true, kCachePolicyNT>(p);
    case 13: return launch_decode_cfg<2, 4, 2, EPI, true, kCachePolicyNT>(p);
    case 14: return launch_decode_cfg<8, 4, 1, EPI, true, kCachePolicyNT>(p);
    case 15: return launch_decode_cfg<8, 2, 2, EPI, true, kCachePolicyNT>(p);
    case 16: return launch_decode_cfg<2, 8, 2, EPI, true, kCachePolicyNT>(p);
    case 17: return launch_decode_cfg<4, 4, 1, EPI, true, kCachePolicyNT>(p);
    case 18: return launch_decode_cfg<2, 8, 1, EPI, true, kCachePolicyNT>(p);
    case 19: return launch_decode_cfg<2, 1, 4, EPI, true, kCachePolicyNT, false, 4>(p);
    case 20: return launch_decode_cfg<2, 1, 2, EPI, true, kCachePolicyNT, false, 2>(p);
    case 21: return launch_decode_cfg<2, 1, 4, EPI, true, kCachePolicyNT, false, 2>(p);
    case 22: return launch_decode_cfg<4, 1, 4, EPI, true, kCachePolicyNT, false, 2>(p);
    case 23: return launch_decode_cfg<2, 1, 4, EPI, true, 0, false, 4>(p);
  }
  return hipErrorInvalidValue;
  }
}

hipError_t launch_decode_bf16(const DecodeArgs& p) {
  switch (p.epi) {
    case EPI_RMS: return launch_decode_epi<EPI_RMS>(p);
    case EPI_GLU: return launch_decode_epi<EPI_GLU>(p);
    case EPI_LN: return launch_decode_epi<EPI_LN>(p);
    case EPI_NONE: return launch_decode_epi<EPI_NONE>(p);
    case EPI_GLU_NOSCALE: return launch_decode_epi<EPI_GLU_NOSCALE>(p);
    case EPI_REGLU: return launch_decode_epi<EPI_REGLU>(p);
    case EPI_BILINEAR: return launch_decode_epi<EPI_BILINEAR>(p);
    case EPI_GLU_DEFER: return launch_decode_epi<EPI_GLU_DEFER>(p);
    case EPI_RELU_DEFER: return launch_decode_epi<EPI_RELU_DEFER>(p);
    case EPI_ROWSCALE: return launch_decode_epi<EPI_ROWSCALE>(p);
    case EPI_ROPE: return launch_decode_epi<EPI_ROPE>(p);
  }
  return hipErrorInvalidValue;
}

}  // namespace fn
