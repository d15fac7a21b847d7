// Large-problem fused norm-then-project kernel for gfx950: a 256 x 256 output
// tile, 8 waves in two groups that take turns ("ping-pong") between a block of
// matrix-core work and a block of memory work, so each SIMD's matrix core is
// fed by one of its two waves while the other issues transfers and LDS reads.
// The per-row sums of squares come from the activation fragments the matrix
// cores consume and the deferred 1/RMS is applied in the epilogue (Prop. 2,
// Cor. 1; App. "Production path" (ii)).
//
// Decomposition.  Group g (waves 4g..4g+3, one per SIMD) owns tile rows
// [128 g, 128 g + 128); wave wn of a group owns packed columns [64 wn, 64 wn + 64),
// i.e. 8 x 4 fragments of 16 x 16.  K advances in steps of 64 (two 32-deep
// fragment blocks, "halves" kh = 0, 1).
//
// Time is cut into intervals separated by workgroup barriers.  Group 0 runs
// memory(t) in interval 2t+1 and compute(t) in interval 2t+2; group 1 runs one
// interval later.  memory(t) issues the wave's global->LDS transfers of a later
// step, reads all of step t's fragments from LDS into registers and waits for
// its transfers of the previous memory phase; compute(t) is 64 matrix-core ops
// plus the wave's share of the row squares, with no memory instructions.
//
// LDS (160 KiB): the weight fragments are read by both groups, the activation
// fragments by one group only, so they live in separate rings:
//   W ring, 3 steps x 32 KiB   [slot][kh][16 column blocks]
//   A ring of group 0, 2 steps x 16 KiB, and of group 1, 2 x 16 KiB   [slot][8 row blocks][2 KiB]
// An activation row block of one step (16 rows x 64 k = 16 rows x 128 bytes) is
// moved by two transfers of 8 whole rows each: lane i takes 16 bytes of row
// i / 8, so every 8 consecutive lanes read one full 128-byte line and the
// address unit coalesces them.  The 16-byte chunks of row r are stored in the
// order chunk ^ swz(r), which keeps the fragment reads free of bank conflicts.
// Transfers of step s go into the slot last used by step s-3 (W) or s-2 (A).
//   group 0, memory(t): W(t+2) half kh=0 and group 1's A(t+1)
//   group 1, memory(t): W(t+2) half kh=1 and group 0's A(t+2)
// Every slot is refilled only after both groups' barriers show its last reader
// done, and every transfer has three intervals to land before it is read: each
// wave waits for its previous memory phase's transfers at the end of the next,
// and the barrier that follows publishes them.
#include <type_traits>

#include "fn_device.h"
#include "fn_epilogue.h"
#include "fn_launch.h"
#include "fn_tile.h"

namespace fn {

namespace pp {
constexpr int BM = 256, BN = 256;
constexpr int FM = 8, FN = 4;              // fragments per wave (rows, columns)
constexpr int kWSlot = 32768;              // one step of weight fragments: 2 halves x 16 blocks
constexpr int kASlot = 16384;              // one step of a group's activations: 2 halves x 8 blocks
constexpr int kWRing = 0;                  // 3 slots
constexpr int kARing0 = 3 * kWSlot;        // group 0: 2 slots
constexpr int kARing1 = kARing0 + 2 * kASlot;  // group 1: 2 slots
constexpr int kLds = kARing1 + 2 * kASlot;     // 160 KiB
constexpr int kBatch = 8;                  // transfers per wave per memory phase
}  // namespace pp

template <int EPI>
__global__ __launch_bounds__(512, 1) void prefill_pp_kernel(
    const __bf16* __restrict__ a, int M, int K, int lda, const __bf16* __restrict__ ws, int NP,
    int KP, int ncols, __bf16* __restrict__ y, int ldy, EpiArgs ep, int tiles_m, int tiles_n) {
  using namespace pp;
  constexpr bool kSS = epi_needs_ss(EPI);
  constexpr bool kSA = EPI == EPI_LN;

  __shared__ __attribute__((aligned(1024))) char smem[kLds];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = wave >> 2, wn = wave & 3;

  int tm, tn;
  tile_of_block(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM;
  const int p0 = tn * BN;
  const int nkb = KP / kKB;       // 32-deep blocks
  const int nsteps = KP / 64;     // 64-deep steps

  const int rows_valid = min(BM, M - m0);
  const i32x4 rs_a = make_rsrc_sgpr(a + (int64_t)m0 * lda,
                                    (uint32_t)(((int64_t)(rows_valid - 1) * lda + K) * 2));
  const int cb0 = p0 / 16;
  const int npb = NP / 16;
  // Column blocks past the packed width (last column tile) read the next block's
  // fragments or zeros; their outputs are never stored.
  const i32x4 rs_w = make_rsrc_sgpr(ws + (int64_t)cb0 * (kFragBytes / 2),
                                    (uint32_t)(((int64_t)nkb * npb - cb0) * kFragBytes));
  const int lrow = lane & 15;
  // Chunk order of row r (0..15) of a row block: distinct over any 8 consecutive
  // rows and over the 8 rows of either parity, so 8 or 16 lanes reading one
  // chunk column of 8 or 16 rows hit distinct LDS banks.
  auto swz = [](int r) { return (r & 7) ^ ((r >> 3) & 1); };
  unsigned a_row_off[2];  // per transfer half h: byte offset of this lane's row and chunk
  int a_chunk[2];         // k offset of this lane's chunk
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int r = h * 8 + (lane >> 3);
    a_chunk[h] = ((lane & 7) ^ swz(r)) * 8;
    a_row_off[h] = (unsigned)(r * lda * 2);
  }
  // LDS offset (inside a row block) of this lane's fragment for half kh:
  // row lrow, chunk kh*4 + lane/16.
  unsigned a_rd[2];
#pragma unroll
  for (int kh = 0; kh < 2; ++kh)
    a_rd[kh] = (unsigned)((lrow * 8 + ((kh * 4 + (lane >> 4)) ^ swz(lrow))) * 16);

  // Rows h*8 .. h*8+7 of tile row block rb, 64 k of step st, into LDS (dst =
  // the row block's 2 KiB + h KiB).  Lane i: row h*8 + i/8, chunk (i%8) ^ swz.
  auto load_a = [&](char* dst, int rb, int h, int st) __attribute__((always_inline)) {
    const int k = st * 64 + a_chunk[h];
    load_lds16(rs_a, dst, k < K ? a_row_off[h] + (unsigned)(rb * 16 * lda * 2 + k * 2) : kOobOffset);
  };
  // One weight fragment (tile column block cb, block kb) into LDS.
  auto load_w = [&](char* dst, int cb, int kb) __attribute__((always_inline)) {
    load_lds16(rs_w, dst, kb < nkb ? (unsigned)((kb * npb + cb) * kFragBytes + lane * 16) : kOobOffset);
  };
  auto w_slot = [&](int s) __attribute__((always_inline)) { return smem + kWRing + (s % 3) * kWSlot; };
  auto a_slot = [&](int g, int s) __attribute__((always_inline)) {
    return smem + (g ? kARing1 : kARing0) + (s & 1) * kASlot;
  };

  // Memory-phase transfers of this wave for step t (kBatch of them): group 0
  // moves weight half 0 of step t+2 and group 1's activations of step t+1;
  // group 1 moves weight half 1 of step t+2 and group 0's activations of t+2.
  auto issue_batch = [&](int t) __attribute__((always_inline)) {
    const int sw = t + 2;
    char* wdst = w_slot(sw) + grp * (kWSlot / 2);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int cb = wn + 4 * i;
      load_w(wdst + cb * kFragBytes, cb, 2 * sw + grp);
    }
    const int sa_ = grp ? t + 2 : t + 1;  // step of the other group's activations
    const int og = grp ^ 1;
    char* adst = a_slot(og, sa_);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int q = wn + 4 * i;  // (rb, h) = (q / 2, q % 2)
      load_a(adst + q * kFragBytes, og * 8 + (q >> 1), q & 1, sa_);
    }
  };

  // Prologue: W(0), W(1), A0(0), A0(1), A1(0): 112 fragments, 14 per wave.
#pragma unroll
  for (int i = 0; i < 14; ++i) {
    const int idx = wave + 8 * i;  // the kind is uniform per i
    if (idx < 64) {
      const int s = idx >> 5, kh = (idx >> 4) & 1, cb = idx & 15;
      load_w(w_slot(s) + kh * (kWSlot / 2) + cb * kFragBytes, cb, 2 * s + kh);
    } else if (idx < 96) {
      const int q = idx - 64, s = q >> 4, r = q & 15;  // r = rb * 2 + h
      load_a(a_slot(0, s) + r * kFragBytes, r >> 1, r & 1, s);
    } else {
      const int r = idx - 96;
      load_a(a_slot(1, 0) + r * kFragBytes, 8 + (r >> 1), r & 1, 0);
    }
  }

  f32x4 acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Row statistics: wave wn squares row blocks wn and wn + 4 of its group.
  float ss[2] = {0.f, 0.f}, sa[2] = {0.f, 0.f};
  bf16x8 af[2][FM], wf[2][FN];

  auto memory_phase = [&](auto wnc, int t) __attribute__((always_inline)) {
    constexpr int WNC = decltype(wnc)::value;  // == wn, known at compile time
    issue_batch(t);
    const char* as = a_slot(grp, t);
    const char* wsl = w_slot(t);
#pragma unroll
    for (int kh = 0; kh < 2; ++kh) {
#pragma unroll
      for (int j = 0; j < FM; ++j)
        af[kh][j] = *reinterpret_cast<const bf16x8*>(as + j * 2 * kFragBytes + a_rd[kh]);
#pragma unroll
      for (int i = 0; i < FN; ++i)
        wf[kh][i] = *reinterpret_cast<const bf16x8*>(wsl + kh * (kWSlot / 2) + (wn * 4 + i) * kFragBytes +
                                                      lane * 16);
    }
    wait_vmcnt<kBatch>();               // previous memory phase's transfers have landed
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): fragments are in registers
    // This wave's share of the row statistics (row blocks wn and wn + 4), on the
    // vector ALU while the other wave of the SIMD runs its matrix-core block.
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        if constexpr (kSS) ss[r] = sumsq8(af[kh][WNC + 4 * r], ss[r]);
        if constexpr (kSA) sa[r] = sum8(af[kh][WNC + 4 * r], sa[r]);
      }
  };
  auto compute_phase = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[kh][i], af[kh][j], acc[i][j], 0, 0, 0);
  };
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  if (grp == 1) __builtin_amdgcn_s_barrier();  // group 1 runs one interval behind
  auto mainloop = [&](auto wnc) __attribute__((always_inline)) {
    for (int t = 0; t < nsteps; ++t) {
      memory_phase(wnc, t);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      compute_phase();
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // One copy of the loop per column-wave index, so the row blocks a wave squares
  // are compile-time register indices (one copy when there are no statistics).
  if constexpr (!kSS && !kSA) {
    mainloop(std::integral_constant<int, 0>{});
  } else switch (wn) {
    case 0: mainloop(std::integral_constant<int, 0>{}); break;
    case 1: mainloop(std::integral_constant<int, 1>{}); break;
    case 2: mainloop(std::integral_constant<int, 2>{}); break;
    default: mainloop(std::integral_constant<int, 3>{}); break;
  }
  if (grp == 0) __builtin_amdgcn_s_barrier();
  wait_vmcnt<0>();  // the trailing (zero-filling) transfers have landed

  // Row totals: lanes l, l^16, l^32, l^48 hold disjoint k of one row; the four
  // waves of a group each hold two of its eight row blocks and share them
  // through LDS (the rings are idle once every transfer has landed).
  float sst[FM], sat[FM];
  if constexpr (kSS || kSA) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      if constexpr (kSS) {
        ss[r] += __shfl_xor(ss[r], 16);
        ss[r] += __shfl_xor(ss[r], 32);
      }
      if constexpr (kSA) {
        sa[r] += __shfl_xor(sa[r], 16);
        sa[r] += __shfl_xor(sa[r], 32);
      }
    }
    float (*row_tot)[BM] = reinterpret_cast<float (*)[BM]>(smem);
    __syncthreads();
    if (lane < 16) {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        row_tot[0][grp * 128 + (wn + 4 * r) * 16 + lane] = ss[r];
        row_tot[1][grp * 128 + (wn + 4 * r) * 16 + lane] = sa[r];
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      sst[j] = row_tot[0][grp * 128 + j * 16 + lrow];
      sat[j] = row_tot[1][grp * 128 + j * 16 + lrow];
    }
  } else {
#pragma unroll
    for (int j = 0; j < FM; ++j) sst[j] = sat[j] = 0.f;
  }

  const int n_lane = (lane >> 4) * 4;
  auto epilogue = [&](auto vec_tag) __attribute__((always_inline)) {
    constexpr bool VEC = decltype(vec_tag)::value;
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      const int mb = m0 + grp * 128 + j * 16;
      const int m = mb + lrow;
      const RowStat st = row_stat<EPI>(sst[j], sat[j], ep);
      if constexpr (EPI == EPI_RMS) {
        if (ep.inv_rms && wn == 0 && lane < 16 && m < M) ep.inv_rms[m] = st.s;
      }
      const bool rows_full = mb + 16 <= M;
      if constexpr (epi_is_glu(EPI)) {
#pragma unroll
        for (int i = 0; i < FN; i += 2) {
          const int fb = (p0 + wn * 64) / 2 + (i / 2) * 16;
          if (rows_full && fb + 16 <= ncols)
            store4_bf16_full<EPI, VEC>(y, ldy, m, fb + n_lane, acc[i][j], acc[i + 1][j], st, ep);
          else
            store4_bf16_edge<EPI, VEC>(y, ldy, M, ncols, m, fb + n_lane, acc[i][j], acc[i + 1][j], st, ep);
        }
      } else {
#pragma unroll
        for (int i = 0; i < FN; ++i) {
          const int pb = p0 + wn * 64 + i * 16;
          if (rows_full && pb + 16 <= ncols)
            store4_bf16_full<EPI, VEC>(y, ldy, m, pb + n_lane, acc[i][j], acc[i][j], st, ep);
          else
            store4_bf16_edge<EPI, VEC>(y, ldy, M, ncols, m, pb + n_lane, acc[i][j], acc[i][j], st, ep);
        }
      }
    }
  };
  if (epi_vec<EPI>(ep) != nullptr)
    epilogue(std::true_type{});
  else
    epilogue(std::false_type{});
}

template <int EPI>
static hipError_t launch_pp(const PrefillArgs& p) {
  const int tiles_m = (p.M + pp::BM - 1) / pp::BM;
  const int tiles_n = (p.NP + pp::BN - 1) / pp::BN;
  hipLaunchKernelGGL((prefill_pp_kernel<EPI>), dim3(tiles_m * tiles_n), dim3(512), 0, p.stream, p.a, p.M,
                     p.K, p.lda, p.ws, p.NP, p.KP, p.ncols, p.y, p.ldy, p.ep, tiles_m, tiles_n);
  return hipGetLastError();
}

hipError_t launch_prefill_pp_bf16(const PrefillArgs& p) {
  switch (p.epi) {
    case EPI_RMS: return launch_pp<EPI_RMS>(p);
    case EPI_GLU: return launch_pp<EPI_GLU>(p);
    case EPI_LN: return launch_pp<EPI_LN>(p);
    case EPI_NONE: return launch_pp<EPI_NONE>(p);
    case EPI_GLU_NOSCALE: return launch_pp<EPI_GLU_NOSCALE>(p);
  }
  return hipErrorInvalidValue;
}

}  // namespace fn
