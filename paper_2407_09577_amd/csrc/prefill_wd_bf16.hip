// Many-row fused norm-then-project kernel for gfx950 with the weight operand
// loaded straight into registers ("weights direct").  The per-row sums of
// squares come from the activation fragments the matrix cores consume and the
// deferred 1/RMS is applied in the epilogue (Prop. 2, Cor. 1; App. "Production
// path" (ii)).
//
// Why.  With both operands staged through LDS, a 256 x 256 tile on 8 waves
// moves 32 KiB into LDS and 96 KiB out of it per 32-deep k block, and the LDS,
// not the matrix cores, sets the pace.  Every weight fragment is a contiguous
// 1 KiB piece of the packed W* (the fold stores it in matrix-core operand
// order), so each wave can load its own weight fragments with one 16-byte load
// per lane; the two waves that share a column block load the same bytes (the
// second request mostly hits the L1).  LDS then carries only the activations:
// 16 KiB in and 64 KiB out per block.
//
// Work split: a BM x BN tile, 8 waves as 2 row bands x 4 column bands, wave
// tile (BM/2) x (BN/4), 16 x 16 fragments: FM = BM/32 activation fragments and
// FN = BN/64 weight fragments per wave and block.  Per block kb, in FN groups:
//   * activations of block kb + kAhead: global -> LDS ring (range-checked
//     buffer loads straight into LDS; rows past M and k past K read zeros);
//   * activation fragments of block kb+1: LDS -> registers (double buffered);
//   * group i: the FM matrix-core ops of weight fragment i, then the register
//     that held it is reloaded with weight fragment i of block kb+2;
//   * the wave's share of the row squares: the 4 waves of a row band hold the
//     same activation fragments, and wave wn squares element pair wn of the
//     four in each lane's 16 bytes, so the band covers every element once with
//     one copy of the loop for all waves.
// A block ends with this wave's transfers of block kb+2 landed and its LDS
// reads done; the barrier opening the next block publishes the transfers.
//
// Activation transfers: lane i moves 16 bytes of row i / 4 of a 16 x 32
// fragment (4 consecutive lanes = 64 contiguous bytes, one coalesced access);
// row r's four 16-byte chunks are stored in the order chunk ^ swz(r), which
// keeps the fragment reads (lane L: row L % 16, chunk L / 16) conflict-free.
#include <type_traits>

#include "fn_device.h"
#include "fn_epilogue.h"
#include "fn_launch.h"
#include "fn_tile.h"

namespace fn {

namespace wd {
constexpr int kSlots = 6;  // LDS ring depth (blocks)
constexpr int kAhead = 4;  // activation transfers run this many blocks ahead
}  // namespace wd

template <int BM, int BN, int EPI>
__global__ __launch_bounds__(512, 1) void prefill_wd_kernel(
    const __bf16* __restrict__ a, int M, int K, int lda, const __bf16* __restrict__ ws, int NP,
    int KP, int ncols, __bf16* __restrict__ y, int ldy, EpiArgs ep, int tiles_m, int tiles_n) {
  using namespace wd;
  constexpr int WM = 2, WN = 4, NW = 8;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 16, FN = TN / 16;
  constexpr int A_FRAGS = BM / 16;              // activation fragments per block
  constexpr int TPW = (A_FRAGS + NW - 1) / NW;  // transfers per wave per block
  constexpr int kSlot = A_FRAGS * kFragBytes;
  constexpr bool kSS = epi_needs_ss(EPI);
  constexpr bool kSA = EPI == EPI_LN;
  static_assert(A_FRAGS % NW == 0, "transfers must split evenly over the waves");
  static_assert(FN >= TPW, "one transfer per group at most");
  static_assert(!epi_is_glu(EPI) || TN % 32 == 0, "GLU needs whole gate/up block pairs per wave");

  __shared__ __attribute__((aligned(1024))) char smem[kSlots * kSlot];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WN, wn = wave % WN;

  int tm, tn;
  tile_of_block(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM;
  const int p0 = tn * BN;
  const int nkb = KP / kKB;  // even

  const int rows_valid = min(BM, M - m0);
  const i32x4 rs_a = make_rsrc_sgpr(a + (int64_t)m0 * lda,
                                    (uint32_t)(((int64_t)(rows_valid - 1) * lda + K) * 2));
  const int npb = NP / 16;
  // Column blocks past the packed width (last column tile) read the next
  // block's fragments or zeros; their outputs are never stored.
  const int cbw = p0 / 16 + wn * FN;  // this wave's first column block
  const __amdgpu_buffer_rsrc_t rs_w =
      make_rsrc(ws + (int64_t)cbw * (kFragBytes / 2), (uint32_t)(((int64_t)nkb * npb - cbw) * kFragBytes));

  const int lrow = lane & 15;
  auto swz = [](int r) { return ((r >> 1) ^ (r >> 3)) & 3; };
  const int t_row = lane >> 2;
  const int t_k = ((lane & 3) ^ swz(t_row)) * 8;
  const unsigned t_row_off = (unsigned)(t_row * lda * 2);
  const unsigned a_rd = (unsigned)((lrow * 4 + ((lane >> 4) ^ swz(lrow))) * 16);
  const unsigned lds0 = lds_addr(smem);

  // Transfer i (0 .. TPW-1) of block kb: activation row block wave + NW i.
  auto transfer = [&](int kb, unsigned slot_off, int i) __attribute__((always_inline)) {
    const int k = kb * kKB + t_k;
    const int rb = wave + NW * i;
    load_lds16_at(rs_a, lds0 + slot_off + rb * kFragBytes,
                  k < K ? t_row_off + (unsigned)(rb * 16 * lda * 2 + k * 2) : kOobOffset);
  };
  auto w_off = [&](int kb, int i) __attribute__((always_inline)) {
    return kb < nkb ? (unsigned)((kb * npb + i) * kFragBytes + lane * 16) : kOobOffset;
  };
  // Ring slots advance one per block (a recurrence, so no address is hoisted
  // per unrolled position).
  auto next_slot = [](unsigned off) __attribute__((always_inline)) {
    off += kSlot;
    return off == kSlots * kSlot ? 0u : off;
  };

  f32x4 acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Row statistics: the WN = 4 waves of a row band hold the same activation
  // fragments; wave wn squares element pair wn (of the four in a lane's 16
  // bytes) of every fragment, so the band's waves cover each element once.
  float ss[FM], sa[FM];
#pragma unroll
  for (int r = 0; r < FM; ++r) ss[r] = sa[r] = 0.f;
  // byte selectors of v_perm: word 1 of {hi, lo} if set, word 0 otherwise
  const unsigned sel_odd = (wn & 1) ? 0x07060504u : 0x03020100u;
  const unsigned sel_high = (wn & 2) ? 0x07060504u : 0x03020100u;
  bf16x8 af[2][FM];
  u32x4 wf[2][FN];

  // Prologue: activations of blocks 0 .. kAhead-1, weights of blocks 0 and 1,
  // activation fragments of block 0.
#pragma unroll
  for (int b = 0; b < kAhead; ++b)
#pragma unroll
    for (int i = 0; i < TPW; ++i) transfer(b, b * kSlot, i);
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int i = 0; i < FN; ++i) wf[b][i] = load_buf16(rs_w, w_off(b, i));
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  const unsigned a_band = wm * FM * kFragBytes + a_rd;
#pragma unroll
  for (int j = 0; j < FM; ++j)
    af[0][j] = *reinterpret_cast<const bf16x8*>(smem + a_band + j * kFragBytes);
  __builtin_amdgcn_s_waitcnt(0xc07f);
  unsigned t_slot = kAhead * kSlot;  // slot of the transfers issued in the next block
  unsigned r_slot = kSlot;           // slot of the fragment reads issued in the next block

  auto block = [&](auto sb, int kb) __attribute__((always_inline)) {
    constexpr int S = decltype(sb)::value;  // register set of block kb (= kb % 2)
    const char* next = smem + r_slot + a_band;
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      if (i < TPW) transfer(kb + kAhead, t_slot, i);
      // this group's share of the next block's activation fragments
#pragma unroll
      for (int j = i * FM / FN; j < (i + 1) * FM / FN; ++j)
        af[S ^ 1][j] = *reinterpret_cast<const bf16x8*>(next + j * kFragBytes);
      const bf16x8 w = __builtin_bit_cast(bf16x8, wf[S][i]);
#pragma unroll
      for (int j = 0; j < FM; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, af[S][j], acc[i][j], 0, 0, 0);
      wf[S][i] = load_buf16(rs_w, w_off(kb + 2, i));  // same fragment, two blocks on
      // row squares of this wave's element pair, FM / FN fragments per group
#pragma unroll
      for (int j = i * FM / FN; j < (i + 1) * FM / FN; ++j) {
        const u32x4 v = __builtin_bit_cast(u32x4, af[S][j]);
        const unsigned p01 = __builtin_amdgcn_perm(v[1], v[0], sel_odd);
        const unsigned p23 = __builtin_amdgcn_perm(v[3], v[2], sel_odd);
        const unsigned pw = __builtin_amdgcn_perm(p23, p01, sel_high);  // pair wn
        const float lo = bf16_lo(pw), hi = bf16_hi(pw);
        if constexpr (kSS) ss[j] = fmaf(hi, hi, fmaf(lo, lo, ss[j]));
        if constexpr (kSA) sa[j] = sa[j] + lo + hi;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // Transfers of block kb+2 (issued in block kb+2-kAhead) have landed.  A
    // block issues, per group i, transfer i (i < TPW) and then weight load i, so
    // after a block's last transfer come FN - TPW + 1 weight loads of that block
    // and then the kAhead - 2 later blocks in full.
    constexpr int kPerBlock = TPW + FN;
    wait_vmcnt<(kAhead - 2) * kPerBlock + FN - TPW + 1>();
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): next fragments in registers
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    t_slot = next_slot(t_slot);
    r_slot = next_slot(r_slot);
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  for (int kb = 0; kb < nkb; kb += 2) {
    block(I0{}, kb);
    block(I1{}, kb + 1);
  }
  wait_vmcnt<0>();  // trailing (zero-filling) transfers and loads have landed

  // Row totals: lanes l, l^16, l^32, l^48 hold disjoint k of one row; each row
  // fragment's total lives in the one wave of the band that squared it.
  float sst[FM], sat[FM];
  if constexpr (kSS || kSA) {
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      if constexpr (kSS) {
        ss[j] += __shfl_xor(ss[j], 16);
        ss[j] += __shfl_xor(ss[j], 32);
      }
      if constexpr (kSA) {
        sa[j] += __shfl_xor(sa[j], 16);
        sa[j] += __shfl_xor(sa[j], 32);
      }
    }
    // partial sums of the WN waves of each band, summed in a fixed order
    static_assert(kSlots * kSlot >= 2 * WN * BM * (int)sizeof(float), "ring too small for row totals");
    float (*part)[WN][BM] = reinterpret_cast<float (*)[WN][BM]>(smem);
    __syncthreads();
    if (lane < 16) {
#pragma unroll
      for (int j = 0; j < FM; ++j) {
        part[0][wn][wm * TM + j * 16 + lane] = ss[j];
        part[1][wn][wm * TM + j * 16 + lane] = sa[j];
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      const int r = wm * TM + j * 16 + lrow;
      sst[j] = (part[0][0][r] + part[0][1][r]) + (part[0][2][r] + part[0][3][r]);
      sat[j] = (part[1][0][r] + part[1][1][r]) + (part[1][2][r] + part[1][3][r]);
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
      const int mb = m0 + wm * TM + j * 16;
      const int m = mb + lrow;
      const RowStat st = row_stat<EPI>(sst[j], sat[j], ep);
      if constexpr (EPI == EPI_RMS) {
        if (ep.inv_rms && wn == 0 && lane < 16 && m < M) ep.inv_rms[m] = st.s;
      }
      const bool rows_full = mb + 16 <= M;
      if constexpr (epi_is_glu(EPI)) {
#pragma unroll
        for (int i = 0; i < FN; i += 2) {
          const int fb = (p0 + wn * TN) / 2 + (i / 2) * 16;
          if (rows_full && fb + 16 <= ncols)
            store4_bf16_full<EPI, VEC>(y, ldy, m, fb + n_lane, acc[i][j], acc[i + 1][j], st, ep);
          else
            store4_bf16_edge<EPI, VEC>(y, ldy, M, ncols, m, fb + n_lane, acc[i][j], acc[i + 1][j], st, ep);
        }
      } else {
#pragma unroll
        for (int i = 0; i < FN; ++i) {
          const int pb = p0 + wn * TN + i * 16;
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

template <int BM, int BN, int EPI>
static hipError_t launch_wd(const PrefillArgs& p) {
  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = (p.NP + BN - 1) / BN;
  hipLaunchKernelGGL((prefill_wd_kernel<BM, BN, EPI>), dim3(tiles_m * tiles_n), dim3(512), 0, p.stream, p.a,
                     p.M, p.K, p.lda, p.ws, p.NP, p.KP, p.ncols, p.y, p.ldy, p.ep, tiles_m, tiles_n);
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_wd_epi(const PrefillArgs& p) {
  switch (p.tile) {
    case TILE_WD_256x256: return launch_wd<256, 256, EPI>(p);
    case TILE_WD_128x256: return launch_wd<128, 256, EPI>(p);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_prefill_wd_bf16(const PrefillArgs& p) {
  switch (p.epi) {
    case EPI_RMS: return launch_wd_epi<EPI_RMS>(p);
    case EPI_GLU: return launch_wd_epi<EPI_GLU>(p);
    case EPI_LN: return launch_wd_epi<EPI_LN>(p);
    case EPI_NONE: return launch_wd_epi<EPI_NONE>(p);
    case EPI_GLU_NOSCALE: return launch_wd_epi<EPI_GLU_NOSCALE>(p);
  }
  return hipErrorInvalidValue;
}

}  // namespace fn
