// Many-row (prefill) fused norm-then-project kernel for gfx950: bf16 matrix
// cores with fp32 accumulation, the per-row statistics accumulated from the very
// activation fragments the matrix cores consume, and the deferred scale applied
// in the epilogue (Prop. 2, Cor. 1; App. "Production path" (ii): accumulating
// the squares during the tile load costs register operations only, no extra
// memory traffic).
//
// Work decomposition.  A workgroup owns a BM x BN output tile (BM activation
// rows x BN packed weight columns) and walks K in steps of 64.  Each step moves
// the activation tile (BM/16 x 2 fragments) and the weight tile (BN/16 x 2
// fragments) straight from HBM into LDS with range-checked buffer loads (rows
// past M, columns past N and k past K read as zero), double buffered, so the
// loads of step t+1 are in flight while the matrix cores work on step t.  The
// WM x WN waves each own a (BM/WM) x (BN/WN) sub-tile.  The matrix multiply runs
// transposed, D' = W*^T a^T, so that one lane's four accumulators are four
// consecutive output columns of one row, and the lane that squares an
// activation fragment holds exactly the row whose outputs it scales.
#include "fn_device.h"
#include "fn_epilogue.h"
#include "fn_launch.h"

namespace fn {

// Workgroup id -> output tile.  Consecutive workgroup ids are dispatched to the
// 8 XCDs in turn, so ids are first regrouped such that each XCD receives a
// contiguous range of logical tiles; logical tiles are then ordered in groups
// of kGroupM tile rows so tiles running together on one XCD share activation
// rows and weight columns in that XCD's L2.
constexpr int kXcds = 8;
constexpr int kGroupM = 4;

__device__ __forceinline__ void tile_of_block(int bid, int nblocks, int tiles_m, int tiles_n,
                                              int& tm, int& tn) {
  const int q = nblocks / kXcds, r = nblocks % kXcds;
  const int x = bid % kXcds, i = bid / kXcds;
  const int logical = x * q + min(x, r) + i;
  const int per_group = kGroupM * tiles_n;
  const int group = logical / per_group;
  const int first_m = group * kGroupM;
  const int gsize = min(tiles_m - first_m, kGroupM);
  const int in_group = logical - group * per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

template <int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(WM* WN * 64, 1) void prefill_bf16_kernel(
    const __bf16* __restrict__ a, int M, int K, int lda, const __bf16* __restrict__ ws, int NP,
    int KP, int ncols, __bf16* __restrict__ y, int ldy, EpiArgs ep, int tiles_m, int tiles_n) {
  constexpr int NW = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;  // wave sub-tile
  constexpr int FM = TM / 16, FN = TN / 16;  // fragments per wave along rows / columns
  constexpr int A_FRAGS = BM / 16 * 2, W_FRAGS = BN / 16 * 2;
  constexpr int A_BYTES = A_FRAGS * kFragBytes;
  constexpr int STAGE = (A_FRAGS + W_FRAGS) * kFragBytes;
  constexpr int A_PER_WAVE = A_FRAGS / NW, W_PER_WAVE = W_FRAGS / NW;
  constexpr int LOADS = A_PER_WAVE + W_PER_WAVE;
  static_assert(A_FRAGS % NW == 0 && W_FRAGS % NW == 0, "fragments must split evenly over waves");
  static_assert(!epi_is_glu(EPI) || TN % 32 == 0, "GLU needs whole gate/up block pairs per wave");
  constexpr bool kSS = epi_needs_ss(EPI);
  constexpr bool kSA = EPI == EPI_LN;

  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;

  int tm, tn;
  tile_of_block(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM;
  const int p0 = tn * BN;
  const int KB = KP / kKB;  // fragments per packed column block

  // Range-checked views of this tile's activation rows and weight column blocks.
  const int rows_valid = min(BM, M - m0);
  const i32x4 rs_a = make_rsrc_sgpr(a + (int64_t)m0 * lda,
                                    (uint32_t)(((int64_t)(rows_valid - 1) * lda + K) * 2));
  const int cb0 = p0 / 16;
  const int cbs_valid = min(BN / 16, NP / 16 - cb0);
  const i32x4 rs_w = make_rsrc_sgpr(ws + (int64_t)cb0 * KB * (kFragBytes / 2),
                                    (uint32_t)(cbs_valid * KB * kFragBytes));

  // Every wave moves A_FRAGS/NW activation and W_FRAGS/NW weight fragments per
  // k step; fragment f covers block f/2 at k half f%2.  The per-lane offsets are
  // fixed except for the k step.
  const int lrow = lane & 15;
  const int lk = (lane >> 4) * 8;
  unsigned a_off[A_PER_WAVE];
  int a_k[A_PER_WAVE];
#pragma unroll
  for (int i = 0; i < A_PER_WAVE; ++i) {
    const int f = wave * A_PER_WAVE + i;
    a_k[i] = (f & 1) * 32 + lk;
    a_off[i] = (unsigned)(((f >> 1) * 16 + lrow) * lda * 2 + a_k[i] * 2);
  }

  auto load_tile = [&](int kt, char* stage) {
#pragma unroll
    for (int i = 0; i < A_PER_WAVE; ++i) {
      const int f = wave * A_PER_WAVE + i;
      const int k = kt * 64 + a_k[i];
      load_lds16(rs_a, stage + f * kFragBytes, k < K ? a_off[i] + kt * 128 : kOobOffset);
    }
#pragma unroll
    for (int i = 0; i < W_PER_WAVE; ++i) {
      const int g = wave * W_PER_WAVE + i;
      const unsigned off = (unsigned)(((g >> 1) * KB + kt * 2 + (g & 1)) * kFragBytes + lane * 16);
      load_lds16(rs_w, stage + A_BYTES + g * kFragBytes, off);
    }
  };

  f32x4 acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float ss[FM], sa[FM];
#pragma unroll
  for (int j = 0; j < FM; ++j) ss[j] = sa[j] = 0.f;

  auto compute = [&](const char* stage) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      bf16x8 wf[FN], af[FM];
#pragma unroll
      for (int i = 0; i < FN; ++i)
        wf[i] = *reinterpret_cast<const bf16x8*>(
            stage + A_BYTES + ((wn * FN + i) * 2 + kb) * kFragBytes + lane * 16);
#pragma unroll
      for (int j = 0; j < FM; ++j)
        af[j] = *reinterpret_cast<const bf16x8*>(stage + ((wm * FM + j) * 2 + kb) * kFragBytes +
                                                 lane * 16);
#pragma unroll
      for (int j = 0; j < FM; ++j) {
        if constexpr (kSS) ss[j] = sumsq8(af[j], ss[j]);
        if constexpr (kSA) sa[j] = sum8(af[j], sa[j]);
      }
#pragma unroll
      for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[i], af[j], acc[i][j], 0, 0, 0);
    }
  };

  // All LDS reads of a stage have been consumed by the matrix cores before the
  // barrier that precedes its next overwrite; the waits below only order the
  // buffer->LDS transfers.
  auto sync_after_loads = [&](bool more) {
    if (more)
      wait_vmcnt<LOADS>();
    else
      wait_vmcnt<0>();
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
  };
  auto sync_after_compute = [&]() {
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_s_barrier();
  };

  const int nkt = KP / 64;
  load_tile(0, smem);
  for (int kt = 0; kt < nkt; ++kt) {
    char* cur = smem + (kt & 1) * STAGE;
    const bool more = kt + 1 < nkt;
    if (more) load_tile(kt + 1, smem + ((kt + 1) & 1) * STAGE);
    sync_after_loads(more);
    compute(cur);
    sync_after_compute();
  }

  // Row statistics: lanes l, l^16, l^32, l^48 hold disjoint k of the same row.
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

  const int n_lane = (lane >> 4) * 4;
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const int m = m0 + wm * TM + j * 16 + lrow;
    const RowStat st = row_stat<EPI>(ss[j], sa[j], ep);
    if constexpr (EPI == EPI_RMS) {
      if (ep.inv_rms && wn == 0 && lane < 16 && m < M) ep.inv_rms[m] = st.s;
    }
    if (m >= M) continue;
    if constexpr (epi_is_glu(EPI)) {
#pragma unroll
      for (int i = 0; i < FN; i += 2) {
        const int f = (p0 + wn * TN) / 2 + (i / 2) * 16 + n_lane;
        store4_bf16<EPI>(y, ldy, ncols, m, f, acc[i][j], acc[i + 1][j], st, ep);
      }
    } else {
#pragma unroll
      for (int i = 0; i < FN; ++i) {
        const int p = p0 + wn * TN + i * 16 + n_lane;
        store4_bf16<EPI>(y, ldy, ncols, m, p, acc[i][j], acc[i][j], st, ep);
      }
    }
  }
}

template <int BM, int BN, int WM, int WN, int EPI>
static hipError_t launch_prefill_cfg(const PrefillArgs& p) {
  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = (p.NP + BN - 1) / BN;
  const int nblocks = tiles_m * tiles_n;
  hipLaunchKernelGGL((prefill_bf16_kernel<BM, BN, WM, WN, EPI>), dim3(nblocks), dim3(WM * WN * 64), 0,
                     p.stream, p.a, p.M, p.K, p.lda, p.ws, p.NP, p.KP, p.ncols, p.y, p.ldy, p.ep,
                     tiles_m, tiles_n);
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_prefill_epi(const PrefillArgs& p) {
  // Shape-specialised tiles: the large tile when it still yields at least one
  // tile per compute unit, a smaller one otherwise.
  const int64_t big = ((int64_t)(p.M + 255) / 256) * ((p.NP + 255) / 256);
  if (p.tile == TILE_256x256 || (p.tile == TILE_AUTO && big >= 256))
    return launch_prefill_cfg<256, 256, 2, 4, EPI>(p);
  if (p.tile == TILE_128x128 || p.tile == TILE_AUTO) return launch_prefill_cfg<128, 128, 2, 2, EPI>(p);
  return hipErrorInvalidValue;
}

hipError_t launch_prefill_bf16(const PrefillArgs& p) {
  switch (p.epi) {
    case EPI_RMS: return launch_prefill_epi<EPI_RMS>(p);
    case EPI_GLU: return launch_prefill_epi<EPI_GLU>(p);
    case EPI_LN: return launch_prefill_epi<EPI_LN>(p);
    case EPI_NONE: return launch_prefill_epi<EPI_NONE>(p);
    case EPI_GLU_NOSCALE: return launch_prefill_epi<EPI_GLU_NOSCALE>(p);
  }
  return hipErrorInvalidValue;
}

}  // namespace fn
