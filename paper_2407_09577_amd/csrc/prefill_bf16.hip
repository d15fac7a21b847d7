// Many-row (prefill) fused norm-then-project kernel for gfx950: bf16 matrix
// cores with fp32 accumulation, the per-row statistics accumulated from the very
// activation fragments the matrix cores consume, and the deferred scale applied
// in the epilogue (Prop. 2, Cor. 1; App. "Production path" (ii): accumulating
// the squares during the tile load costs register operations only, no extra
// memory traffic).
//
// Work decomposition.  A workgroup owns a BM x BN output tile (BM activation
// rows x BN packed weight columns) and walks K in blocks of 32.  Each block's
// activation fragments (BM/16) and weight fragments (BN/16) move straight from
// HBM into an LDS ring of STAGES blocks with range-checked buffer loads (rows
// past M, columns past N and k past K read as zero), issued several blocks
// ahead of the matrix cores.  The WM x WN waves each own a (BM/WM) x (BN/WN)
// sub-tile.  The matrix multiply runs
// transposed, D' = W*^T a^T, so that one lane's four accumulators are four
// consecutive output columns of one row, and the lane that squares an
// activation fragment holds exactly the row whose outputs it scales.
#include <type_traits>

#include "fn_device.h"
#include "fn_epilogue.h"
#include "fn_launch.h"
#include "fn_tile.h"
#include "prefill_w4_step.inc"

namespace fn {

// Activation fragment order in LDS (see the kernel): half-wave-major when true,
// row-major with an XOR swizzle when false.  Measured on MI355X, the half-wave order's
// faster fragment reads do not shorten the Llama-7B QKV projection (319.6 vs 318.3 us)
// and its two-row transfer groups cost the 128-row tiles 3-6%, so row-major stays.
constexpr bool kActHalfWave = false;

// Wait until at most `ahead` k blocks of this wave's ring transfers (LOADS each)
// are still outstanding, i.e. everything issued before them has landed.
// `ahead` is wave-uniform and at most A; the counter needs an immediate, so the
// exact value is selected by a chain of uniform branches.
template <int LOADS, int A>
__device__ __forceinline__ void wait_ahead(int ahead) {
  if constexpr (A == 0) {
    wait_vmcnt<0>();
  } else {
    if (ahead >= A)
      wait_vmcnt<A * LOADS>();
    else
      wait_ahead<LOADS, A - 1>(ahead);
  }
}

// KCHK: activation transfers check k < K lane by lane.  Only needed when K is
// not a multiple of 64: otherwise every k of a block that is multiplied lies
// below K, and the transfers of the blocks past the end (never multiplied) are
// range-checked reads that stay inside the activation buffer or return zeros.
// KD: 32-deep k fragments per ring step (1, or 2 for 64-deep steps: half the
// barriers and waits per k; the accumulation order is unchanged).
template <int BM, int BN, int WM, int WN, int STAGES, bool PF, int EPI, bool SPREAD = false, bool GS = false,
          bool KCHK = true, int KD = 1>
__global__ __launch_bounds__(WM* WN * 64, 1) void prefill_bf16_kernel(
    const __bf16* __restrict__ a, int M, int K, int lda, const __bf16* __restrict__ ws, int NP,
    int KP, int ncols, __bf16* __restrict__ y, int ldy, EpiArgs ep, int tiles_m, int tiles_n) {
  constexpr int NW = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;  // wave sub-tile
  constexpr int FM = TM / 16, FN = TN / 16;  // fragments per wave along rows / columns
  constexpr int A_RB = BM / 16, W_CB = BN / 16;     // row / column blocks of the tile
  constexpr int A_FRAGS = A_RB * KD, W_FRAGS = W_CB * KD;  // per ring step (KD x 32 deep)
  constexpr int T_FRAGS = A_FRAGS + W_FRAGS;
  constexpr int A_BYTES = A_FRAGS * kFragBytes;
  constexpr int STAGE = T_FRAGS * kFragBytes;
  constexpr int LOADS = (T_FRAGS + NW - 1) / NW;     // loads per wave per stage
  constexpr bool kUneven = T_FRAGS % NW != 0;        // some waves pad with a dummy load
  constexpr int FMK = FM * KD, FNK = FN * KD;        // operand fragments per wave per step
  constexpr int NMF = FN * FM * KD;                  // matrix-core ops per wave per step
  constexpr int NRD = FNK + FMK;                     // LDS fragment reads per wave per step
  static_assert(KD == 1 || (KD == 2 && !GS && FM % WN == 0),
                "64-deep steps: no run-time g; each row block's statistics stay with one wave");
  static_assert(TM % 16 == 0 && TN % 16 == 0, "wave tile must be whole fragments");
  static_assert(!epi_is_glu(EPI) || TN % 32 == 0, "GLU needs whole gate/up block pairs per wave");
  static_assert(STAGES >= 3 && (STAGES - 2) * LOADS < 64, "ring depth / vmcnt range");
  static_assert(NRD <= NMF && LOADS <= NRD, "schedule needs at least one op per group");
  constexpr bool kSS = epi_needs_ss(EPI);
  constexpr bool kSA = EPI == EPI_LN;
  // GS: the normalisation weight g is applied at run time to the activation
  // tiles (unfolded W; Remark "Unfolded case"), once per workgroup: every
  // fragment of block kb+2 is scaled in LDS during block kb by the wave that owns
  // its row block, which also takes the row's squares from the raw values.
  static_assert(!GS || (PF && A_FRAGS % NW == 0 && (EPI == EPI_RMS || EPI == EPI_GLU) && STAGES >= 4),
                "run-time g: prefetching ring, even split of row blocks, RMS kinds");
  constexpr int SPW = GS ? A_FRAGS / NW : 0;  // row blocks each wave scales
  static_assert(SPW < NRD, "run-time g: one matrix-core group per scaled fragment after the first");

  // STAGES ring of k blocks, plus one slot that absorbs padding loads.
  __shared__ __attribute__((aligned(1024))) char smem[STAGES * STAGE + (kUneven ? kFragBytes : 0)];
  // Run-time g (GS), staged once: g[k] for k < K, zeros up to kGsMaxK + 64.
  __shared__ __attribute__((aligned(16))) float g_lds[GS ? kGsMaxK + 64 : 4];
  // Fused QKV kinds: each row's scale and token position, for the staged copy-out.
  constexpr bool kRowLds = EPI == EPI_ROPE || EPI == EPI_HEADNORM;
  __shared__ float row_s[kRowLds ? BM : 1];
  __shared__ int row_pos[kRowLds ? BM : 1];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WN, wn = wave % WN;

  int tm, tn;
  tile_of_block(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM;
  const int p0 = tn * BN;
  const int nkb = KP / (kKB * KD);  // ring steps (KP is a multiple of 64: even for KD = 1)

  // Range-checked views of this tile's activation rows and weight column blocks.
  const int rows_valid = min(BM, M - m0);
  const i32x4 rs_a = make_rsrc_sgpr(a + (int64_t)m0 * lda,
                                    (uint32_t)(((int64_t)(rows_valid - 1) * lda + K) * 2));
  const int cb0 = p0 / 16;
  const int npb = NP / 16;  // column blocks per k block of the packed weight
  const i32x4 rs_w = make_rsrc_sgpr(ws + (int64_t)cb0 * (kFragBytes / 2),
                                    (uint32_t)(((int64_t)(KP / kKB) * npb - cb0) * kFragBytes));

  // Fragment f of a stage: f < A_FRAGS is activation row block f, otherwise weight
  // column block f - A_FRAGS.  Wave w moves fragments w, w + NW, ...
  const int lrow = lane & 15;
  // Activation fragment layout in LDS.  A transfer writes lane i's 16 bytes to unit i
  // of the fragment, and the matrix-core operand needs lane L to read row L % 16,
  // k chunk L / 16.  Half-wave-major order: unit u holds row (u / 2) % 16, chunk
  // 2 (u / 32) + u % 2, so two consecutive transfer lanes read 32 contiguous bytes of
  // one row, and the fragment reads (unit 32 (q / 2) + 2 m + q % 2 for row m, chunk q)
  // run at ~185 B/clk per CU on MI355X.  Row-major orders (unit 4 r + chunk, with or
  // without an XOR swizzle of the chunks) let four lanes read one 64-byte row segment
  // but their fragment reads run at ~125 B/clk (linear unit order: ~230).
  const int t_row = kActHalfWave ? (lane >> 1) & 15 : lane >> 2;  // row of this lane's transfer
  auto swz = [](int r) { return ((r >> 1) ^ (r >> 3)) & 3; };
  const int lk = kActHalfWave ? (2 * (lane >> 5) + (lane & 1)) * 8            // k offset of the chunk
                              : ((lane & 3) ^ swz(t_row)) * 8;
  const unsigned a_rd = kActHalfWave
                            ? (unsigned)((32 * (lane >> 5) + 2 * lrow + ((lane >> 4) & 1)) * 16)
                            : (unsigned)((lrow * 4 + ((lane >> 4) ^ swz(lrow))) * 16);
  // Weight column blocks past the packed width (last column tile only) read the
  // next k block's fragments, or zeros past the buffer's end; the columns they
  // feed lie beyond every output column and are never stored.
  // With KD = 2, fragment f covers k half f / A_RB (activations) or
  // (f - A_FRAGS) / W_CB (weights) of the 64-deep step.
  unsigned off0[LOADS];
  int lkh[LOADS];  // k offset of this lane's activation chunk within the step
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    const int f = wave + NW * i;
    if (A_FRAGS % NW == 0 ? i < A_FRAGS / NW : f < A_FRAGS) {
      lkh[i] = (f / A_RB) * kKB + lk;
      off0[i] = (unsigned)(((f % A_RB) * 16 + t_row) * lda * 2 + lkh[i] * 2);
    } else {
      const int wf = f - A_FRAGS;
      lkh[i] = 0;
      off0[i] = (unsigned)(((wf / W_CB) * npb + wf % W_CB) * kFragBytes + lane * 16);
    }
  }

  // Transfer i of block kb into its ring slot.  Every wave issues exactly LOADS
  // transfers per block, also for blocks past the end of K (their slots are
  // never multiplied), so the outstanding-transfer count of every step is the
  // same.  When the activation fragments split evenly over the waves, transfer i
  // is an activation fragment exactly when i < A_FRAGS / NW (known at compile
  // time).  The ring is addressed by 32-bit LDS offsets from one base, so a
  // transfer costs one scalar add for its destination and one vector add for
  // its source: weight offsets past the packed buffer read zeros, and the
  // activations need a lane check only with KCHK.
  constexpr bool kSplitA = A_FRAGS % NW == 0;
  const unsigned lds_ring = lds_addr(smem);
  auto load_one = [&](int kb, int i) __attribute__((always_inline)) {
    const unsigned st = lds_ring + (unsigned)((kb % STAGES) * STAGE);
    const int f = wave + NW * i;
    if (kSplitA ? i < A_FRAGS / NW : f < A_FRAGS) {
      const unsigned off = off0[i] + (unsigned)(kb * (KD * kKB * 2));
      load_lds16_at(rs_a, st + f * kFragBytes, (!KCHK || kb * (KD * kKB) + lkh[i] < K) ? off : kOobOffset);
    } else if (!kUneven || f < T_FRAGS) {
      load_lds16_at(rs_w, st + f * kFragBytes, off0[i] + (unsigned)(kb * KD * npb) * kFragBytes);
    } else {
      load_lds16_at(rs_w, lds_ring + STAGES * STAGE, kOobOffset);
    }
  };

  f32x4 acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Row sums.  In the K loop a wave keeps only the row blocks whose statistics it
  // takes (row block WNC + WN t is its t-th, see multiply_interleaved); after the loop
  // ss / sa hold the totals of all FM row blocks of its sub-tile.
  //
  // The RMS kinds take the sums of squares on the matrix cores, from the activation
  // fragments the product consumes: for a fragment F (16 rows m x 32 k) the product
  // F F^T is the 16 x 16 Gram block whose diagonal holds each row's sum of squares over
  // the fragment; added block after block they give the totals over K.  Measured on
  // MI355X, one extra 16x16x32 op per fragment costs about a third of the four packed
  // dot products it replaces, which compete for the same pipe.  Row m's diagonal
  // element sits in lane 20 (m / 4) + m % 4, component m % 4.
  //
  // LayerNorm (sums and squares) keeps packed dot products: fp32 partials of four
  // 32-deep k blocks (32 elements per lane, whose squares and sums are exact in fp32
  // when the values are of one magnitude, the case where the variance would cancel)
  // flushed into fp64 totals.  The grouping is by 32-deep blocks whatever the ring step
  // depth, so both depths round alike.  (Its Gram and all-ones products need 16 more
  // registers in the loop than the 256-wide tile has.)
  using ST = StatT<EPI>;
  static_assert(!(kSS || kSA) || GS || FM % WN == 0, "each wave takes whole row blocks' statistics");
  constexpr int TW = (FM / WN) > 0 ? FM / WN : 1;
  constexpr bool kGram = kSS && !kSA && !GS;
  f32x4 gsq[kGram ? TW : 1];
  float tss[kSA ? TW : 1], tsa[kSA ? TW : 1];
  ST ssw[TW], saw[TW];
#pragma unroll
  for (int t = 0; t < TW; ++t) ssw[t] = saw[t] = ST(0);
#pragma unroll
  for (int t = 0; t < (kGram ? TW : 1); ++t) gsq[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < (kSA ? TW : 1); ++t) tss[t] = tsa[t] = 0.0f;
  // This lane's Gram component: the diagonal one when the lane holds a diagonal element.
  auto diag_of = [&](const f32x4& g) __attribute__((always_inline)) {
    return (lane & 2) ? ((lane & 1) ? g[3] : g[2]) : ((lane & 1) ? g[1] : g[0]);
  };
  ST ss[FM], sa[FM];
#pragma unroll
  for (int j = 0; j < FM; ++j) ss[j] = sa[j] = ST(0);

  bf16x8 af0[FMK], wf0[FNK];
  bf16x8 af1[PF ? FMK : 1], wf1[PF ? FNK : 1];

  // Fragment r of step kb (r < FMK: activations, else weights; k half r / FM or
  // (r - FMK) / FN) into registers.
  auto read_one = [&](int kb, int r, bf16x8 (&af)[FMK], bf16x8 (&wf)[FNK]) __attribute__((always_inline)) {
    const char* st = smem + (kb % STAGES) * STAGE;
    if (r < FMK) {
      af[r] = *reinterpret_cast<const bf16x8*>(st + ((r / FM) * A_RB + wm * FM + r % FM) * kFragBytes + a_rd);
    } else {
      const int q = r - FMK;
      wf[q] = *reinterpret_cast<const bf16x8*>(st + A_BYTES + ((q / FN) * W_CB + wn * FN + q % FN) * kFragBytes +
                                               lane * 16);
    }
  };

  // Row statistics of fragment j (row block j % FM): its Gram block added on the
  // matrix cores (RMS kinds), or its squares and sums as packed bf16 dot products
  // (LayerNorm).  j % FM is WNC + WN t for this wave's mainloop copy WNC.
  auto stats_one = [&](int j, const bf16x8 (&af)[FMK]) __attribute__((always_inline)) {
    const int t = (j % FM) / WN;
    if constexpr (kSA) {
      tss[t] = sumsq8(af[j], tss[t]);
      tsa[t] = sum8(af[j], tsa[t]);
    } else if constexpr (kGram) {
      gsq[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[j], af[j], gsq[t], 0, 0, 0);
    }
  };
  auto flush_ln = [&]() __attribute__((always_inline)) {
    if constexpr (kSA) {
#pragma unroll
      for (int t = 0; t < TW; ++t) {
        ssw[t] += (double)tss[t];
        saw[t] += (double)tsa[t];
        tss[t] = tsa[t] = 0.0f;
      }
    }
  };

  // GS: scale the activation fragments of block b in place, g applied per k
  // (each product rounded once to bf16), and take the row squares from the raw
  // values.  The lane handles the 16 bytes it transferred: row t_row of the row
  // block, k chunk lk of the block (the transfer layout of the ring).  The LDS
  // reads go out right after the barrier (scale_fetch) and the arithmetic and
  // write-back run between the matrix-core groups of the block (scale_store),
  // so the read latency and the VALU work overlap the matrix cores.
  float ss_own[SPW > 0 ? SPW : 1];
  u32x4 sc_raw[SPW > 0 ? SPW : 1];
  f32x4 sc_g0, sc_g1;
  int sc_slot = 0;
#pragma unroll
  for (int t = 0; t < (SPW > 0 ? SPW : 1); ++t) ss_own[t] = 0.f;
  auto scale_fetch = [&](int b) __attribute__((always_inline)) {
    if constexpr (GS) {
      sc_slot = (b % STAGES) * STAGE;
      const float* gk = g_lds + b * kKB + lk;
      sc_g0 = *reinterpret_cast<const f32x4*>(gk);
      sc_g1 = *reinterpret_cast<const f32x4*>(gk + 4);
#pragma unroll
      for (int t = 0; t < SPW; ++t)
        sc_raw[t] = *reinterpret_cast<const u32x4*>(smem + sc_slot + (wave + NW * t) * kFragBytes + lane * 16);
    }
  };
  auto scale_store = [&](int t) __attribute__((always_inline)) {
    if constexpr (GS) {
      const bf16x8 v = __builtin_bit_cast(bf16x8, sc_raw[t]);
      ss_own[t] = sumsq8(v, ss_own[t]);
      float o[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o[e] = (float)v[e] * sc_g0[e];
        o[4 + e] = (float)v[4 + e] * sc_g1[e];
      }
      const u32x2 lo = pack4_bf16(*reinterpret_cast<const float(*)[4]>(o));
      const u32x2 hi = pack4_bf16(*reinterpret_cast<const float(*)[4]>(o + 4));
      *reinterpret_cast<u32x4*>(smem + sc_slot + (wave + NW * t) * kFragBytes + lane * 16) =
          u32x4{lo[0], lo[1], hi[0], hi[1]};
    }
  };
  auto scale_block = [&](int b) __attribute__((always_inline)) {
    scale_fetch(b);
#pragma unroll
    for (int t = 0; t < SPW; ++t) scale_store(t);
  };

  auto sync_block = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS reads have landed
    __builtin_amdgcn_s_barrier();
  };

  // Wave priorities on the 256 x 256 tile.  Its two waves on a SIMD share one
  // matrix-core pipe; the arbiter favours the older wave, which then reached the
  // block barrier ~550 cycles ahead of its partner (s_memtime probe on MI355X,
  // Llama-7B QKV shape), leaving the pipe to one wave for the end of every block.
  // A priority that falls with the progress through the block (3 in the first
  // quarter of the groups, down to 0 in the last) hands the pipe to whichever wave
  // lags: the lead shrank to ~130 cycles and the projection ran 1.2% faster (308.8
  // vs 312.6 us; LayerNorm 4096^3 -0.9%).  The 128-row tiles measured no gain.
  constexpr bool kProgressPrio = BM == 256 && NW == 8;
  auto progress_prio = [](int g) __attribute__((always_inline)) {
    if constexpr (kProgressPrio) {
      switch (3 - (4 * g) / NRD) {  // g is a compile-time constant after unrolling
        case 3: __builtin_amdgcn_s_setprio(3); break;
        case 2: __builtin_amdgcn_s_setprio(2); break;
        case 1: __builtin_amdgcn_s_setprio(1); break;
        default: __builtin_amdgcn_s_setprio(0); break;
      }
    }
  };

  // One k block of work for the matrix cores.  First this wave's share of the
  // row statistics, as one clump of dot products: the waves of a row band split
  // its fragments at compile time (the wave with column index WNC takes
  // fragments WNC, WNC + WN, ...), over the whole of K.  Measured on MI355X, a
  // clump at the start of the block costs next to nothing, while the same work
  // spread between the matrix-core ops costs several percent.  Then NRD groups:
  // group g holds its share of the NMF matrix-core ops, LDS read g of the next
  // block (PF) and, spread over the block, transfer i of block kb+STAGES.  The
  // scheduling fences keep this interleaving, so memory traffic overlaps the
  // matrix cores.
  auto multiply_interleaved = [&](auto wnc, int kb, const bf16x8 (&afc)[FMK], const bf16x8 (&wfc)[FNK],
                                  bf16x8 (&afn)[FMK], bf16x8 (&wfn)[FNK], bool more, bool scale = false)
                                  __attribute__((always_inline)) {
    constexpr int WNC = decltype(wnc)::value;
    if constexpr (!GS) {
#pragma unroll
      for (int j = WNC; j < FMK; j += WN) stats_one(j, afc);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int g = 0; g < NRD; ++g) {
      progress_prio(g);
#pragma unroll
      for (int t = g * NMF / NRD; t < (g + 1) * NMF / NRD; ++t) {
        const int h = t / (FN * FM), i = t % (FN * FM) / FM, j = t % FM;  // k half, column, row
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wfc[h * FN + i], afc[h * FM + j], acc[i][j], 0, 0, 0);
      }
      // GS: fragment t of the block being scaled is finished in group t + 1.
      if constexpr (GS) {
        if (scale && g >= 1 && g - 1 < SPW) scale_store(g - 1);
      }
      // Transfer i goes out in group i * LSTEP: spread over the block (SPREAD),
      // so the workgroup's transfers reach the address unit at the rate it
      // drains them, or in the first groups.
      constexpr int LSTEP = SPREAD ? NRD / LOADS : 1;
      if (more) {
        if (g % LSTEP == 0 && g / LSTEP < LOADS) load_one(kb + STAGES, g / LSTEP);
        read_one(kb + 1, g, afn, wfn);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Ring discipline.  Block kb lives in slot kb % STAGES.
  //  PF: LDS->register reads run one block ahead of the matrix cores, and
  //   global->LDS transfers STAGES blocks ahead.  Before step kb every wave
  //   waits until its transfers of block kb+1 have landed (those of the
  //   STAGES-2 blocks after it may stay outstanding) and for its own reads of
  //   block kb; the barrier then makes block kb+1 visible to all waves and
  //   guarantees that every wave has finished reading block kb, whose slot the
  //   transfer of block kb+STAGES issued during step kb overwrites.
  //  !PF: transfers run STAGES-1 blocks ahead; step kb waits for block kb,
  //   barriers (every wave is done with block kb-1, whose slot block
  //   kb+STAGES-1 takes), then reads and multiplies block kb.
  static_assert(!PF || (STAGES - 1) * LOADS < 64, "vmcnt range");
#pragma unroll
  for (int s = 0; s < (PF ? STAGES : STAGES - 1); ++s)
#pragma unroll
    for (int i = 0; i < LOADS; ++i) load_one(s, i);
  // GS: the run-time g goes to LDS once (zeros past K), after the first
  // transfers are on their way.
  if constexpr (GS) {
    for (int i = threadIdx.x; i < kGsMaxK + 64; i += NW * 64) g_lds[i] = i < K ? ep.g_rt[i] : 0.f;
  }
  // GS needs block kb+2 landed (and scaled during block kb) before block kb+1
  // reads it; otherwise block kb+1 must have landed before step kb.
  constexpr int kAheadWait = GS ? (STAGES - 3) * LOADS : (STAGES - 2) * LOADS;
  // The 4-wave 256 x 256 tile (one wave of 128 x 128 per SIMD) with K a multiple of 64:
  // each k block is one hand-scheduled inline-asm sequence (prefill_w4_step.inc, written by
  // gen_prefill_w4_step.py) that interleaves the block's 64 matrix-core ops (and the Gram
  // ops of the RMS kinds) with the next block's LDS reads, a later block's transfers and
  // their address arithmetic; the compiler allocates its operands, the accumulators in
  // AGPRs.  Compiled from the loop above, one wave per SIMD ran ~12% behind the 8-wave
  // tile; the sequence runs 1-2% ahead of it (Llama-7B QKV shape, MI355X).  The wave keeps
  // its own copy of the ring slot offsets and transfer offsets, which the sequence advances.
  constexpr bool kAsmW4 = BM == 256 && BN == 256 && WM == 2 && WN == 2 && PF && !GS && KD == 1 && STAGES == 4 &&
                          !KCHK && (EPI == EPI_RMS || EPI == EPI_GLU || EPI == EPI_NONE);
  static_assert(!kAsmW4 || (STAGE == 0x8000 && FMK == 8 && FNK == 8 && (!kGram || TW == 4) && LOADS == 8 &&
                            A_FRAGS / NW == 4),
                "the asm step's fixed geometry");
  unsigned w4_sn = 0x8000, w4_sl = 0, w4_vo[8];  // read slot of block kb+1, transfer slot of block kb+4
  const unsigned w4_aconst = lds_ring + (unsigned)(wm * FM * kFragBytes) + a_rd;
  const unsigned w4_wconst = lds_ring + (unsigned)(A_BYTES + wn * FN * kFragBytes + lane * 16);
  const unsigned w4_mbase = __builtin_amdgcn_readfirstlane(lds_ring + (unsigned)(wave * kFragBytes));
  const unsigned w4_dw = __builtin_amdgcn_readfirstlane((unsigned)npb * kFragBytes);
  auto w4_init = [&]() __attribute__((always_inline)) {
    if constexpr (kAsmW4) {
#pragma unroll
      for (int i = 0; i < 8; ++i)  // the transfers of block STAGES (issued during block 0)
        w4_vo[i] = i < A_FRAGS / NW ? off0[i] + (unsigned)(STAGES * (kKB * 2))
                                    : off0[i] + (unsigned)(STAGES * npb) * kFragBytes;
    }
  };
  // One k block: the asm sequence on the 4-wave tile, else the compiled schedule.
  auto mstep = [&](auto wnc, int kb, bf16x8 (&afc)[FMK], bf16x8 (&wfc)[FNK], bf16x8 (&afn)[FMK],
                   bf16x8 (&wfn)[FNK], bool more, bool scale = false) __attribute__((always_inline)) {
    if constexpr (kAsmW4) {
      constexpr int WNC = decltype(wnc)::value;
      u32x4 ca[8], cw[8], na[8], nw[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        ca[r] = __builtin_bit_cast(u32x4, afc[r]);
        cw[r] = __builtin_bit_cast(u32x4, wfc[r]);
      }
      f32x4 gnone[4];
      f32x4 (&g4)[4] = *reinterpret_cast<f32x4(*)[4]>(kGram ? &gsq[0] : &gnone[0]);
      if (more) {
        if constexpr (kGram && WNC == 0)
          w4_step_full_gram0(acc, g4, na, nw, ca, cw, w4_vo, w4_sn, w4_sl, w4_aconst, w4_wconst, w4_mbase, w4_dw, rs_a,
                             rs_w);
        else if constexpr (kGram)
          w4_step_full_gram1(acc, g4, na, nw, ca, cw, w4_vo, w4_sn, w4_sl, w4_aconst, w4_wconst, w4_mbase, w4_dw, rs_a,
                             rs_w);
        else
          w4_step_full_plain(acc, g4, na, nw, ca, cw, w4_vo, w4_sn, w4_sl, w4_aconst, w4_wconst, w4_mbase, w4_dw, rs_a,
                             rs_w);
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          afn[r] = __builtin_bit_cast(bf16x8, na[r]);
          wfn[r] = __builtin_bit_cast(bf16x8, nw[r]);
        }
      } else {
        if constexpr (kGram && WNC == 0) w4_step_last_gram0(acc, g4, ca, cw);
        else if constexpr (kGram) w4_step_last_gram1(acc, g4, ca, cw);
        else w4_step_last_plain(acc, g4, ca, cw);
        // Wait states between the last matrix-core ops and the first reads of their results
        // (the compiler does not see the asm's ops).
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
      }
    } else {
      multiply_interleaved(wnc, kb, afc, wfc, afn, wfn, more, scale);
    }
  };

  auto mainloop = [&](auto wnc) __attribute__((always_inline)) {
    constexpr int WNC = decltype(wnc)::value;
    if constexpr (PF) {
      if constexpr (GS) {
        wait_vmcnt<(STAGES - 2) * LOADS>();  // blocks 0 and 1
        sync_block();
        scale_block(0);
        scale_block(1);
        sync_block();
      } else {
        wait_vmcnt<(STAGES - 1) * LOADS>();
        sync_block();
      }
#pragma unroll
      for (int r = 0; r < NRD; ++r) read_one(0, r, af0, wf0);
      w4_init();
      for (int kb = 0; kb < nkb - 2; kb += 2) {
        wait_vmcnt<kAheadWait>();
        sync_block();
        scale_fetch(kb + 2);
        mstep(wnc, kb, af0, wf0, af1, wf1, true, true);
        wait_vmcnt<kAheadWait>();
        sync_block();
        scale_fetch(kb + 3);
        mstep(wnc, kb + 1, af1, wf1, af0, wf0, true, true);
        if (((kb + 2) * KD) % 4 == 0) flush_ln();  // every fourth 32-deep block
      }
      auto tail_even = [&]() __attribute__((always_inline)) {
        wait_vmcnt<kAheadWait>();
        sync_block();
        mstep(wnc, nkb - 2, af0, wf0, af1, wf1, true);
        __builtin_amdgcn_s_waitcnt(0xc07f);
        mstep(wnc, nkb - 1, af1, wf1, af0, wf0, false);
      };
      if constexpr (KD == 1) {
        tail_even();  // nkb is even
      } else if (nkb % 2 == 0) {
        tail_even();
      } else {
        // Odd step count: the loop (or, for one step, the prologue) has read the
        // last step into af0.
        __builtin_amdgcn_s_waitcnt(0xc07f);
        mstep(wnc, nkb - 1, af0, wf0, af1, wf1, false);
      }
      flush_ln();
    } else {
      for (int kb = 0; kb < nkb; ++kb) {
        wait_vmcnt<(STAGES - 2) * LOADS>();
        sync_block();
#pragma unroll
        for (int i = 0; i < LOADS; ++i) load_one(kb + STAGES - 1, i);
#pragma unroll
        for (int r = 0; r < NRD; ++r) read_one(kb, r, af0, wf0);
#pragma unroll
        for (int j = WNC; j < FMK; j += WN) stats_one(j, af0);
#pragma unroll
        for (int t = 0; t < NMF; ++t) {
          const int h = t / (FN * FM), i = t % (FN * FM) / FM, j = t % FM;
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf0[h * FN + i], af0[h * FM + j], acc[i][j], 0, 0, 0);
        }
        if (((kb + 1) * KD) % 4 == 0) flush_ln();
      }
      flush_ln();
    }
  };
  // One copy of the main loop per column-wave index (wave-uniform dispatch); a
  // single copy when there are no row statistics to split (or GS takes them).
  static_assert(WN <= 4, "mainloop dispatch covers up to 4 column waves");
  if constexpr ((!kSS && !kSA) || GS) {
    mainloop(std::integral_constant<int, 0>{});
  } else switch (wn) {
    case 0: mainloop(std::integral_constant<int, 0>{}); break;
    case 1: if constexpr (WN > 1) mainloop(std::integral_constant<int, 1>{}); break;
    case 2: if constexpr (WN > 2) mainloop(std::integral_constant<int, 2>{}); break;
    default: if constexpr (WN > 3) mainloop(std::integral_constant<int, 3>{}); break;
  }

  if constexpr (kProgressPrio) __builtin_amdgcn_s_setprio(0);

  // GS: the squares were taken by the wave that scaled each row block: the four
  // transfer lanes of row r (half-wave order: 2r, 2r+1, 2r+32, 2r+33; row-major:
  // 4r .. 4r+3) hold disjoint k of it.  Totals reach the waves through LDS.
  if constexpr (GS) {
    float (*row_tot)[BM] = reinterpret_cast<float (*)[BM]>(smem);
#pragma unroll
    for (int t = 0; t < SPW; ++t) {
      ss_own[t] += __shfl_xor(ss_own[t], 1);
      ss_own[t] += __shfl_xor(ss_own[t], kActHalfWave ? 32 : 2);
    }
    wait_vmcnt<0>();
    __syncthreads();
    if ((lane & (kActHalfWave ? 33 : 3)) == 0) {
#pragma unroll
      for (int t = 0; t < SPW; ++t) row_tot[0][(wave + NW * t) * 16 + t_row] = ss_own[t];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < FM; ++j) ss[j] = row_tot[0][wm * TM + j * 16 + lrow];
  } else
  // Row statistics.  Gram: row m's sum of squares is in the diagonal lane
  // 20 (m / 4) + m % 4 and is broadcast to the lanes of row m (m = lane % 16).  Dot
  // products: lanes l, l^16, l^32, l^48 hold disjoint k of the same row.  Row block
  // WN t + wn's totals live in this wave (the one of the row band that took them); they
  // reach the other WN-1 waves through LDS.
  if constexpr (kSS || kSA) {
    const int diag_lane = (lane & 15) + 16 * ((lane & 15) >> 2);
#pragma unroll
    for (int t = 0; t < TW; ++t) {
      if constexpr (kGram) {
        ssw[t] = __shfl(diag_of(gsq[t]), diag_lane);
      } else {
        ssw[t] += __shfl_xor(ssw[t], 16);
        ssw[t] += __shfl_xor(ssw[t], 32);
        if constexpr (kSA) {
          saw[t] += __shfl_xor(saw[t], 16);
          saw[t] += __shfl_xor(saw[t], 32);
        }
      }
    }
    if constexpr (WN > 1) {
      // The totals reuse the ring: wait for this wave's last (zero-filling)
      // transfers, and for every wave to finish reading the last block.
      static_assert(STAGES * STAGE >= 2 * BM * (int)sizeof(ST), "ring too small for row totals");
      ST (*row_tot)[BM] = reinterpret_cast<ST (*)[BM]>(smem);
      wait_vmcnt<0>();
      __syncthreads();
      if (lane < 16) {
#pragma unroll
        for (int t = 0; t < TW; ++t) {
          row_tot[0][wm * TM + (wn + WN * t) * 16 + lane] = ssw[t];
          row_tot[1][wm * TM + (wn + WN * t) * 16 + lane] = saw[t];
        }
      }
      __syncthreads();
#pragma unroll
      for (int j = 0; j < FM; ++j) {
        ss[j] = row_tot[0][wm * TM + j * 16 + lrow];
        sa[j] = row_tot[1][wm * TM + j * 16 + lrow];
      }
    } else {
#pragma unroll
      for (int j = 0; j < FM; ++j) {
        ss[j] = ssw[j];
        sa[j] = saw[j];
      }
    }
  }

  // Epilogue.  A tile that lies wholly inside the output (and a 16-byte
  // aligned row pitch) is staged through LDS and written as whole rows, 16
  // bytes per lane.  Otherwise one uniform decision per 16 x 16 fragment picks
  // the plain store or the guarded edge store.  The optional per-column vector
  // is dispatched once for the whole tile.
  constexpr int OUT_COLS = epi_is_glu(EPI) ? BN / 2 : BN;  // output columns of a tile
  constexpr int UPR = OUT_COLS / 8;                       // 16-byte units per output row
  constexpr bool kStageable = OUT_COLS % 8 == 0 && stage_bytes<BM, UPR>() <= STAGES * STAGE;
  // Fused QKV kinds: the fp32 accumulators are staged (in passes of RP rows when the
  // tile does not fit the ring at once) and finished on the copy to HBM.
  constexpr int F32U = OUT_COLS / 4;                       // 16-byte fp32 units per row
  constexpr bool kF32Xor = F32U % 16 == 0;                 // else rows padded by one unit
  constexpr int F32_ROW = (kF32Xor ? F32U : F32U + 1) * 16;  // bytes per staged row
  constexpr int RP = (BM * F32_ROW <= STAGES * STAGE) ? BM : BM / 2;
  constexpr bool kF32Stage = (EPI == EPI_ROPE || EPI == EPI_HEADNORM) && OUT_COLS % 8 == 0 && RP % TM == 0 &&
                            BM % RP == 0 && RP * F32_ROW <= STAGES * STAGE;
  // The per-head norms need whole heads in one tile and the fp32 staging: every tile
  // (also at the ragged edges, with guarded stores) takes the staged path.
  static_assert(EPI != EPI_HEADNORM || (kF32Stage && (RP * (OUT_COLS / 8)) % (NW * 64) == 0),
                "per-head norms: fp32 staging and a uniform copy-out loop");
  const int n0 = epi_is_glu(EPI) ? p0 / 2 : p0;
  const int n_lane = (lane >> 4) * 4;
  auto write_inv_rms = [&](int j, const RowStat& st) __attribute__((always_inline)) {
    if constexpr (epi_exports_s(EPI)) {
      const int m = m0 + wm * TM + j * 16 + lrow;
      if (ep.inv_rms && wn == 0 && lane < 16 && m < M) ep.inv_rms[m] = st.s;
    }
  };
  // Kinds that read per-row data (a row scale, a token position) take the
  // statistics of all the lane's rows first, so that every such load is in flight
  // at once; the others compute them row by row (fewer live registers).
  constexpr bool kRowData = EPI == EPI_ROWSCALE || EPI == EPI_ROPE || EPI == EPI_HEADNORM;
  auto row_stats = [&](RowStat (&sts)[kRowData ? FM : 1]) __attribute__((always_inline)) {
    if constexpr (kRowData) {
#pragma unroll
      for (int j = 0; j < FM; ++j) sts[j] = row_stat_at<EPI>(ss[j], sa[j], ep, m0 + wm * TM + j * 16 + lrow, M);
    }
  };
  auto staged = [&](auto vec_tag) __attribute__((always_inline)) {
    constexpr bool VEC = decltype(vec_tag)::value;
    RowStat sts[kRowData ? FM : 1];
    row_stats(sts);
    wait_vmcnt<0>();  // the ring's last (zero-filling) transfers have landed
    __syncthreads();  // every wave is done with the ring and the row totals
    if constexpr (kF32Stage) {
      // Read in the matrix-core layout, a lane's 16 rows are 16 tokens, so every angle
      // load would touch 16 table rows.  Here the fp32 accumulators go through LDS
      // and the copy to HBM rotates them: a thread takes 8 consecutive columns of one
      // row, and the threads of a row read its angles contiguously.
      auto f32_pos = [](int r, int u) { return kF32Xor ? r * F32U + (u ^ (r & 15)) : r * (F32U + 1) + u; };
      constexpr int U8 = OUT_COLS / 8;  // 8-column output units per row
#pragma unroll
      for (int pass = 0; pass < BM / RP; ++pass) {
        if (pass > 0) __syncthreads();  // the previous pass's rows have been copied out
        if (wm * TM / RP == pass) {
#pragma unroll
          for (int j = 0; j < FM; ++j) {
            const int r = wm * TM + j * 16 + lrow - pass * RP;  // row within the pass
            write_inv_rms(j, sts[j]);
            if (wn == 0 && lane < 16) {
              row_s[r + pass * RP] = sts[j].s;
              row_pos[r + pass * RP] = sts[j].pos;
            }
#pragma unroll
            for (int i = 0; i < FN; ++i) {
              const int u = (wn * TN + i * 16 + n_lane) / 4;
              *reinterpret_cast<f32x4*>(smem + f32_pos(r, u) * 16) = acc[i][j];
            }
          }
        }
        __syncthreads();
#pragma unroll
        for (int q = threadIdx.x; q < RP * U8; q += NW * 64) {
          const int r = q / U8, v = q % U8;
          const int row = pass * RP + r;
          const RowStat st{row_s[row], 0.0f, row_pos[row]};
          float o[8];
          if constexpr (EPI == EPI_HEADNORM) {
            headnorm8(n0 + v * 8, *reinterpret_cast<const f32x4*>(smem + f32_pos(r, 2 * v) * 16),
                      *reinterpret_cast<const f32x4*>(smem + f32_pos(r, 2 * v + 1) * 16), st, ep, o);
          } else {
#pragma unroll
            for (int hlf = 0; hlf < 2; ++hlf) {
              const int n = n0 + v * 8 + hlf * 4;
              const f32x4 a4 = *reinterpret_cast<const f32x4*>(smem + f32_pos(r, 2 * v + hlf) * 16);
              f32x4 vec = {0.f, 0.f, 0.f, 0.f};
              if constexpr (VEC) vec = *reinterpret_cast<const f32x4*>(ep.bias + n);
              float h4[4];
              rope_apply<VEC>(n, a4, vec, st, rope_tab(n, st, ep), ep, h4);
#pragma unroll
              for (int e = 0; e < 4; ++e) o[hlf * 4 + e] = h4[e];
            }
          }
          // whole tiles, or (per-head norms) rows and columns inside the output
          if (m0 + row < M && n0 + v * 8 < ncols) {
            const u32x2 lo = pack4_bf16(*reinterpret_cast<const float(*)[4]>(o));
            const u32x2 hi = pack4_bf16(*reinterpret_cast<const float(*)[4]>(o + 4));
            store_out16(y + (int64_t)(m0 + row) * ldy + n0 + v * 8, u32x4{lo[0], lo[1], hi[0], hi[1]});
          }
        }
      }
      return;
    } else if constexpr (EPI == EPI_ROPE) {
      // The angles of RB rows at a time are loaded before any of them is used, so
      // their latencies overlap (the lane's rows hold different tokens).
      constexpr int RB = FM >= 2 ? 2 : FM;
      static_assert(FM % RB == 0, "row batches");
      f32x4 bv[FN];
#pragma unroll
      for (int i = 0; i < FN; ++i) {
        bv[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        if constexpr (VEC) bv[i] = *reinterpret_cast<const f32x4*>(ep.bias + n0 + wn * TN + i * 16 + n_lane);
      }
#pragma unroll
      for (int jb = 0; jb < FM; jb += RB) {
        RopeTab tb[RB][FN];
#pragma unroll
        for (int jj = 0; jj < RB; ++jj)
#pragma unroll
          for (int i = 0; i < FN; ++i) tb[jj][i] = rope_tab(n0 + wn * TN + i * 16 + n_lane, sts[jb + jj], ep);
#pragma unroll
        for (int jj = 0; jj < RB; ++jj) {
          const int j = jb + jj;
          const int r = wm * TM + j * 16 + lrow;
          write_inv_rms(j, sts[j]);
#pragma unroll
          for (int i = 0; i < FN; ++i) {
            const int c = wn * TN + i * 16 + n_lane;
            stage4<UPR>(smem, r, c, rope4_bf16<VEC>(n0 + c, acc[i][j], bv[i], sts[j], tb[jj][i], ep));
          }
        }
      }
    } else
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      const int r = wm * TM + j * 16 + lrow;
      RowStat st;
      if constexpr (kRowData) st = sts[j];
      else st = row_stat_at<EPI>(ss[j], sa[j], ep, m0 + r, M);
      write_inv_rms(j, st);
      if constexpr (epi_is_glu(EPI)) {
#pragma unroll
        for (int i = 0; i < FN; i += 2) {
          const int c = wn * (TN / 2) + (i / 2) * 16 + n_lane;
          stage4<UPR>(smem, r, c, epi4_bf16<EPI, VEC>(n0 + c, acc[i][j], acc[i + 1][j], st, ep));
        }
      } else {
#pragma unroll
        for (int i = 0; i < FN; ++i) {
          const int c = wn * TN + i * 16 + n_lane;
          stage4<UPR>(smem, r, c, epi4_bf16<EPI, VEC>(n0 + c, acc[i][j], acc[i][j], st, ep));
        }
      }
    }
    __syncthreads();
    copy_tile_out<BM, UPR, NW * 64>(smem, y, ldy, m0, n0, threadIdx.x);
  };
  auto direct = [&](auto vec_tag) __attribute__((always_inline)) {
    constexpr bool VEC = decltype(vec_tag)::value;
    RowStat sts[kRowData ? FM : 1];
    row_stats(sts);
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      const int mb = m0 + wm * TM + j * 16;
      const int m = mb + lrow;
      RowStat st;
      if constexpr (kRowData) st = sts[j];
      else st = row_stat_at<EPI>(ss[j], sa[j], ep, m, M);
      write_inv_rms(j, st);
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
  // Workgroup-uniform: every wave takes the same branch (the staged path has barriers).
  if constexpr (EPI == EPI_HEADNORM) {
    staged(std::false_type{});
  } else {
    const bool whole = kStageable && m0 + BM <= M && n0 + OUT_COLS <= ncols && (ldy & 7) == 0;
    const bool vec = epi_vec<EPI>(ep) != nullptr;
    if constexpr (kStageable) {
      if (whole) {
        if (vec) staged(std::true_type{});
        else staged(std::false_type{});
        return;
      }
    }
    if (vec)
      direct(std::true_type{});
    else
      direct(std::false_type{});
  }
}

// LEAN: the automatically chosen tiles also have an instantiation without the
// activation lane check (KCHK = false), launched when K is a multiple of 64.
template <int BM, int BN, int WM, int WN, int STAGES, bool PF, int EPI, bool SPREAD = false, bool GS = false,
          bool LEAN = false, int KD = 1>
static hipError_t launch_prefill_cfg(const PrefillArgs& p) {
  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = (p.NP + BN - 1) / BN;
  const int nblocks = tiles_m * tiles_n;
  auto go = [&](auto kchk) {
    hipLaunchKernelGGL((prefill_bf16_kernel<BM, BN, WM, WN, STAGES, PF, EPI, SPREAD, GS, decltype(kchk)::value, KD>),
                       dim3(nblocks), dim3(WM * WN * 64), 0, p.stream, p.a, p.M, p.K, p.lda, p.ws, p.NP, p.KP,
                       p.ncols, p.y, p.ldy, p.ep, tiles_m, tiles_n);
  };
  if constexpr (LEAN) {
    if (p.K % kKPad == 0) {
      go(std::false_type{});
      return hipGetLastError();
    }
  }
  go(std::true_type{});
  return hipGetLastError();
}

// The automatically chosen configurations.
template <int BM, int BN, int WM, int WN, int EPI, bool SPREAD = false, bool GS = false, int KD = 1>
static hipError_t launch_auto_cfg(const PrefillArgs& p) {
  return launch_prefill_cfg<BM, BN, WM, WN, 4, true, EPI, SPREAD, GS, true, KD>(p);
}

// Shape-specialised tile choice (measured on MI355X).  The 256 x 256 tile with 8
// waves, register prefetch and transfers spread over the k block when it still
// yields at least one tile per compute unit.  Otherwise 128-row tiles with 8 waves, 128 or 96 columns wide, whichever
// fills the 256 compute units best (whole rounds of tiles); 96 is not used for a
// GLU, whose wave tiles must hold whole gate/up block pairs.
static int auto_tile(int M, int NP, bool glu) {
  constexpr int kCUs = 256;
  const int64_t big = ((int64_t)(M + 255) / 256) * ((NP + 255) / 256);
  if (big >= kCUs) return TILE_256x256_W8_PF_SP;
  if (glu) return TILE_128x128_W8T;
  const int64_t t128 = ((int64_t)(M + 127) / 128) * ((NP + 127) / 128);
  const int64_t t96 = ((int64_t)(M + 127) / 128) * ((NP + 95) / 96);
  // fill = tiles / (CUs x rounds); compare t96 * rounds128 against t128 * rounds96.
  const int64_t r128 = (t128 + kCUs - 1) / kCUs, r96 = (t96 + kCUs - 1) / kCUs;
  return t96 * r128 > t128 * r96 ? TILE_128x96_W8 : TILE_128x128_W8T;
}

// 64-deep ring steps on the 128-row tiles, for the core non-GLU kinds.
// Measured on MI355X (interleaved runs): 128 x 96 tiles 2048 x 4096 -> 1024
// -2.3%, 4096 x 5120 -> 576 -1.6%, 2048 x 576 -> 1536 -0.6%; 128 x 128 tiles
// 1024 x 4096 -> 4096 -4%, 512 x 8192 -> 8192 -6.6%, but 2048 x 576 -> 1536 +1%
// (and a GLU +2..+14% at any K).
constexpr int kK64MinK96 = 512;
constexpr int kK64MinK128 = 2048;

template <int EPI>
static hipError_t launch_prefill_epi(const PrefillArgs& p) {
  int tile = p.tile;
  if (tile == TILE_AUTO) {
    tile = auto_tile(p.M, p.NP, epi_is_glu(EPI));
    // Large shapes of the core RMS kinds (and the unfused baseline's GEMM) with K a multiple
    // of 64 take the 4-wave tile with the hand-scheduled k block.
    if constexpr (EPI == EPI_RMS || EPI == EPI_GLU || EPI == EPI_NONE) {
      if (!p.gs && tile == TILE_256x256_W8_PF_SP && p.K % kKPad == 0) tile = TILE_256x256;
    }
    if constexpr (EPI == EPI_RMS || EPI == EPI_LN || EPI == EPI_NONE) {
      if (!p.gs && tile == TILE_128x96_W8 && p.K >= kK64MinK96) tile = TILE_128x96_W8_K64;
      if (!p.gs && tile == TILE_128x128_W8T && p.K >= kK64MinK128) tile = TILE_128x128_W8T_K64;
    }
  }
  if constexpr (EPI == EPI_RMS || EPI == EPI_GLU) {
    if (p.gs) {  // run-time g: the automatically chosen tiles only
      switch (tile) {
        case TILE_256x256_W8_PF_SP: return launch_auto_cfg<256, 256, 2, 4, EPI, true, true>(p);
        case TILE_128x128_W8T: return launch_auto_cfg<128, 128, 4, 2, EPI, false, true>(p);
        case TILE_128x96_W8:
          if constexpr (epi_is_glu(EPI)) return launch_auto_cfg<128, 128, 4, 2, EPI, false, true>(p);
          else return launch_auto_cfg<128, 96, 4, 2, EPI, false, true>(p);
      }
      return hipErrorInvalidValue;
    }
  } else {
    if (p.gs) return hipErrorInvalidValue;
  }
  if constexpr (EPI == EPI_HEADNORM) {
    // Whole heads per tile: 256 columns, or 128 when that fills the chip better and
    // holds whole heads.
    if (tile == TILE_256x256_W8_PF_SP || p.ep.head_h > 128)
      return launch_auto_cfg<256, 256, 2, 4, EPI, true>(p);
    return launch_auto_cfg<128, 128, 4, 2, EPI>(p);
  } else if constexpr (EPI >= EPI_REGLU) {
    // The epilogue family beyond the core kinds is built for the automatically
    // chosen tiles only.
    switch (tile) {
      case TILE_256x256_W8_PF_SP: return launch_auto_cfg<256, 256, 2, 4, EPI, true>(p);
      case TILE_128x128_W8T: return launch_auto_cfg<128, 128, 4, 2, EPI>(p);
      case TILE_128x96_W8:
        if constexpr (epi_is_glu(EPI)) return launch_auto_cfg<128, 128, 2, 2, EPI>(p);
        else return launch_auto_cfg<128, 96, 4, 2, EPI>(p);
    }
    return hipErrorInvalidValue;
  } else {
  switch (tile) {
    case TILE_256x256: return launch_prefill_cfg<256, 256, 2, 2, 4, true, EPI, false, false, true>(p);  // asm steps when K % 64 == 0
    case TILE_128x128: return launch_prefill_cfg<128, 128, 2, 2, 4, true, EPI>(p);
    case TILE_256x256_W8: return launch_prefill_cfg<256, 256, 2, 4, 4, false, EPI>(p);
    case TILE_128x96_W8:
      if constexpr (epi_is_glu(EPI)) return launch_auto_cfg<128, 128, 2, 2, EPI>(p);
      else return launch_auto_cfg<128, 96, 4, 2, EPI>(p);
    case TILE_256x128: return launch_prefill_cfg<256, 128, 2, 2, 4, true, EPI>(p);
    case TILE_128x256: return launch_prefill_cfg<128, 256, 2, 2, 4, true, EPI>(p);
    case TILE_128x64: return launch_prefill_cfg<128, 64, 2, 2, 4, true, EPI>(p);
    case TILE_64x128: return launch_prefill_cfg<64, 128, 2, 2, 4, true, EPI>(p);
    case TILE_128x128_NOPF: return launch_prefill_cfg<128, 128, 2, 2, 4, false, EPI>(p);
    case TILE_256x256_W8_PF: return launch_prefill_cfg<256, 256, 2, 4, 4, true, EPI>(p);
    case TILE_256x256_W8_PF5: return launch_prefill_cfg<256, 256, 2, 4, 5, true, EPI>(p);
    case TILE_128x128_W8: return launch_prefill_cfg<128, 128, 2, 4, 4, true, EPI>(p);
    case TILE_128x128_W8T: return launch_auto_cfg<128, 128, 4, 2, EPI>(p);
    case TILE_128x96:
      // 48-column wave tiles cannot hold whole gate/up pairs: a GLU takes 128 x 128.
      if constexpr (epi_is_glu(EPI)) return launch_prefill_cfg<128, 128, 2, 2, 4, true, EPI>(p);
      else return launch_prefill_cfg<128, 96, 2, 2, 4, true, EPI>(p);
    case TILE_256x256_W8_PF_SP: return launch_auto_cfg<256, 256, 2, 4, EPI, true>(p);
    case TILE_128x128_W8T_SP: return launch_prefill_cfg<128, 128, 4, 2, 4, true, EPI, true>(p);
    case TILE_128x96_W8_SP:
      if constexpr (epi_is_glu(EPI)) return launch_prefill_cfg<128, 128, 4, 2, 4, true, EPI, true>(p);
      else return launch_prefill_cfg<128, 96, 4, 2, 4, true, EPI, true>(p);
    case TILE_128x96_W8_K64:
      if constexpr (epi_is_glu(EPI)) return launch_auto_cfg<128, 128, 4, 2, EPI, false, false, 2>(p);
      else return launch_auto_cfg<128, 96, 4, 2, EPI, false, false, 2>(p);
    case TILE_128x128_W8T_K64: return launch_auto_cfg<128, 128, 4, 2, EPI, false, false, 2>(p);
  }
  return hipErrorInvalidValue;
  }
}

hipError_t launch_prefill_bf16(const PrefillArgs& p) {
  switch (p.epi) {
    case EPI_RMS: return launch_prefill_epi<EPI_RMS>(p);
    case EPI_GLU: return launch_prefill_epi<EPI_GLU>(p);
    case EPI_LN: return launch_prefill_epi<EPI_LN>(p);
    case EPI_NONE: return launch_prefill_epi<EPI_NONE>(p);
    case EPI_GLU_NOSCALE: return launch_prefill_epi<EPI_GLU_NOSCALE>(p);
    case EPI_REGLU: return launch_prefill_epi<EPI_REGLU>(p);
    case EPI_BILINEAR: return launch_prefill_epi<EPI_BILINEAR>(p);
    case EPI_GLU_DEFER: return launch_prefill_epi<EPI_GLU_DEFER>(p);
    case EPI_RELU_DEFER: return launch_prefill_epi<EPI_RELU_DEFER>(p);
    case EPI_ROWSCALE: return launch_prefill_epi<EPI_ROWSCALE>(p);
    case EPI_ROPE: return launch_prefill_epi<EPI_ROPE>(p);
    case EPI_HEADNORM: return launch_prefill_epi<EPI_HEADNORM>(p);
  }
  return hipErrorInvalidValue;
}

}  // namespace fn
