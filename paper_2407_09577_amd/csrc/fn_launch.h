// Host-side launch interface between the C ABI (api.hip) and the kernel files.
// Arguments reaching these functions have already been validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fn_device.h"

namespace fn {

// Prefill tile configurations (selected automatically, or forced through the
// high byte of the path argument for tuning).
enum Tile : int {
  TILE_AUTO = 0,
  TILE_256x256 = 1,       // 4 waves of 128 x 128, 4-stage ring, register prefetch; hand-scheduled
                          // k blocks (inline asm) when K is a multiple of 64
  TILE_128x128 = 2,       // 4 waves of 64 x 64, 4-stage ring, register prefetch
  TILE_256x256_W8 = 3,    // 8 waves of 128 x 64, 4-stage ring
  TILE_128x96_W8 = 4,     // 8 waves of 32 x 48, register prefetch (GLU: 128 x 128)
  TILE_256x128 = 5,       // 4 waves of 128 x 64
  TILE_128x256 = 6,       // 4 waves of 64 x 128
  TILE_128x64 = 7,        // 4 waves of 64 x 32
  TILE_64x128 = 8,        // 4 waves of 32 x 64
  TILE_128x128_NOPF = 9,  // as TILE_128x128 without register prefetch
  TILE_256x256_W8_PF = 10,   // 8 waves of 128 x 64, 4-stage ring, register prefetch
  TILE_256x256_W8_PF5 = 11,  // 8 waves of 128 x 64, 5-stage ring, register prefetch
  TILE_128x128_W8 = 12,      // 8 waves of 64 x 32, register prefetch
  TILE_128x128_W8T = 13,     // 8 waves of 32 x 64, register prefetch
  TILE_128x96 = 14,          // 4 waves of 64 x 48, register prefetch (GLU: 128 x 128)
  TILE_256x256_W8_PF_SP = 15,  // TILE_256x256_W8_PF, transfers spread over the k block
  TILE_128x128_W8T_SP = 16,    // TILE_128x128_W8T, transfers spread over the k block
  TILE_128x96_W8_SP = 17,      // TILE_128x96_W8, transfers spread over the k block
  TILE_128x96_W8_K64 = 18,     // TILE_128x96_W8 with 64-deep ring steps (GLU: 128 x 128)
  TILE_128x128_W8T_K64 = 19,   // TILE_128x128_W8T with 64-deep ring steps
  TILE_COUNT
};

// Packed-layout geometry shared by the fold and the kernels.
inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
// Packed column count: N for a linear layer, 2 * round_up(F, 16) for a GLU with N = 2F.
inline int64_t packed_cols(int64_t N, int glu) {
  return glu ? 2 * round_up(N / 2, kNPad) : round_up(N, kNPad);
}
inline int64_t packed_rows(int64_t K) { return round_up(K, kKPad); }

// Largest K of the bf16 run-time-g prefill path: g is staged once in LDS
// (kGsMaxK + 64 floats beside a 128 KiB ring fill the 160 KiB).
constexpr int kGsMaxK = 8128;

struct PrefillArgs {
  const __bf16* a;
  int M, K, lda;
  const __bf16* ws;
  int NP, KP;
  int ncols;  // logical output columns (N, or F for a GLU)
  __bf16* y;
  int ldy;
  int epi;
  int tile;
  EpiArgs ep;
  hipStream_t stream;
  bool gs;  // run-time g (ep.g_rt) applied to the activations; unfolded W
};
hipError_t launch_prefill_bf16(const PrefillArgs& p);

struct DecodeArgs {
  const __bf16* a;
  int M, K, lda;
  const __bf16* ws;
  int NP, KP;
  int ncols;
  __bf16* y;
  int ldy;
  int epi;
  int cfg;  // decode configuration (0 = automatic), see launch_decode_bf16
  EpiArgs ep;
  hipStream_t stream;
  bool gs;  // run-time g (ep.g_rt) applied to the activations; unfolded W
};
hipError_t launch_decode_bf16(const DecodeArgs& p);
constexpr int kDecodeCfgCount = 24;

struct F32Args {
  const float* a;
  int M, K, lda;
  const float* ws;  // [KP][NP] row-major fp32, columns in packed order
  int NP, KP;
  int ncols;
  float* y;
  int ldy;
  int epi;
  EpiArgs ep;
  hipStream_t stream;
  bool gs;      // run-time g (ep.g_rt) applied to the activations; unfolded W
  int cfg = 0;  // tile configuration (0 = automatic), see launch_f32
};
hipError_t launch_f32(const F32Args& p);
// fp32 tile configurations: 0 automatic, 1 = 64-row tiles, 2 = 16-row tiles with four k groups,
// 3 = 16-row tiles 4 to 64 columns wide with K split over up to 64 thread groups.
constexpr int kF32CfgCount = 4;

struct FoldArgs {
  const void* W;
  int64_t sk, sn;  // element (k, n) of the logical weight is W[k * sk + n * sn]
  int w_dtype;  // 0 fp32, 1 bf16
  const float* g;
  const float* beta;
  int64_t K, N;
  int glu;
  void* ws;
  int ws_dtype;
  float* colsum;
  float* cstar;
  hipStream_t stream;
};
hipError_t launch_fold(const FoldArgs& p);
hipError_t launch_unpack(const void* ws, int64_t K, int64_t N, int glu, int ws_dtype, void* out,
                         int64_t ldo, hipStream_t stream);

// Unfused baseline normalisation: x = RMSNorm(a; g) or LayerNorm(a; g, beta), dtype of a.
hipError_t launch_norm_rows(const void* a, int M, int K, int lda, int dtype, const float* g,
                            const float* beta, float eps, void* x, int ldx, hipStream_t stream);

// Unfused baseline per-head norms (+ RoPE): the first ncols columns of y in place
// (EPI_HEADNORM arguments in ep; ncols a multiple of the head width).
hipError_t launch_headnorm_rows(void* y, int M, int ldy, int ncols, const EpiArgs& ep, hipStream_t stream);

// Unfused baseline RoPE: rotate the Q and K heads (first qk columns) of y in place.
hipError_t launch_rope_rows(void* y, int M, int ldy, int dtype, int qk, int q_end, int h, const int* pos,
                            const float* cos_tab, const float* sin_tab, int P, float q_scale, hipStream_t stream);

// MLA latent pass (Sec. 3.3): in place over y after the projection, the latent
// RMSNorm of the first L columns (u * rsqrt(mean(u^2) + eps_lat s^2) * g_lat, s from
// s_row or 1 without it) and RoPE of the R columns after them (one head of width R).
// L % 8 == 0, L <= 2048; R % 8 == 0, R <= 512; y rows 16-byte aligned.
hipError_t launch_mla_latent_rows(void* y, int M, int ldy, int dtype, int L, int R, const float* g_lat,
                                  float eps_lat, const float* s_row, const int* pos, const float* cos_tab,
                                  const float* sin_tab, int P, hipStream_t stream);

}  // namespace fn
