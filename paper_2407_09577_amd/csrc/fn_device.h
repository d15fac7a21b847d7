// Device-side building blocks shared by the FlashNorm gfx950 kernels.
//
// Packed weight layout ("fragment-major"), written by fold_weights and read by
// every bf16 kernel.  A logical column n is first mapped to a packed column p
// (identity for a linear layer; for a GLU, gate feature f goes to
// 32*(f/16) + f%16 and up feature f to 32*(f/16) + 16 + f%16, so a gate block of
// 16 columns is immediately followed by its up block).  Packed columns are padded
// to NP (a multiple of 16) and rows to KP (a multiple of 64) with zeros.  The
// packed buffer is a sequence of 1 KiB fragments, k-block major:
//   fragment (cb, kb) = columns [16 cb, 16 cb + 16) x rows [32 kb, 32 kb + 32),
//   at byte offset (kb * NP/16 + cb) * 1024; inside it, lane L = 16 * ((k%32)/8) + p%16
//   holds the 8 consecutive rows k..k+7 (k%8 == 0) of column p as 16 bytes.
// That is exactly the per-lane operand of one v_mfma_f32_16x16x32_bf16, so a
// wave moves a fragment global -> LDS -> registers with one 16-byte access per
// lane.  All column blocks of one 32-row k block are contiguous, so workgroups
// that advance through K together read one contiguous region at a time (spread
// over every HBM channel), and a prefill tile's weight columns for one k block
// are one contiguous run.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fn {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
typedef __attribute__((ext_vector_type(2))) unsigned int u32x2;

constexpr int kFragBytes = 1024;  // one 16 x 32 bf16 operand fragment
constexpr int kKB = 32;           // k extent of a fragment
constexpr int kKPad = 64;         // packed K is padded to this
constexpr int kNPad = 16;         // packed columns are padded to this
constexpr int kDtypeF32 = 0;      // element type codes of the C ABI
constexpr int kDtypeBf16 = 1;

// dword 3 of a CDNA buffer resource: 32-bit raw data, no swizzle, range checked.
constexpr int kBufferRsrcWord3 = 0x00020000;
// A voffset this large is outside every buffer the kernels build (all extents < 2^31),
// so the load returns zeros.
constexpr unsigned kOobOffset = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           kBufferRsrcWord3);
}

typedef __attribute__((ext_vector_type(4))) int i32x4;

// Buffer resource as four SGPRs, for the LDS-DMA loads issued through inline asm.
__device__ __forceinline__ i32x4 make_rsrc_sgpr(const void* base, uint32_t bytes) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  i32x4 r;
  r[0] = (int)(uint32_t)p;
  r[1] = (int)(uint32_t)(p >> 32) & 0xffff;  // stride 0
  r[2] = (int)bytes;                          // num_records (bytes)
  r[3] = kBufferRsrcWord3;
  r[0] = __builtin_amdgcn_readfirstlane(r[0]);
  r[1] = __builtin_amdgcn_readfirstlane(r[1]);
  r[2] = __builtin_amdgcn_readfirstlane(r[2]);
  r[3] = __builtin_amdgcn_readfirstlane(r[3]);
  return r;
}

// 16 bytes per lane from a range-checked buffer straight into LDS: lane i of the
// wave writes lds_base + 16 * i; out-of-range lanes write zeros.  Issued through
// inline asm so the compiler does not add a conservative wait for these writes
// before unrelated LDS reads: the kernels order them with explicit vmcnt waits
// and barriers.  lds_base must be wave-uniform.  M0 is written here without being
// declared (the compiler reserves it and rejects the clobber); these kernels use
// M0 for nothing else, which tests/test_lds_dma_m0.py checks on the built code
// object (every M0 write feeds the transfer right after it, no implicit M0 reader).
__device__ __forceinline__ void load_lds16(i32x4 rsrc, const void* lds_base, unsigned voffset) {
  const unsigned m0 = __builtin_amdgcn_readfirstlane(
      (unsigned)(uintptr_t)(const __attribute__((address_space(3))) void*)lds_base);
  // The descriptor is wave-uniform; re-assert it so it is allocated to SGPRs.
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane(rsrc[0]);
  r[1] = __builtin_amdgcn_readfirstlane(rsrc[1]);
  r[2] = __builtin_amdgcn_readfirstlane(rsrc[2]);
  r[3] = __builtin_amdgcn_readfirstlane(rsrc[3]);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(m0), "v"(voffset), "s"(r)
               : "memory");
}

// As load_lds16, with the LDS destination given as a 32-bit LDS byte address.
__device__ __forceinline__ void load_lds16_at(i32x4 rsrc, unsigned lds_addr, unsigned voffset) {
  const unsigned m0 = __builtin_amdgcn_readfirstlane(lds_addr);
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane(rsrc[0]);
  r[1] = __builtin_amdgcn_readfirstlane(rsrc[1]);
  r[2] = __builtin_amdgcn_readfirstlane(rsrc[2]);
  r[3] = __builtin_amdgcn_readfirstlane(rsrc[3]);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(m0), "v"(voffset), "s"(r)
               : "memory");
}

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ unsigned lds_addr(const void* p) {
  return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Cache-policy operand of the buffer loads: the non-temporal hint, for data
// streamed exactly once (the decode weight stream).
constexpr int kCachePolicyNT = 2;

// 16 bytes per lane from a range-checked buffer into registers.
template <int CPOL = 0>
__device__ __forceinline__ u32x4 load_buf16(__amdgpu_buffer_rsrc_t rsrc, unsigned voffset) {
  return __builtin_amdgcn_raw_buffer_load_b128(rsrc, voffset, 0, CPOL);
}

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding:
// vmcnt[3:0] and [15:14], expcnt[6:4], lgkmcnt[11:8]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}


// fp32 -> bf16 bits, round to nearest even (NaN stays NaN).
__device__ __forceinline__ unsigned f32_to_bf16_bits(float f) {
  unsigned u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ unsigned pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

// sum of squares and plain sum of the 8 bf16 values of one operand fragment lane,
// via packed bf16 dot products accumulated in fp32.
__device__ __forceinline__ float sumsq8(const bf16x8& v, float acc) {
  bf16x2 p0 = {v[0], v[1]}, p1 = {v[2], v[3]}, p2 = {v[4], v[5]}, p3 = {v[6], v[7]};
  acc = __builtin_amdgcn_fdot2_f32_bf16(p0, p0, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(p1, p1, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(p2, p2, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(p3, p3, acc, false);
  return acc;
}

// bf16 halves of a 32-bit word, widened exactly to fp32.
__device__ __forceinline__ float bf16_lo(unsigned w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(unsigned w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float sum8(const bf16x8& v, float acc) {
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
  bf16x2 p0 = {v[0], v[1]}, p1 = {v[2], v[3]}, p2 = {v[4], v[5]}, p3 = {v[6], v[7]};
  acc = __builtin_amdgcn_fdot2_f32_bf16(p0, one, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(p1, one, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(p2, one, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(p3, one, acc, false);
  return acc;
}

__device__ __forceinline__ float silu(float t) { return t / (1.0f + __expf(-t)); }

// Epilogue kinds of the fused kernels.  s = 1/RMSe(a) = rsqrt(eps + sum a^2/K).
enum Epi : int {
  EPI_RMS = 0,          // y = acc * s (+ bias)
  EPI_GLU = 1,          // out = silu(s * gate) * (s * up)                  (Fig. 3(a))
  EPI_LN = 2,           // y = (acc - mu * colsum) * rstd + c*
  EPI_NONE = 3,         // y = acc                      (unfused baseline GEMM)
  EPI_GLU_NOSCALE = 4,  // out = silu(gate) * up        (unfused baseline GEMM)
  EPI_REGLU = 5,        // out = relu(gate) * up * s^2  (both scales merged: 1/MSe)
  EPI_BILINEAR = 6,     // out = gate * up * s^2
  EPI_GLU_DEFER = 7,    // out = silu(s * gate) * up, s exported        (Fig. 3(b))
  EPI_RELU_DEFER = 8,   // y = relu(acc), s exported                    (Fig. 2(b))
  EPI_ROWSCALE = 9,     // y = acc * row_scale[m]   (applies a deferred scale)
  EPI_ROPE = 10,        // fused QKV: RoPE on Q and K with s folded into the tables (Fig. 5(b))
  EPI_HEADNORM = 11,    // fused QKV: per-head RMSNorm of Q, K (and V), input scale dropped (Prop. 3)
};

constexpr bool epi_is_glu(int e) {
  return e == EPI_GLU || e == EPI_GLU_NOSCALE || e == EPI_REGLU || e == EPI_BILINEAR || e == EPI_GLU_DEFER;
}
constexpr bool epi_needs_ss(int e) {
  return e == EPI_RMS || e == EPI_GLU || e == EPI_LN || e == EPI_REGLU || e == EPI_BILINEAR ||
         e == EPI_GLU_DEFER || e == EPI_RELU_DEFER || e == EPI_ROPE || e == EPI_HEADNORM;
}
// Kinds whose per-row scale s = 1/RMSe(a) can be written to the inv_rms output.
constexpr bool epi_exports_s(int e) {
  return e == EPI_RMS || e == EPI_GLU || e == EPI_GLU_DEFER || e == EPI_RELU_DEFER || e == EPI_ROPE ||
         e == EPI_HEADNORM;
}

struct EpiArgs {
  float eps;
  float inv_k;          // 1/K
  double inv_kd;        // 1/K in fp64 (LayerNorm statistics)
  const float* bias;    // EPI_RMS: optional [N]
  const float* colsum;  // EPI_LN: [N]
  const float* cstar;   // EPI_LN: optional [N]
  float* inv_rms;       // optional [M] output of s (kinds with epi_exports_s)
  const float* row_scale;  // EPI_ROWSCALE: [M]
  const float* g_rt;       // run-time normalisation weight [K] (unfolded W), or nullptr
  // Fused QKV kinds (EPI_ROPE, EPI_HEADNORM): output columns [0, q_end) are Q heads,
  // [q_end, k_end) K heads, the rest V; heads are head_h wide; Q is also multiplied by
  // q_scale.  Row m is a token at position rope_pos[m], whose angles are rope_cos /
  // rope_sin [rope_P][head_h / 2] (EPI_HEADNORM: rope_pos == nullptr, no rotation).
  const int* rope_pos;
  const float* rope_cos;
  const float* rope_sin;
  int head_h, rope_P, q_end, k_end;
  float head_inv_h;  // 1/h in fp32
  float q_scale;
  // EPI_HEADNORM: per-head norm weights [h] of Q, K and (optional, QKV-normalization) V,
  // and the heads' epsilon.
  const float* hn_gq;
  const float* hn_gk;
  const float* hn_gv;
  float hn_eps;
};

}  // namespace fn
