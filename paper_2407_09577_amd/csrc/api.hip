// C ABI of the FlashNorm library: argument validation (before anything is
// launched), shape-specialised kernel selection, and launches on the caller's
// stream.  No allocation, no synchronisation, no mutable global state.
#include <math.h>
#include <stdint.h>

#include <mutex>

#include "flashnorm.h"
#include "fn_launch.h"

// The one piece of library-owned device memory: the workspace of
// baseline_rmsnorm_linear_noalloc, for callers that cannot allocate (see the header).
// Every GPU the library runs on holds its own copy until the process ends.  In host
// code this name is only a handle: its device address comes from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[FN_NOALLOC_SCRATCH_BYTES];

namespace {

// Device address of `scratch` on the current device, looked up once per device (with
// that device current) and kept; nullptr if the lookup fails.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

using fn::EpiArgs;

constexpr int64_t kMaxLd = int64_t(1) << 21;    // leading dimensions, K (keeps tile extents < 2^31)
constexpr int64_t kMaxRows = int64_t(1) << 30;  // M, N
// Packed weight buffer: the matrix-core kernels address it with 32-bit byte
// offsets and use offsets >= 2^31 as out-of-range (zero-returning) loads.
constexpr int64_t kMaxPackedBytes = (int64_t(1) << 31) - 1;
// Strides of the weight view fold_weights reads: with K <= 2^21 and N <= 2^30 every
// element offset stays below 2^62.
constexpr int64_t kMaxFoldStrideK = int64_t(1) << 40;
constexpr int64_t kMaxFoldStrideN = int64_t(1) << 31;

int64_t packed_bytes(int64_t K, int64_t N, bool glu, int64_t elem) {
  return fn::packed_rows(K) * fn::packed_cols(N, glu) * elem;
}

bool dtype_ok(int d) { return d == FN_F32 || d == FN_BF16; }
int64_t elem_size(int d) { return d == FN_BF16 ? 2 : 4; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
int64_t row_align(int d) { return 16 / elem_size(d); }

bool overlaps(const void* p, int64_t pbytes, const void* q, int64_t qbytes) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(p), b0 = reinterpret_cast<uintptr_t>(q);
  return a0 < b0 + (uintptr_t)qbytes && b0 < a0 + (uintptr_t)pbytes;
}

int64_t extent_bytes(int64_t rows, int64_t cols, int64_t ld, int dtype) {
  return rows > 0 ? ((rows - 1) * ld + cols) * elem_size(dtype) : 0;
}

// Common checks of an activation-like operand [M, K] with leading dimension ld.
int check_matrix(const void* p, int64_t M, int64_t K, int64_t ld, int dtype, bool required) {
  if (M < 0 || K <= 0 || M > kMaxRows) return FN_ERR_SHAPE;
  if (ld < K) return FN_ERR_SHAPE;
  if (ld > kMaxLd) return FN_ERR_SIZE;
  if (required && M > 0 && !p) return FN_ERR_NULL;
  if (!aligned16(p) || ld % row_align(dtype)) return FN_ERR_ALIGN;
  return FN_OK;
}

int check_eps(float eps) { return (isfinite(eps) && eps >= 0.0f) ? FN_OK : FN_ERR_VALUE; }

int status_of(hipError_t e) { return e == hipSuccess ? FN_OK : FN_ERR_HIP; }

struct OpDesc {
  const void* a;
  int64_t M, K, lda;
  int dtype;
  const void* ws;
  int64_t ncols;  // N, or F for a GLU
  int glu;
  void* y;
  int64_t ldy;
  int epi;
  EpiArgs ep;
  int path;
  hipStream_t stream;
  bool gs = false;  // run-time g in ep.g_rt, unfolded packed W
};

// Validation shared by the three fused ops (and the baselines' matrix multiply).
int validate_op(const OpDesc& d, int y_dtype) {
  if (!dtype_ok(d.dtype) || !dtype_ok(y_dtype)) return FN_ERR_DTYPE;
  if (y_dtype != d.dtype) return FN_ERR_DTYPE;
  const int base_path = d.path & 0xff, tile = d.path >> FN_PATH_TILE_SHIFT;
  if (base_path < FN_PATH_AUTO || base_path > FN_PATH_DECODE) return FN_ERR_VALUE;
  if (tile < 0 || tile >= (base_path == FN_PATH_DECODE ? fn::kDecodeCfgCount
                            : d.dtype == FN_F32        ? fn::kF32CfgCount
                                                       : (int)fn::TILE_COUNT))
    return FN_ERR_VALUE;
  if (d.K > kMaxLd) return FN_ERR_SIZE;
  if (d.K % (d.dtype == FN_BF16 ? 8 : 4)) return FN_ERR_SHAPE;
  int s = check_matrix(d.a, d.M, d.K, d.lda, d.dtype, true);
  if (s) return s;
  if (d.ncols <= 0 || d.ncols > kMaxRows) return FN_ERR_SHAPE;
  s = check_matrix(d.y, d.M, d.ncols, d.ldy, d.dtype, true);
  if (s) return s;
  if (packed_bytes(d.K, d.glu ? 2 * d.ncols : d.ncols, d.glu, elem_size(d.dtype)) > kMaxPackedBytes)
    return FN_ERR_SIZE;
  if (!d.ws) return FN_ERR_NULL;
  if (!aligned16(d.ws)) return FN_ERR_ALIGN;
  s = check_eps(d.ep.eps);
  if (s) return s;
  if (d.M > 0) {
    const int64_t ybytes = extent_bytes(d.M, d.ncols, d.ldy, d.dtype);
    const int64_t N = d.glu ? 2 * d.ncols : d.ncols;
    const int64_t wbytes = fold_weights_size(d.K, N, d.glu ? FN_LAYOUT_GLU : FN_LAYOUT_LINEAR, d.dtype);
    if (overlaps(d.y, ybytes, d.a, extent_bytes(d.M, d.K, d.lda, d.dtype))) return FN_ERR_ALIAS;
    if (overlaps(d.y, ybytes, d.ws, wbytes)) return FN_ERR_ALIAS;
  }
  if (base_path == FN_PATH_DECODE && (d.dtype != FN_BF16 || d.M > FN_DECODE_MAX_M)) return FN_ERR_UNSUPPORTED;
  return FN_OK;
}

int run_op(const OpDesc& d) {
  if (d.M == 0) return FN_OK;
  const int64_t N = d.glu ? 2 * d.ncols : d.ncols;
  const int NP = (int)fn::packed_cols(N, d.glu), KP = (int)fn::packed_rows(d.K);
  if (d.dtype == FN_F32) {
    fn::F32Args p{(const float*)d.a, (int)d.M, (int)d.K, (int)d.lda, (const float*)d.ws, NP, KP,
                  (int)d.ncols, (float*)d.y, (int)d.ldy, d.epi, d.ep, d.stream, d.gs};
    p.cfg = d.path >> FN_PATH_TILE_SHIFT;
    return status_of(fn::launch_f32(p));
  }
  const int base_path = d.path & 0xff;
  // The per-head norms need whole heads in one workgroup: always the tile kernel.
  const bool decode = d.epi != fn::EPI_HEADNORM &&
                      (base_path == FN_PATH_DECODE || (base_path == FN_PATH_AUTO && d.M <= FN_DECODE_MAX_M));
  if (decode) {
    fn::DecodeArgs p{(const __bf16*)d.a, (int)d.M, (int)d.K, (int)d.lda, (const __bf16*)d.ws, NP, KP,
                     (int)d.ncols, (__bf16*)d.y, (int)d.ldy, d.epi, d.path >> FN_PATH_TILE_SHIFT, d.ep,
                     d.stream, d.gs};
    return status_of(fn::launch_decode_bf16(p));
  }
  fn::PrefillArgs p{(const __bf16*)d.a, (int)d.M, (int)d.K, (int)d.lda, (const __bf16*)d.ws, NP, KP,
                    (int)d.ncols, (__bf16*)d.y, (int)d.ldy, d.epi, d.path >> FN_PATH_TILE_SHIFT, d.ep,
                    d.stream, d.gs};
  return status_of(fn::launch_prefill_bf16(p));
}

EpiArgs make_ep(float eps, int64_t K) {
  EpiArgs ep{};
  ep.eps = eps;
  ep.inv_k = 1.0f / (float)K;
  ep.inv_kd = 1.0 / (double)K;
  return ep;
}

}  // namespace

extern "C" {

size_t fold_weights_size(int64_t K, int64_t N, int layout, int ws_dtype) {
  if (K <= 0 || N <= 0 || K > kMaxLd || N > kMaxRows || !dtype_ok(ws_dtype)) return 0;
  if (layout != FN_LAYOUT_LINEAR && layout != FN_LAYOUT_GLU) return 0;
  if (layout == FN_LAYOUT_GLU && N % 2) return 0;
  const int64_t bytes = packed_bytes(K, N, layout == FN_LAYOUT_GLU, elem_size(ws_dtype));
  return bytes > kMaxPackedBytes ? 0 : (size_t)bytes;
}

int fold_weights(const void* W, int64_t stride_k, int64_t stride_n, int w_dtype, const float* g,
                 const float* beta, int64_t K, int64_t N, int layout, void* W_star, int ws_dtype,
                 float* colsum, float* c_star, void* stream) {
  if (!dtype_ok(w_dtype) || !dtype_ok(ws_dtype)) return FN_ERR_DTYPE;
  if (layout != FN_LAYOUT_LINEAR && layout != FN_LAYOUT_GLU) return FN_ERR_VALUE;
  if (K <= 0 || N <= 0 || stride_k < 0 || stride_n < 0 || (layout == FN_LAYOUT_GLU && N % 2))
    return FN_ERR_SHAPE;
  if (K > kMaxLd || N > kMaxRows || stride_k >= kMaxFoldStrideK || stride_n >= kMaxFoldStrideN)
    return FN_ERR_SIZE;
  if (packed_bytes(K, N, layout == FN_LAYOUT_GLU, elem_size(ws_dtype)) > kMaxPackedBytes) return FN_ERR_SIZE;
  if (!W || !W_star) return FN_ERR_NULL;
  if (c_star && !beta) return FN_ERR_NULL;
  if (layout == FN_LAYOUT_GLU && (colsum || c_star)) return FN_ERR_UNSUPPORTED;
  if (!aligned16(W_star) || (reinterpret_cast<uintptr_t>(W) % elem_size(w_dtype))) return FN_ERR_ALIGN;
  const int64_t wsb = (int64_t)fold_weights_size(K, N, layout, ws_dtype);
  // Bytes spanned by the strided view (the largest element offset is below 2^62).
  const int64_t wext = ((K - 1) * stride_k + (N - 1) * stride_n + 1) * elem_size(w_dtype);
  if (overlaps(W_star, wsb, W, wext)) return FN_ERR_ALIAS;
  fn::FoldArgs p{W, stride_k, stride_n, w_dtype, g, beta, K, N, layout == FN_LAYOUT_GLU, W_star, ws_dtype,
                 colsum, c_star, (hipStream_t)stream};
  return status_of(fn::launch_fold(p));
}

int unpack_weights(const void* W_star, int64_t K, int64_t N, int layout, int ws_dtype, void* out,
                   int64_t ldo, void* stream) {
  if (!dtype_ok(ws_dtype)) return FN_ERR_DTYPE;
  if (layout != FN_LAYOUT_LINEAR && layout != FN_LAYOUT_GLU) return FN_ERR_VALUE;
  if (K <= 0 || N <= 0 || ldo < N || (layout == FN_LAYOUT_GLU && N % 2)) return FN_ERR_SHAPE;
  if (K > kMaxLd || N > kMaxRows) return FN_ERR_SIZE;
  if (packed_bytes(K, N, layout == FN_LAYOUT_GLU, elem_size(ws_dtype)) > kMaxPackedBytes) return FN_ERR_SIZE;
  if (!W_star || !out) return FN_ERR_NULL;
  if (!aligned16(W_star) || (reinterpret_cast<uintptr_t>(out) % elem_size(ws_dtype))) return FN_ERR_ALIGN;
  const int64_t wsb = (int64_t)fold_weights_size(K, N, layout, ws_dtype);
  if (overlaps(out, extent_bytes(K, N, ldo, ws_dtype), W_star, wsb)) return FN_ERR_ALIAS;
  return status_of(fn::launch_unpack(W_star, K, N, layout == FN_LAYOUT_GLU, ws_dtype, out, ldo,
                                     (hipStream_t)stream));
}

int flashnorm_linear_ex(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const void* W_star,
                        int64_t N, float eps, const float* bias, void* y, int64_t ldy, int y_dtype,
                        float* inv_rms, int path, void* stream) {
  OpDesc d{a, M, K, lda, a_dtype, W_star, N, 0, y, ldy, fn::EPI_RMS, make_ep(eps, K), path, (hipStream_t)stream};
  d.ep.bias = bias;
  d.ep.inv_rms = inv_rms;
  int s = validate_op(d, y_dtype);
  if (s) return s;
  if (!aligned16(bias)) return FN_ERR_ALIGN;
  return run_op(d);
}

int flashnorm_linear(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const void* W_star,
                     int64_t N, float eps, const float* bias, void* y, int64_t ldy, int y_dtype,
                     float* inv_rms, void* stream) {
  return flashnorm_linear_ex(a, M, K, lda, a_dtype, W_star, N, eps, bias, y, ldy, y_dtype, inv_rms,
                             FN_PATH_AUTO, stream);
}

int flashnorm_glu_ex(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const void* W_star_gu,
                     int64_t F, float eps, void* out, int64_t ldo, int out_dtype, int path, void* stream) {
  OpDesc d{a, M, K, lda, a_dtype, W_star_gu, F, 1, out, ldo, fn::EPI_GLU, make_ep(eps, K), path,
           (hipStream_t)stream};
  int s = validate_op(d, out_dtype);
  if (s) return s;
  return run_op(d);
}

int flashnorm_glu(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const void* W_star_gu,
                  int64_t F, float eps, void* out, int64_t ldo, int out_dtype, void* stream) {
  return flashnorm_glu_ex(a, M, K, lda, a_dtype, W_star_gu, F, eps, out, ldo, out_dtype, FN_PATH_AUTO,
                          stream);
}

int flashnorm_layernorm_linear_ex(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                                  const void* W_star, const float* colsum, const float* c_star, int64_t N,
                                  float eps, void* y, int64_t ldy, int y_dtype, int path, void* stream) {
  OpDesc d{a, M, K, lda, a_dtype, W_star, N, 0, y, ldy, fn::EPI_LN, make_ep(eps, K), path, (hipStream_t)stream};
  d.ep.colsum = colsum;
  d.ep.cstar = c_star;
  int s = validate_op(d, y_dtype);
  if (s) return s;
  if (!colsum) return FN_ERR_NULL;
  if (!aligned16(colsum) || !aligned16(c_star)) return FN_ERR_ALIGN;
  return run_op(d);
}

int flashnorm_layernorm_linear(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                               const void* W_star, const float* colsum, const float* c_star, int64_t N,
                               float eps, void* y, int64_t ldy, int y_dtype, void* stream) {
  return flashnorm_layernorm_linear_ex(a, M, K, lda, a_dtype, W_star, colsum, c_star, N, eps, y, ldy,
                                       y_dtype, FN_PATH_AUTO, stream);
}

// The epilogue family beyond the core kinds runs with the automatic configuration
// of the chosen path only.
static int check_auto_config(int path) {
  return (path >> FN_PATH_TILE_SHIFT) ? FN_ERR_UNSUPPORTED : FN_OK;
}

int flashnorm_glu_act(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const void* W_star_gu,
                      int64_t F, float eps, int act, void* out, int64_t ldo, int out_dtype, float* inv_rms,
                      int path, void* stream) {
  int epi;
  switch (act) {
    case FN_GLU_SWIGLU: epi = fn::EPI_GLU; break;
    case FN_GLU_REGLU: epi = fn::EPI_REGLU; break;
    case FN_GLU_BILINEAR: epi = fn::EPI_BILINEAR; break;
    case FN_GLU_SWIGLU_DEFER_UP: epi = fn::EPI_GLU_DEFER; break;
    default: return FN_ERR_VALUE;
  }
  OpDesc d{a, M, K, lda, a_dtype, W_star_gu, F, 1, out, ldo, epi, make_ep(eps, K), path, (hipStream_t)stream};
  d.ep.inv_rms = inv_rms;
  int s = validate_op(d, out_dtype);
  if (s) return s;
  if ((s = check_auto_config(path))) return s;
  if (act == FN_GLU_SWIGLU_DEFER_UP && M > 0 && !inv_rms) return FN_ERR_NULL;
  if ((act == FN_GLU_REGLU || act == FN_GLU_BILINEAR) && inv_rms) return FN_ERR_VALUE;
  return run_op(d);
}

int flashnorm_linear_relu(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const void* W_star,
                          int64_t N, float eps, void* y, int64_t ldy, int y_dtype, float* inv_rms, int path,
                          void* stream) {
  OpDesc d{a, M, K, lda, a_dtype, W_star, N, 0, y, ldy, fn::EPI_RELU_DEFER, make_ep(eps, K), path,
           (hipStream_t)stream};
  d.ep.inv_rms = inv_rms;
  int s = validate_op(d, y_dtype);
  if (s) return s;
  if ((s = check_auto_config(path))) return s;
  if (M > 0 && !inv_rms) return FN_ERR_NULL;
  return run_op(d);
}

int rowscale_linear(const void* x, int64_t M, int64_t K, int64_t ldx, int x_dtype, const void* W_packed,
                    int64_t N, const float* row_scale, void* y, int64_t ldy, int y_dtype, int path,
                    void* stream) {
  OpDesc d{x, M, K, ldx, x_dtype, W_packed, N, 0, y, ldy, fn::EPI_ROWSCALE, make_ep(0.0f, K), path,
           (hipStream_t)stream};
  d.ep.row_scale = row_scale;
  int s = validate_op(d, y_dtype);
  if (s) return s;
  if ((s = check_auto_config(path))) return s;
  if (M > 0 && !row_scale) return FN_ERR_NULL;
  return run_op(d);
}

// Fused QKV projection with RoPE on Q and K (Sec. 4.2, Fig. 5(b)).
int flashnorm_qkv_rope(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const void* W_star_qkv,
                       int64_t Hq, int64_t Hkv, int64_t h, float eps, const float* bias, const int32_t* positions,
                       const float* cos_tab, const float* sin_tab, int64_t P, float q_scale, void* y, int64_t ldy,
                       int y_dtype, float* inv_rms, int path, void* stream) {
  if (Hq < 1 || Hkv < 0 || h < 4 || h % 4 || P < 1) return FN_ERR_SHAPE;
  if (Hq > kMaxRows || Hkv > kMaxRows || h > kMaxRows) return FN_ERR_SHAPE;
  if (P > INT32_MAX / h) return FN_ERR_SIZE;
  if (!isfinite(q_scale)) return FN_ERR_VALUE;
  const int64_t N = (Hq + 2 * Hkv) * h;
  if (N >= (int64_t(1) << 24)) return FN_ERR_SHAPE;  // the head arithmetic runs in fp32
  OpDesc d{a, M, K, lda, a_dtype, W_star_qkv, N, 0, y, ldy, fn::EPI_ROPE, make_ep(eps, K), path,
           (hipStream_t)stream};
  d.ep.bias = bias;
  d.ep.inv_rms = inv_rms;
  d.ep.rope_pos = positions;
  d.ep.rope_cos = cos_tab;
  d.ep.rope_sin = sin_tab;
  d.ep.head_h = (int)h;
  d.ep.head_inv_h = 1.0f / (float)h;
  d.ep.rope_P = (int)P;
  d.ep.q_end = (int)(Hq * h);
  d.ep.k_end = (int)((Hq + Hkv) * h);
  d.ep.q_scale = q_scale;
  int s = validate_op(d, y_dtype);
  if (s) return s;
  if ((s = check_auto_config(path))) return s;
  if (M == 0) return FN_OK;
  if (!positions || !cos_tab || !sin_tab) return FN_ERR_NULL;
  if (!aligned16(bias) || !aligned16(cos_tab) || !aligned16(sin_tab) || !aligned16(positions)) return FN_ERR_ALIGN;
  const int64_t ybytes = extent_bytes(M, N, ldy, a_dtype), tbytes = P * (h / 2) * (int64_t)sizeof(float);
  if (overlaps(y, ybytes, cos_tab, tbytes) || overlaps(y, ybytes, sin_tab, tbytes) ||
      overlaps(y, ybytes, positions, M * (int64_t)sizeof(int32_t)))
    return FN_ERR_ALIAS;
  return run_op(d);
}

// Fused QKV projection with per-head RMSNorm of Q and K (and V), Prop. 3 / Sec. 4.3.
int flashnorm_qkv_headnorm(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const void* W_star_qkv,
                           int64_t Hq, int64_t Hkv, int64_t h, float eps, const float* gq, const float* gk,
                           const float* gv, float eps_head, const int32_t* positions, const float* cos_tab,
                           const float* sin_tab, int64_t P, float q_scale, void* y, int64_t ldy, int y_dtype,
                           float* inv_rms, int path, void* stream) {
  if (Hq < 1 || Hkv < 0 || Hq > kMaxRows || Hkv > kMaxRows) return FN_ERR_SHAPE;
  if (h != 8 && h != 16 && h != 32 && h != 64 && h != 128 && h != 256) return FN_ERR_SHAPE;
  if (positions && (P < 1 || P > INT32_MAX / h)) return P < 1 ? FN_ERR_SHAPE : FN_ERR_SIZE;
  if (!isfinite(q_scale) || !(eps_head >= 0.0f) || !isfinite(eps_head)) return FN_ERR_VALUE;
  const int64_t N = (Hq + 2 * Hkv) * h;
  if (N >= (int64_t(1) << 24)) return FN_ERR_SHAPE;
  OpDesc d{a, M, K, lda, a_dtype, W_star_qkv, N, 0, y, ldy, fn::EPI_HEADNORM, make_ep(eps, K), path,
           (hipStream_t)stream};
  d.ep.inv_rms = inv_rms;
  d.ep.rope_pos = positions;
  d.ep.rope_cos = cos_tab;
  d.ep.rope_sin = sin_tab;
  d.ep.head_h = (int)h;
  d.ep.head_inv_h = 1.0f / (float)h;
  d.ep.rope_P = positions ? (int)P : 0;
  d.ep.q_end = (int)(Hq * h);
  d.ep.k_end = (int)((Hq + Hkv) * h);
  d.ep.q_scale = q_scale;
  d.ep.hn_gq = gq;
  d.ep.hn_gk = gk;
  d.ep.hn_gv = gv;
  d.ep.hn_eps = eps_head;
  int s = validate_op(d, y_dtype);
  if (s) return s;
  if (a_dtype == FN_F32 && h > 64) return FN_ERR_UNSUPPORTED;  // the fp32 tile is 64 columns wide
  if ((s = check_auto_config(path))) return s;
  if (M == 0) return FN_OK;
  if (!gq || !gk) return FN_ERR_NULL;
  if (positions && (!cos_tab || !sin_tab)) return FN_ERR_NULL;
  if (!aligned16(gq) || !aligned16(gk) || !aligned16(gv) || !aligned16(positions) || !aligned16(cos_tab) ||
      !aligned16(sin_tab))
    return FN_ERR_ALIGN;
  const int64_t ybytes = extent_bytes(M, N, ldy, a_dtype), wb = h * (int64_t)sizeof(float);
  const int64_t tbytes = positions ? P * (h / 2) * (int64_t)sizeof(float) : 0;
  if (overlaps(y, ybytes, gq, wb) || overlaps(y, ybytes, gk, wb) || (gv && overlaps(y, ybytes, gv, wb)) ||
      (positions && (overlaps(y, ybytes, cos_tab, tbytes) || overlaps(y, ybytes, sin_tab, tbytes) ||
                     overlaps(y, ybytes, positions, M * (int64_t)sizeof(int32_t)))))
    return FN_ERR_ALIAS;
  return run_op(d);
}

// Arguments of the MLA latent pass over y [M, L + R] (latent, then rotary key).
static int check_mla_pass(const void* y, int64_t M, int64_t ldy, int dtype, int64_t L, int64_t R,
                          const float* g_lat, float eps_lat, const int32_t* positions, const float* cos_tab,
                          const float* sin_tab, int64_t P, const float* s_row) {
  if (L < 8 || L % 8 || L > 2048 || R < 0 || R % 8 || R > 512) return FN_ERR_SHAPE;
  if (R > 0 && P < 1) return FN_ERR_SHAPE;
  if (R > 0 && P > INT32_MAX / R) return FN_ERR_SIZE;
  int s = check_eps(eps_lat);
  if (s) return s;
  if (M == 0) return FN_OK;
  if (!g_lat || (R > 0 && (!positions || !cos_tab || !sin_tab))) return FN_ERR_NULL;
  if (!aligned16(g_lat) || !aligned16(positions) || !aligned16(cos_tab) || !aligned16(sin_tab)) return FN_ERR_ALIGN;
  const int64_t ybytes = extent_bytes(M, L + R, ldy, dtype), tbytes = P * (R / 2) * (int64_t)sizeof(float);
  if (overlaps(y, ybytes, g_lat, L * (int64_t)sizeof(float)) ||
      (s_row && overlaps(y, ybytes, s_row, M * (int64_t)sizeof(float))) ||
      (R > 0 && (overlaps(y, ybytes, cos_tab, tbytes) || overlaps(y, ybytes, sin_tab, tbytes) ||
                 overlaps(y, ybytes, positions, M * (int64_t)sizeof(int32_t)))))
    return FN_ERR_ALIAS;
  return FN_OK;
}

// MLA down-projection with latent normalization (Sec. 3.3; Prop. 3): the fused
// projection (with the deferred scale when a rotary key needs it, none otherwise),
// then the latent pass.
int flashnorm_mla_latent(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const void* W_star,
                         int64_t L, int64_t R, const float* g_lat, float eps_lat, float eps, const int32_t* positions,
                         const float* cos_tab, const float* sin_tab, int64_t P, void* y, int64_t ldy, int y_dtype,
                         float* inv_rms, int path, void* stream) {
  if (L < 8 || R < 0 || L > kMaxRows || R > kMaxRows) return FN_ERR_SHAPE;
  OpDesc d{a, M, K, lda, a_dtype, W_star, L + R, 0, y, ldy, R > 0 ? fn::EPI_RMS : fn::EPI_NONE, make_ep(eps, K),
           path, (hipStream_t)stream};
  d.ep.inv_rms = R > 0 ? inv_rms : nullptr;
  int s = validate_op(d, y_dtype);
  if (s) return s;
  if ((s = check_mla_pass(y, M, ldy, a_dtype, L, R, g_lat, eps_lat, positions, cos_tab, sin_tab, P,
                          R > 0 ? inv_rms : nullptr)))
    return s;
  if (M == 0) return FN_OK;
  if (R > 0 && !inv_rms) return FN_ERR_NULL;
  if ((s = run_op(d))) return s;
  return fn::launch_mla_latent_rows(y, (int)M, (int)ldy, a_dtype, (int)L, (int)R, g_lat, eps_lat,
                                    R > 0 ? inv_rms : nullptr, positions, cos_tab, sin_tab, (int)P,
                                    (hipStream_t)stream) == hipSuccess
             ? FN_OK
             : FN_ERR_HIP;
}

// Run-time g (unfolded W): g must be given, 16-byte aligned; the bf16 tile path
// stages g in LDS and takes K <= fn::kGsMaxK.
static int check_runtime_g(const OpDesc& d, const float* g) {
  if (d.M > 0 && !g) return FN_ERR_NULL;
  if (!aligned16(g)) return FN_ERR_ALIGN;
  if (d.M > 0 && overlaps(d.y, extent_bytes(d.M, d.ncols, d.ldy, d.dtype), g, d.K * (int64_t)sizeof(float)))
    return FN_ERR_ALIAS;
  const int base_path = d.path & 0xff;
  const bool decode = base_path == FN_PATH_DECODE || (base_path == FN_PATH_AUTO && d.M <= FN_DECODE_MAX_M);
  if (d.dtype == FN_BF16 && !decode && d.K > fn::kGsMaxK) return FN_ERR_UNSUPPORTED;
  return check_auto_config(d.path);
}

int flashnorm_linear_unfolded(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const float* g,
                              const void* W_packed, int64_t N, float eps, const float* bias, void* y, int64_t ldy,
                              int y_dtype, float* inv_rms, int path, void* stream) {
  OpDesc d{a, M, K, lda, a_dtype, W_packed, N, 0, y, ldy, fn::EPI_RMS, make_ep(eps, K), path, (hipStream_t)stream};
  d.ep.bias = bias;
  d.ep.inv_rms = inv_rms;
  d.ep.g_rt = g;
  d.gs = true;
  int s = validate_op(d, y_dtype);
  if (s) return s;
  if (!aligned16(bias)) return FN_ERR_ALIGN;
  if ((s = check_runtime_g(d, g))) return s;
  return run_op(d);
}

int flashnorm_glu_unfolded(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const float* g,
                           const void* W_packed_gu, int64_t F, float eps, void* out, int64_t ldo, int out_dtype,
                           int path, void* stream) {
  OpDesc d{a, M, K, lda, a_dtype, W_packed_gu, F, 1, out, ldo, fn::EPI_GLU, make_ep(eps, K), path,
           (hipStream_t)stream};
  d.ep.g_rt = g;
  d.gs = true;
  int s = validate_op(d, out_dtype);
  if (s) return s;
  if ((s = check_runtime_g(d, g))) return s;
  return run_op(d);
}

// Unfused baselines: normalise into the workspace, then the plain matrix multiply.
static int baseline_common(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const float* g,
                           const float* beta, const void* Wp, int64_t ncols, int glu, float eps, void* x_ws,
                           void* y, int64_t ldy, int path, void* stream) {
  OpDesc d{x_ws, M, K, K, a_dtype, Wp, ncols, glu, y, ldy, glu ? fn::EPI_GLU_NOSCALE : fn::EPI_NONE,
           make_ep(eps, K), path, (hipStream_t)stream};
  int s = validate_op(d, a_dtype);
  if (s) return s;
  s = check_matrix(a, M, K, lda, a_dtype, true);
  if (s) return s;
  if (!g) return FN_ERR_NULL;
  if (M == 0) return FN_OK;
  const int64_t xb = extent_bytes(M, K, K, a_dtype);
  if (overlaps(x_ws, xb, a, extent_bytes(M, K, lda, a_dtype)) ||
      overlaps(x_ws, xb, y, extent_bytes(M, ncols, ldy, a_dtype)))
    return FN_ERR_ALIAS;
  s = status_of(fn::launch_norm_rows(a, (int)M, (int)K, (int)lda, a_dtype, g, beta, eps, x_ws, (int)K,
                                     (hipStream_t)stream));
  if (s) return s;
  return run_op(d);
}

int baseline_rmsnorm_linear(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const float* g,
                            const void* W_packed, int64_t N, float eps, void* x_ws, void* y, int64_t ldy,
                            int path, void* stream) {
  return baseline_common(a, M, K, lda, a_dtype, g, nullptr, W_packed, N, 0, eps, x_ws, y, ldy, path, stream);
}

int baseline_rmsnorm_linear_noalloc(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const float* g,
                                    const void* W_packed, int64_t N, float eps, void* y, int64_t ldy, int path,
                                    void* stream) {
  if (!dtype_ok(a_dtype)) return FN_ERR_DTYPE;
  if (M < 0 || K <= 0) return FN_ERR_SHAPE;
  if (M == 0)  // validated and done, without touching the device
    return baseline_common(a, M, K, lda, a_dtype, g, nullptr, W_packed, N, 0, eps, nullptr, y, ldy, path, stream);
  if (M * K * elem_size(a_dtype) > FN_NOALLOC_SCRATCH_BYTES) return FN_ERR_SIZE;
  void* ws = scratch_on_current_device();
  if (!ws) return FN_ERR_HIP;
  // The normalisation kernel writes every element of the [M, K] workspace before the
  // product reads it, so nothing needs clearing between calls.
  return baseline_common(a, M, K, lda, a_dtype, g, nullptr, W_packed, N, 0, eps, ws, y, ldy, path, stream);
}

int baseline_rmsnorm_glu(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const float* g,
                         const void* W_packed_gu, int64_t F, float eps, void* x_ws, void* out, int64_t ldo,
                         int path, void* stream) {
  return baseline_common(a, M, K, lda, a_dtype, g, nullptr, W_packed_gu, F, 1, eps, x_ws, out, ldo, path,
                         stream);
}

int baseline_layernorm_linear(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype, const float* g,
                              const float* beta, const void* W_packed, int64_t N, float eps, void* x_ws,
                              void* y, int64_t ldy, int path, void* stream) {
  if (!beta) return FN_ERR_NULL;
  return baseline_common(a, M, K, lda, a_dtype, g, beta, W_packed, N, 0, eps, x_ws, y, ldy, path, stream);
}

int baseline_rope(void* y, int64_t M, int64_t ldy, int y_dtype, int64_t Hq, int64_t Hkv, int64_t h,
                  const int32_t* positions, const float* cos_tab, const float* sin_tab, int64_t P, float q_scale,
                  void* stream) {
  if (!dtype_ok(y_dtype)) return FN_ERR_DTYPE;
  if (Hq < 1 || Hkv < 0 || h < 4 || h % 4 || P < 1) return FN_ERR_SHAPE;
  if (Hq > kMaxRows || Hkv > kMaxRows || h > kMaxRows || (Hq + Hkv) * h > kMaxLd) return FN_ERR_SHAPE;
  if (P > INT32_MAX / h) return FN_ERR_SIZE;
  if (!isfinite(q_scale)) return FN_ERR_VALUE;
  const int64_t qk = (Hq + Hkv) * h;
  int s = check_matrix(y, M, qk, ldy, y_dtype, true);
  if (s) return s;
  if (M == 0) return FN_OK;
  if (!positions || !cos_tab || !sin_tab) return FN_ERR_NULL;
  if (!aligned16(cos_tab) || !aligned16(sin_tab) || !aligned16(positions)) return FN_ERR_ALIGN;
  const int64_t ybytes = extent_bytes(M, qk, ldy, y_dtype), tbytes = P * (h / 2) * (int64_t)sizeof(float);
  if (overlaps(y, ybytes, cos_tab, tbytes) || overlaps(y, ybytes, sin_tab, tbytes) ||
      overlaps(y, ybytes, positions, M * (int64_t)sizeof(int32_t)))
    return FN_ERR_ALIAS;
  return fn::launch_rope_rows(y, (int)M, (int)ldy, y_dtype, (int)qk, (int)(Hq * h), (int)h, positions, cos_tab,
                              sin_tab, (int)P, q_scale, (hipStream_t)stream) == hipSuccess
             ? FN_OK
             : FN_ERR_HIP;
}

int baseline_mla_latent(void* y, int64_t M, int64_t ldy, int y_dtype, int64_t L, int64_t R, const float* g_lat,
                        float eps_lat, const int32_t* positions, const float* cos_tab, const float* sin_tab,
                        int64_t P, void* stream) {
  if (!dtype_ok(y_dtype)) return FN_ERR_DTYPE;
  int s = check_matrix(y, M, L + R, ldy, y_dtype, true);
  if (s) return s;
  if ((s = check_mla_pass(y, M, ldy, y_dtype, L, R, g_lat, eps_lat, positions, cos_tab, sin_tab, P, nullptr)))
    return s;
  if (M == 0) return FN_OK;
  return fn::launch_mla_latent_rows(y, (int)M, (int)ldy, y_dtype, (int)L, (int)R, g_lat, eps_lat, nullptr,
                                    positions, cos_tab, sin_tab, (int)P, (hipStream_t)stream) == hipSuccess
             ? FN_OK
             : FN_ERR_HIP;
}

int baseline_qkv_headnorm(void* y, int64_t M, int64_t ldy, int y_dtype, int64_t Hq, int64_t Hkv, int64_t h,
                          const float* gq, const float* gk, const float* gv, float eps_head, const int32_t* positions,
                          const float* cos_tab, const float* sin_tab, int64_t P, float q_scale, void* stream) {
  if (y_dtype != FN_BF16) return dtype_ok(y_dtype) ? FN_ERR_UNSUPPORTED : FN_ERR_DTYPE;
  if (Hq < 1 || Hkv < 0 || Hq > kMaxRows || Hkv > kMaxRows) return FN_ERR_SHAPE;
  if (h != 8 && h != 16 && h != 32 && h != 64 && h != 128 && h != 256) return FN_ERR_SHAPE;
  if (positions && (P < 1 || P > INT32_MAX / h)) return P < 1 ? FN_ERR_SHAPE : FN_ERR_SIZE;
  if (!isfinite(q_scale) || !(eps_head >= 0.0f) || !isfinite(eps_head)) return FN_ERR_VALUE;
  const int64_t ncols = (Hq + Hkv + (gv ? Hkv : 0)) * h;
  if ((Hq + 2 * Hkv) * h >= (int64_t(1) << 24)) return FN_ERR_SHAPE;
  int s = check_matrix(y, M, ncols, ldy, y_dtype, true);
  if (s) return s;
  if (M == 0) return FN_OK;
  if (!gq || !gk || (positions && (!cos_tab || !sin_tab))) return FN_ERR_NULL;
  if (!aligned16(gq) || !aligned16(gk) || !aligned16(gv) || !aligned16(positions) || !aligned16(cos_tab) ||
      !aligned16(sin_tab))
    return FN_ERR_ALIGN;
  EpiArgs ep{};
  ep.rope_pos = positions;
  ep.rope_cos = cos_tab;
  ep.rope_sin = sin_tab;
  ep.head_h = (int)h;
  ep.head_inv_h = 1.0f / (float)h;
  ep.rope_P = positions ? (int)P : 0;
  ep.q_end = (int)(Hq * h);
  ep.k_end = (int)((Hq + Hkv) * h);
  ep.q_scale = q_scale;
  ep.hn_gq = gq;
  ep.hn_gk = gk;
  ep.hn_gv = gv;
  ep.hn_eps = eps_head;
  return fn::launch_headnorm_rows(y, (int)M, (int)ldy, (int)ncols, ep, (hipStream_t)stream) == hipSuccess
             ? FN_OK
             : FN_ERR_HIP;
}

const char* flashnorm_status_string(int status) {
  switch (status) {
    case FN_OK: return "FN_OK";
    case FN_ERR_NULL: return "FN_ERR_NULL: a required pointer is NULL";
    case FN_ERR_SHAPE: return "FN_ERR_SHAPE: invalid shape or leading dimension";
    case FN_ERR_DTYPE: return "FN_ERR_DTYPE: unknown or mismatched dtype";
    case FN_ERR_ALIGN: return "FN_ERR_ALIGN: pointer or leading dimension breaks 16-byte alignment";
    case FN_ERR_UNSUPPORTED: return "FN_ERR_UNSUPPORTED: request not implemented by the library";
    case FN_ERR_VALUE: return "FN_ERR_VALUE: invalid eps, layout or path";
    case FN_ERR_HIP: return "FN_ERR_HIP: HIP runtime error at launch";
    case FN_ERR_ALIAS: return "FN_ERR_ALIAS: output overlaps an input";
    case FN_ERR_SIZE: return "FN_ERR_SIZE: tensor extent beyond the kernels' 32-bit addressing";
  }
  return "unknown fn_status";
}

}  // extern "C"
