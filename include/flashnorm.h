/*
 * flashnorm.h -- C ABI of the FlashNorm norm-then-project library for AMD MI355X (gfx950).
 *
 * FlashNorm ("FlashNorm: Fast Normalization for Transformers", arXiv 2407.09577)
 * computes an RMSNorm followed by a linear layer, z = RMSNorm(a; g) W (Sec. 3.1),
 * in the deferred form z = (a W*) * (1 / RMS(a)) with W* = diag(g) W folded once,
 * offline (Prop. 1 "weightless normalization", Prop. 2 "deferred normalization").
 * The per-row sum of squares is accumulated from the same activation tiles the
 * matrix multiply consumes, so the two run side by side (Cor. 1) and a single
 * per-row scale is applied in the epilogue.
 *
 * Notation: a[M,K] holds M activation rows of width K (the paper's n);
 * W[K,N] maps K inputs to N outputs (the paper's k).  eps sits inside the root,
 * RMSe(a) = sqrt(eps + (1/K) sum_k a_k^2) (App. "RMS with epsilon").
 *
 * Conventions shared by every entry point:
 *  - Pointers to tensors are DEVICE pointers owned by the caller.  The library
 *    never allocates device memory, never synchronises, and keeps no mutable
 *    global state: calls on different streams may run concurrently.
 *  - Tensors are row-major with an explicit leading dimension (elements between
 *    consecutive rows).  Every tensor pointer (including the fp32 per-column
 *    vectors bias, colsum and c_star) must be 16-byte aligned and every leading
 *    dimension a multiple of 8 elements for bf16, 4 for fp32.
 *  - Arguments are validated on the host before anything is launched; on any
 *    error nothing is written and a negative fn_status is returned.  M == 0 is
 *    a valid no-op.  Kernel launch failures return FN_ERR_HIP; faults during
 *    execution surface at the caller's next synchronisation.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream).
 *  - Results are deterministic: no atomics and no split reductions across
 *    workgroups, so repeated calls give bitwise-identical outputs.
 *  - The packed weight layout written by fold_weights is opaque; only the
 *    library reads it.  One buffer serves both the many-row (matrix-core) and
 *    the few-row (bandwidth-bound) kernels.
 */
#ifndef FLASHNORM_H
#define FLASHNORM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FN_OK = 0,
  FN_ERR_NULL = -1,        /* a required pointer is NULL */
  FN_ERR_SHAPE = -2,       /* M < 0, K <= 0, N <= 0, leading dimension too small, K not a multiple of 8 (bf16) or 4 (fp32) */
  FN_ERR_DTYPE = -3,       /* unknown dtype, or dtypes that do not match */
  FN_ERR_ALIGN = -4,       /* a pointer is not 16-byte aligned or a leading dimension breaks row alignment */
  FN_ERR_UNSUPPORTED = -5, /* valid request the library does not implement (e.g. a forced path that cannot run it) */
  FN_ERR_VALUE = -6,       /* eps negative or not finite; unknown layout or path */
  FN_ERR_HIP = -7,         /* the HIP runtime reported an error while launching */
  FN_ERR_ALIAS = -8,       /* the output overlaps an input */
  FN_ERR_SIZE = -9         /* a tensor exceeds the 32-bit byte extents the kernels address
                              (leading dimensions and K above 2^21, M or N above 2^30,
                              or a packed weight buffer of 2^31 bytes or more) */
} fn_status;

typedef enum { FN_F32 = 0, FN_BF16 = 1 } fn_dtype;

/* FN_LAYOUT_GLU: the logical weight is [K, 2F] = [Wg | Wu] (gate columns first,
 * then up columns, Sec. 4.1 Fig. 3(a)); the packed layout pairs each gate column
 * with its up column so one workgroup owns both. */
typedef enum { FN_LAYOUT_LINEAR = 0, FN_LAYOUT_GLU = 1 } fn_layout;

/* Kernel selection (Sec. 6 and App. "Production path": shape-specialised dispatch).
 * AUTO picks by M; PREFILL forces the matrix-core tile kernel (any M);
 * DECODE forces the bandwidth-bound few-row kernel (bf16, M <= 16, else
 * FN_ERR_UNSUPPORTED).  fp32 always runs the fp32 kernel. */
typedef enum { FN_PATH_AUTO = 0, FN_PATH_PREFILL = 1, FN_PATH_DECODE = 2 } fn_path;

/* Tuning override: bits 8..15 of a path argument may name one of the library's
 * kernel configurations for the selected path (prefill tile shapes, or decode
 * work splits with FN_PATH_DECODE; for fp32 operands, 1 = 64-row tiles,
 * 2 = 16-row tiles with K split over four thread groups, 3 = the few-row kernel:
 * 16-row tiles of 4, 8 or 16 columns (8 or 16 for a GLU, 64 with per-head norms,
 * the width chosen by the workgroup count) with K split over 256 / width thread
 * groups; 0 = automatic choice);
 * values it does not know return FN_ERR_VALUE.  Results are identical for every configuration up to
 * floating-point summation order. */
#define FN_PATH_TILE_SHIFT 8

/* Largest M the DECODE path accepts. */
#define FN_DECODE_MAX_M 16

/* Bytes of the packed weight buffer that fold_weights writes for a logical
 * weight with K rows and N columns (N = 2F for FN_LAYOUT_GLU) stored as
 * ws_dtype.  Returns 0 for invalid arguments and for buffers of 2^31 bytes or
 * more (FN_ERR_SIZE).  Host only; no device work. */
size_t fold_weights_size(int64_t K, int64_t N, int layout, int ws_dtype);

/* Fold the normalisation weights into the linear layer, once, offline
 * (Prop. 1: W*[k,n] = g_k W[k,n]; Sec. 3.4: c* = beta W).
 *   W       logical [K, N] weight, dtype w_dtype (fp32 or bf16): element (k, n) is at
 *           W[k * stride_k + n * stride_n] (strides in elements, each >= 0, stride_k
 *           below 2^40 and stride_n below 2^31, else FN_ERR_SIZE; negative: FN_ERR_SHAPE).
 *           A row-major [K, N] tensor has (stride_k, stride_n) = (ld, 1); a framework's
 *           [N, K] linear-layer weight is folded in place, with no transposed copy,
 *           as (1, ld).  Only read; views whose elements overlap are allowed.
 *           For FN_LAYOUT_GLU, N = 2F and W = [Wg | Wu].
 *   g       [K] fp32, or NULL for g = 1 (plain packing of W, used by the unfused baseline).
 *   beta    [K] fp32 LayerNorm bias, or NULL; needed only for c_star.
 *   W_star  output, fold_weights_size(K, N, layout, ws_dtype) bytes, 16-byte aligned.
 *           Each element is the exact product g_k W[k,n] rounded once
 *           (to nearest, ties to even) to ws_dtype; padding is zero.
 *           ws_dtype must equal the dtype of the activations it will be used with.
 *   colsum  optional [N] fp32: sum over k of the STORED W*[k,n] (the mean correction
 *           of the deferred LayerNorm), accumulated in fp64 and rounded once.
 *   c_star  optional [N] fp32: sum over k of beta_k W[k,n] with the unfolded W,
 *           accumulated in fp64 and rounded once; requires beta.
 *   colsum and c_star are available for FN_LAYOUT_LINEAR only. */
int fold_weights(const void* W, int64_t stride_k, int64_t stride_n, int w_dtype, const float* g,
                 const float* beta, int64_t K, int64_t N, int layout, void* W_star, int ws_dtype,
                 float* colsum, float* c_star, void* stream);

/* Inverse of the packing: write the logical [K, N] weight held in W_star (as
 * written by fold_weights with the same K, N, layout, ws_dtype) to out, row-major
 * with leading dimension ldo >= N, in ws_dtype.  Inspection and tests only. */
int unpack_weights(const void* W_star, int64_t K, int64_t N, int layout, int ws_dtype, void* out,
                   int64_t ldo, void* stream);

/* Deferred RMSNorm -> linear (Prop. 2; with a bias, the Remark "Bias case": the
 * scale is applied before the bias is added):
 *   y[m,n] = (sum_k a[m,k] W*[k,n]) * s_m  (+ bias[n]),  s_m = 1/sqrt(eps + ss_m/K),
 *   ss_m = sum_k a[m,k]^2 accumulated from the tiles the product reads.
 *   a       [M, K] activations, leading dimension lda >= K, dtype a_dtype.
 *   W_star  packed by fold_weights(..., N, FN_LAYOUT_LINEAR, a_dtype, ...).
 *   bias    optional [N] fp32 output bias.
 *   y       [M, N] output, leading dimension ldy >= N, dtype y_dtype == a_dtype;
 *           computed in fp32 and rounded once (to nearest even) on the store.
 *   inv_rms optional [M] fp32 side output of s_m (for consumers that defer the scale further). */
int flashnorm_linear(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                     const void* W_star, int64_t N, float eps, const float* bias, void* y,
                     int64_t ldy, int y_dtype, float* inv_rms, void* stream);

/* RMSNorm -> SwiGLU FFN input projection with both branch scales deferred to the
 * products (Sec. 4.1, Fig. 3(a)):
 *   out[m,f] = silu(s_m (a W*g)[m,f]) * (s_m (a W*u)[m,f]),  silu(t) = t / (1 + e^-t).
 *   W_star_gu  packed by fold_weights(..., 2F, FN_LAYOUT_GLU, a_dtype, ...).
 *   out        [M, F], leading dimension ldo >= F, dtype out_dtype == a_dtype. */
int flashnorm_glu(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                  const void* W_star_gu, int64_t F, float eps, void* out, int64_t ldo,
                  int out_dtype, void* stream);

/* Deferred LayerNorm -> linear.  LayerNorm is centering followed by RMS scaling
 * with g and the bias beta (Sec. 2); beta moves past W as c* = beta W (Sec. 3.4),
 * g folds into W* (Prop. 1), the 1/sigma scale is deferred (Prop. 2) and the
 * centering is exchanged with the sum over k as in Sec. 3.5:
 *   y[m,n] = ((a W*)[m,n] - mu_m colsum[n]) / sigma_m + c_star[n],
 *   mu_m = sa_m/K, sigma_m = sqrt(ss_m/K - mu_m^2 + eps), sa and ss accumulated
 *   from the tiles the product reads.
 *   colsum  [N] fp32 from fold_weights (required);  c_star  [N] fp32 or NULL (= 0).
 *   The one-pass variance loses precision when |mu| >> sigma (relative error of
 *   order (mu/sigma)^2 * 2^-24 in fp32). */
int flashnorm_layernorm_linear(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                               const void* W_star, const float* colsum, const float* c_star,
                               int64_t N, float eps, void* y, int64_t ldy, int y_dtype,
                               void* stream);

/* The same three operations with an explicit kernel selection (fn_path). */
int flashnorm_linear_ex(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                        const void* W_star, int64_t N, float eps, const float* bias, void* y,
                        int64_t ldy, int y_dtype, float* inv_rms, int path, void* stream);
int flashnorm_glu_ex(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                     const void* W_star_gu, int64_t F, float eps, void* out, int64_t ldo,
                     int out_dtype, int path, void* stream);
int flashnorm_layernorm_linear_ex(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                                  const void* W_star, const float* colsum, const float* c_star,
                                  int64_t N, float eps, void* y, int64_t ldy, int y_dtype,
                                  int path, void* stream);

/* Gate nonlinearity of a GLU-variant FFN input projection (Sec. 4.1 and App. "FFN with
 * ReGLU and Bilinear GLU").  SWIGLU_DEFER_UP is SwiGLU with the up-branch scale left
 * for the FFN output (Fig. 3(b)). */
typedef enum {
  FN_GLU_SWIGLU = 0,
  FN_GLU_REGLU = 1,
  FN_GLU_BILINEAR = 2,
  FN_GLU_SWIGLU_DEFER_UP = 3
} fn_glu_act;

/* RMSNorm -> GLU-variant FFN input projection with the normalisation deferred past
 * the products; s_m = 1/sqrt(eps + ss_m/K) as in flashnorm_linear:
 *   FN_GLU_SWIGLU:          out = silu(s_m hg) * (s_m hu)            (Fig. 3(a))
 *   FN_GLU_REGLU:           out = relu(hg) * hu * s_m^2              (Fig. 4(b))
 *   FN_GLU_BILINEAR:        out = hg * hu * s_m^2                    (Fig. 4(b))
 *   FN_GLU_SWIGLU_DEFER_UP: out = silu(s_m hg) * hu                  (Fig. 3(b))
 * with hg = (a W*g)[m,f], hu = (a W*u)[m,f].  For ReGLU and the bilinear GLU both
 * branch scales merge into one factor s^2 = 1/MSe(a) because ReLU(s t) = s ReLU(t)
 * for s >= 0 (App. "FFN with ReGLU and Bilinear GLU").
 *   W_star_gu  packed by fold_weights(..., 2F, FN_LAYOUT_GLU, a_dtype, ...).
 *   out        [M, F], leading dimension ldo >= F, dtype out_dtype == a_dtype.
 *   inv_rms    [M] fp32 output of s_m: required for FN_GLU_SWIGLU_DEFER_UP (the
 *              consumer, e.g. rowscale_linear for the down projection, applies it),
 *              optional for FN_GLU_SWIGLU, and must be NULL for ReGLU and bilinear
 *              (FN_ERR_VALUE), whose output carries the whole scale.
 *   path       FN_PATH_AUTO / PREFILL / DECODE with the automatic configuration
 *              (bits 8..15 zero, else FN_ERR_UNSUPPORTED). */
int flashnorm_glu_act(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                      const void* W_star_gu, int64_t F, float eps, int act, void* out,
                      int64_t ldo, int out_dtype, float* inv_rms, int path, void* stream);

/* RMSNorm -> up projection of a ReLU FFN with the normalisation deferred all the
 * way to the FFN output (App. "FFN with ReLU", Fig. 2(b): ReLU(s t) = s ReLU(t) for
 * s >= 0, so the scale passes the ReLU and the down projection):
 *   y[m,n] = relu((a W*)[m,n])   and   inv_rms[m] = s_m (required).
 * The FFN output is rowscale_linear(y, W_down, inv_rms).  Arguments as for
 * flashnorm_linear; path as for flashnorm_glu_act. */
int flashnorm_linear_relu(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                          const void* W_star, int64_t N, float eps, void* y, int64_t ldy,
                          int y_dtype, float* inv_rms, int path, void* stream);

/* Linear layer applying a per-row scale deferred from an earlier normalisation
 * (Prop. 2 carried to the FFN output, Fig. 2(b) and Fig. 3(b)):
 *   y[m,n] = (sum_k x[m,k] W[k,n]) * row_scale[m].
 *   x          [M, K] (e.g. the output of flashnorm_linear_relu or of
 *              flashnorm_glu_act with FN_GLU_SWIGLU_DEFER_UP), dtype x_dtype.
 *   W_packed   packed by fold_weights(..., N, FN_LAYOUT_LINEAR, x_dtype, ...); pass
 *              g = NULL unless a per-input-channel weight should be folded in.
 *   row_scale  [M] fp32 (required), e.g. the inv_rms side output of the producer.
 *   y          [M, N], leading dimension ldy >= N, dtype y_dtype == x_dtype.
 *   path as for flashnorm_glu_act. */
int rowscale_linear(const void* x, int64_t M, int64_t K, int64_t ldx, int x_dtype,
                    const void* W_packed, int64_t N, const float* row_scale, void* y,
                    int64_t ldy, int y_dtype, int path, void* stream);

/* RMSNorm -> fused QKV projection -> RoPE (Sec. 4.2, Fig. 5).  W_star_qkv is
 * [Wq | Wk | Wv] folded with g (FN_LAYOUT_LINEAR, N = (Hq + 2 Hkv) h columns: Hq
 * query heads, then Hkv key heads, then Hkv value heads, each h wide).  Row m is a
 * token at position positions[m].  With t = (a W*) s_m (+ bias, added before the
 * rotation), s_m = 1/RMSe(a_m):
 *   Q and K heads:  y_2j = t_2j cos - t_2j+1 sin,  y_2j+1 = t_2j sin + t_2j+1 cos,
 *                   cos = cos_tab[positions[m]][j], sin = sin_tab[positions[m]][j],
 *                   j the pair index within the head (consecutive pairs, as in the
 *                   RoPE paper); Q also times q_scale (e.g. 1/sqrt(h), the
 *                   attention-score scale folded into the same multiply);
 *   V heads:        y = t.
 * Without a bias the kernels fold s_m (and q_scale) into the token's table values,
 * cos*s and sin*s, as in Fig. 5(b).
 *   positions  [M] int32, 16-byte aligned.  A position outside [0, P) makes that
 *              row's Q and K outputs NaN (V is still written).
 *   cos_tab, sin_tab  [P][h/2] fp32 row-major, 16-byte aligned, shared by all heads.
 *   h          a multiple of 4 (FN_ERR_SHAPE otherwise); Hq >= 1, Hkv >= 0.
 *   bias       optional [N] fp32, 16-byte aligned.  inv_rms optional [M] output of s.
 *   path       as for flashnorm_glu_act (automatic configuration only).
 * The output may not overlap the tables or positions (FN_ERR_ALIAS). */
int flashnorm_qkv_rope(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                       const void* W_star_qkv, int64_t Hq, int64_t Hkv, int64_t h, float eps,
                       const float* bias, const int32_t* positions, const float* cos_tab,
                       const float* sin_tab, int64_t P, float q_scale, void* y, int64_t ldy,
                       int y_dtype, float* inv_rms, int path, void* stream);

/* Deferred normalisation with the UNFOLDED weight (Remark "Unfolded case": the
 * deferral of Prop. 2 needs only that 1/RMS is a per-token scalar, so it serves a
 * checkpoint as it is, with g applied at run time instead of folded into W):
 *   flashnorm_linear_unfolded:  y = (sum_k bf(a[m,k] g_k) W[k,n]) * s_m (+ bias[n])
 *   flashnorm_glu_unfolded:     out = silu(s_m hg) * (s_m hu), hg/hu from bf(a g) [Wg | Wu]
 * where s_m = 1/sqrt(eps + ss_m/K) with ss_m the squares of the RAW activations, and
 * bf() is the activation dtype: each product a_k g_k is rounded once to it before
 * the matrix multiply (the folded path instead rounds g_k W[k,n] once).
 *   g         [K] fp32 (required), 16-byte aligned.
 *   W_packed  the unfolded weight packed by fold_weights(..., g = NULL, ...), with
 *             FN_LAYOUT_LINEAR or FN_LAYOUT_GLU respectively.
 * Other arguments as for flashnorm_linear / flashnorm_glu; path as for
 * flashnorm_glu_act.  The bf16 tile path stages g in LDS and takes K <= 8128
 * (FN_ERR_UNSUPPORTED beyond; the decode and fp32 paths have no such limit). */
int flashnorm_linear_unfolded(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                              const float* g, const void* W_packed, int64_t N, float eps,
                              const float* bias, void* y, int64_t ldy, int y_dtype, float* inv_rms,
                              int path, void* stream);
int flashnorm_glu_unfolded(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                           const float* g, const void* W_packed_gu, int64_t F, float eps, void* out,
                           int64_t ldo, int out_dtype, int path, void* stream);

/* Unfused baselines in the same library (the sequential RMSNorm -> GEMM of Fig. 1(a)
 * and Sec. 6): a normalisation kernel writes the normalised activations
 * x = RMSNorm(a; g) (or LayerNorm(a; g, beta)) to the caller's workspace x_ws
 * ([M, K], leading dimension K, dtype a_dtype), then the same matrix-multiply
 * kernels run on x without any normalisation epilogue.
 *   W_packed is the UNFOLDED weight packed by fold_weights with g = NULL.
 *   baseline_layernorm_linear adds no c*: beta enters through x. */
int baseline_rmsnorm_linear(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                            const float* g, const void* W_packed, int64_t N, float eps, void* x_ws,
                            void* y, int64_t ldy, int path, void* stream);
/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): baseline_rmsnorm_linear without the
 * x_ws argument.  The normalised activations go to a workspace the library holds in a
 * static device array of FN_NOALLOC_SCRATCH_BYTES (32 MiB) on each GPU it runs on,
 * kept until the process ends; the call itself allocates nothing (no hipMalloc, no
 * hipFree, no allocating library routine).
 *   M * K * sizeof(a_dtype) above FN_NOALLOC_SCRATCH_BYTES: FN_ERR_SIZE, nothing launched.
 *   The first call on a device looks up that device's array (FN_ERR_HIP if that fails).
 *   Every call on one GPU shares that GPU's array: calls that overlap on one GPU (on
 *   different streams, or from different threads) race and give undefined results;
 *   calls on one stream are ordered and safe.  The array keeps the last call's
 *   normalised activations; each call overwrites all it reads, so nothing needs clearing.
 * Other arguments, results and errors as for baseline_rmsnorm_linear. */
#define FN_NOALLOC_SCRATCH_BYTES (32 * 1024 * 1024)
int baseline_rmsnorm_linear_noalloc(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                                    const float* g, const void* W_packed, int64_t N, float eps,
                                    void* y, int64_t ldy, int path, void* stream);
int baseline_rmsnorm_glu(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                         const float* g, const void* W_packed_gu, int64_t F, float eps,
                         void* x_ws, void* out, int64_t ldo, int path, void* stream);
int baseline_layernorm_linear(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                              const float* g, const float* beta, const void* W_packed, int64_t N,
                              float eps, void* x_ws, void* y, int64_t ldy, int path, void* stream);

/* RMSNorm -> fused QKV projection -> per-head RMSNorm of the Q and K heads (QK-norm,
 * Sec. 4.3) or of Q, K and V (QKV-normalization, Sec. 3.3) -> RoPE on Q and K.
 * By Prop. 3 ("RMSNorm cancellation") the input norm's scale cancels in every
 * normalised head, so those heads are normalised straight from t = a W*
 * (W_star_qkv folded with the input g, FN_LAYOUT_LINEAR, heads ordered as for
 * flashnorm_qkv_rope):
 *   Q head:  y = RoPE(t_head / sqrt(eps_head + mean(t_head^2)) * gq) * q_scale
 *   K head:  y = RoPE(t_head / sqrt(eps_head + mean(t_head^2)) * gk)
 *   V head:  with gv, as K without the rotation (the input RMSNorm is then
 *            eliminated entirely); without gv (QK-norm), y = t_head * s_m with
 *            s_m = 1/RMSe(a_m) as in flashnorm_linear.
 * With eps_head > 0 this differs from the standard form (input RMSNorm first) by
 * the epsilon caveat of Sec. 3.3, negligible unless a head's energy is tiny.
 *   gq, gk     [h] fp32 (required), shared by all heads; gv [h] or NULL.  16-byte aligned.
 *   eps_head   >= 0, finite.  h in {8, 16, 32, 64, 128, 256}.
 *   positions  [M] int32 or NULL (no rotation); cos_tab, sin_tab, P as for
 *              flashnorm_qkv_rope (required with positions).
 *   inv_rms    optional [M] output of s_m.
 * bf16: every M runs on the tile kernel (a workgroup must hold whole heads).
 * fp32: h <= 64 (the fp32 tile is 64 columns wide; FN_ERR_UNSUPPORTED beyond).
 * path as for flashnorm_glu_act. */
int flashnorm_qkv_headnorm(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                           const void* W_star_qkv, int64_t Hq, int64_t Hkv, int64_t h, float eps,
                           const float* gq, const float* gk, const float* gv, float eps_head,
                           const int32_t* positions, const float* cos_tab, const float* sin_tab,
                           int64_t P, float q_scale, void* y, int64_t ldy, int y_dtype,
                           float* inv_rms, int path, void* stream);

/* MLA down-projection with latent normalization (Sec. 3.3, the paragraph on
 * multi-head latent attention; Prop. 3, Fig. 6(b)).  W_star is the down-projection
 * [W_lat | W_rope] folded with the input norm's g (fold_weights, linear layout,
 * N = L + R columns).  With t = a W*, row m of y gets
 *   y[m, 0:L)     = t / sqrt(eps_lat + mean(t^2)) * g_lat      (the latent RMSNorm)
 *   y[m, L:L+R)   = RoPE(t * s_m) at positions[m]               (the rotary key)
 * where s_m = 1/RMSe(a_m).  By Prop. 3 the input RMSNorm cancels in the normalised
 * latent (exactly when eps_lat = 0; with eps_lat > 0 this is the cancelled form,
 * which differs from input RMSNorm -> projection -> latent RMSNorm by the epsilon
 * caveat of Sec. 3.3).  The rotary key is followed by no norm and keeps s_m; it is
 * one head of width R, pairs (2j, 2j+1) turned by cos_tab/sin_tab [P][R/2] as in
 * flashnorm_qkv_rope; a position outside [0, P) makes it NaN.  With R = 0 no
 * statistics of a are taken at all: the input norm is gone.
 *   L          latent width, a multiple of 8, 8 <= L <= 2048.
 *   R          rotary width, a multiple of 8, 0 <= R <= 512.
 *   g_lat      [L] fp32 latent norm weight (required), 16-byte aligned.
 *   eps_lat    latent epsilon, >= 0 and finite; eps is the input norm's.
 *   positions, cos_tab, sin_tab, P: required when R > 0 (16-byte aligned).
 *   inv_rms    [M] fp32, required when R > 0: receives s_m, which the latent pass
 *              reads; ignored (may be NULL) when R = 0.
 *   y          [M, L + R], leading dimension ldy; dtype of a.
 *   path       as for flashnorm_linear (it selects the projection's kernel).
 * Two launches on the stream: the fused projection, then one wave per row for the
 * latent norm and the rotation (in place in y). */
int flashnorm_mla_latent(const void* a, int64_t M, int64_t K, int64_t lda, int a_dtype,
                         const void* W_star, int64_t L, int64_t R, const float* g_lat, float eps_lat,
                         float eps, const int32_t* positions, const float* cos_tab,
                         const float* sin_tab, int64_t P, void* y, int64_t ldy, int y_dtype,
                         float* inv_rms, int path, void* stream);

/* Unfused baseline of the MLA latent stage (the standard form: input RMSNorm ->
 * projection -> latent RMSNorm, rotary key rotated): applied in place to y [M, L + R]
 * holding the projection of the normalised input; y[:, 0:L) becomes
 * y / sqrt(eps_lat + mean(y^2)) * g_lat and y[:, L:L+R) is turned by RoPE.
 * Arguments as for flashnorm_mla_latent.  Run after baseline_rmsnorm_linear. */
int baseline_mla_latent(void* y, int64_t M, int64_t ldy, int y_dtype, int64_t L, int64_t R,
                        const float* g_lat, float eps_lat, const int32_t* positions,
                        const float* cos_tab, const float* sin_tab, int64_t P, void* stream);

/* Unfused baseline of flashnorm_qkv_rope's rotation (Fig. 5(a)): RoPE applied in
 * place to the first (Hq + Hkv) h columns of y (the Q and K heads of a QKV
 * projection output, leading dimension ldy), Q also times q_scale; arguments as
 * for flashnorm_qkv_rope.  Run after baseline_rmsnorm_linear for the three-kernel
 * chain norm -> projection -> rotation. */
int baseline_rope(void* y, int64_t M, int64_t ldy, int y_dtype, int64_t Hq, int64_t Hkv, int64_t h,
                  const int32_t* positions, const float* cos_tab, const float* sin_tab, int64_t P,
                  float q_scale, void* stream);

/* Unfused baseline of flashnorm_qkv_headnorm's per-head stage (the standard form:
 * input RMSNorm -> projection -> per-head norms -> RoPE): applied in place to the
 * Q and K heads of y (and V heads when gv is given), Q times q_scale; arguments as
 * for flashnorm_qkv_headnorm; bf16 only.  Run after baseline_rmsnorm_linear. */
int baseline_qkv_headnorm(void* y, int64_t M, int64_t ldy, int y_dtype, int64_t Hq, int64_t Hkv,
                          int64_t h, const float* gq, const float* gk, const float* gv, float eps_head,
                          const int32_t* positions, const float* cos_tab, const float* sin_tab,
                          int64_t P, float q_scale, void* stream);

/* Human-readable name of a status code (static string; never NULL). */
const char* flashnorm_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* FLASHNORM_H */
