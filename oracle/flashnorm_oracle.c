/*
 * FlashNorm CPU oracle — TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 implementation of what the norm-then-project hot path
 * computes, written from the paper "FlashNorm: Fast Normalization for
 * Transformers" (arXiv 2407.09577).  Only the test suite, the smoke check and
 * the benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the GPU library; neither side includes or links
 * the other.
 *
 * Conventions (paper notation -> ours): the paper's activation row a in R^n and
 * weight W in R^{n x k} (Sec. 3.1) become a[M,K] row-major (K = paper n, the
 * reduction width) and W[K,N] row-major (N = paper k, the output width).
 * Every function takes fp64 copies of exactly the values the GPU receives.
 *
 * Row subsets: every op takes an optional list `rows` of nrows row indices of
 * `a`; output row r of `y` is the result for input row rows[r].  rows == NULL
 * means all M rows in order (nrows must then equal M).  This lets the tests
 * check sampled rows of the full-size workloads one by one.
 *
 * Parity pins: every function here is pinned by tests (closed forms, exact
 * rational worked examples, library reductions, identities); none is
 * "parity unpinned".
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_EXPORT __attribute__((visibility("default")))

/* Threads the OpenMP loops below use (reported with CPU timings). */
ORACLE_EXPORT int fn_oracle_num_threads(void) { return omp_get_max_threads(); }

static int64_t row_of(const int64_t* rows, int64_t r) { return rows ? rows[r] : r; }

/* RMS with the epsilon inside the root (App. "RMS with epsilon"):
 *   RMSe(a) = sqrt(eps + (1/K) * sum_k a_k^2).
 * eps = 0 gives the plain RMS of Sec. 3.1. */
ORACLE_EXPORT double fn_oracle_rms(const double* a, int64_t K, double eps) {
  double ss = 0.0;
  for (int64_t k = 0; k < K; ++k) ss += a[k] * a[k];
  return sqrt(eps + ss / (double)K);
}

/* Standard form (a), Sec. 3.1 and Fig. 1(a):
 *   x_k = a_k / RMSe(a) * g_k,   y_n = sum_k x_k W[k,n]   (+ c_n if bias).
 * With a bias the normalisation precedes the bias addition (Remark "Bias case"). */
ORACLE_EXPORT void fn_oracle_rmsnorm_linear(const double* a, int64_t M, int64_t K,
                                            const double* g, const double* W, int64_t N,
                                            double eps, const double* bias,
                                            const int64_t* rows, int64_t nrows, double* y) {
  (void)M;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < nrows; ++r) {
    const double* ar = a + row_of(rows, r) * K;
    double* yr = y + r * N;
    double* x = (double*)malloc(sizeof(double) * (size_t)K);
    double rms = fn_oracle_rms(ar, K, eps);
    for (int64_t k = 0; k < K; ++k) x[k] = ar[k] / rms * g[k];
    for (int64_t n = 0; n < N; ++n) yr[n] = 0.0;
    for (int64_t k = 0; k < K; ++k) {
      const double* wk = W + k * N;
      for (int64_t n = 0; n < N; ++n) yr[n] += x[k] * wk[n];
    }
    if (bias)
      for (int64_t n = 0; n < N; ++n) yr[n] += bias[n];
    free(x);
  }
}

/* Form (b), weightless normalisation (Prop. 1, Fig. 1(b)):
 *   W*[k,n] = g_k W[k,n] (exact fp64 product),  y = (a / RMSe(a)) W*  (+ c).
 * Self-check only: used to show forms (a), (b), (c) agree. */
ORACLE_EXPORT void fn_oracle_weightless(const double* a, int64_t M, int64_t K, const double* g,
                                        const double* W, int64_t N, double eps,
                                        const double* bias, const int64_t* rows, int64_t nrows,
                                        double* y) {
  (void)M;
  double* Ws = (double*)malloc(sizeof(double) * (size_t)(K * N));
  for (int64_t k = 0; k < K; ++k)
    for (int64_t n = 0; n < N; ++n) Ws[k * N + n] = g[k] * W[k * N + n];
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < nrows; ++r) {
    const double* ar = a + row_of(rows, r) * K;
    double* yr = y + r * N;
    double rms = fn_oracle_rms(ar, K, eps);
    for (int64_t n = 0; n < N; ++n) yr[n] = 0.0;
    for (int64_t k = 0; k < K; ++k) {
      double xk = ar[k] / rms;
      for (int64_t n = 0; n < N; ++n) yr[n] += xk * Ws[k * N + n];
    }
    if (bias)
      for (int64_t n = 0; n < N; ++n) yr[n] += bias[n];
  }
  free(Ws);
}

/* Form (c), deferred normalisation (Prop. 2, Fig. 1(c), Cor. 1):
 *   y = (a W*) * (1 / RMSe(a))   and, with a bias, + c after the scaling.
 * Self-check only. */
ORACLE_EXPORT void fn_oracle_deferred(const double* a, int64_t M, int64_t K, const double* g,
                                      const double* W, int64_t N, double eps, const double* bias,
                                      const int64_t* rows, int64_t nrows, double* y) {
  (void)M;
  double* Ws = (double*)malloc(sizeof(double) * (size_t)(K * N));
  for (int64_t k = 0; k < K; ++k)
    for (int64_t n = 0; n < N; ++n) Ws[k * N + n] = g[k] * W[k * N + n];
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < nrows; ++r) {
    const double* ar = a + row_of(rows, r) * K;
    double* yr = y + r * N;
    for (int64_t n = 0; n < N; ++n) yr[n] = 0.0;
    for (int64_t k = 0; k < K; ++k)
      for (int64_t n = 0; n < N; ++n) yr[n] += ar[k] * Ws[k * N + n];
    double inv = 1.0 / fn_oracle_rms(ar, K, eps);
    for (int64_t n = 0; n < N; ++n) yr[n] *= inv;
    if (bias)
      for (int64_t n = 0; n < N; ++n) yr[n] += bias[n];
  }
  free(Ws);
}

static double silu(double t) { return t / (1.0 + exp(-t)); }

/* RMSNorm followed by a SwiGLU FFN input projection (Sec. 4.1, Fig. 3(a)):
 *   x = RMSNorm(a; g),  h_g = x Wg,  h_u = x Wu,  out = silu(h_g) * h_u,
 * with silu(t) = t * sigmoid(t).  Wgu is [K, 2F] = [Wg | Wu] row-major. */
ORACLE_EXPORT void fn_oracle_rmsnorm_swiglu(const double* a, int64_t M, int64_t K,
                                            const double* g, const double* Wgu, int64_t F,
                                            double eps, const int64_t* rows, int64_t nrows,
                                            double* out) {
  (void)M;
  const int64_t N2 = 2 * F;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < nrows; ++r) {
    const double* ar = a + row_of(rows, r) * K;
    double* x = (double*)malloc(sizeof(double) * (size_t)K);
    double* h = (double*)calloc((size_t)N2, sizeof(double));
    double rms = fn_oracle_rms(ar, K, eps);
    for (int64_t k = 0; k < K; ++k) x[k] = ar[k] / rms * g[k];
    for (int64_t k = 0; k < K; ++k) {
      const double* wk = Wgu + k * N2;
      for (int64_t n = 0; n < N2; ++n) h[n] += x[k] * wk[n];
    }
    for (int64_t f = 0; f < F; ++f) out[r * F + f] = silu(h[f]) * h[F + f];
    free(x);
    free(h);
  }
}

/* Gate nonlinearities of the GLU variants: 0 = SwiGLU (silu), 1 = ReGLU (ReLU),
 * 2 = bilinear GLU (identity); and 3 = the plain ReLU of a non-gated FFN. */
static double glu_act(int act, double t) {
  if (act == 0) return silu(t);
  if (act == 1 || act == 3) return t > 0.0 ? t : 0.0;
  return t;
}

/* RMSNorm followed by a GLU-variant FFN input projection, standard form
 * (Sec. 4.1, Fig. 3(a); App. "FFN with ReGLU and Bilinear GLU", Fig. 4(a)):
 *   x = RMSNorm(a; g),  h_g = x Wg,  h_u = x Wu,  out = act(h_g) * h_u,
 * act = silu (0), ReLU (1) or the identity (2).  Wgu = [Wg | Wu], [K, 2F]. */
ORACLE_EXPORT void fn_oracle_rmsnorm_glu_act(const double* a, int64_t M, int64_t K,
                                             const double* g, const double* Wgu, int64_t F,
                                             double eps, int act, const int64_t* rows,
                                             int64_t nrows, double* out) {
  (void)M;
  const int64_t N2 = 2 * F;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < nrows; ++r) {
    const double* ar = a + row_of(rows, r) * K;
    double* x = (double*)malloc(sizeof(double) * (size_t)K);
    double* h = (double*)calloc((size_t)N2, sizeof(double));
    double rms = fn_oracle_rms(ar, K, eps);
    for (int64_t k = 0; k < K; ++k) x[k] = ar[k] / rms * g[k];
    for (int64_t k = 0; k < K; ++k) {
      const double* wk = Wgu + k * N2;
      for (int64_t n = 0; n < N2; ++n) h[n] += x[k] * wk[n];
    }
    for (int64_t f = 0; f < F; ++f) out[r * F + f] = glu_act(act, h[f]) * h[F + f];
    free(x);
    free(h);
  }
}

/* The same with the normalisation deferred past the projections (self-check
 * only): W* = diag(g) W in fp64 (Prop. 1), and the per-token scale s = 1/RMSe(a)
 * applied after the matrix multiply (Prop. 2).  For ReGLU and the bilinear GLU
 * both branch scales merge into one factor s^2 = 1/MSe(a) = 1/(eps + sum a^2/K)
 * on the product (App. "FFN with ReGLU and Bilinear GLU": ReLU(s t) = s ReLU(t)
 * for s >= 0); SwiGLU keeps the scale inside the silu (Fig. 3). */
ORACLE_EXPORT void fn_oracle_glu_act_deferred(const double* a, int64_t M, int64_t K,
                                              const double* g, const double* Wgu, int64_t F,
                                              double eps, int act, const int64_t* rows,
                                              int64_t nrows, double* out) {
  (void)M;
  const int64_t N2 = 2 * F;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < nrows; ++r) {
    const double* ar = a + row_of(rows, r) * K;
    double* h = (double*)calloc((size_t)N2, sizeof(double));
    double ss = 0.0;
    for (int64_t k = 0; k < K; ++k) ss += ar[k] * ar[k];
    const double ms = eps + ss / (double)K;
    for (int64_t k = 0; k < K; ++k) {
      const double* wk = Wgu + k * N2;
      for (int64_t n = 0; n < N2; ++n) h[n] += ar[k] * (g[k] * wk[n]);
    }
    for (int64_t f = 0; f < F; ++f) {
      if (act == 0) {
        const double s = 1.0 / sqrt(ms);
        out[r * F + f] = silu(s * h[f]) * (s * h[F + f]);
      } else {
        out[r * F + f] = glu_act(act, h[f]) * h[F + f] / ms;
      }
    }
    free(h);
  }
}

/* A whole FFN after an RMSNorm, standard form: x = RMSNorm(a; g), then
 *   act 3 (App. "FFN with ReLU", Fig. 2(a)):  h = ReLU(x Wup), Wup [K, F];
 *   act 0/1/2 (Fig. 3(a), Fig. 4(a)):         h = act(x Wg) * (x Wu), Wup = [Wg | Wu], [K, 2F];
 * and y = h Wdown, Wdown [F, N]. */
ORACLE_EXPORT void fn_oracle_rmsnorm_ffn(const double* a, int64_t M, int64_t K, const double* g,
                                         const double* Wup, int64_t F, const double* Wdown,
                                         int64_t N, double eps, int act, const int64_t* rows,
                                         int64_t nrows, double* y) {
  (void)M;
  const int64_t NU = act == 3 ? F : 2 * F;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < nrows; ++r) {
    const double* ar = a + row_of(rows, r) * K;
    double* x = (double*)malloc(sizeof(double) * (size_t)K);
    double* u = (double*)calloc((size_t)NU, sizeof(double));
    double* h = (double*)malloc(sizeof(double) * (size_t)F);
    double rms = fn_oracle_rms(ar, K, eps);
    for (int64_t k = 0; k < K; ++k) x[k] = ar[k] / rms * g[k];
    for (int64_t k = 0; k < K; ++k) {
      const double* wk = Wup + k * NU;
      for (int64_t n = 0; n < NU; ++n) u[n] += x[k] * wk[n];
    }
    for (int64_t f = 0; f < F; ++f) h[f] = act == 3 ? glu_act(3, u[f]) : glu_act(act, u[f]) * u[F + f];
    double* yr = y + r * N;
    for (int64_t n = 0; n < N; ++n) yr[n] = 0.0;
    for (int64_t f = 0; f < F; ++f) {
      const double* wf = Wdown + f * N;
      for (int64_t n = 0; n < N; ++n) yr[n] += h[f] * wf[n];
    }
    free(x);
    free(u);
    free(h);
  }
}

/* LayerNorm followed by a linear layer, standard form (Sec. 2 "Normalization in
 * transformers": centering, then RMS scaling with g, then the bias beta; the
 * epsilon sits inside the root as in App. "RMS with epsilon"):
 *   mu = (1/K) sum a_k,  v = (1/K) sum (a_k - mu)^2   (two passes),
 *   x_k = (a_k - mu) / sqrt(v + eps) * g_k + beta_k,  y = x W (+ c). */
ORACLE_EXPORT void fn_oracle_layernorm_linear(const double* a, int64_t M, int64_t K,
                                              const double* g, const double* beta,
                                              const double* W, int64_t N, double eps,
                                              const double* bias, const int64_t* rows,
                                              int64_t nrows, double* y) {
  (void)M;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < nrows; ++r) {
    const double* ar = a + row_of(rows, r) * K;
    double* yr = y + r * N;
    double* x = (double*)malloc(sizeof(double) * (size_t)K);
    double mu = 0.0;
    for (int64_t k = 0; k < K; ++k) mu += ar[k];
    mu /= (double)K;
    double v = 0.0;
    for (int64_t k = 0; k < K; ++k) v += (ar[k] - mu) * (ar[k] - mu);
    v /= (double)K;
    double sigma = sqrt(v + eps);
    for (int64_t k = 0; k < K; ++k) x[k] = (ar[k] - mu) / sigma * g[k] + beta[k];
    for (int64_t n = 0; n < N; ++n) yr[n] = 0.0;
    for (int64_t k = 0; k < K; ++k) {
      const double* wk = W + k * N;
      for (int64_t n = 0; n < N; ++n) yr[n] += x[k] * wk[n];
    }
    if (bias)
      for (int64_t n = 0; n < N; ++n) yr[n] += bias[n];
    free(x);
  }
}

/* Deferred LayerNorm -> linear, self-check only.  Composed from the paper's
 * pieces: the normalisation bias moves past W as c* = c + beta W (Sec. 3.4),
 * g folds into W* (Prop. 1), the scalar 1/sigma is deferred to the output
 * (Prop. 2), and the centering term is exchanged with the sum over k as in the
 * row-sum step of Sec. 3.5:  sum_k (a_k - mu) W*[k,n] = (a W*)_n - mu colsum(W*)_n.
 *   y_n = ((a W*)_n - mu * colsum(W*)_n) / sigma + c*_n. */
ORACLE_EXPORT void fn_oracle_layernorm_linear_deferred(const double* a, int64_t M, int64_t K,
                                                       const double* g, const double* beta,
                                                       const double* W, int64_t N, double eps,
                                                       const double* bias, const int64_t* rows,
                                                       int64_t nrows, double* y) {
  (void)M;
  double* Ws = (double*)malloc(sizeof(double) * (size_t)(K * N));
  double* colsum = (double*)calloc((size_t)N, sizeof(double));
  double* cstar = (double*)calloc((size_t)N, sizeof(double));
  for (int64_t k = 0; k < K; ++k)
    for (int64_t n = 0; n < N; ++n) {
      Ws[k * N + n] = g[k] * W[k * N + n];
      colsum[n] += Ws[k * N + n];
      cstar[n] += beta[k] * W[k * N + n];
    }
  if (bias)
    for (int64_t n = 0; n < N; ++n) cstar[n] += bias[n];
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < nrows; ++r) {
    const double* ar = a + row_of(rows, r) * K;
    double* yr = y + r * N;
    double sa = 0.0, ss = 0.0;
    for (int64_t k = 0; k < K; ++k) {
      sa += ar[k];
      ss += ar[k] * ar[k];
    }
    double mu = sa / (double)K;
    double var = ss / (double)K - mu * mu;
    double inv_sigma = 1.0 / sqrt(var + eps);
    for (int64_t n = 0; n < N; ++n) yr[n] = 0.0;
    for (int64_t k = 0; k < K; ++k)
      for (int64_t n = 0; n < N; ++n) yr[n] += ar[k] * Ws[k * N + n];
    for (int64_t n = 0; n < N; ++n) yr[n] = (yr[n] - mu * colsum[n]) * inv_sigma + cstar[n];
  }
  free(Ws);
  free(colsum);
  free(cstar);
}

/* Round a double to the nearest bfloat16 value, ties to even, returned as a
 * double.  bfloat16 keeps fp32's 8-bit exponent and 8 significant bits
 * (7 stored).  Written from the format's definition: scale x into [2^7, 2^8)
 * (or, below fp32's normal range, to bfloat16's fixed subnormal spacing
 * 2^-133), round the significand to an integer with ties to even, scale back. */
ORACLE_EXPORT double fn_oracle_round_bf16(double x) {
  if (x == 0.0 || isnan(x) || isinf(x)) return x;
  int e2;
  (void)frexp(fabs(x), &e2); /* |x| = m * 2^e2, m in [0.5, 1) */
  int q = e2 - 8;            /* spacing of 8-bit significands at this binade */
  if (q < -133) q = -133;    /* subnormal spacing of bfloat16 */
  double s = ldexp(x, -q);   /* exact: power-of-two scaling */
  double r = nearbyint(s);   /* default rounding mode: nearest, ties to even */
  double out = ldexp(r, q);
  if (fabs(out) > 3.3895313892515355e38) out = copysign(INFINITY, x); /* beyond max bf16 */
  return out;
}

/* Round a double to the nearest fp32 value, ties to even (C's conversion in the
 * default rounding mode). */
ORACLE_EXPORT double fn_oracle_round_f32(double x) { return (double)(float)x; }

/* Expected result of folding the normalisation weights into the linear layer
 * (Prop. 1: W*[k,n] = g_k W[k,n]) when W* is stored in a finite precision:
 * the exact product, rounded once to the storage type (0 = fp32,
 * 1 = bfloat16).  Also the LayerNorm extras: colsum[n] = sum_k of the STORED
 * W*[k,n] (what the matrix multiply actually sees), and
 * c*[n] = sum_k beta_k W[k,n] with the unfolded W (Sec. 3.4).  Any of
 * Ws_out, colsum, cstar may be NULL; beta may be NULL (then cstar is not
 * written). */
ORACLE_EXPORT void fn_oracle_fold(const double* W, const double* g, const double* beta, int64_t K,
                                  int64_t N, int storage, double* Ws_out, double* colsum,
                                  double* cstar) {
  if (colsum)
    for (int64_t n = 0; n < N; ++n) colsum[n] = 0.0;
  if (cstar && beta)
    for (int64_t n = 0; n < N; ++n) cstar[n] = 0.0;
  for (int64_t k = 0; k < K; ++k)
    for (int64_t n = 0; n < N; ++n) {
      double p = g[k] * W[k * N + n];
      double st = storage == 1 ? fn_oracle_round_bf16(p) : fn_oracle_round_f32(p);
      if (Ws_out) Ws_out[k * N + n] = st;
      if (colsum) colsum[n] += st;
      if (cstar && beta) cstar[n] += beta[k] * W[k * N + n];
    }
}
