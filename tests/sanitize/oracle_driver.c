/*
 * Sanitizer driver of the fp64 CPU oracle (test infrastructure): built with
 * -fsanitize=address,undefined together with oracle/flashnorm_oracle.c and run by
 * tests/test_sanitizers.py.  Every buffer is allocated at exactly the size its
 * function documents, so an out-of-bounds access or undefined behaviour in the oracle
 * aborts the run.  A few closed forms are checked on the way (the worked example of
 * Sec. 3.1, the agreement of the standard, weightless and deferred forms of
 * Props. 1 and 2, the LayerNorm exchange of Sec. 3.5), with edge shapes (K = 1,
 * N = 1, M = 1) and row subsets.  Exit status 0 = clean.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void fn_oracle_rmsnorm_linear(const double*, int64_t, int64_t, const double*, const double*, int64_t, double,
                              const double*, const int64_t*, int64_t, double*);
void fn_oracle_weightless(const double*, int64_t, int64_t, const double*, const double*, int64_t, double,
                          const double*, const int64_t*, int64_t, double*);
void fn_oracle_deferred(const double*, int64_t, int64_t, const double*, const double*, int64_t, double,
                        const double*, const int64_t*, int64_t, double*);
void fn_oracle_rmsnorm_swiglu(const double*, int64_t, int64_t, const double*, const double*, int64_t, double,
                              const int64_t*, int64_t, double*);
void fn_oracle_rmsnorm_glu_act(const double*, int64_t, int64_t, const double*, const double*, int64_t, double, int,
                               const int64_t*, int64_t, double*);
void fn_oracle_glu_act_deferred(const double*, int64_t, int64_t, const double*, const double*, int64_t, double, int,
                                const int64_t*, int64_t, double*);
void fn_oracle_rmsnorm_ffn(const double*, int64_t, int64_t, const double*, const double*, int64_t, const double*,
                           int64_t, double, int, const int64_t*, int64_t, double*);
void fn_oracle_layernorm_linear(const double*, int64_t, int64_t, const double*, const double*, const double*, int64_t,
                                double, const double*, const int64_t*, int64_t, double*);
void fn_oracle_layernorm_linear_deferred(const double*, int64_t, int64_t, const double*, const double*,
                                         const double*, int64_t, double, const double*, const int64_t*, int64_t,
                                         double*);
double fn_oracle_rms(const double*, int64_t, double);
double fn_oracle_round_bf16(double);
double fn_oracle_round_f32(double);
void fn_oracle_fold(const double*, const double*, const double*, int64_t, int64_t, int, double*, double*, double*);

static int failures = 0;
static void check(int ok, const char* what) {
  if (!ok) {
    fprintf(stderr, "FAIL: %s\n", what);
    ++failures;
  }
}

static double* vec(int64_t n) { return (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1)); }

static uint64_t state = 0x9e3779b97f4a7c15ull;
static double rnd(void) {  /* splitmix64 -> uniform [-1, 1) */
  uint64_t z = (state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z ^= z >> 31;
  return (double)(z >> 11) / 4503599627370496.0 - 1.0;
}
static double* rvec(int64_t n, double lo, double hi) {
  double* v = vec(n);
  for (int64_t i = 0; i < n; ++i) v[i] = lo + (hi - lo) * 0.5 * (rnd() + 1.0);
  return v;
}
static double maxdiff(const double* x, const double* y, int64_t n) {
  double d = 0.0;
  for (int64_t i = 0; i < n; ++i) d = fmax(d, fabs(x[i] - y[i]));
  return d;
}

/* All linear-layer forms and the LayerNorm forms on one shape and row subset. */
static void shapes(int64_t M, int64_t K, int64_t N, int use_rows) {
  double *a = rvec(M * K, -2, 2), *g = rvec(K, 0.5, 1.5), *W = rvec(K * N, -1, 1), *bias = rvec(N, -1, 1);
  double* beta = rvec(K, -0.5, 0.5);
  int64_t rows[2] = {M - 1, 0};
  const int64_t* rp = use_rows ? rows : NULL;
  const int64_t nr = use_rows ? (M > 1 ? 2 : 1) : M;
  double *y0 = vec(nr * N), *y1 = vec(nr * N), *y2 = vec(nr * N);
  fn_oracle_rmsnorm_linear(a, M, K, g, W, N, 1e-6, bias, rp, nr, y0);
  fn_oracle_weightless(a, M, K, g, W, N, 1e-6, bias, rp, nr, y1);
  fn_oracle_deferred(a, M, K, g, W, N, 1e-6, bias, rp, nr, y2);
  check(maxdiff(y0, y1, nr * N) < 1e-12 && maxdiff(y0, y2, nr * N) < 1e-12, "forms (a) = (b) = (c)");
  fn_oracle_layernorm_linear(a, M, K, g, beta, W, N, 1e-5, bias, rp, nr, y0);
  fn_oracle_layernorm_linear_deferred(a, M, K, g, beta, W, N, 1e-5, bias, rp, nr, y1);
  check(maxdiff(y0, y1, nr * N) < 1e-11, "LayerNorm standard = deferred");
  free(a), free(g), free(W), free(bias), free(beta), free(y0), free(y1), free(y2);
}

static void glu_shapes(int64_t M, int64_t K, int64_t F) {
  double *a = rvec(M * K, -2, 2), *g = rvec(K, 0.5, 1.5), *Wgu = rvec(K * 2 * F, -1, 1);
  double *Wdown = rvec(F * 3, -1, 1), *o0 = vec(M * F), *o1 = vec(M * F), *y = vec(M * 3);
  int64_t rows[1] = {M - 1};
  fn_oracle_rmsnorm_swiglu(a, M, K, g, Wgu, F, 1e-6, NULL, M, o0);
  fn_oracle_rmsnorm_glu_act(a, M, K, g, Wgu, F, 1e-6, 0, NULL, M, o1);
  check(maxdiff(o0, o1, M * F) < 1e-13, "SwiGLU = GLU act 0");
  for (int act = 0; act < 3; ++act) {
    fn_oracle_rmsnorm_glu_act(a, M, K, g, Wgu, F, 1e-6, act, rows, 1, o0);
    fn_oracle_glu_act_deferred(a, M, K, g, Wgu, F, 1e-6, act, rows, 1, o1);
    check(maxdiff(o0, o1, F) < 1e-11, "GLU standard = deferred");
  }
  for (int act = 0; act < 4; ++act) fn_oracle_rmsnorm_ffn(a, M, K, g, Wgu, F, Wdown, 3, 1e-6, act, NULL, M, y);
  free(a), free(g), free(Wgu), free(Wdown), free(o0), free(o1), free(y);
}

int main(void) {
  /* Sec. 3.1 worked example: a = (3, 4, 0, 0), eps = 0: RMS = 5/2; g = (1, 2, 1, 1), W = I
     gives y = (6/5, 16/5, 0, 0). */
  double* a = vec(4);
  double* g = vec(4);
  double* W = vec(16);
  double* y = vec(4);
  const double av[4] = {3, 4, 0, 0}, gv[4] = {1, 2, 1, 1};
  for (int i = 0; i < 4; ++i) a[i] = av[i], g[i] = gv[i];
  for (int i = 0; i < 16; ++i) W[i] = (i % 5 == 0) ? 1.0 : 0.0;
  check(fn_oracle_rms(a, 4, 0.0) == 2.5, "RMS(3, 4, 0, 0) = 5/2");
  fn_oracle_rmsnorm_linear(a, 1, 4, g, W, 4, 0.0, NULL, NULL, 1, y);
  check(fabs(y[0] - 1.2) < 1e-15 && fabs(y[1] - 3.2) < 1e-15 && y[2] == 0.0 && y[3] == 0.0, "worked example");
  free(a), free(g), free(W), free(y);

  shapes(1, 1, 1, 0);
  shapes(3, 5, 7, 1);
  shapes(4, 16, 1, 0);
  shapes(2, 33, 9, 1);
  glu_shapes(1, 1, 1);
  glu_shapes(3, 12, 5);

  /* Rounding helpers and the fold (Prop. 1; Sec. 3.4) in both storage types. */
  check(fn_oracle_round_bf16(1.0 + 0x1p-8) == 1.0, "bf16 tie to even");
  check(fn_oracle_round_bf16(1.0 + 3 * 0x1p-9) == 1.0 + 0x1p-7, "bf16 round up");
  check(fn_oracle_round_f32(1.0 + 0x1p-30) == 1.0, "fp32 rounding");
  for (int storage = 0; storage < 2; ++storage) {
    const int64_t K = 7, N = 3;
    double *Wf = rvec(K * N, -1, 1), *gf = rvec(K, 0.5, 1.5), *bf = rvec(K, -1, 1);
    double *Ws = vec(K * N), *cs = vec(N), *cb = vec(N);
    fn_oracle_fold(Wf, gf, bf, K, N, storage, Ws, cs, cb);
    fn_oracle_fold(Wf, gf, NULL, K, N, storage, Ws, cs, NULL);
    double s0 = 0.0;
    for (int64_t k = 0; k < K; ++k) s0 += Ws[k * N];
    check(fabs(s0 - cs[0]) < 1e-12, "colsum of the stored W*");
    free(Wf), free(gf), free(bf), free(Ws), free(cs), free(cb);
  }
  if (failures) {
    fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  printf("oracle sanitizer driver: clean\n");
  return 0;
}
