// Host-only sanitizer driver of the C ABI (test infrastructure): calls the entry points
// of include/flashnorm.h with invalid and valid arguments (addresses that are never
// dereferenced on the host) and checks the returned status, that invalid calls launch
// nothing, and what the valid ones would launch.  Built with ASan/UBSan against the
// launch stubs; run by tests/test_sanitizers.py.  Exit status 0 = clean.
#include <stdint.h>
#include <stdio.h>

#include "abi_stub_record.h"
#include "flashnorm.h"

static int failures = 0;
#define CHECK(cond)                                              \
  do {                                                           \
    if (!(cond)) {                                               \
      fprintf(stderr, "FAIL line %d: %s\n", __LINE__, #cond);    \
      ++failures;                                                \
    }                                                            \
  } while (0)

static void* P(uintptr_t x) { return reinterpret_cast<void*>(x); }
static float* PF(uintptr_t x) { return reinterpret_cast<float*>(x); }
static const uintptr_t A = 0x100000, W = 0x10000000, Y = 0x20000000, X = 0x30000000, B = 0x40000000;

// An invalid call returns `status` and launches nothing.
#define REJECT(status, call)             \
  do {                                   \
    const int before = fnstub_launches;  \
    CHECK((call) == (status));           \
    CHECK(fnstub_launches == before);    \
  } while (0)

int main() {
  // flashnorm_linear: shapes, dtypes, alignment, eps, aliasing, sizes.
  auto lin = [](int64_t M, int64_t K, int64_t lda, int dt, uintptr_t a, uintptr_t y, int64_t ldy, float eps, int path) {
    return flashnorm_linear_ex(P(a), M, K, lda, dt, P(W), 64, eps, nullptr, P(y), ldy, dt, nullptr, path, nullptr);
  };
  REJECT(FN_ERR_SHAPE, lin(-1, 128, 128, FN_BF16, A, Y, 64, 1e-6f, 0));
  REJECT(FN_ERR_SHAPE, lin(4, 0, 128, FN_BF16, A, Y, 64, 1e-6f, 0));
  REJECT(FN_ERR_SHAPE, lin(4, 128, 64, FN_BF16, A, Y, 64, 1e-6f, 0));
  REJECT(FN_ERR_SHAPE, lin(4, 124, 128, FN_BF16, A, Y, 64, 1e-6f, 0));  // bf16 K % 8
  REJECT(FN_ERR_DTYPE, lin(4, 128, 128, 9, A, Y, 64, 1e-6f, 0));
  REJECT(FN_ERR_ALIGN, lin(4, 128, 128, FN_BF16, A + 2, Y, 64, 1e-6f, 0));
  REJECT(FN_ERR_VALUE, lin(4, 128, 128, FN_BF16, A, Y, 64, -1.0f, 0));
  REJECT(FN_ERR_VALUE, lin(4, 128, 128, FN_BF16, A, Y, 64, 1e-6f, 7));
  REJECT(FN_ERR_VALUE, lin(4, 128, 128, FN_F32, A, Y, 64, 1e-6f, 4 << FN_PATH_TILE_SHIFT));
  REJECT(FN_ERR_ALIAS, lin(4, 128, 128, FN_BF16, A, A + 64, 64, 1e-6f, 0));
  REJECT(FN_ERR_SIZE, lin(4, 1 << 22, 1 << 22, FN_BF16, A, Y, 64, 1e-6f, 0));
  REJECT(FN_ERR_UNSUPPORTED, lin(32, 128, 128, FN_BF16, A, Y, 64, 1e-6f, FN_PATH_DECODE));
  CHECK(lin(0, 128, 128, FN_BF16, 0, 0, 64, 1e-6f, 0) == FN_OK);  // M = 0: no-op

  // Valid calls: the kernel chosen and the packed geometry it is given.
  CHECK(lin(300, 200, 208, FN_BF16, A, Y, 64, 1e-6f, 0) == FN_OK);
  CHECK(fnstub_last.kind == 1 && fnstub_last.M == 300 && fnstub_last.K == 200 && fnstub_last.lda == 208);
  CHECK(fnstub_last.NP == 64 && fnstub_last.KP == 256 && fnstub_last.ncols == 64 && fnstub_last.cfg == 0);
  CHECK(lin(16, 200, 208, FN_BF16, A, Y, 64, 1e-6f, 0) == FN_OK && fnstub_last.kind == 2);  // M <= 16: decode
  CHECK(lin(16, 200, 208, FN_BF16, A, Y, 64, 1e-6f, FN_PATH_PREFILL | (19 << FN_PATH_TILE_SHIFT)) == FN_OK);
  CHECK(fnstub_last.kind == 1 && fnstub_last.cfg == 19);
  CHECK(lin(16, 200, 200, FN_F32, A, Y, 64, 1e-6f, 2 << FN_PATH_TILE_SHIFT) == FN_OK);
  CHECK(fnstub_last.kind == 3 && fnstub_last.cfg == 2);

  // GLU: F columns out, 2F packed with gate/up pairs.
  CHECK(flashnorm_glu(P(A), 40, 128, 128, FN_BF16, P(W), 45, 1e-6f, P(Y), 48, FN_BF16, nullptr) == FN_OK);
  CHECK(fnstub_last.kind == 1 && fnstub_last.NP == 2 * 48 && fnstub_last.ncols == 45);

  // LayerNorm needs colsum; c* is optional.
  REJECT(FN_ERR_NULL, flashnorm_layernorm_linear(P(A), 4, 64, 64, FN_BF16, P(W), nullptr, nullptr, 32, 1e-5f, P(Y),
                                                 32, FN_BF16, nullptr));
  CHECK(flashnorm_layernorm_linear(P(A), 4, 64, 64, FN_BF16, P(W), PF(X), nullptr, 32, 1e-5f, P(Y), 32, FN_BF16,
                                   nullptr) == FN_OK);

  // fold_weights: strided views, aliasing of the strided extent, sizes.
  auto fold = [](const void* w, int64_t sk, int64_t sn, int64_t K, int64_t N, uintptr_t ws) {
    return fold_weights(w, sk, sn, FN_BF16, PF(X), nullptr, K, N, FN_LAYOUT_LINEAR, P(ws), FN_BF16, nullptr,
                        nullptr, nullptr);
  };
  REJECT(FN_ERR_SHAPE, fold(P(A), -1, 1, 64, 32, W));
  REJECT(FN_ERR_SIZE, fold(P(A), int64_t(1) << 40, 1, 64, 32, W));
  REJECT(FN_ERR_ALIAS, fold(P(A), 1, 64, 64, 32, A + 4096 - 16));  // transposed view's last element
  CHECK(fold(P(A), 1, 64, 64, 32, A + 4096) == FN_OK);
  CHECK(fnstub_last.kind == 4 && fnstub_last.sk == 1 && fnstub_last.sn == 64 && fnstub_last.K == 64);
  CHECK(fold_weights_size(64, 32, FN_LAYOUT_LINEAR, FN_BF16) == 64 * 32 * 2);
  CHECK(fold_weights_size(0, 32, FN_LAYOUT_LINEAR, FN_BF16) == 0);

  // Unfused baselines: workspace checks, then the norm kernel and the product.
  REJECT(FN_ERR_NULL, baseline_rmsnorm_linear(P(A), 4, 64, 64, FN_BF16, PF(X), P(W), 32, 1e-6f, nullptr, P(Y), 32, 0,
                                              nullptr));
  REJECT(FN_ERR_ALIAS, baseline_rmsnorm_linear(P(A), 4, 64, 64, FN_BF16, PF(X), P(W), 32, 1e-6f, P(A), P(Y), 32, 0,
                                               nullptr));
  const int before = fnstub_launches;
  CHECK(baseline_rmsnorm_linear(P(A), 4, 64, 64, FN_BF16, PF(X), P(W), 32, 1e-6f, P(B), P(Y), 32, 0, nullptr) == FN_OK);
  CHECK(fnstub_launches == before + 2 && fnstub_last.kind == 2);

  // The no-allocation entry point refuses inputs beyond its array before any device call.
  const int hip_before = fnstub_hip_calls;
  REJECT(FN_ERR_SIZE, baseline_rmsnorm_linear_noalloc(P(A), 4097, 4096, 4096, FN_BF16, PF(X), P(W), 64, 1e-6f, P(Y),
                                                      64, 0, nullptr));
  CHECK(baseline_rmsnorm_linear_noalloc(P(A), 0, 4096, 4096, FN_BF16, PF(X), P(W), 64, 1e-6f, P(Y), 64, 0,
                                        nullptr) == FN_OK);
  CHECK(fnstub_hip_calls == hip_before);

  // Attention-side entry points: head geometry and position tables.
  REJECT(FN_ERR_SHAPE, flashnorm_qkv_rope(P(A), 4, 64, 64, FN_BF16, P(W), 2, 1, 6, 1e-6f, nullptr, nullptr, PF(X),
                                          PF(B), 8, 0.5f, P(Y), 64, FN_BF16, nullptr, 0, nullptr));
  CHECK(flashnorm_qkv_rope(P(A), 40, 64, 64, FN_BF16, P(W), 2, 1, 16, 1e-6f, nullptr,
                           reinterpret_cast<const int32_t*>(B), PF(X), PF(X + 4096), 8, 0.25f, P(Y), 64, FN_BF16,
                           nullptr, 0, nullptr) == FN_OK);

  for (int s = 1; s >= -9; --s) CHECK(flashnorm_status_string(s) != nullptr);
  if (failures) {
    fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  printf("ABI sanitizer driver: clean (%d launches recorded)\n", fnstub_launches);
  return 0;
}
