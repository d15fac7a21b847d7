// Launch stubs for the host-only sanitizer build of the C ABI (test infrastructure):
// every kernel launcher the ABI calls records its arguments and returns success, so
// the argument validation and translation in api.hip run on a machine without a GPU.
#include "abi_stub_record.h"
#include "fn_launch.h"

fnstub_record fnstub_last;
int fnstub_launches = 0;
int fnstub_hip_calls = 0;

static hipError_t rec(int kind, int64_t M, int64_t K, int64_t lda, int64_t NP, int64_t KP, int64_t ncols,
                      int64_t ldy, int64_t cfg, int64_t epi, int64_t sk = 0, int64_t sn = 0) {
  fnstub_last = fnstub_record{kind, M, K, lda, NP, KP, ncols, ldy, cfg, epi, sk, sn};
  ++fnstub_launches;
  return hipSuccess;
}

namespace fn {
hipError_t launch_prefill_bf16(const PrefillArgs& p) {
  return rec(1, p.M, p.K, p.lda, p.NP, p.KP, p.ncols, p.ldy, p.tile, p.epi);
}
hipError_t launch_decode_bf16(const DecodeArgs& p) {
  return rec(2, p.M, p.K, p.lda, p.NP, p.KP, p.ncols, p.ldy, p.cfg, p.epi);
}
hipError_t launch_f32(const F32Args& p) { return rec(3, p.M, p.K, p.lda, p.NP, p.KP, p.ncols, p.ldy, p.cfg, p.epi); }
hipError_t launch_fold(const FoldArgs& p) { return rec(4, 0, p.K, 0, 0, 0, p.N, 0, 0, p.glu, p.sk, p.sn); }
hipError_t launch_unpack(const void*, int64_t K, int64_t N, int glu, int, void*, int64_t ldo, hipStream_t) {
  return rec(5, 0, K, 0, 0, 0, N, ldo, 0, glu);
}
hipError_t launch_norm_rows(const void*, int M, int K, int lda, int, const float*, const float*, float, void*, int ldx,
                            hipStream_t) {
  return rec(6, M, K, lda, 0, 0, 0, ldx, 0, 0);
}
hipError_t launch_headnorm_rows(void*, int M, int ldy, int ncols, const EpiArgs&, hipStream_t) {
  return rec(7, M, 0, 0, 0, 0, ncols, ldy, 0, 0);
}
hipError_t launch_rope_rows(void*, int M, int ldy, int, int qk, int, int h, const int*, const float*, const float*, int,
                            float, hipStream_t) {
  return rec(8, M, h, 0, 0, 0, qk, ldy, 0, 0);
}
hipError_t launch_mla_latent_rows(void*, int M, int ldy, int, int L, int R, const float*, float, const float*,
                                  const int*, const float*, const float*, int, hipStream_t) {
  return rec(9, M, L, R, 0, 0, L + R, ldy, 0, 0);
}
}  // namespace fn
