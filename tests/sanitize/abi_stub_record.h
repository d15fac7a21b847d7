/* What the launch stubs of the host-only sanitizer build record about the last launch
 * the C ABI asked for (test infrastructure). */
#pragma once
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif
typedef struct {
  int kind;  /* 1 prefill, 2 decode, 3 fp32, 4 fold, 5 unpack, 6 norm rows, 7 head norm, 8 rope, 9 mla */
  int64_t M, K, lda, NP, KP, ncols, ldy, cfg, epi, sk, sn;
} fnstub_record;
extern fnstub_record fnstub_last;
extern int fnstub_launches;     /* launches requested since the start */
extern int fnstub_hip_calls;    /* HIP runtime calls made by the library (device lookups) */
#ifdef __cplusplus
}
#endif
