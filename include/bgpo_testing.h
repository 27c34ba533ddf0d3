/*
 * bgpo_testing.h - test hooks of libbgpo, not part of the ELBO-head API.
 */
#ifndef BGPO_TESTING_H_
#define BGPO_TESTING_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The bf16 MFMA GEMM core alone, used to test it in isolation:
 *   C[m][n] = sum_k A[m][k] * B[n][k]   (fp32 result, fp32 accumulation)
 * A bf16 [M, K], B bf16 [N, K], C float [M, N], all row-major device memory.
 * Requires M, N >= 1 and K a positive multiple of 64.  Returns 0, -1 (invalid
 * argument) or -3 (HIP error).  Enqueued on `stream` (hipStream_t). */
int bgpo_test_gemm_nt(const uint16_t* A, const uint16_t* B, float* C, int32_t M, int32_t N,
                      int32_t K, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BGPO_TESTING_H_ */
