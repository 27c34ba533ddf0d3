/*
 * bgpo_testing.h - test hooks of libbgpo, not part of the ELBO-head API.
 */
#ifndef BGPO_TESTING_H_
#define BGPO_TESTING_H_

#include <stddef.h>
#include <stdint.h>

#include "bgpo.h"

#ifdef __cplusplus
extern "C" {
#endif

/* The bf16 MFMA GEMM core of the production kernels alone (the kernel of the
 * dX GEMM, in its operand layouts), used to test it in isolation:
 *   C[m][n] = sum_k A[m][k] * B[n][k]   (fp32 result, fp32 accumulation)
 * A bf16 M x K in the library's K-slab-major operand layout (element (m, k)
 * at index ((k / 64) M + m) 64 + k % 64, i.e. [K/64][M][64]); B bf16 [N, K]
 * row-major; C float [M, N] row-major; all device memory.
 * Requires M, N >= 1 and K a positive multiple of 64.  Returns 0, -1 (invalid
 * argument) or -3 (HIP error).  Enqueued on `stream` (hipStream_t). */
int bgpo_test_gemm_nt(const uint16_t* A, const uint16_t* B, float* C, int32_t M, int32_t N,
                      int32_t K, void* stream);

/* The same core with K split into n_split slices (1 <= n_split <= 255), as
 * the dX GEMM splits the vocabulary: slice s covers K range
 * [s * ks, min(K, (s + 1) * ks)) with ks = ceil(K / n_split) rounded up to a
 * multiple of 64, and its product is written to C + s * M * N (C holds
 * n_split blocks of M x N floats; slices past K are stored as zeros).  Same
 * shape rules and return codes as bgpo_test_gemm_nt. */
int bgpo_test_gemm_split(const uint16_t* A, const uint16_t* B, float* C, int32_t M, int32_t N,
                         int32_t K, int32_t n_split, void* stream);

/* The dW GEMM's kernel alone, in its operand layouts: A is read with its
 * indices' roles swapped (the layout of the kept exponentials, M contiguous
 * within 64-wide slabs, through the transposing LDS reads) and the product
 * is added to C:
 *   C[n][m] += sum_k A[m][k] * B[n][k]   (fp32 accumulation into C)
 * A bf16 with element (m, k) at index ((m / 64) K + k) 64 + m % 64, i.e.
 * [M/64][K][64]; B bf16 in the K-slab-major layout, element (n, k) at
 * ((k / 64) N + n) 64 + k % 64, i.e. [K/64][N][64]; C float [N, M]
 * row-major, read and written; all device memory.  Requires N >= 1 and M, K
 * positive multiples of 64.  Returns 0, -1 (invalid argument) or -3 (HIP
 * error).  Enqueued on `stream` (hipStream_t). */
int bgpo_test_gemm_tn(const uint16_t* A, const uint16_t* B, float* C, int32_t M, int32_t N,
                      int32_t K, void* stream);

/* The multi-block form of the mask and compaction step (the three passes the
 * library uses above 65536 positions: mask words with per-block counts, a
 * one-block scan of the counts, a scatter), run at any size, with the same
 * arguments and outputs as bgpo_sample_masks; `scratch` is device memory of
 * at least bgpo_test_mask_scratch_bytes(prob) bytes, 256-byte aligned
 * (BGPO_ERR_WORKSPACE otherwise). */
size_t bgpo_test_mask_scratch_bytes(const bgpo_problem* prob);
int bgpo_test_mask_multiblock(const bgpo_problem* prob, const uint8_t* resp_mask, int32_t j,
                              int32_t* idx, int32_t* n_masked, float* t_out, void* scratch,
                              size_t scratch_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BGPO_TESTING_H_ */
