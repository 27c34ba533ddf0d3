/*
 * bgpo_testing.h - test hooks of libbgpo, not part of the ELBO-head API.
 */
#ifndef BGPO_TESTING_H_
#define BGPO_TESTING_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The bf16 MFMA GEMM core of the production kernels alone, used to test it in
 * isolation:
 *   C[m][n] = sum_k A[m][k] * B[n][k]   (fp32 result, fp32 accumulation)
 * A bf16 [M, K], B bf16 [N, K], C float [M, N], all row-major device memory.
 * Requires M, N >= 1 and K a positive multiple of 64.  Returns 0, -1 (invalid
 * argument) or -3 (HIP error).  Enqueued on `stream` (hipStream_t). */
int bgpo_test_gemm_nt(const uint16_t* A, const uint16_t* B, float* C, int32_t M, int32_t N,
                      int32_t K, void* stream);

/* Tile-configuration variants of the GEMM (fp32 store), for tuning; 0-17 are
 * the earlier core on 32x32x16 MFMAs (compiler-scheduled, accumulators in
 * VGPRs):
 * variant 0: 256x256 tile, K slab 32, 4-stage LDS ring (four waves of 128x128)
 *         1: 5 stages, 2: K slab 64 in 2 stages,
 *         3: 256x128 tile, 3 stages, two workgroups per compute unit
 *         4: 128x256 tile, 3 stages, two workgroups per compute unit
 *         5: 256x256 tile, K slab 64, 2 stages, 8 waves of 128x64
 *         6: as 5 with 8 waves of 64x128
 *         7: as 2 with the 256-byte LDS swizzle; 8: as 5 with that swizzle (the
 *            earlier production configuration)
 *         9: 8 waves of 128x64, K slab 32, 4 stages; 10: as 9 with 5 stages
 *         11: as 6 with the 256-byte swizzle
 *         12: 256x128 tile, K slab 32, 3 stages, 256-byte swizzle, two
 *             independent 4-wave workgroups per compute unit; 13: 128x256
 *         14: 4 waves of 128x128, K slab 32, 4 stages, 256-byte swizzle;
 *         15: as 14 with 5 stages
 *         16: as 9 with the 256-byte swizzle; 17: as 10 with that swizzle
 *         18: four waves of 128x128 on 16x16x32 MFMAs, K slab 64 in 2 stages,
 *             256-byte swizzle (the production kernel, as bgpo_test_gemm_nt)
 *         19: as 18 on a 4-stage ring of 32-deep slabs (same LDS, one barrier
 *             per 32-deep MFMA sub-step instead of per two)
 * flags bit 0: M tiles consecutive in the tile walk (else N tiles);
 *       bit 1: plain workgroup order (no XCD grouping);
 *       bits 8-15: if nonzero, band height (M tiles) of the tile walk;
 *       bits 16-23: if > 1, split K into that many slices, slice s written to
 *                   C + s * M * N (C then holds that many M x N blocks).
 * Same shape rules and return codes as bgpo_test_gemm_nt. */
int bgpo_test_gemm_variant(const uint16_t* A, const uint16_t* B, float* C, int32_t M, int32_t N,
                           int32_t K, int32_t variant, int32_t flags, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BGPO_TESTING_H_ */
