/*
 * spz_testing.h -- test hooks of libspz.so (not part of the update API).
 *
 * Direct access to the matrix-product kernels the update is built from, for
 * unit tests against a host reference. All pointers are DEVICE pointers owned
 * by the caller; row-major layouts as in the update:
 *   mode 0 (forward):   C[M, N] = act(A[M, K] . B[N, K]^T + bias[N]), act = ReLU if relu
 *   mode 1 (dgrad):     C[M, N] = (A[M, K] . B[K, N]) * (mask[M, N] > 0 if mask)
 *   mode 2 (wgrad):     C[M, N] = A[K, M]^T . B[K, N]   (split over K in `splits` slices,
 *                                                        reduced in slice order)
 * bf16 != 0: A, B, mask (and C unless out_f32 or mode 2) are bfloat16; else float32.
 * Leading dimensions are in elements. Shapes must satisfy the kernels' tiling
 * contract (M and N multiples of 32 with M % 128 == 0 for modes 0 and 1, K a
 * multiple of 32 * splits); otherwise SPZ_EINVAL. Synchronous.
 */
#ifndef SPZ_TESTING_H
#define SPZ_TESTING_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int spzt_gemm(int32_t bf16, int32_t mode, int32_t M, int32_t N, int32_t K, int32_t splits, const void* A,
              int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc, const float* bias,
              const void* mask, int64_t ldm, int32_t relu, int32_t out_f32);

#ifdef __cplusplus
}
#endif

#endif /* SPZ_TESTING_H */
