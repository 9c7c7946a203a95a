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
 * bf16 mode 1: the hook also builds the transposed image of B (a temporary device
 * buffer), which the large-tile kernel reads. mode 3: mode 1 with B passed through its
 * transposed image in either precision (the k-contiguous input-gradient path the
 * library takes for hidden layers).
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

/*
 * Fused epilogues of the large-tile bf16 kernel (bf16 operands; the whole product
 * must fit that kernel: M % 256 == 0, N % 128 == 0, K % 32 == 0; else SPZ_EINVAL).
 * Bit c % 32 of word bits[(c / 32) * ldbits + r] is mask element (r, c).
 *   mode 0: C = ReLU(A . B^T + bias) in bf16 (bias may be null);
 *           bits_out (or null): bits of C > 0;
 *           rdot_w [N] bf16 (or null): rdot_part[p * ldrd + r] = sum over columns c of
 *             group p (spzt_rdot_cols(M, N) columns each) of C[r, c] * rdot_w[c];
 *           no_store: C is not written (requires rdot_w).
 *   mode 1: C = (A . B) * bit(r, c) in bf16 (bits required; the hook builds the
 *           transposed image of B that the kernel reads);
 *           colsum (or null): colsum[t * ldcs + c] = sum of stored C[r, c] over the
 *             256 rows r of row tile t.
 * Synchronous.
 */
int spzt_gemm_fused(int32_t mode, int32_t M, int32_t N, int32_t K, const void* A, int64_t lda, const void* B,
                    int64_t ldb, void* C, int64_t ldc, const float* bias, uint32_t* bits_out, const uint32_t* bits,
                    int64_t ldbits, const void* rdot_w, float* rdot_part, int64_t ldrd, int32_t no_store,
                    float* colsum, int64_t ldcs);
/*
 * Input-gradient product C = (A . B) [* bit(r, c) with bits] restricted to the first
 * m_rows rows by a device-side row count (the form the library's SAC actor row split
 * uses; m_rows a multiple of 256, at most M): rows from m_rows on are not written.
 * Same operand conventions as spzt_gemm mode 1 (bf16 builds B's transposed image).
 * Synchronous.
 */
int spzt_gemm_dgrad_rows(int32_t bf16, int32_t M, int32_t N, int32_t K, const void* A, int64_t lda,
                         const void* B, int64_t ldb, void* C, int64_t ldc, const uint32_t* bits, int64_t ldbits,
                         int32_t out_f32, int32_t m_rows);
/* Columns per row-dot partial of an M x N forward product (its column tile over 2). */
int spzt_rdot_cols(int32_t M, int32_t N);
/*
 * The deferred reduction kernel on n <= 24 jobs in one launch (host arrays of the
 * per-job fields; part[i], out[i] device pointers): out[r * ldo + c] = sum over slices
 * z < slices of part[z * zstride + r * ld + c] for r < rows, c < cols, summed in a
 * fixed order: thread g of `groups` (a power of two up to 256) adds slices g,
 * g + groups, ... in turn, then the group sums are added in g order; vec (4 or 1)
 * columns per piece (4: cols, ld, ldo, zstride multiples of 4, 16-byte aligned
 * pointers). SPZ_EINVAL on a bad job. Synchronous.
 */
int spzt_reduce_jobs(int32_t n, const float* const* part, float* const* out, const int64_t* zstride,
                     const int64_t* ld, const int64_t* ldo, const int32_t* rows, const int32_t* cols,
                     const int32_t* slices, const int32_t* groups, const int32_t* vec);
/*
 * Checks the device float32 -> bfloat16 rounding used by every kernel against an
 * integer round-to-nearest-even over the float bit patterns [begin, begin + count)
 * (begin + count <= 2^32); a NaN input must give a NaN. *mismatches receives the
 * number of failing patterns.
 */
int spzt_bf16_round_check(uint64_t begin, uint64_t count, uint64_t* mismatches);

#ifdef __cplusplus
}
#endif

#endif /* SPZ_TESTING_H */
