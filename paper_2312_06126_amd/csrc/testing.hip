// Test hooks (include/spz_testing.h): the GEMM kernels on caller-owned device memory.
#include "../../include/spz_testing.h"
#include "internal.h"

using namespace spz;

extern "C" int spzt_gemm(int32_t bf16, int32_t mode, int32_t M, int32_t N, int32_t K, int32_t splits,
                         const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
                         const float* bias, const void* mask, int64_t ldm, int32_t relu, int32_t out_f32) {
  if (mode < 0 || mode > 2 || splits < 1 || !A || !B || !C) return SPZ_EINVAL;
  GemmArgs g{};
  g.A = A; g.lda = lda; g.B = B; g.ldb = ldb; g.C = C; g.ldc = ldc;
  g.bias = bias; g.mask = mask; g.ldm = ldm; g.M = M; g.N = N; g.K = K;
  g.relu = relu; g.out_f32 = out_f32; g.splits = splits;
  float* part = nullptr;
  if (mode == GEMM_WGRAD) {
    if (hipMalloc(&part, (size_t)splits * M * N * 4) != hipSuccess) return SPZ_ENOMEM;
    g.C = part;
    g.ldc = N;
  }
  hipError_t e = gemm(bf16 != 0, (GemmMode)mode, g, nullptr);
  if (e == hipSuccess && mode == GEMM_WGRAD) e = splitk_reduce(part, splits, M, N, N, (float*)C, ldc, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (part) (void)hipFree(part);
  if (e == hipErrorInvalidValue) return SPZ_EINVAL;
  return e == hipSuccess ? SPZ_OK : SPZ_EHIP;
}
