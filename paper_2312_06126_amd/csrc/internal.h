// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/spz.h"

namespace spz {

// ----------------------------------------------------------------------------- numerics
typedef uint16_t bf16_t;  // bfloat16 storage

__host__ __device__ inline float bf2f(bf16_t h) {
  union { uint32_t u; float f; } v;
  v.u = (uint32_t)h << 16;
  return v.f;
}

// float32 -> bfloat16, round to nearest, ties to even; NaN stays NaN.
__host__ __device__ inline bf16_t f2bf(float f) {
  union { uint32_t u; float f; } v;
  v.f = f;
  if ((v.u & 0x7F800000u) == 0x7F800000u && (v.u & 0x007FFFFFu)) return (bf16_t)0x7FC0;
  uint32_t r = v.u + 0x7FFFu + ((v.u >> 16) & 1u);
  return (bf16_t)(r >> 16);
}

template <typename T> __host__ __device__ inline float to_f(T x);
template <> __host__ __device__ inline float to_f<float>(float x) { return x; }
template <> __host__ __device__ inline float to_f<bf16_t>(bf16_t x) { return bf2f(x); }
template <typename T> __host__ __device__ inline T from_f(float x);
template <> __host__ __device__ inline float from_f<float>(float x) { return x; }
template <> __host__ __device__ inline bf16_t from_f<bf16_t>(float x) { return f2bf(x); }

// ----------------------------------------------------------------------------- Philox4x32-10
// Salmon et al., SC'11. Round: (hi, lo) of M0*c0 and M1*c2; output
// (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); key bumped by two Weyl constants.
struct U4 { uint32_t x, y, z, w; };

__host__ __device__ inline uint32_t mulhi32(uint32_t a, uint32_t b) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __umulhi(a, b);
#else
  return (uint32_t)(((uint64_t)a * b) >> 32);
#endif
}

__host__ __device__ inline U4 philox(U4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    const uint32_t hi0 = mulhi32(0xD2511F53u, c.x), lo0 = 0xD2511F53u * c.x;
    const uint32_t hi1 = mulhi32(0xCD9E8D57u, c.z), lo1 = 0xCD9E8D57u * c.z;
    c = U4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
  }
  return c;
}

__host__ __device__ inline uint32_t philox_word(uint64_t seed, uint64_t i, uint32_t step,
                                                uint32_t purpose, uint32_t tensor) {
  U4 o = philox(U4{(uint32_t)(i >> 2), step, purpose, tensor}, (uint32_t)seed, (uint32_t)(seed >> 32));
  switch (i & 3) { case 0: return o.x; case 1: return o.y; case 2: return o.z; default: return o.w; }
}

enum Purpose : uint32_t { P_INIT = 0, P_IDX = 1, P_NOISE_TGT = 2, P_NOISE_POL = 3 };

// ----------------------------------------------------------------------------- GEMM
enum GemmMode { GEMM_FWD = 0, GEMM_DGRAD = 1, GEMM_WGRAD = 2 };

struct GemmArgs {
  const void* A; int64_t lda;
  const void* B; int64_t ldb;
  void* C; int64_t ldc;
  const float* bias;           // FWD: bias [N] (fp32)
  const void* mask; int64_t ldm;  // DGRAD: C *= (mask > 0) when non-null (operand type)
  int M, N, K;                 // WGRAD: K is the batch extent split over gridDim.z
  int relu;                    // FWD
  int out_f32;                 // FWD / DGRAD: store float32 instead of the operand type
  int splits;                  // WGRAD: number of K slices; C gets splits * M * ldc floats
  float* colsum; int64_t ldcs; // DGRAD (bf16 large-tile only): column sums of the stored C
                               // per 256-row tile, colsum[M / 256, ldcs]
};

// C = A B with A: [M, K] k-contiguous (FWD, DGRAD) or [K, M] (WGRAD),
// B: [N, K] (FWD) or [K, N] (DGRAD, WGRAD). Returns a hipError_t.
hipError_t gemm(bool bf16, GemmMode mode, const GemmArgs& g, hipStream_t s);
// Sum `splits` float slices [splits, M, ldc] into out [M, ldo].
hipError_t splitk_reduce(const float* part, int splits, int M, int N, int64_t ldc, float* out,
                         int64_t ldo, hipStream_t s);
// Choose a split count for a WGRAD of (M, N, K) and return it (K % (32*splits) == 0).
int wgrad_splits(bool bf16, int M, int N, int K);
// Large-tile bf16 kernel (gemm_big.hip): M % 256 == 0, N % 128 == 0, K slices of 32.
bool big_gemm_fits(GemmMode mode, int M, int N, int K, int splits);
// True when gemm() with these arguments can produce the fused column sums (GemmArgs::colsum).
bool gemm_colsum_fused(bool bf16, GemmMode mode, int M, int N, int K);
bool big_gemm_colsum(GemmMode mode, int M, int N, int K);
hipError_t gemm_big(GemmMode mode, const GemmArgs& g, hipStream_t s);

}  // namespace spz
