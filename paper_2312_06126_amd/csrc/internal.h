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

// float32 -> bfloat16, round to nearest, ties to even (subnormals kept); NaN stays
// NaN. On the device this is the hardware conversion (v_cvt_pk_bf16_f32).
__host__ __device__ inline bf16_t f2bf(float f) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_bit_cast(bf16_t, (__bf16)f);
#else
  union { uint32_t u; float f; } v;
  v.f = f;
  if ((v.u & 0x7F800000u) == 0x7F800000u && (v.u & 0x007FFFFFu)) return (bf16_t)0x7FC0;
  uint32_t r = v.u + 0x7FFFu + ((v.u >> 16) & 1u);
  return (bf16_t)(r >> 16);
#endif
}

// Two values rounded as f2bf, lo in the low half (one instruction on the device).
__host__ __device__ inline uint32_t pack_bf16x2(float lo, float hi) {
#if defined(__HIP_DEVICE_COMPILE__)
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
#else
  return (uint32_t)f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
#endif
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

enum Purpose : uint32_t { P_INIT = 0, P_IDX = 1, P_NOISE_TGT = 2, P_NOISE_POL = 3, P_ACT = 4 };

// ----------------------------------------------------------------------------- device math
constexpr float LN2F = 0.69314718055994531f;
constexpr float HALF_LN_2PI_F = 0.91893853320467274f;

__device__ inline float softplusf(float x) { return x > 0.0f ? x + log1pf(expf(-x)) : log1pf(expf(x)); }

// Clamp that keeps a NaN operand (fminf / fmaxf would drop it), so that a non-finite
// network output reaches the loss record as it does in exact arithmetic.
__device__ inline float clamp_keep_nan(float x, float lo, float hi) { return x < lo ? lo : (x > hi ? hi : x); }

// Standard normal deviate for flat element i of the stream (seed, step, purpose):
// Box-Muller on words (0,1) -> lanes 0,1 and (2,3) -> lanes 2,3 of each Philox block.
__device__ inline float normal_at(uint64_t seed, uint64_t i, uint32_t step, uint32_t purpose) {
  const U4 w = philox(U4{(uint32_t)(i >> 2), step, purpose, 0u}, (uint32_t)seed, (uint32_t)(seed >> 32));
  const int lane = (int)(i & 3);
  const uint32_t wa = lane < 2 ? w.x : w.z, wb = lane < 2 ? w.y : w.w;
  const float u1 = (float)((wa >> 8) + 1u) * 5.9604644775390625e-8f;  // (0, 1]
  const float u2 = (float)(wb >> 8) * 5.9604644775390625e-8f;          // [0, 1)
  const float rad = sqrtf(-2.0f * logf(u1));
  float sn, cs;
  sincospif(2.0f * u2, &sn, &cs);
  return rad * ((lane & 1) ? sn : cs);
}

// ----------------------------------------------------------------------------- SAC head
// z = [mu | l] per row -> a = tanh(mu + exp(clip(l)) eps), written into the action
// columns of the next operand tensor x, and the tanh-Gaussian log-density of a.
struct SacHeadArgs {
  const float* z; int ldz; int A, B;
  uint64_t seed; const int64_t* step; uint32_t purpose;
  float lmin, lmax;
  void* x; int64_t ldx; int xoff;      // action columns of the next operand tensor
  float* logp;
  float *th, *se, *lm;                 // backward cache [B, A] (null for the target side)
};

// Element (row b, action j) of the SAC head from its mean mu, log-std l and deviate eps
// (normal_at of element b A + j at the step's counter word): stores the action (and the backward cache) and returns
// the element's log-density term, in the overflow-free form of log(1 - tanh^2 u) =
// 2 (ln 2 - u - softplus(-2u)). Shared by the head kernel and the head product's fused
// epilogue, so both compute the same bits.
template <typename T>
__device__ inline float sac_head_element(const SacHeadArgs& h, float mu, float l, int b, int j, float eps) {
  const uint64_t e = (uint64_t)b * h.A + j;
  const float lc = clamp_keep_nan(l, h.lmin, h.lmax);
  const float sig = expf(lc);
  const float u = mu + sig * eps;
  const float a = tanhf(u);
  static_cast<T*>(h.x)[(int64_t)b * h.ldx + h.xoff + j] = from_f<T>(a);
  if (h.th) {
    h.th[e] = a;
    h.se[e] = sig * eps;
    h.lm[e] = (l >= h.lmin && l <= h.lmax) ? 1.0f : 0.0f;
  }
  return -0.5f * eps * eps - lc - HALF_LN_2PI_F - 2.0f * (LN2F - u - softplusf(-2.0f * u));
}

// ----------------------------------------------------------------------------- GEMM
enum GemmMode { GEMM_FWD = 0, GEMM_DGRAD = 1, GEMM_WGRAD = 2 };

struct GemmArgs {
  const void* A; int64_t lda;
  const void* B; int64_t ldb;
  // DGRAD: the same B operand transposed, Bt[N, K] (row n = column n of B), read
  // instead of B (k-contiguous, like the forward's weight). The bf16 large-tile kernel
  // needs it: without it the product runs on the generic kernel (and the large-tile
  // epilogue features are refused).
  const void* Bt; int64_t ldbt;
  void* C; int64_t ldc;
  const float* bias;           // FWD: bias [N] (fp32; 16-byte aligned for the large-tile kernel)
  const void* mask; int64_t ldm;  // DGRAD: C *= (mask > 0) when non-null (operand type)
  int M, N, K;                 // WGRAD: K is the batch extent split over gridDim.z
  int relu;                    // FWD
  int out_f32;                 // FWD / DGRAD: store float32 instead of the operand type
  int splits;                  // WGRAD: number of K slices; C gets splits * M * ldc floats
  float* colsum; int64_t ldcs; // DGRAD (bf16 large-tile only): column sums of the stored C
                               // per 256-row tile, colsum[M / 256, ldcs]
  // Large-tile bf16 epilogue features (the whole product must run on that kernel,
  // see gemm_fused_ok). Bit c % 32 of word bits[(c / 32) * ldbits + r] is element
  // (r, c) of a ReLU mask.
  uint32_t* bits_out;          // FWD with relu: mask of the stored C (C[r, c] > 0)
  const uint32_t* bits;        // DGRAD: C *= mask bit (instead of mask)
  int64_t ldbits;
  const void* rdot_w;          // FWD with relu: rdot_part[p, r] = sum over the p-th group of
  float* rdot_part;            // gemm_rdot_cols(M, N) columns c of stored C[r, c] * rdot_w[c]
  int64_t ldrd;
  int no_store;                // FWD with rdot_w: C is not written
  // DGRAD: when set, only rows [0, *m_dyn) of C are computed (a device-side count,
  // a multiple of 256 and at most M); the launch is still sized by M and the
  // blocks past the count exit at once. Rows from *m_dyn on are left untouched.
  const int32_t* m_dyn;
};

enum EpilogueFlag : int {
  EPI_F32 = 1, EPI_RELU = 2, EPI_MASK = 4, EPI_BITS = 8, EPI_BITS_OUT = 16, EPI_CSUM = 32,
  EPI_RDOT = 64, EPI_NOSTORE = 128
};

__host__ __device__ inline int epilogue_flags(GemmMode mode, const GemmArgs& g) {
  if (mode == GEMM_WGRAD) return EPI_F32;
  int f = g.out_f32 ? EPI_F32 : 0;
  if (mode == GEMM_FWD) {
    if (g.relu) f |= EPI_RELU;
    if (g.bits_out) f |= EPI_BITS_OUT;
    if (g.rdot_w) f |= EPI_RDOT;
    if (g.no_store) f |= EPI_NOSTORE;
  } else {
    if (g.mask) f |= EPI_MASK;
    if (g.bits) f |= EPI_BITS;
    if (g.colsum) f |= EPI_CSUM;
  }
  return f;
}

// C = A B with A: [M, K] k-contiguous (FWD, DGRAD) or [K, M] (WGRAD),
// B: [N, K] (FWD) or [K, N] (DGRAD, WGRAD). Returns a hipError_t.
hipError_t gemm(bool bf16, GemmMode mode, const GemmArgs& g, hipStream_t s);
// Two independent products of one mode: a single large-tile launch when gemm_pairs
// holds, else gemm() twice.
hipError_t gemm_pair(bool bf16, GemmMode mode, const GemmArgs& g0, const GemmArgs& g1, hipStream_t s);
// Both products run on the large-tile kernel with the same launch shape and one of them
// alone would leave compute units idle (fewer workgroups than 256).
bool gemm_pairs(bool bf16, GemmMode mode, const GemmArgs& g0, const GemmArgs& g1);
// Threads per output piece of the split-K reduction of an M x N product from `splits`
// slices (the grouping ReduceJob::groups reproduces).
int splitk_groups(int M, int N, int splits);
// Sum `splits` float slices [splits, M, ldc] into out [M, ldo].
hipError_t splitk_reduce(const float* part, int splits, int M, int N, int64_t ldc, float* out,
                         int64_t ldo, hipStream_t s);
// Choose a split count for a WGRAD of (M, N, K) and return it (K % (32*splits) == 0).
int wgrad_splits(bool bf16, int M, int N, int K);
// Large-tile bf16 kernel (gemm_big.hip): M % 256 == 0, N >= 128 with N % 8 == 0 (a
// ragged last column tile reads zeros and stores nothing past N), K slices of 32.
bool big_gemm_fits(GemmMode mode, int M, int N, int K, int splits);
// Its column tile: 256 when N % 256 == 0 (forward and input gradient: only while the
// grid still has a workgroup per CU, else 128); with fused epilogue features 128 (they
// need N % 128 == 0); otherwise 256 above N = 256 and 128 below.
int big_bn(GemmMode mode, int M, int N, bool fused);
// True when gemm() with these arguments can produce the fused column sums (GemmArgs::colsum).
bool gemm_colsum_fused(bool bf16, GemmMode mode, int M, int N, int K);
bool big_gemm_colsum(GemmMode mode, int M, int N, int K);
// Leading dimensions the large-tile kernel addresses (forward and input gradient:
// below 2^22 elements).
bool big_gemm_ld_ok(GemmMode mode, const GemmArgs& g);
hipError_t gemm_big(GemmMode mode, const GemmArgs& g, hipStream_t s);
// Two products of the same mode, shape, epilogue and split count in one launch of the
// large-tile kernel (the second's tiles after the first's); each must satisfy the
// single-product contract. GemmPair is the kernel's argument.
struct GemmPair { GemmArgs g[2]; int n; };
hipError_t gemm_big_pair(GemmMode mode, const GemmArgs& g0, const GemmArgs& g1, hipStream_t s);
// Workgroups of one large-tile launch of this product.
int big_gemm_tiles(GemmMode mode, const GemmArgs& g);
// True when a product of this shape runs entirely on the large-tile kernel, so that
// bits_out / bits / rdot_w / no_store / colsum may be used.
bool gemm_fused_ok(bool bf16, GemmMode mode, int M, int N, int K);
// Columns per row-dot partial for an M x N forward (N / gemm_rdot_cols partials; at
// least N / 64, the most any shape uses).
int gemm_rdot_cols(int M, int N);
// True when the large-tile kernel has an epilogue for these flags.
bool big_epilogue_supported(GemmMode mode, int flags);
// The actor's output product z = X W^T + b with the SAC head fused into its epilogue
// (z itself is not stored; h.z is ignored): every row's outputs must fall in one tile,
// 2 A <= N with N one of 32, 64; M % 128 == 0 and K % 32 == 0 as for gemm().
bool gemm_sac_head_ok(int M, int N, int K, int A);
hipError_t gemm_fwd_sac_head(bool bf16, const GemmArgs& g, const SacHeadArgs& h, hipStream_t s);

}  // namespace spz
