// Test hooks (include/spz_testing.h): the GEMM kernels on caller-owned device memory.
#include "../../include/spz_testing.h"
#include "kernels.h"

using namespace spz;

namespace {
// The transposed image Bt [N, K] of an input-gradient operand B [K, N] (ldb), which
// the large-tile kernel and the generic kernel's k-contiguous input-gradient path read;
// *bt must be freed by the caller.
hipError_t make_bt(bool bf16, const void* B, int64_t ldb, int K, int N, void** bt) {
  *bt = nullptr;
  if (K <= 0 || N <= 0) return hipErrorInvalidValue;
  TransposeJob job{0, 0, ldb, K, K, N, 0};
  TransposeJob* dj = nullptr;
  hipError_t e = hipMalloc(bt, (size_t)K * N * (bf16 ? 2 : 4));
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&dj), sizeof(job));
  if (e == hipSuccess) e = hipMemcpy(dj, &job, sizeof(job), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = launch_transpose(bf16, B, *bt, dj, 1, transpose_tiles(K, N), nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (dj) (void)hipFree(dj);
  if (e != hipSuccess && *bt) {
    (void)hipFree(*bt);
    *bt = nullptr;
  }
  return e;
}
}  // namespace

extern "C" int spzt_gemm(int32_t bf16, int32_t mode, int32_t M, int32_t N, int32_t K, int32_t splits,
                         const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
                         const float* bias, const void* mask, int64_t ldm, int32_t relu, int32_t out_f32) {
  if (mode < 0 || mode > 3 || splits < 1 || !A || !B || !C) return SPZ_EINVAL;
  // mode 3: the input gradient with B passed as its transposed image (bf16 mode 1 does
  // that always: the large-tile kernel needs it)
  const bool via_bt = mode == 3 || (bf16 && mode == GEMM_DGRAD);
  if (mode == 3) mode = GEMM_DGRAD;
  GemmArgs g{};
  g.A = A; g.lda = lda; g.B = B; g.ldb = ldb; g.C = C; g.ldc = ldc;
  g.bias = bias; g.mask = mask; g.ldm = ldm; g.M = M; g.N = N; g.K = K;
  g.relu = relu; g.out_f32 = out_f32; g.splits = splits;
  float* part = nullptr;
  void* bt = nullptr;
  if (mode == GEMM_WGRAD) {
    if (hipMalloc(&part, (size_t)splits * M * N * 4) != hipSuccess) return SPZ_ENOMEM;
    g.C = part;
    g.ldc = N;
  }
  hipError_t e = hipSuccess;
  if (via_bt && (e = make_bt(bf16 != 0, B, ldb, K, N, &bt)) == hipSuccess) {
    g.Bt = bt;
    g.ldbt = K;
  }
  if (e == hipSuccess) e = gemm(bf16 != 0, (GemmMode)mode, g, nullptr);
  if (e == hipSuccess && mode == GEMM_WGRAD) e = splitk_reduce(part, splits, M, N, N, (float*)C, ldc, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (part) (void)hipFree(part);
  if (bt) (void)hipFree(bt);
  if (e == hipErrorInvalidValue) return SPZ_EINVAL;
  return e == hipSuccess ? SPZ_OK : SPZ_EHIP;
}

extern "C" int spzt_gemm_fused(int32_t mode, int32_t M, int32_t N, int32_t K, const void* A, int64_t lda,
                               const void* B, int64_t ldb, void* C, int64_t ldc, const float* bias,
                               uint32_t* bits_out, const uint32_t* bits, int64_t ldbits, const void* rdot_w,
                               float* rdot_part, int64_t ldrd, int32_t no_store, float* colsum, int64_t ldcs) {
  if ((mode != GEMM_FWD && mode != GEMM_DGRAD) || !A || !B || !C) return SPZ_EINVAL;
  if (mode == GEMM_DGRAD && !bits) return SPZ_EINVAL;
  GemmArgs g{};
  g.A = A; g.lda = lda; g.B = B; g.ldb = ldb; g.C = C; g.ldc = ldc;
  g.M = M; g.N = N; g.K = K;
  if (mode == GEMM_FWD) {
    g.bias = bias; g.relu = 1;
    g.bits_out = bits_out;
    g.rdot_w = rdot_w; g.rdot_part = rdot_part; g.ldrd = ldrd;
    g.no_store = no_store;
  } else {
    g.bits = bits;
    g.colsum = colsum; g.ldcs = ldcs;
  }
  g.ldbits = ldbits;
  if (!gemm_fused_ok(true, (GemmMode)mode, M, N, K)) return SPZ_EINVAL;
  void* bt = nullptr;
  hipError_t e = hipSuccess;
  if (mode == GEMM_DGRAD && (e = make_bt(true, B, ldb, K, N, &bt)) == hipSuccess) {
    g.Bt = bt;
    g.ldbt = K;
  }
  if (e == hipSuccess) e = gemm(true, (GemmMode)mode, g, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (bt) (void)hipFree(bt);
  if (e == hipErrorInvalidValue) return SPZ_EINVAL;
  return e == hipSuccess ? SPZ_OK : SPZ_EHIP;
}

extern "C" int spzt_gemm_dgrad_rows(int32_t bf16, int32_t M, int32_t N, int32_t K, const void* A, int64_t lda,
                                    const void* B, int64_t ldb, void* C, int64_t ldc, const uint32_t* bits,
                                    int64_t ldbits, int32_t out_f32, int32_t m_rows) {
  if (!A || !B || !C || m_rows < 0 || m_rows > M || m_rows % 256) return SPZ_EINVAL;
  GemmArgs g{};
  g.A = A; g.lda = lda; g.B = B; g.ldb = ldb; g.C = C; g.ldc = ldc;
  g.M = M; g.N = N; g.K = K; g.out_f32 = out_f32;
  g.bits = bits; g.ldbits = ldbits;
  int32_t* rows = nullptr;
  void* bt = nullptr;
  hipError_t e = hipMalloc(reinterpret_cast<void**>(&rows), sizeof(int32_t));
  if (e != hipSuccess) return SPZ_ENOMEM;
  e = hipMemcpy(rows, &m_rows, sizeof(int32_t), hipMemcpyHostToDevice);
  g.m_dyn = rows;
  if (e == hipSuccess && bf16 && (e = make_bt(true, B, ldb, K, N, &bt)) == hipSuccess) {
    g.Bt = bt;
    g.ldbt = K;
  }
  if (e == hipSuccess) e = gemm(bf16 != 0, GEMM_DGRAD, g, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (bt) (void)hipFree(bt);
  (void)hipFree(rows);
  if (e == hipErrorInvalidValue) return SPZ_EINVAL;
  return e == hipSuccess ? SPZ_OK : SPZ_EHIP;
}

extern "C" int spzt_rdot_cols(int32_t M, int32_t N) { return gemm_rdot_cols(M, N); }

extern "C" int spzt_reduce_jobs(int32_t n, const float* const* part, float* const* out, const int64_t* zstride,
                                const int64_t* ld, const int64_t* ldo, const int32_t* rows, const int32_t* cols,
                                const int32_t* slices, const int32_t* groups, const int32_t* vec) {
  if (n < 1 || n > MAX_REDUCE_JOBS || !part || !out || !zstride || !ld || !ldo || !rows || !cols || !slices ||
      !groups || !vec)
    return SPZ_EINVAL;
  ReduceJobs J{};
  J.n = n;
  for (int i = 0; i < n; ++i) {
    if (!part[i] || !out[i]) return SPZ_EINVAL;
    J.j[i] = ReduceJob{part[i], out[i], zstride[i], ld[i], ldo[i], rows[i], cols[i], slices[i], groups[i], vec[i], 0};
  }
  hipError_t e = launch_reduce_jobs(J, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e == hipErrorInvalidValue) return SPZ_EINVAL;
  return e == hipSuccess ? SPZ_OK : SPZ_EHIP;
}

// Rounding check of the device float32 -> bfloat16 conversion against an integer
// round-to-nearest-even written out here: every input bit pattern in
// [begin, begin + count) must give the same 16 bits, except that a NaN input only
// has to give a NaN.
namespace {
__device__ inline uint32_t rne_bf16_ref(uint32_t u) {
  const uint32_t mant = u & 0xFFFFu, keep = u >> 16;
  const bool up = mant > 0x8000u || (mant == 0x8000u && (keep & 1u));
  return (keep + (up ? 1u : 0u)) & 0xFFFFu;
}

__global__ void k_round_check(uint64_t begin, uint64_t count, unsigned long long* bad) {
  const uint64_t base = begin + ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) * 16;
  unsigned n = 0;
  for (int t = 0; t < 16; ++t) {
    const uint64_t x = base + t;
    if (x >= begin + count) break;
    const uint32_t u = (uint32_t)x;
    const float f = __uint_as_float(u);
    const uint32_t hw = f2bf(f);
    const uint32_t pk = pack_bf16x2(f, -f);
    const bool nan = (u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu);
    if (nan) {
      const bool ok = (hw & 0x7F80u) == 0x7F80u && (hw & 0x7Fu) && (pk & 0x7F80u) == 0x7F80u && (pk & 0x7Fu);
      n += ok ? 0 : 1;
    } else {
      const uint32_t ref = rne_bf16_ref(u), refn = rne_bf16_ref(u ^ 0x80000000u);
      n += (hw != ref || (pk & 0xFFFFu) != ref || (pk >> 16) != refn) ? 1 : 0;
    }
  }
  if (n) atomicAdd(bad, (unsigned long long)n);
}
}  // namespace

extern "C" int spzt_bf16_round_check(uint64_t begin, uint64_t count, uint64_t* mismatches) {
  if (!mismatches || count == 0 || begin + count > (1ull << 32)) return SPZ_EINVAL;
  unsigned long long* d = nullptr;
  if (hipMalloc(&d, sizeof(*d)) != hipSuccess) return SPZ_ENOMEM;
  hipError_t e = hipMemset(d, 0, sizeof(*d));
  const uint64_t threads = (count + 15) / 16;
  if (e == hipSuccess) {
    k_round_check<<<(unsigned)((threads + 255) / 256), 256>>>(begin, count, d);
    e = hipGetLastError();
  }
  unsigned long long h = 0;
  if (e == hipSuccess) e = hipMemcpy(&h, d, sizeof(h), hipMemcpyDeviceToHost);
  (void)hipFree(d);
  *mismatches = h;
  return e == hipSuccess ? SPZ_OK : SPZ_EHIP;
}
