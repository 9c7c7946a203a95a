// MFMA GEMMs of the MLP forward, input-gradient (dgrad) and weight-gradient
// (wgrad) products, with their elementwise epilogues fused.
//
//   FWD   C[m, n] = act( sum_k X[m, k] W[n, k] + b[n] )       X [M, K], W [N, K]
//   DGRAD C[m, n] = (sum_k dZ[m, k] W[k, n]) * (H[m, n] > 0)   dZ [M, K], W [K, N]
//   WGRAD C[s, m, n] = sum_{k in slice s} dZ[k, m] X[k, n]     dZ [K, M], X [K, N]
//
// All operands are row-major. A workgroup owns a BM x BN tile; its waves (2x2,
// 2x1, 1x2 or 1x1) each own TM x TN blocks of 32x32 and step through K in
// slices of BK = 32 staged in LDS (register prefetch of the next slice while the
// current one is consumed). Each lane feeds the matrix core with consecutive k
// values of one row: operands that are k-contiguous in memory are read from LDS
// as 16-byte vectors, operands that are m/n-contiguous are read element-wise
// down an LDS column. A and B use the same k-to-lane assignment, which is all
// the instruction needs. Accumulation is float32 in both precisions:
//   fp32: v_mfma_f32_32x32x2_f32, 4 instructions per 8 k (one float4 per lane)
//   bf16: v_mfma_f32_32x32x16_bf16, 1 instruction per 16 k
// Dimensions are multiples of the tile (the caller pads features to 32 and the
// batch to 256), so the kernel carries no bounds checks; the host verifies the
// divisibility before every launch.
#include "internal.h"

namespace spz {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int BK = 32;

template <typename T> struct Traits;
template <> struct Traits<float> { static constexpr int VEC = 4, PAD = 4; };
template <> struct Traits<bf16_t> { static constexpr int VEC = 8, PAD = 8; };

// One operand tile (ROWS along m or n, BK along k) moving global -> registers -> LDS.
// KC: global element (r, k) at base[(r0 + r) * ld + k0 + k]; LDS [ROWS][BK + PAD].
// !KC: global element (r, k) at base[(k0 + k) * ld + r0 + r]; LDS [BK][ROWS + PAD].
template <typename T, bool KC, int ROWS, int NT>
struct Tile {
  static constexpr int VEC = Traits<T>::VEC;
  static constexpr int LD = KC ? (BK + Traits<T>::PAD) : (ROWS + Traits<T>::PAD);
  static constexpr int SIZE = (KC ? ROWS : BK) * LD;
  static constexpr int NVEC = ROWS * BK / VEC;
  static constexpr int PER = (NVEC + NT - 1) / NT;
  static constexpr int VPR = (KC ? BK : ROWS) / VEC;
  u32x4 r[PER];

  // RG: the tile may reach past the operand's `lim` rows (KC) or columns (m/n-contiguous;
  // lim % VEC == 0); those are read from row lim - 1 or columns lim - VEC instead. Their
  // products land only in output rows / columns that are not stored.
  template <bool RG = false>
  __device__ inline void load(const T* __restrict__ base, int64_t ld, int r0, int k0, int tid, int lim = 0) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      if (NVEC % NT == 0 || v < NVEC) {
        int a = v / VPR, b = (v % VPR) * VEC;
        if constexpr (RG) {
          if (KC && r0 + a >= lim) a = lim - 1 - r0;
          if (!KC && r0 + b >= lim) b = lim - VEC - r0;
        } else {
          (void)lim;
        }
        const T* src = KC ? base + (int64_t)(r0 + a) * ld + (k0 + b)
                          : base + (int64_t)(k0 + a) * ld + (r0 + b);
        r[p] = *reinterpret_cast<const u32x4*>(src);
      }
    }
  }
  __device__ inline void store(T* lds, int tid) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      if (NVEC % NT == 0 || v < NVEC) {
        const int a = v / VPR, b = (v % VPR) * VEC;
        *reinterpret_cast<u32x4*>(lds + a * LD + b) = r[p];
      }
    }
  }
};

// bf16 fragment: lane supplies 8 consecutive k (ks + 8*(lane/32) ...) of row rb + lane%32.
template <bool KC, int LD>
__device__ inline bf16x8 frag_bf16(const bf16_t* lds, int rb, int ks, int lane) {
  const int row = rb + (lane & 31), kb = ks + 8 * (lane >> 5);
  if constexpr (KC) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(lds + row * LD + kb));
  } else {
    u16x8 t;
#pragma unroll
    for (int j = 0; j < 8; ++j) t[j] = lds[(kb + j) * LD + row];
    return __builtin_bit_cast(bf16x8, t);
  }
}

// fp32 fragment: lane supplies 4 consecutive k (ks + 4*(lane/32) ...) of row rb + lane%32,
// one per instruction.
template <bool KC, int LD>
__device__ inline float4 frag_f32(const float* lds, int rb, int ks, int lane) {
  const int row = rb + (lane & 31), kb = ks + 4 * (lane >> 5);
  if constexpr (KC) {
    return *reinterpret_cast<const float4*>(lds + row * LD + kb);
  } else {
    return make_float4(lds[kb * LD + row], lds[(kb + 1) * LD + row], lds[(kb + 2) * LD + row],
                       lds[(kb + 3) * LD + row]);
  }
}

constexpr int gemm_threads(int bm, int bn) { return 64 * (bm >= 64 ? 2 : 1) * (bn >= 64 ? 2 : 1); }

template <int BM, int BN> struct Shape {
  static constexpr int WM = BM >= 64 ? 2 : 1, WN = BN >= 64 ? 2 : 1;
  static constexpr int NT = 64 * WM * WN;
  static constexpr int TM = BM / (32 * WM), TN = BN / (32 * WN);
};

// RG: a last row tile (weight gradient) or column tile may reach past M or N (both
// multiples of 32); operand reads there are clamped and the epilogue stores nothing there.
// BT (input gradient): B is the transposed weight image [N, K], read k-contiguous like
// the forward's weight (16-byte fragment reads instead of element-wise ones).
// HEAD (forward, the actor's output layer): the SAC head runs in the epilogue on whole
// rows of z (the tile spans all N columns) instead of z being stored; h describes it.
template <typename T, int MODE, int BM, int BN, bool RG, bool BT, bool HEAD = false>
__global__ void __launch_bounds__(gemm_threads(BM, BN)) k_gemm(GemmArgs g, SacHeadArgs h) {
  using S = Shape<BM, BN>;
  constexpr int TM = S::TM, TN = S::TN, NT = S::NT;
  constexpr bool AKC = MODE != GEMM_WGRAD;
  constexpr bool BKC = MODE == GEMM_FWD || BT;
  using TA = Tile<T, AKC, BM, NT>;
  using TB = Tile<T, BKC, BN, NT>;
  __shared__ __attribute__((aligned(16))) T lds_a[TA::SIZE];
  __shared__ __attribute__((aligned(16))) T lds_b[TB::SIZE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / S::WN, wn = wave % S::WN;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
  if constexpr (MODE == GEMM_DGRAD) {
    if (g.m_dyn && m0 >= *g.m_dyn) return;
  }
  int kbeg = 0, kend = g.K;
  if constexpr (MODE == GEMM_WGRAD) {
    const int ks = g.K / g.splits;
    kbeg = blockIdx.z * ks;
    kend = kbeg + ks;
  }
  const T* __restrict__ A = static_cast<const T*>(g.A);
  const T* __restrict__ B = static_cast<const T*>(g.B);

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;

  TA ta;
  TB tb;
  ta.template load<RG>(A, g.lda, m0, kbeg, tid, g.M);
  tb.template load<RG>(B, g.ldb, n0, kbeg, tid, g.N);
  for (int k0 = kbeg; k0 < kend; k0 += BK) {
    __syncthreads();
    ta.store(lds_a, tid);
    tb.store(lds_b, tid);
    __syncthreads();
    if (k0 + BK < kend) {
      ta.template load<RG>(A, g.lda, m0, k0 + BK, tid, g.M);
      tb.template load<RG>(B, g.ldb, n0, k0 + BK, tid, g.N);
    }
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int ks = 0; ks < BK; ks += 16) {
        bf16x8 af[TM], bw[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) af[i] = frag_bf16<AKC, TA::LD>(lds_a, (wm * TM + i) * 32, ks, lane);
#pragma unroll
        for (int j = 0; j < TN; ++j) bw[j] = frag_bf16<BKC, TB::LD>(lds_b, (wn * TN + j) * 32, ks, lane);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bw[j], acc[i][j], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < BK; ks += 8) {
        float4 af[TM], bw[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) af[i] = frag_f32<AKC, TA::LD>(lds_a, (wm * TM + i) * 32, ks, lane);
#pragma unroll
        for (int j = 0; j < TN; ++j) bw[j] = frag_f32<BKC, TB::LD>(lds_b, (wn * TN + j) * 32, ks, lane);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i].x, bw[j].x, acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i].y, bw[j].y, acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i].z, bw[j].z, acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i].w, bw[j].w, acc[i][j], 0, 0, 0);
          }
      }
    }
  }

  // Epilogue. 32x32 accumulator layout: lane holds column lane%32; register q holds
  // row 8*(q/4) + 4*(lane/32) + q%4.
  if constexpr (HEAD) {
    // z = acc + b for the tile's rows goes to LDS (the value a stored z would hold), then
    // one thread per (row, action) element runs the head and each row's log-density
    // terms are added in action order, as the head kernel does.
    static_assert(MODE == GEMM_FWD && !RG && !BT, "the head follows the forward product");
    constexpr int ZP = BN + 1;
    __shared__ float zt[HEAD ? BM * ZP : 1];
    __shared__ float lt[HEAD ? BM * (BN / 2) : 1];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int cl = (wn * TN + j) * 32 + (lane & 31);
        const int rl = (wm * TM + i) * 32 + 4 * (lane >> 5);
        const float bias = g.bias ? g.bias[cl] : 0.0f;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          float v = acc[i][j][q];
          v += bias;
          zt[(rl + 8 * (q >> 2) + (q & 3)) * ZP + cl] = v;
        }
      }
    __syncthreads();
    const int rows = min(BM, h.B - m0);
    const uint32_t t = (uint32_t)(*h.step + 1);
    for (int e = tid; e < rows * h.A; e += NT) {
      const int r = e / h.A, j = e - r * h.A;
      const int b = m0 + r;
      lt[e] = sac_head_element<T>(h, zt[r * ZP + j], zt[r * ZP + h.A + j], b, j,
                                  normal_at(h.seed, (uint64_t)b * h.A + j, t, h.purpose));
    }
    __syncthreads();
    if (tid < rows) {
      float lp = 0.0f;
      for (int j = 0; j < h.A; ++j) lp += lt[tid * h.A + j];
      h.logp[m0 + tid] = lp;
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + (wn * TN + j) * 32 + (lane & 31);
      const int rowb = m0 + (wm * TM + i) * 32 + 4 * (lane >> 5);
      if constexpr (RG) {
        // 32-column and 32-row blocks are whole (M, N multiples of 32)
        if (n0 + (wn * TN + j) * 32 >= g.N || m0 + (wm * TM + i) * 32 >= g.M) continue;
      }
      float bias = 0.0f;
      if constexpr (MODE == GEMM_FWD) bias = g.bias ? g.bias[col] : 0.0f;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int row = rowb + 8 * (q >> 2) + (q & 3);
        float v = acc[i][j][q];
        if constexpr (MODE == GEMM_WGRAD) {
          static_cast<float*>(g.C)[((int64_t)blockIdx.z * g.M + row) * g.ldc + col] = v;
        } else {
          if constexpr (MODE == GEMM_FWD) {
            v += bias;
            if (g.relu) v = v < 0.0f ? 0.0f : v;
          } else {
            if (g.mask) {
              const float h = to_f<T>(static_cast<const T*>(g.mask)[(int64_t)row * g.ldm + col]);
              if (!(h > 0.0f)) v = 0.0f;
            }
          }
          if (g.out_f32) static_cast<float*>(g.C)[(int64_t)row * g.ldc + col] = v;
          else static_cast<T*>(g.C)[(int64_t)row * g.ldc + col] = from_f<T>(v);
        }
      }
    }
}

// out[m, n] = sum over slices z in order of part[z, m, n]; 4 columns per thread.
__global__ void k_splitk_reduce(const float* __restrict__ part, int splits, int M, int N, int64_t ldc,
                                float* __restrict__ out, int64_t ldo) {
  const int nv = N / 4;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)M * nv) return;
  const int m = (int)(i / nv), n = (int)(i % nv) * 4;
  float4 s = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  for (int z = 0; z < splits; ++z) {
    const float4 v = *reinterpret_cast<const float4*>(part + ((int64_t)z * M + m) * ldc + n);
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  *reinterpret_cast<float4*>(out + (int64_t)m * ldo + n) = s;
}

// The same for small outputs with many slices: RG_GROUPS threads per 16-byte output
// piece take every RG_GROUPS-th slice, and the group sums are added in group order
// (a fixed order, as above), so the grid has RG_GROUPS times more threads.
constexpr int RG_GROUPS = 8;
__global__ void __launch_bounds__(256) k_splitk_reduce_grouped(const float* __restrict__ part, int splits, int M,
                                                               int N, int64_t ldc, float* __restrict__ out,
                                                               int64_t ldo) {
  constexpr int COLS = 256 / RG_GROUPS;
  __shared__ float4 sh[RG_GROUPS][COLS];
  const int nv = N / 4, grp = threadIdx.x / COLS, col = threadIdx.x % COLS;
  const int64_t i = (int64_t)blockIdx.x * COLS + col;
  const bool valid = i < (int64_t)M * nv;
  const int m = valid ? (int)(i / nv) : 0, n = valid ? (int)(i % nv) * 4 : 0;
  float4 s = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  if (valid) {
    for (int z = grp; z < splits; z += RG_GROUPS) {
      const float4 v = *reinterpret_cast<const float4*>(part + ((int64_t)z * M + m) * ldc + n);
      s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
  }
  sh[grp][col] = s;
  __syncthreads();
  if (grp != 0 || !valid) return;
#pragma unroll
  for (int q = 1; q < RG_GROUPS; ++q) {
    const float4 v = sh[q][col];
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  *reinterpret_cast<float4*>(out + (int64_t)m * ldo + n) = s;
}

int pick_tile(int n) { return n % 128 == 0 ? 128 : n % 64 == 0 ? 64 : n % 32 == 0 ? 32 : 0; }

// Widest tile (128, 64 or 32) for a dimension of n (a multiple of 32) whose padding to
// whole tiles wastes at most 10% (416 -> 64: 7.7%; 32-wide tiles run fp32 products at
// about 45% of the matrix peak against about 60% for 64-wide ones).
int fit_tile(int n) {
  if (n <= 0 || n % 32) return 0;
  for (int t = 128; t > 32; t /= 2)
    if ((int64_t)((n + t - 1) / t) * t * 10 <= (int64_t)n * 11) return t;
  return 32;
}

template <typename T, int MODE, int BM, int BN, bool BT>
hipError_t launch_rg(const GemmArgs& g, hipStream_t s) {
  dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM, MODE == GEMM_WGRAD ? g.splits : 1);
  if (g.N % BN || g.M % BM) k_gemm<T, MODE, BM, BN, true, BT><<<grid, Shape<BM, BN>::NT, 0, s>>>(g, SacHeadArgs{});
  else k_gemm<T, MODE, BM, BN, false, BT><<<grid, Shape<BM, BN>::NT, 0, s>>>(g, SacHeadArgs{});
  return hipGetLastError();
}

template <typename T, int MODE, int BM, int BN>
hipError_t launch(const GemmArgs& g, hipStream_t s) {
  if constexpr (MODE == GEMM_DGRAD) {
    if (g.Bt) {
      GemmArgs t = g;
      t.B = g.Bt;
      t.ldb = g.ldbt;
      return launch_rg<T, MODE, BM, BN, true>(t, s);
    }
  }
  return launch_rg<T, MODE, BM, BN, false>(g, s);
}

template <typename T, int MODE, int BM>
hipError_t launch_bn(const GemmArgs& g, int bn, hipStream_t s) {
  switch (bn) {
    case 128: return launch<T, MODE, BM, 128>(g, s);
    case 64: return launch<T, MODE, BM, 64>(g, s);
    case 32: return launch<T, MODE, BM, 32>(g, s);
  }
  return hipErrorInvalidValue;
}

// Largest K-split the weight-gradient product allows: K % (32 s) == 0 with at
// least 256 batch rows per slice.
int max_splits(int K) {
  int s = 1;
  while (K % (2 * s * BK) == 0 && K / (2 * s) >= 256) s *= 2;
  return s;
}

// Tile of a generic-kernel product: the widest (up to 128 x 128, fit_tile) whose grid
// still gives about two workgroups per CU (512), halving the larger side first. A 128 x
// 128 tile over a batch of 8192 and 256 features is only 128 workgroups of one wave per
// SIMD: half the CUs idle and a quarter of the matrix-core issue slots used.
constexpr int GEN_TARGET_WGS = 512;
void generic_tiles(GemmMode mode, int M, int N, int K, int* bm, int* bn) {
  *bm = mode == GEMM_WGRAD ? fit_tile(M) : 128;
  *bn = fit_tile(N);
  if (!*bm || !*bn) return;
  const int64_t s = mode == GEMM_WGRAD ? max_splits(K) : 1;
  auto wgs = [&] { return (int64_t)((M + *bm - 1) / *bm) * ((N + *bn - 1) / *bn) * s; };
  while (wgs() < GEN_TARGET_WGS && (*bm > 32 || *bn > 32)) {
    if (*bm >= *bn && *bm > 32) *bm /= 2;
    else *bn /= 2;
  }
}

template <typename T, int MODE>
hipError_t launch_mode(const GemmArgs& g, hipStream_t s) {
  int bm = 0, bn = 0;
  generic_tiles((GemmMode)MODE, g.M, g.N, g.K, &bm, &bn);
  switch (bm) {
    case 128: return launch_bn<T, MODE, 128>(g, bn, s);
    case 64: return launch_bn<T, MODE, 64>(g, bn, s);
    case 32: return launch_bn<T, MODE, 32>(g, bn, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

bool gemm_sac_head_ok(int M, int N, int K, int A) {
  return (N == 32 || N == 64) && A >= 1 && 2 * A <= N && M > 0 && M % 128 == 0 && K > 0 && K % BK == 0;
}

namespace {
template <typename T, int BM, int BN>
hipError_t launch_head(const GemmArgs& g, const SacHeadArgs& h, hipStream_t s) {
  k_gemm<T, GEMM_FWD, BM, BN, false, false, true><<<dim3(1, g.M / BM), Shape<BM, BN>::NT, 0, s>>>(g, h);
  return hipGetLastError();
}
template <typename T, int BN>
hipError_t launch_head_bm(const GemmArgs& g, const SacHeadArgs& h, int bm, hipStream_t s) {
  return bm == 64 ? launch_head<T, 64, BN>(g, h, s) : launch_head<T, 32, BN>(g, h, s);
}
template <typename T>
hipError_t launch_head_t(const GemmArgs& g, const SacHeadArgs& h, int bm, hipStream_t s) {
  return g.N == 64 ? launch_head_bm<T, 64>(g, h, bm, s) : launch_head_bm<T, 32>(g, h, bm, s);
}
}  // namespace

hipError_t gemm_fwd_sac_head(bool bf16, const GemmArgs& g, const SacHeadArgs& h, hipStream_t s) {
  if (!gemm_sac_head_ok(g.M, g.N, g.K, h.A) || h.B < 0 || h.B > g.M || !h.step || !h.x || !h.logp)
    return hipErrorInvalidValue;
  const int vec = bf16 ? 8 : 4;
  if (g.lda % vec || g.ldb % vec || g.lda < g.K || g.ldb < g.K) return hipErrorInvalidValue;
  // Row tiles of 64 (the z tile and the log-density terms stay within static LDS), or 32
  // while the grid is short of two workgroups per CU.
  const int bm = g.M / 64 >= GEN_TARGET_WGS ? 64 : 32;
  return bf16 ? launch_head_t<bf16_t>(g, h, bm, s) : launch_head_t<float>(g, h, bm, s);
}

int wgrad_splits(bool bf16, int M, int N, int K) {
  int tiles, target;
  if (bf16 && big_gemm_fits(GEMM_WGRAD, M, N, K, 1)) {
    // large-tile kernel: about one workgroup per CU
    const int bn = big_bn(GEMM_WGRAD, M, N, false);
    tiles = (M / 256) * ((N + bn - 1) / bn);
    target = 256;
  } else {
    int bm = 0, bn = 0;
    generic_tiles(GEMM_WGRAD, M, N, K, &bm, &bn);
    if (!bm || !bn) return 1;
    tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
    target = 1024;
  }
  int s = 1;
  while (tiles * s < target && K % (2 * s * BK) == 0 && K / (2 * s) >= 256) s *= 2;
  return s;
}

namespace {

hipError_t gemm_generic(bool bf16, GemmMode mode, const GemmArgs& g, hipStream_t s) {
  if (!pick_tile(g.N)) return hipErrorInvalidValue;
  if (mode == GEMM_WGRAD) {
    if (!pick_tile(g.M) || g.splits < 1 || g.K % (g.splits * BK)) return hipErrorInvalidValue;
  } else {
    if (g.M % 128 || g.K % BK) return hipErrorInvalidValue;
    if (mode == GEMM_DGRAD && g.Bt && (g.ldbt % (bf16 ? 8 : 4) || g.ldbt < g.K)) return hipErrorInvalidValue;
  }
  if (bf16) {
    switch (mode) {
      case GEMM_FWD: return launch_mode<bf16_t, GEMM_FWD>(g, s);
      case GEMM_DGRAD: return launch_mode<bf16_t, GEMM_DGRAD>(g, s);
      case GEMM_WGRAD: return launch_mode<bf16_t, GEMM_WGRAD>(g, s);
    }
  } else {
    switch (mode) {
      case GEMM_FWD: return launch_mode<float, GEMM_FWD>(g, s);
      case GEMM_DGRAD: return launch_mode<float, GEMM_DGRAD>(g, s);
      case GEMM_WGRAD: return launch_mode<float, GEMM_WGRAD>(g, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace

bool gemm_colsum_fused(bool bf16, GemmMode mode, int M, int N, int K) {
  return bf16 && N % 128 == 0 && big_gemm_colsum(mode, M, N, K);
}

bool gemm_fused_ok(bool bf16, GemmMode mode, int M, int N, int K) {
  return bf16 && N % 128 == 0 && big_gemm_fits(mode, M, N, K, 1);
}

namespace {

// The launch contract of gemm(): hipSuccess when the product is valid; *big tells
// whether it runs on the large-tile kernel.
hipError_t route(bool bf16, GemmMode mode, const GemmArgs& g, bool* big) {
  if (g.colsum && !gemm_colsum_fused(bf16, mode, g.M, g.N, g.K)) return hipErrorInvalidValue;
  // A device-side row count: input-gradient products only, whole 256-row tiles, and
  // no per-tile column sums (the skipped tiles would leave theirs unwritten).
  if (g.m_dyn && (mode != GEMM_DGRAD || g.colsum || g.M % 256)) return hipErrorInvalidValue;
  // Epilogue features of the large-tile kernel only: the whole product must run there.
  const bool fused = g.bits_out || g.bits || g.rdot_w || g.no_store;
  if ((fused || g.colsum) && ((mode == GEMM_DGRAD && !g.Bt) || !big_gemm_ld_ok(mode, g))) return hipErrorInvalidValue;
  if (fused) {
    if (mode == GEMM_WGRAD || !gemm_fused_ok(bf16, mode, g.M, g.N, g.K)) return hipErrorInvalidValue;
    if ((g.bits_out || g.bits) && (g.ldbits < g.M || ((uintptr_t)(g.bits_out ? (const void*)g.bits_out : g.bits) & 3)))
      return hipErrorInvalidValue;
    if (g.rdot_w && (!g.rdot_part || g.ldrd < g.M || ((uintptr_t)g.rdot_w & 15))) return hipErrorInvalidValue;
    if (g.no_store && !g.rdot_w) return hipErrorInvalidValue;
    if (g.bits && g.mask) return hipErrorInvalidValue;
    if (!big_epilogue_supported(mode, epilogue_flags(mode, g))) return hipErrorInvalidValue;
  }
  // Shape contract: tiles divide the problem, K slices are whole BK steps,
  // operand rows are 16-byte aligned.
  if (g.M <= 0 || g.N <= 0 || g.K <= 0) return hipErrorInvalidValue;
  const int vec = bf16 ? 8 : 4;
  if (g.lda % vec || g.ldb % vec) return hipErrorInvalidValue;
  if (mode == GEMM_WGRAD && (g.splits < 1 || g.K % g.splits)) return hipErrorInvalidValue;
  *big = bf16 && big_gemm_fits(mode, g.M, g.N, g.K, mode == GEMM_WGRAD ? g.splits : 1) &&
         big_epilogue_supported(mode, epilogue_flags(mode, g)) && (mode != GEMM_DGRAD || g.Bt) &&
         big_gemm_ld_ok(mode, g);
  return hipSuccess;
}

}  // namespace

hipError_t gemm(bool bf16, GemmMode mode, const GemmArgs& g, hipStream_t s) {
  bool big = false;
  const hipError_t e = route(bf16, mode, g, &big);
  if (e != hipSuccess) return e;
  return big ? gemm_big(mode, g, s) : gemm_generic(bf16, mode, g, s);
}

hipError_t gemm_pair(bool bf16, GemmMode mode, const GemmArgs& g0, const GemmArgs& g1, hipStream_t s) {
  bool big0 = false, big1 = false;
  hipError_t e = route(bf16, mode, g0, &big0);
  if (e == hipSuccess) e = route(bf16, mode, g1, &big1);
  if (e != hipSuccess) return e;
  // One launch when both take the large-tile kernel with the same launch shape and one
  // product alone leaves compute units idle (fewer workgroups than 256).
  if (big0 && big1 && gemm_pairs(bf16, mode, g0, g1)) return gemm_big_pair(mode, g0, g1, s);
  e = gemm(bf16, mode, g0, s);
  return e != hipSuccess ? e : gemm(bf16, mode, g1, s);
}

bool gemm_pairs(bool bf16, GemmMode mode, const GemmArgs& g0, const GemmArgs& g1) {
  bool big0 = false, big1 = false;
  if (route(bf16, mode, g0, &big0) != hipSuccess || route(bf16, mode, g1, &big1) != hipSuccess || !big0 || !big1)
    return false;
  return g0.M == g1.M && g0.N == g1.N && g0.K == g1.K && epilogue_flags(mode, g0) == epilogue_flags(mode, g1) &&
         (mode != GEMM_WGRAD || g0.splits == g1.splits) && (!g0.m_dyn) == (!g1.m_dyn) &&
         big_gemm_tiles(mode, g0) < 256;
}

int splitk_groups(int M, int N, int splits) {
  // Small outputs (under 64K 16-byte pieces) from many slices: split the slices too.
  return (int64_t)M * (N / 4) < 4 * 256 * 64 && splits >= 4 * RG_GROUPS ? RG_GROUPS : 1;
}

hipError_t splitk_reduce(const float* part, int splits, int M, int N, int64_t ldc, float* out,
                         int64_t ldo, hipStream_t s) {
  if (N % 4 || ldc % 4 || ldo % 4) return hipErrorInvalidValue;
  const int64_t n = (int64_t)M * (N / 4);
  if (splitk_groups(M, N, splits) > 1) {
    constexpr int COLS = 256 / RG_GROUPS;
    k_splitk_reduce_grouped<<<(unsigned)((n + COLS - 1) / COLS), 256, 0, s>>>(part, splits, M, N, ldc, out, ldo);
    return hipGetLastError();
  }
  k_splitk_reduce<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(part, splits, M, N, ldc, out, ldo);
  return hipGetLastError();
}

}  // namespace spz
