// Large-tile bfloat16 MFMA GEMM for the wide layers (256-row tiles).
//
// Same three products and epilogues as the generic kernel (gemm.hip), for
// bf16 operands whose tile dimensions are multiples of 256 (rows) and 256 or
// 128 (columns). Design points for gfx950:
//   * 512 threads = 8 waves (two per SIMD) in a 4x2 grid; each wave owns
//     64 x BN/2 of the output as 2 x (BN/64) blocks of v_mfma_f32_32x32x16_bf16
//     (128 or 64 float32 accumulators per lane). Two waves per SIMD let one
//     wave's LDS reads and global loads overlap the other's matrix work, which
//     measured faster than one wave per SIMD with 128 x 128 wave tiles.
//   * Forward and input-gradient products (both operands k-contiguous; the input
//     gradient reads the transposed weight image GemmArgs::Bt): 64-deep chunks go
//     straight from global memory into LDS (buffer_load ... lds, 128-byte row
//     segments, chunk-swizzled rows) in two stages, one barrier per chunk; see
//     chunk_main_loop.
//   * Register-staged operands are copied global -> registers -> LDS in their
//     memory layout (16-byte vector loads and stores, no shuffles). An
//     m/n-contiguous (k-major) tile is read with two ds_read_b64_tr_b16
//     transposing reads per fragment: within each 16-lane group, lane i addresses
//     4 consecutive values of row k0 + i/4 at column m0 + 4(i%4), and lane j
//     receives column m0 + j for the 4 rows.
//   * Weight-gradient product (both operands register-staged): three LDS stages
//     of one 32-deep k slice each, one barrier per slice. In slice k: the
//     registers holding slice k+2 go to the stage freed by slice k-1, the global
//     loads of slice k+3 are issued, the first 16-deep half of slice k
//     is multiplied while the fragments of its second half are read, the barrier
//     publishes slice k+1, and the second half is multiplied while the fragments
//     of slice k+1's first half are read. The matrix cores never wait for an LDS
//     read after the barrier, and the barrier sits between two runs of MFMAs.
//     Instruction groups are interleaved explicitly (one LDS access per MFMA).
//   * XCD-aware tile order: workgroup b runs on XCD b % 8, so logical tiles are
//     handed out in contiguous ranges per XCD; the column tiles of one row panel
//     (and the split-K slices of one weight-gradient tile) share an L2.
//   * Epilogue: the forward's bias starts the accumulators; blocks leave in pairs
//     through a per-wave LDS scratch as 16-byte row pieces (whole 128-byte lines per
//     store); ReLU, mask bits, column sums and row dots work on rounded bf16 pairs
//     (the epilogue is VALU-heavy); see epi_pair. Forward products that do not store
//     C take transposed accumulators instead (each lane holds a row) and need no
//     scratch; see epilogue_trans.
#include "internal.h"

namespace spz {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int16_t i16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
#define LDS_AS __attribute__((address_space(3)))

constexpr int BM = 256, BK = 32, NT = 512, WM = 4, WN = 2, STAGES = 3;

template <bool KC, int ROWS>
struct BigTile {
  // Row pitch in elements. k-contiguous rows of 80 bytes put the 16 rows read by
  // one 16-lane phase of a 16-byte read on distinct 4-bank groups; k-major rows of
  // 2*ROWS + 64 bytes shift consecutive k rows by 16 banks, so the two 16-lane
  // groups of a transposing read (4 rows x 32 bytes each) never share a bank.
  static constexpr int PITCH = KC ? BK + 8 : ROWS + 32;
  static constexpr int ELEMS = (KC ? ROWS : BK) * PITCH;
  static constexpr int NV = ROWS * BK / 8;
  static constexpr int PER = NV / NT;
  static constexpr int VPR = (KC ? BK : ROWS) / 8;
  static_assert(NV % NT == 0, "tile must split evenly over the workgroup");
  u32x4 r[PER];

  // RG (ragged last tile of N, N % 8 == 0): rows (KC) or columns (m/n-contiguous)
  // at or beyond lim read as zero. Separate instantiation: the predicate in the
  // main loop costs the whole-tile products several percent.
  template <bool RG>
  __device__ inline void load(const bf16_t* __restrict__ base, int64_t ld, int r0, int k0, int tid, int lim) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      const int a = v / VPR, b = (v % VPR) * 8;
      const bf16_t* src = KC ? base + (int64_t)(r0 + a) * ld + (k0 + b) : base + (int64_t)(k0 + a) * ld + (r0 + b);
      if constexpr (RG) {
        const bool ok = KC ? r0 + a < lim : r0 + b < lim;
        r[p] = ok ? *reinterpret_cast<const u32x4*>(src) : u32x4{0u, 0u, 0u, 0u};
      } else {
        (void)lim;
        r[p] = *reinterpret_cast<const u32x4*>(src);
      }
    }
  }
  __device__ inline void store(bf16_t* lds, int tid) const {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      const int a = v / VPR, b = (v % VPR) * 8;
      *reinterpret_cast<u32x4*>(lds + a * PITCH + b) = r[p];
    }
  }
};

template <bool KC, int PITCH>
__device__ inline bf16x8 frag(const bf16_t* lds, int rb, int ks, int lane) {
  if constexpr (KC) {
    const int row = rb + (lane & 31), k = ks + 8 * (lane >> 5);
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(lds + row * PITCH + k));
  } else {
    const int g = lane >> 4, i = lane & 15;
    const int m0 = rb + 16 * (g & 1), k0 = ks + 8 * (g >> 1);
    const bf16_t* p = lds + (k0 + (i >> 2)) * PITCH + m0 + 4 * (i & 3);
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LDS_AS bf16x4*)(p));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((LDS_AS bf16x4*)(p + 4 * PITCH));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  }
}

// Forward-product operands (both k-contiguous) are loaded 64 deep at a time straight
// into LDS (buffer_load_dwordx4 ... lds, 16 bytes per lane), so that every row
// contributes one 128-byte segment per load: half the L2 requests of 64-byte segments,
// which measured clearly faster, and no register staging or LDS store instructions.
// The buffer form, not global_load_lds: the compiler treats a global (FLAT-encoded)
// load into LDS as possibly reaching LDS through the flat aperture, and then waits for
// every outstanding LDS read (lgkmcnt 0) before each MFMA that consumes a fragment,
// which put an LDS round trip in front of every 16-deep step; with the buffer form the
// waits stay partial (2-6% faster on the forward and input-gradient products).
constexpr int CK = 64;   // k depth of one forward chunk
// Word 3 of a raw (stride 0) buffer resource on gfx9-family targets: 32-bit data
// format, no swizzle, no index stride.
constexpr int BUF_DW3 = 0x00020000;

// Chunk swizzle of the 128-byte LDS rows of a forward chunk (eight 16-byte chunks):
// chunk c of row r sits at position c ^ csw(r), so the 16 rows read by one 16-lane
// phase of a fragment read fall on 16 distinct 16-byte bank groups.
__host__ __device__ constexpr int csw(int r) { return (r >> 1) & 7; }

// ROWS x 64 operand chunk: one wave instruction fills 1 KB of LDS (lane l at byte
// 16 l) = 8 rows. Each chunk gets its own buffer resource, starting at element
// (r0, k0) and ending with row lim - 1, so the per-lane offsets do not change from
// chunk to chunk (they stay in registers) and the hardware range check turns reads
// past the end of the operand into zeros: the k beyond the last column of a row read
// the next row's values (never read back), and chunks past the end of the product
// read nothing. RG rows at or beyond lim (ragged last tile of N) are loaded from row
// lim - 1 (their products land only in columns not stored). Offsets are 32-bit: 256
// rows of the operand stay below 2 GiB (big_gemm_ld_ok).
template <int ROWS>
struct FwdChunk {
  static constexpr int BYTES = ROWS * CK * 2;
  static constexpr int PER = BYTES / 1024 / (NT / 64);   // instructions per wave
  static_assert(PER * 1024 * (NT / 64) == BYTES, "chunk must split evenly over the waves");
  template <bool RG>
  __device__ static inline void issue(const bf16_t* __restrict__ base, int64_t ld, int r0, int k0, uint8_t* lds,
                                      int wave, int lane, int lim) {
    int64_t nrec = ((int64_t)lim - r0) * ld * 2 - (int64_t)k0 * 2;
    nrec = nrec < 0 ? 0 : (nrec < 0x7fffffff ? nrec : 0x7fffffff);
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void*)(base + (int64_t)r0 * ld + k0), (short)0, (int)nrec, BUF_DW3);
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int idx = wave + p * (NT / 64);
      const int rr = idx * 8 + (lane >> 3);
      int row = rr;
      if constexpr (RG) row = r0 + row < lim ? row : lim - 1 - r0;
      const int voff = (row * (int)ld + 8 * ((lane & 7) ^ csw(rr))) * 2;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (LDS_AS void*)(lds + idx * 1024), 16, voff, 0, 0, 0);
    }
  }
};

// Fragment (32 rows x 16 k, lane layout of frag<true, ...>) at k offset ks of a chunk.
__device__ inline bf16x8 cfrag(const uint8_t* lds, int rb, int ks, int lane) {
  const int row = rb + (lane & 31);
  const int c = (ks >> 3) + (lane >> 5);
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(lds + row * 128 + (c ^ csw(row)) * 16));
}

// Workgroup barrier after this wave's loads into LDS have landed but for the N most
// recent ones (loads complete in issue order) and its LDS reads are done. A plain
// __syncthreads would also wait for the loads still meant to be in flight.
template <int N>
__device__ inline void sync_loads() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | ((N >> 4) << 14));   // vmcnt N, expcnt 7, lgkmcnt 0
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Epilogue. Accumulator blocks leave in pairs of horizontally adjacent 32x32 blocks
// (64 columns) through a per-wave LDS scratch, so that each lane handles 8
// consecutive columns of one row and the 8 lanes of a row cover 128 bytes of bf16
// output: 16-byte loads of mask and bias, 16-byte (bf16) or 32-byte (fp32) stores,
// whole 128-byte lines per row and store. 32x32 accumulator layout: lane holds
// column lane%32; register q holds row 8*(q/4) + 4*(lane/32) + q%4 of the block.
//   CSUM (dgrad): column sums of the stored (rounded) values over the tile's 256
//     rows go to g.colsum[mt, :]: per lane over its rows, a fixed butterfly over the
//     8 lanes of a column group, then the WM waves of the column in order via LDS.
//   BITS_OUT (fwd): one bit per stored value (> 0), 32 columns per word, words of
//     one 32-column block stored row-contiguously.
//   BITS (dgrad): the same bits as the mask.
//   RDOT (fwd): per row, the dot product of the stored values of the wave's
//     BN/WN columns with rdot_w, one partial per (column tile, wave column).
//   NOSTORE (fwd): C itself is not written.
constexpr int SCR_ROWS = 8;     // scratch rows per wave (one pass of a block pair)
constexpr int SCR_PITCH = 68;   // floats per scratch row
// Floats of the per-wave scratches and the column-sum area [WM][BN]; the staged
// epilogue inputs follow.
template <int BN>
constexpr int scr_floats() { return (NT / 64) * SCR_ROWS * SCR_PITCH + WM * BN; }

// Epilogue inputs of one tile, staged in LDS (after the scratch) so that each
// 32x32 block reads them with LDS latency: bias [BN] fp32, output-layer weights
// [BN] bf16 (as BN/2 words), and mask bits [BN/32 word columns][BM rows] (read by
// the input gradient, written by the forward and stored to memory at the end).
template <int BN>
struct EpiLds {
  static constexpr int BIAS = 0, RDW = BN, BITS = BN + BN / 2;
  static constexpr int WORDS = BN + BN / 2 + (BN / 32) * BM;
};

// Global loads of the staged inputs, issued before the last slice's MFMAs so their
// latency is hidden; 16-byte loads.
template <int MODE, int BN, int F>
struct EpiPrefetch {
  static constexpr bool BIAS = false, RDOT = (F & EPI_RDOT) != 0, BITS = (F & EPI_BITS) != 0;   // bias: in the accumulators
  static constexpr int NBITS = (BN / 32) * BM / 4;   // 16-byte pieces of the bits tile
  static constexpr int NBP = (NBITS + NT - 1) / NT;   // ... per thread
  u32x4 bits[NBP], rdw;
  float4 bias;
  __device__ inline void load(const GemmArgs& g, int m0, int n0, int tid) {
    if constexpr (BIAS) {
      if (g.bias && tid < BN / 4 && n0 + 4 * tid < g.N) bias = *reinterpret_cast<const float4*>(g.bias + n0 + 4 * tid);
      else bias = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
    if constexpr (RDOT) {
      if (tid < BN / 8) rdw = *reinterpret_cast<const u32x4*>(static_cast<const bf16_t*>(g.rdot_w) + n0 + 8 * tid);
    }
    if constexpr (BITS) {
#pragma unroll
      for (int p = 0; p < NBP; ++p) {
        const int t = tid + p * NT;
        if (t < NBITS) {
          const int wc = t / (BM / 4), r4 = (t % (BM / 4)) * 4;
          bits[p] = *reinterpret_cast<const u32x4*>(g.bits + (int64_t)(n0 / 32 + wc) * g.ldbits + m0 + r4);
        }
      }
    }
  }
  __device__ inline void store(uint32_t* lds, int tid) const {
    using L = EpiLds<BN>;
    if constexpr (BIAS) {
      if (tid < BN / 4) *reinterpret_cast<float4*>(lds + L::BIAS + 4 * tid) = bias;
    }
    if constexpr (RDOT) {
      if (tid < BN / 8) *reinterpret_cast<u32x4*>(lds + L::RDW + 4 * tid) = rdw;
    }
    if constexpr (BITS) {
#pragma unroll
      for (int p = 0; p < NBP; ++p)
        if (tid + p * NT < NBITS) *reinterpret_cast<u32x4*>(lds + L::BITS + 4 * (tid + p * NT)) = bits[p];
    }
  }
};

// Blocks (i, 2 jp) and (i, 2 jp + 1) of the wave, in four passes of 8 rows: cs
// accumulates the column sums of the lane's 8 columns, rd[p] the row dots of its
// row in pass p.
template <int MODE, int BN, int F>
__device__ inline void epi_pair(const GemmArgs& g, const f32x16& a0, const f32x16& a1, int i, int jp, int m0,
                                int n0, int wm, int wn, int lane, int z, float* scr, const uint32_t* in,
                                float (&cs)[8], float (&rd)[4]) {
  using L = EpiLds<BN>;
  constexpr int WCOLS = BN / WN;
  constexpr bool OUTF32 = F & EPI_F32, RELU = F & EPI_RELU, MASK = F & EPI_MASK, BITS = F & EPI_BITS;
  constexpr bool BITS_OUT = F & EPI_BITS_OUT, CSUM = F & EPI_CSUM, RDOT = F & EPI_RDOT;
  constexpr bool STORE = !(F & EPI_NOSTORE);
  const int cgrp = lane & 7, rsub = lane >> 3;
  const int cb = wn * WCOLS + 64 * jp + 8 * cgrp;   // lane's first column in the tile
  uint32_t ww[4] = {0u, 0u, 0u, 0u};   // output-layer weights of the lane's 8 columns, packed bf16
  if constexpr (RDOT) {
    const u32x4 w4 = *reinterpret_cast<const u32x4*>(in + L::RDW + cb / 2);
    ww[0] = w4[0]; ww[1] = w4[1]; ww[2] = w4[2]; ww[3] = w4[3];
  }
  // Mask words of the lane's 32-column block; its 8 columns are bits 8 (cgrp % 4) on.
  uint32_t* bits_lds = const_cast<uint32_t*>(in) + L::BITS + (cb >> 5) * BM;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
#pragma unroll
    for (int q = 4 * p; q < 4 * p + 4; ++q) {
      scr[(4 * (lane >> 5) + (q & 3)) * SCR_PITCH + (lane & 31)] = a0[q];
      scr[(4 * (lane >> 5) + (q & 3)) * SCR_PITCH + 32 + (lane & 31)] = a1[q];
    }
    const int rl = wm * (BM / WM) + 32 * i + 8 * p + rsub;   // row within the tile
    const int64_t row = m0 + rl;
    const float4 x0 = *reinterpret_cast<const float4*>(scr + rsub * SCR_PITCH + 8 * cgrp);
    const float4 x1 = *reinterpret_cast<const float4*>(scr + rsub * SCR_PITCH + 8 * cgrp + 4);
    float v[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
    if (n0 + cb >= g.N) continue;   // ragged last column tile (N % 8 == 0)
    if constexpr (MODE == GEMM_WGRAD) {
      float* dst = static_cast<float*>(g.C) + ((int64_t)z * g.M + row) * g.ldc + n0 + cb;
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      *reinterpret_cast<float4*>(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
      continue;
    }
    // The forward's bias is already in the accumulators (k_gemm_big). ReLU of a bf16
    // output is taken on the rounded values (below).
    if constexpr (RELU && OUTF32) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = v[e] < 0.0f ? 0.0f : v[e];
    }
    // Row offsets within the tile in 32-bit arithmetic (leading dimensions below 2^22,
    // big_gemm_ld_ok), added to the tile's base address.
    if constexpr (MASK) {
      const uint4 mk = *reinterpret_cast<const uint4*>(static_cast<const bf16_t*>(g.mask) + (int64_t)m0 * g.ldm + n0 +
                                                        (rl * (int)g.ldm + cb));
      const uint32_t mw[4] = {mk.x, mk.y, mk.z, mk.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float h = bf2f((bf16_t)((mw[e >> 1] >> (16 * (e & 1))) & 0xFFFFu));
        v[e] = h > 0.0f ? v[e] : 0.0f;
      }
    }
    if constexpr (BITS && OUTF32) {
      const uint32_t wd = bits_lds[rl] >> (8 * (cgrp & 3));
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (wd >> e) & 1u ? v[e] : 0.0f;
    }
    if constexpr (OUTF32) {
      float* dst = static_cast<float*>(g.C) + (int64_t)m0 * g.ldc + n0 + (rl * (int)g.ldc + cb);
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      *reinterpret_cast<float4*>(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
    } else {
      // bf16 output. The epilogue is VALU-bound, so the per-value work is done on the
      // rounded pairs where that is exact: ReLU (a bf16 is negative exactly when its
      // bits are as int16; a rounded -0.0 becomes +0.0), the mask bits (masking before
      // or after rounding gives the same bits), the mask bits out (after ReLU a value
      // is > 0 exactly when its bits are nonzero); column sums and the row dot take
      // both values of a pair with one v_dot2_f32_bf16 (products by 1, 0 are exact).
      static_assert(!BITS_OUT || RELU, "mask bits out are taken of ReLU outputs");
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        w[e] = pack_bf16x2(v[2 * e], v[2 * e + 1]);
        if constexpr (RELU)
          w[e] = __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(i16x2, w[e]), i16x2{0, 0}));
      }
      if constexpr (BITS) {
        const int wd = (int)(bits_lds[rl] >> (8 * (cgrp & 3)));
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] &= (0x0000FFFFu & (uint32_t)__builtin_amdgcn_sbfe(wd, 2 * e, 1)) |
                  (0xFFFF0000u & (uint32_t)__builtin_amdgcn_sbfe(wd, 2 * e + 1, 1));
      }
      if constexpr (CSUM) {
        // (1, 0) and (0, 1) from registers: folded into an inline constant, (1, 0) was
        // encoded as the 32-bit 1.0f, which the packed operand reads as (0, 1).
        uint32_t k_lo = 0x00003F80u, k_hi = 0x3F800000u;
        asm volatile("" : "+v"(k_lo), "+v"(k_hi));
        const bf16x2 lo1 = __builtin_bit_cast(bf16x2, k_lo), hi1 = __builtin_bit_cast(bf16x2, k_hi);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          cs[2 * e] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), lo1, cs[2 * e], false);
          cs[2 * e + 1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), hi1, cs[2 * e + 1], false);
        }
      }
      if constexpr (RDOT) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          rd[p] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), __builtin_bit_cast(bf16x2, ww[e]), rd[p],
                                                  false);
      }
      if constexpr (BITS_OUT) {
        // halves clamped to 0 / 1, pair e at bits 2e (low) and 16 + 2e (high)
        uint32_t t = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t m;
          // one packed min (the compiler splits the vector form into compares and selects)
          // (1, 1) from a register: an inline constant would give the high half 0
          asm("v_pk_min_u16 %0, %1, %2" : "=v"(m) : "v"(w[e]), "s"(0x00010001u));
          t |= m << (2 * e);
        }
        // Each of the four lanes of a row and 32-column block owns one byte of its word.
        reinterpret_cast<uint8_t*>(bits_lds + rl)[cgrp & 3] = (uint8_t)((t | (t >> 15)) & 0xFFu);
      }
      // Non-temporal: the stored activations are re-read by later kernels, not by
      // this one (measured faster per update step than plain stores).
      if constexpr (STORE)
        __builtin_nontemporal_store(u32x4{w[0], w[1], w[2], w[3]},
                                    reinterpret_cast<u32x4*>(static_cast<bf16_t*>(g.C) + (int64_t)m0 * g.ldc + n0 +
                                                             (rl * (int)g.ldc + cb)));
    }
  }
}

// Epilogue over the wave's blocks, in pairs (epi_pair). Bias, output-layer weights
// and mask bits come from the LDS staging area (EpiLds). Pairs go column-major when
// column sums accumulate over row blocks and row-major otherwise, so that only the
// running sums of one block row or column stay live. BITS_OUT words are gathered in
// LDS and written to memory with one 16-byte store per thread at the end.
template <int MODE, int BN, int F>
__device__ inline void epilogue(const GemmArgs& g, const f32x16 (&acc)[BM / WM / 32][BN / WN / 32], int m0,
                                int n0, int wm, int wn, int lane, int wave, int z, int mt, float* smem_f,
                                uint32_t* in) {
  constexpr int TM_ = BM / WM / 32, TN_ = BN / WN / 32, WCOLS = BN / WN;
  static_assert(TN_ % 2 == 0, "blocks leave in horizontal pairs");
  float* scr = smem_f + wave * (SCR_ROWS * SCR_PITCH);
  float* csh = smem_f + (NT / 64) * SCR_ROWS * SCR_PITCH;   // [WM][BN]
  const int cgrp = lane & 7, rsub = lane >> 3;
  if constexpr ((F & EPI_CSUM) != 0) {
#pragma unroll
    for (int jp = 0; jp < TN_ / 2; ++jp) {
      float cs[8], rd[4];
#pragma unroll
      for (int e = 0; e < 8; ++e) cs[e] = 0.0f;
#pragma unroll
      for (int i = 0; i < TM_; ++i)
        epi_pair<MODE, BN, F>(g, acc[i][2 * jp], acc[i][2 * jp + 1], i, jp, m0, n0, wm, wn, lane, z, scr, in, cs,
                              rd);
      // Reduce-scatter over lane bits 3, 4, 5 (the 8 rows of a column group; each
      // exchange halves the columns a lane keeps).
      const bool b3 = lane & 8, b4 = lane & 16, b5 = lane & 32;
      float t4[4], t2[2];
#pragma unroll
      for (int e = 0; e < 4; ++e) t4[e] = (b3 ? cs[4 + e] : cs[e]) + __shfl_xor(b3 ? cs[e] : cs[4 + e], 8);
#pragma unroll
      for (int e = 0; e < 2; ++e) t2[e] = (b4 ? t4[2 + e] : t4[e]) + __shfl_xor(b4 ? t4[e] : t4[2 + e], 16);
      const float t1 = (b5 ? t2[1] : t2[0]) + __shfl_xor(b5 ? t2[0] : t2[1], 32);
      csh[wm * BN + wn * WCOLS + 64 * jp + 8 * cgrp + 4 * b3 + 2 * b4 + (b5 ? 1 : 0)] = t1;
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    for (int c = threadIdx.x; c < BN; c += NT) {
      float t = 0.0f;
#pragma unroll
      for (int w = 0; w < WM; ++w) t += csh[w * BN + c];
      g.colsum[(int64_t)mt * g.ldcs + n0 + c] = t;
    }
  } else {
#pragma unroll
    for (int i = 0; i < TM_; ++i) {
      float cs[8], rd[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int jp = 0; jp < TN_ / 2; ++jp) {
        epi_pair<MODE, BN, F>(g, acc[i][2 * jp], acc[i][2 * jp + 1], i, jp, m0, n0, wm, wn, lane, z, scr, in, cs,
                              rd);
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr ((F & EPI_RDOT) != 0) {
        const int part = (n0 + wn * WCOLS) / WCOLS;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          float t = rd[p];
          t += __shfl_xor(t, 1);
          t += __shfl_xor(t, 2);
          t += __shfl_xor(t, 4);
          if (cgrp == 0) g.rdot_part[(int64_t)part * g.ldrd + m0 + wm * (BM / WM) + 32 * i + 8 * p + rsub] = t;
        }
      }
    }
  }
  if constexpr ((F & EPI_BITS_OUT) != 0) {
    // The tile's mask words, one 16-byte piece per thread, row-contiguous per word column.
    __syncthreads();
    constexpr int NB = (BN / 32) * BM / 4;
    for (int t = threadIdx.x; t < NB; t += NT) {
      const int wc = t / (BM / 4), r4 = (t % (BM / 4)) * 4;
      *reinterpret_cast<u32x4*>(g.bits_out + (int64_t)(n0 / 32 + wc) * g.ldbits + m0 + r4) =
          *reinterpret_cast<const u32x4*>(in + EpiLds<BN>::BITS + 4 * t);
    }
  }
}

// Forward products that do not store C (row dots with the output layer, mask bits) take
// the transposed accumulator layout: the MFMA computes the 32 x 32 block of C^T
// (operands swapped), so lane l holds row l % 32 of the block and register q column
// 8 (q / 4) + 4 (l / 32) + q % 4, and a row's dot product and mask word need no LDS
// round trip (the scratch path costs these variants about 7% of the kernel). With a
// stored C the same layout would write each 128-byte line in four 32-byte pieces from
// four instructions, which measured 15-75% slower than whole-line stores (non-temporal
// or plain), so those variants keep the scratch path.
__host__ __device__ constexpr bool trans_epilogue(int mode, int f) {
  return mode == GEMM_FWD && (f & EPI_NOSTORE);
}

// Swap the upper half-wave's x with the lower half-wave's y (v_permlane32_swap).
__device__ inline void swap_halves(uint32_t& x, uint32_t& y) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, y, false, false);
  x = r[0];
  y = r[1];
}

template <int BN, int F, bool RG>
__device__ inline void epilogue_trans(const GemmArgs& g, const f32x16 (&acc)[BM / WM / 32][BN / WN / 32], int m0,
                                      int n0, int wm, int wn, int lane, uint32_t* in) {
  using L = EpiLds<BN>;
  constexpr int TM = BM / WM / 32, TN = BN / WN / 32, WCOLS = BN / WN;
  constexpr bool RELU = F & EPI_RELU, BITS_OUT = F & EPI_BITS_OUT, RDOT = F & EPI_RDOT;
  static_assert(F & EPI_NOSTORE, "C is not stored in this layout");
  static_assert(!BITS_OUT || RELU, "mask bits out are taken of ReLU outputs");
  static_assert(!RG, "fused epilogue features need whole column tiles");
  const int h = lane >> 5, r = lane & 31;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int rl = wm * (BM / WM) + 32 * i + r;   // row within the tile
    float rd = 0.0f;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int cb = wn * WCOLS + 32 * j;   // block's first column within the tile
      // w[2 q4 + t]: columns 8 q4 + 4 h + 2 t and + 1, rounded to bf16 as a stored C
      // would be (ReLU on the rounded pair: a bf16 is negative exactly when its bits are
      // as int16)
      uint32_t w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        w[e] = pack_bf16x2(acc[i][j][2 * e], acc[i][j][2 * e + 1]);
        if constexpr (RELU)
          w[e] = __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(i16x2, w[e]), i16x2{0, 0}));
      }
      if constexpr (RDOT) {
        // Output-layer weights of the lane's 16 columns, packed bf16 pairs.
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const uint2 ww = *reinterpret_cast<const uint2*>(in + L::RDW + (cb + 8 * q4 + 4 * h) / 2);
          rd = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[2 * q4]), __builtin_bit_cast(bf16x2, ww.x),
                                               rd, false);
          rd = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[2 * q4 + 1]),
                                               __builtin_bit_cast(bf16x2, ww.y), rd, false);
        }
      }
      if constexpr (BITS_OUT) {
        // After ReLU a value is > 0 exactly when its bits are nonzero: halves clamped to
        // 0 / 1 by one packed min, column c of the block at bit c.
        uint32_t t = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          uint32_t m;
          asm("v_pk_min_u16 %0, %1, %2" : "=v"(m) : "v"(w[e]), "s"(0x00010001u));
          const int c = 8 * (e >> 1) + 4 * h + 2 * (e & 1);
          t |= ((m & 1u) << c) | ((m >> 16) << (c + 1));
        }
        uint32_t u = t;
        swap_halves(t, u);   // lower half-wave: own word in t, the upper's in u
        if (h == 0) in[L::BITS + (cb >> 5) * BM + rl] = t | u;
      }
    }
    if constexpr (RDOT) {
      // per row, the sum over the wave's WCOLS columns; one partial per (column tile,
      // wave column)
      uint32_t a = __builtin_bit_cast(uint32_t, rd), b = a;
      swap_halves(a, b);
      const float o = __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
      const int part = (n0 + wn * WCOLS) / WCOLS;
      if (h == 0) g.rdot_part[(int64_t)part * g.ldrd + m0 + rl] = o;
    }
  }
  if constexpr (BITS_OUT) {
    // The tile's mask words, one 16-byte piece per thread, row-contiguous per word column.
    __syncthreads();
    constexpr int NB = (BN / 32) * BM / 4;
    for (int t = threadIdx.x; t < NB; t += NT) {
      const int wc = t / (BM / 4), r4 = (t % (BM / 4)) * 4;
      *reinterpret_cast<u32x4*>(g.bits_out + (int64_t)(n0 / 32 + wc) * g.ldbits + m0 + r4) =
          *reinterpret_cast<const u32x4*>(in + L::BITS + 4 * t);
    }
  }
}

// Chunked main loop of the forward and input-gradient products, C = A . B^T with A
// [M, K] and B [N, K] both k-contiguous (the input gradient takes the transposed
// weight image): 64-deep chunks in two LDS stages, one barrier per chunk. Chunk c
// is multiplied in four 16-deep steps, each step's MFMAs overlapping the fragment
// reads of the next step; the barrier sits between steps 2 and 3: it publishes
// chunk c + 1 (whose loads, issued right after the previous barrier, have had four
// steps to land) and retires every wave's reads of chunk c, whose stage then
// receives chunk c + 2 while step 3 runs. An odd number of 32-deep slices ends with
// a half chunk of two steps.
template <int BN>
struct ChunkLds {
  static constexpr int ABYTES = FwdChunk<BM>::BYTES;
  static constexpr int BYTES = ABYTES + FwdChunk<BN>::BYTES;
};

template <int BN, bool RG, bool TRANS>
__device__ inline void chunk_main_loop(const GemmArgs& g, f32x16 (&acc)[BM / WM / 32][BN / WN / 32], int m0,
                                       int n0, int wm, int wn, int wave, int lane, uint8_t* smem) {
  constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
  using CA = FwdChunk<BM>;
  using CB = FwdChunk<BN>;
  constexpr int ABYTES = ChunkLds<BN>::ABYTES;
  constexpr int SB = ChunkLds<BN>::BYTES;     // bytes per stage: A chunk then B chunk
  constexpr int LPC = CA::PER + CB::PER;      // load instructions per wave and chunk
  constexpr int NR = TM + TN;                 // fragment reads per step
  const bf16_t* __restrict__ A = static_cast<const bf16_t*>(g.A);
  const bf16_t* __restrict__ B = static_cast<const bf16_t*>(g.B);
  const int nk = g.K / BK;                    // 32-deep slices
  const int nfull = nk >> 1;
  wave = __builtin_amdgcn_readfirstlane(wave);   // LDS destinations (M0) from scalar registers
  auto stage = [&](int c) { return smem + (c & 1) * SB; };
  auto issue = [&](int c) {
    CA::template issue<false>(A, g.lda, m0, c * CK, stage(c), wave, lane, g.M);
    CB::template issue<RG>(B, g.ldb, n0, c * CK, stage(c) + ABYTES, wave, lane, g.N);
  };
  bf16x8 fa0[TM], fb0[TN], fa1[TM], fb1[TN];
  auto read_step = [&](const uint8_t* st, int ks, bf16x8 (&fa)[TM], bf16x8 (&fb)[TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[i] = cfrag(st, (wm * TM + i) * 32, ks, lane);
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[j] = cfrag(st + ABYTES, (wn * TN + j) * 32, ks, lane);
  };
  auto mma = [&](const bf16x8 (&fa)[TM], const bf16x8 (&fb)[TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = TRANS ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0)
                          : __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  };
  // One LDS read per MFMA (sched_group_barrier masks: 0x008 MFMA, 0x020 global load,
  // 0x100 LDS read).
  auto interleave_reads = [&]() {
#pragma unroll
    for (int t = 0; t < NR; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
  };
  issue(0);
  asm volatile("" ::: "memory");
  issue(1);
  sync_loads<LPC>();   // chunk 0 landed
  read_step(stage(0), 0, fa0, fb0);
  for (int c = 0; c < nfull; ++c) {
    const uint8_t* st = stage(c);
    read_step(st, 16, fa1, fb1);
    mma(fa0, fb0);
    interleave_reads();
    read_step(st, 32, fa0, fb0);
    mma(fa1, fb1);
    interleave_reads();
    read_step(st, 48, fa1, fb1);
    mma(fa0, fb0);
    interleave_reads();
    sync_loads<0>();   // chunk c + 1 landed (the only loads in flight)
    issue(c + 2);
    read_step(stage(c + 1), 0, fa0, fb0);
    mma(fa1, fb1);
#pragma unroll
    for (int t = 0; t < LPC; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
    interleave_reads();
  }
  if (nk & 1) {   // half chunk nfull, published by the last barrier
    read_step(stage(nfull), 16, fa1, fb1);
    mma(fa0, fb0);
    interleave_reads();
    mma(fa1, fb1);
  }
}

// One kernel per (product, column tile, epilogue variant): a runtime switch over the
// variants inside one kernel let common code move above the switch and raised the
// register pressure of every variant to the point of spilling. A launch runs one
// product or two of the same shape and epilogue (GemmPair: the twin critics' layers),
// the second's tiles after the first's.
template <int MODE, int BN, int F, bool RG>
__global__ void __launch_bounds__(NT, 1) k_gemm_big(GemmPair pr, int tiles_m, int tiles_n) {
  constexpr bool AKC = MODE != GEMM_WGRAD;
  constexpr bool BKC = MODE == GEMM_FWD;
  using TA = BigTile<AKC, BM>;
  using TB = BigTile<BKC, BN>;
  constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
  constexpr int SE = TA::ELEMS + TB::ELEMS;   // elements per stage: A tile then B tile
  constexpr bool TRANS = trans_epilogue(MODE, F);
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  bf16_t* S = reinterpret_cast<bf16_t*>(smem);

  // Tiles of each product. A device-side row count (input gradient) leaves only its
  // leading row tiles; the tiles of both products are spread over the XCDs as one range.
  const int per = tiles_m * tiles_n * (MODE == GEMM_WGRAD ? pr.g[0].splits : 1);
  int t0 = per, t1 = pr.n > 1 ? per : 0;
  if constexpr (MODE == GEMM_DGRAD) {
    if (pr.g[0].m_dyn) t0 = (*pr.g[0].m_dyn / BM) * tiles_n;
    if (pr.n > 1 && pr.g[1].m_dyn) t1 = (*pr.g[1].m_dyn / BM) * tiles_n;
  }
  const int total = t0 + t1;
  if ((int)blockIdx.x >= total) return;
  // XCD-aware logical tile: contiguous logical ranges per XCD, column tiles fastest.
  int L = blockIdx.x;
  if ((total & 7) == 0) L = (blockIdx.x & 7) * (total >> 3) + (blockIdx.x >> 3);
  const int pi = L >= t0 ? 1 : 0;
  const GemmArgs& g = pr.g[pi];
  L -= pi * t0;
  const int nt = L % tiles_n;
  const int mt = (L / tiles_n) % tiles_m;
  const int z = L / (tiles_n * tiles_m);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = mt * BM, n0 = nt * BN;
  int kbeg = 0, kend = g.K;
  if constexpr (MODE == GEMM_WGRAD) {
    const int ks = g.K / g.splits;
    kbeg = z * ks;
    kend = kbeg + ks;
  }
  const bf16_t* __restrict__ A = static_cast<const bf16_t*>(g.A);
  const bf16_t* __restrict__ B = static_cast<const bf16_t*>(g.B);

  // The forward's bias starts the accumulators (accumulator column = lane % 32; with
  // transposed accumulators, register q holds column 8 (q / 4) + 4 (lane / 32) + q % 4).
  f32x16 acc[TM][TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    if constexpr (TRANS) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int n = n0 + wn * (BN / WN) + 32 * j + 8 * q4 + 4 * (lane >> 5);
        float4 b = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (g.bias && n < g.N) b = *reinterpret_cast<const float4*>(g.bias + n);   // N % 8 == 0
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          acc[i][j][4 * q4] = b.x;
          acc[i][j][4 * q4 + 1] = b.y;
          acc[i][j][4 * q4 + 2] = b.z;
          acc[i][j][4 * q4 + 3] = b.w;
        }
      }
    } else {
      float b = 0.0f;
      if constexpr (MODE == GEMM_FWD) {
        const int n = n0 + wn * (BN / WN) + 32 * j + (lane & 31);
        if (g.bias && n < g.N) b = g.bias[n];
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[i][j][q] = b;
    }
  }

  EpiPrefetch<MODE, BN, F> pre;
  if constexpr (MODE != GEMM_WGRAD) {
    chunk_main_loop<BN, RG, TRANS>(g, acc, m0, n0, wm, wn, wave, lane, smem);
    pre.load(g, m0, n0, tid);
    sync_loads<0>();   // the trailing (unused) chunk loads must land before LDS is reused
  } else {
    TA ta;
    TB tb;
    const int nk = (kend - kbeg) / BK;
    // Prologue: slices 0 and 1 in stages 0 and 1, slice 2 in registers.
    ta.template load<false>(A, g.lda, m0, kbeg, tid, g.M);
    tb.template load<RG>(B, g.ldb, n0, kbeg, tid, g.N);
    ta.store(S, tid);
    tb.store(S + TA::ELEMS, tid);
    if (nk > 1) {
      ta.template load<false>(A, g.lda, m0, kbeg + BK, tid, g.M);
      tb.template load<RG>(B, g.ldb, n0, kbeg + BK, tid, g.N);
      ta.store(S + SE, tid);
      tb.store(S + SE + TA::ELEMS, tid);
    }
    if (nk > 2) {
      ta.template load<false>(A, g.lda, m0, kbeg + 2 * BK, tid, g.M);
      tb.template load<RG>(B, g.ldb, n0, kbeg + 2 * BK, tid, g.N);
    }
    __syncthreads();
    bf16x8 fa0[TM], fb0[TN], fa1[TM], fb1[TN];
  #pragma unroll
    for (int i = 0; i < TM; ++i) fa0[i] = frag<AKC, TA::PITCH>(S, (wm * TM + i) * 32, 0, lane);
  #pragma unroll
    for (int j = 0; j < TN; ++j) fb0[j] = frag<BKC, TB::PITCH>(S + TA::ELEMS, (wn * TN + j) * 32, 0, lane);
    // LDS read / write and global load instruction counts of one slice, for the
    // interleave pattern (a transposing fragment read is two instructions).
    constexpr int NR = (AKC ? TM : 2 * TM) + (BKC ? TN : 2 * TN);
    constexpr int NW = TA::PER + TB::PER;
    int sc = 0;   // stage of slice kt
    for (int kt = 0; kt < nk; ++kt) {
      if (kt == nk - 1) pre.load(g, m0, n0, tid);
      const int s1 = sc == STAGES - 1 ? 0 : sc + 1;   // stage of slice kt + 1
      const int s2 = s1 == STAGES - 1 ? 0 : s1 + 1;   // stage of slice kt + 2 (= that of kt - 1)
      const bf16_t* Sc = S + sc * SE;
      if (kt + 2 < nk) {
        ta.store(S + s2 * SE, tid);
        tb.store(S + s2 * SE + TA::ELEMS, tid);
      }
      if (kt + 3 < nk) {
        ta.template load<false>(A, g.lda, m0, kbeg + (kt + 3) * BK, tid, g.M);
        tb.template load<RG>(B, g.ldb, n0, kbeg + (kt + 3) * BK, tid, g.N);
      }
  #pragma unroll
      for (int i = 0; i < TM; ++i) fa1[i] = frag<AKC, TA::PITCH>(Sc, (wm * TM + i) * 32, 16, lane);
  #pragma unroll
      for (int j = 0; j < TN; ++j) fb1[j] = frag<BKC, TB::PITCH>(Sc + TA::ELEMS, (wn * TN + j) * 32, 16, lane);
  #pragma unroll
      for (int i = 0; i < TM; ++i)
  #pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa0[i], fb0[j], acc[i][j], 0, 0, 0);
      // sched_group_barrier masks: 0x008 MFMA, 0x020 global load, 0x100 LDS read, 0x200 LDS write.
  #pragma unroll
      for (int t = 0; t < NW; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
  #pragma unroll
      for (int t = 0; t < NW; ++t) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
  #pragma unroll
      for (int t = 0; t < NR; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
      // Publishes slice kt + 1 (stored one slice earlier) and retires every wave's
      // reads of slice kt - 1, whose stage the next slice overwrites.
      __syncthreads();
      if (kt + 1 < nk) {
        const bf16_t* Sn = S + s1 * SE;
  #pragma unroll
        for (int i = 0; i < TM; ++i) fa0[i] = frag<AKC, TA::PITCH>(Sn, (wm * TM + i) * 32, 0, lane);
  #pragma unroll
        for (int j = 0; j < TN; ++j) fb0[j] = frag<BKC, TB::PITCH>(Sn + TA::ELEMS, (wn * TN + j) * 32, 0, lane);
      }
  #pragma unroll
      for (int i = 0; i < TM; ++i)
  #pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa1[i], fb1[j], acc[i][j], 0, 0, 0);
  #pragma unroll
      for (int t = 0; t < NR; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      }
      sc = s1;
    }
  }
  // The barrier of the last slice came after every wave's last LDS read, so the
  // epilogue may reuse LDS: scratch first, then the staged inputs.
  float* scratch = reinterpret_cast<float*>(smem);
  uint32_t* in = reinterpret_cast<uint32_t*>(scratch + scr_floats<BN>());
  if constexpr (MODE != GEMM_WGRAD) {
    pre.store(in, tid);
    __syncthreads();
  }
  if constexpr (TRANS)
    epilogue_trans<BN, F, RG>(g, acc, m0, n0, wm, wn, lane, in);
  else
    epilogue<MODE, BN, F>(g, acc, m0, n0, wm, wn, lane, wave, z, mt, scratch, in);
}

template <int MODE, int BN, int F, bool RG>
hipError_t launch_big_f(const GemmPair& p, hipStream_t s) {
  const GemmArgs& g = p.g[0];
  using TA = BigTile<MODE != GEMM_WGRAD, BM>;
  using TB = BigTile<MODE == GEMM_FWD, BN>;
  const size_t tiles = MODE != GEMM_WGRAD ? 2 * ChunkLds<BN>::BYTES
                                          : STAGES * (TA::ELEMS + TB::ELEMS) * sizeof(bf16_t);
  const size_t scratch = (scr_floats<BN>() + EpiLds<BN>::WORDS) * sizeof(float);
  const size_t lds = tiles > scratch ? tiles : scratch;
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)k_gemm_big<MODE, BN, F, RG>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int tiles_m = g.M / BM, tiles_n = (g.N + BN - 1) / BN;
  const int splits = MODE == GEMM_WGRAD ? g.splits : 1;
  k_gemm_big<MODE, BN, F, RG><<<tiles_m * tiles_n * splits * p.n, NT, lds, s>>>(p, tiles_m, tiles_n);
  return hipGetLastError();
}

template <int MODE, int BN>
hipError_t launch_big(const GemmPair& p, hipStream_t s) {
  const GemmArgs& g = p.g[0];
  const bool rg = g.N % BN != 0;
#define SPZ_CASE(F) \
  case (F): return rg ? launch_big_f<MODE, BN, (F), true>(p, s) : launch_big_f<MODE, BN, (F), false>(p, s)
#define SPZ_CASE_WHOLE(F) \
  case (F): return rg ? hipErrorInvalidValue : launch_big_f<MODE, BN, (F), false>(p, s)
  if constexpr (MODE == GEMM_WGRAD) {
    return rg ? launch_big_f<MODE, BN, EPI_F32, true>(p, s) : launch_big_f<MODE, BN, EPI_F32, false>(p, s);
  } else if constexpr (MODE == GEMM_FWD) {
    switch (epilogue_flags((GemmMode)MODE, g)) {
      SPZ_CASE(EPI_F32);
      SPZ_CASE(0);
      SPZ_CASE(EPI_RELU);
      SPZ_CASE_WHOLE(EPI_RELU | EPI_BITS_OUT);
      SPZ_CASE_WHOLE(EPI_RELU | EPI_RDOT);
      SPZ_CASE_WHOLE(EPI_RELU | EPI_RDOT | EPI_NOSTORE);
      SPZ_CASE_WHOLE(EPI_RELU | EPI_BITS_OUT | EPI_RDOT);
      SPZ_CASE_WHOLE(EPI_RELU | EPI_BITS_OUT | EPI_RDOT | EPI_NOSTORE);
    }
  } else {
    switch (epilogue_flags((GemmMode)MODE, g)) {
      SPZ_CASE(EPI_F32);
      SPZ_CASE(0);
      SPZ_CASE(EPI_MASK);
      SPZ_CASE_WHOLE(EPI_MASK | EPI_CSUM);
      SPZ_CASE_WHOLE(EPI_CSUM);
      SPZ_CASE_WHOLE(EPI_BITS);
      SPZ_CASE_WHOLE(EPI_BITS | EPI_CSUM);
    }
  }
#undef SPZ_CASE
#undef SPZ_CASE_WHOLE
  return hipErrorInvalidValue;
}

}  // namespace

int gemm_rdot_cols(int M, int N) { return big_bn(GEMM_FWD, M, N, true) / WN; }

bool big_epilogue_supported(GemmMode mode, int f) {
  switch (mode) {
    case GEMM_WGRAD: return f == EPI_F32;
    case GEMM_FWD:
      switch (f) {
        case EPI_F32: case 0: case EPI_RELU: case EPI_RELU | EPI_BITS_OUT: case EPI_RELU | EPI_RDOT:
        case EPI_RELU | EPI_RDOT | EPI_NOSTORE: case EPI_RELU | EPI_BITS_OUT | EPI_RDOT:
        case EPI_RELU | EPI_BITS_OUT | EPI_RDOT | EPI_NOSTORE:
          return true;
      }
      return false;
    case GEMM_DGRAD:
      switch (f) {
        case EPI_F32: case 0: case EPI_MASK: case EPI_MASK | EPI_CSUM: case EPI_CSUM: case EPI_BITS:
        case EPI_BITS | EPI_CSUM:
          return true;
      }
      return false;
  }
  return false;
}

bool big_gemm_colsum(GemmMode mode, int M, int N, int K) {
  return mode == GEMM_DGRAD && big_gemm_fits(mode, M, N, K, 1);
}

int big_bn(GemmMode mode, int M, int N, bool fused) {
  // 256-wide unless that grid leaves CUs idle: a 16384 x 256 forward is 64 workgroups of
  // 256 x 256 on 256 CUs (the weight gradient splits K to fill the GPU instead).
  if (N % 256 == 0) return mode == GEMM_WGRAD || (int64_t)(M / BM) * (N / 256) >= 256 ? 256 : 128;
  if (fused) return 128;          // fused epilogues need whole column tiles (N % 128 == 0)
  return N > 256 ? 256 : 128;     // ragged last column tile
}

bool big_gemm_fits(GemmMode mode, int M, int N, int K, int splits) {
  (void)mode;
  // Below 128 columns the generic kernel's small tiles waste less work.
  if (M % BM || N % 8 || N < 128) return false;
  const int kk = mode == GEMM_WGRAD ? K / splits : K;
  return kk % BK == 0 && kk > 0;
}

bool big_gemm_ld_ok(GemmMode mode, const GemmArgs& g) {
  // Forward and input-gradient tiles are read through buffer resources with 32-bit
  // byte offsets: 256 rows of the widest operand must stay below 2 GiB.
  constexpr int64_t LIM = (int64_t)1 << 22;
  if (mode == GEMM_WGRAD) return true;
  // The epilogue addresses rows of C (and of a stored mask) within a tile the same way.
  return g.lda < LIM && (mode == GEMM_FWD ? g.ldb : g.ldbt) < LIM && g.ldc < LIM && (!g.mask || g.ldm < LIM);
}

namespace {

// Checks one product against the large-tile kernel's launch contract; its launch form
// (the input gradient reads the transposed weight image as B) goes to *t.
hipError_t big_prepare(GemmMode mode, const GemmArgs& g, GemmArgs* t) {
  if (!big_gemm_ld_ok(mode, g)) return hipErrorInvalidValue;
  // The forward reads its bias four columns at a time.
  if (mode == GEMM_FWD && g.bias && ((uintptr_t)g.bias & 15)) return hipErrorInvalidValue;
  const int f = epilogue_flags(mode, g);
  const bool fused = f & (EPI_BITS | EPI_BITS_OUT | EPI_RDOT | EPI_CSUM | EPI_NOSTORE);
  if (fused && g.N % 128) return hipErrorInvalidValue;
  *t = g;
  if (mode == GEMM_DGRAD) {
    // The input-gradient product reads the weight as Bt [N, K] (k-contiguous).
    if (!g.Bt || g.ldbt % 8 || g.ldbt < g.K) return hipErrorInvalidValue;
    t->B = g.Bt;
    t->ldb = g.ldbt;
  }
  return hipSuccess;
}

hipError_t big_launch(GemmMode mode, const GemmPair& p, hipStream_t s) {
  const GemmArgs& g = p.g[0];
  const int f = epilogue_flags(mode, g);
  const bool fused = f & (EPI_BITS | EPI_BITS_OUT | EPI_RDOT | EPI_CSUM | EPI_NOSTORE);
  const bool bn256 = big_bn(mode, g.M, g.N, fused) == 256;
  switch (mode) {
    case GEMM_FWD: return bn256 ? launch_big<GEMM_FWD, 256>(p, s) : launch_big<GEMM_FWD, 128>(p, s);
    case GEMM_DGRAD: return bn256 ? launch_big<GEMM_DGRAD, 256>(p, s) : launch_big<GEMM_DGRAD, 128>(p, s);
    case GEMM_WGRAD: return bn256 ? launch_big<GEMM_WGRAD, 256>(p, s) : launch_big<GEMM_WGRAD, 128>(p, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t gemm_big(GemmMode mode, const GemmArgs& g, hipStream_t s) {
  GemmPair p{};
  p.n = 1;
  const hipError_t e = big_prepare(mode, g, &p.g[0]);
  return e != hipSuccess ? e : big_launch(mode, p, s);
}

int big_gemm_tiles(GemmMode mode, const GemmArgs& g) {
  const int f = epilogue_flags(mode, g);
  const bool fused = f & (EPI_BITS | EPI_BITS_OUT | EPI_RDOT | EPI_CSUM | EPI_NOSTORE);
  const int bn = big_bn(mode, g.M, g.N, fused);
  return (g.M / BM) * ((g.N + bn - 1) / bn) * (mode == GEMM_WGRAD ? g.splits : 1);
}

hipError_t gemm_big_pair(GemmMode mode, const GemmArgs& g0, const GemmArgs& g1, hipStream_t s) {
  if (g0.M != g1.M || g0.N != g1.N || g0.K != g1.K || epilogue_flags(mode, g0) != epilogue_flags(mode, g1) ||
      (mode == GEMM_WGRAD && g0.splits != g1.splits) || (!g0.m_dyn) != (!g1.m_dyn))
    return hipErrorInvalidValue;
  GemmPair p{};
  p.n = 2;
  hipError_t e = big_prepare(mode, g0, &p.g[0]);
  if (e == hipSuccess) e = big_prepare(mode, g1, &p.g[1]);
  return e != hipSuccess ? e : big_launch(mode, p, s);
}

}  // namespace spz
