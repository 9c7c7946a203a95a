// Argument blocks and launchers of the non-GEMM kernels (kernels.hip).
#pragma once

#include "internal.h"

namespace spz {

constexpr int COLSUM_CHUNK = 256;  // rows per first-pass block of the column sums

struct GatherArgs {
  const uint8_t* buf; int64_t row_bytes;
  int off_a, off_s2, off_r, off_d;   // byte offsets inside a ring row (obs at 0)
  int O, A, Ka, Kc, B;
  uint64_t seed; uint32_t size; const int64_t* step;
  void* xsa; void* xs2; void* xsp;   // [Bp, Kc] operand tensors (xsp may be null: not written)
  float* r; float* d; int32_t* idx;
  // When set, a copy of the sampled actions [B, A] (operand type): on one stream the
  // actor part later overwrites xsa's action columns with its own sample.
  void* abuf;
};

struct PackArgs {
  uint8_t* buf; int64_t row_bytes; int off_a, off_s2, off_r, off_d;
  int O, A; int64_t n, ptr, capacity;
  const float *obs, *act, *rew, *done, *nobs;   // device staging
};

struct Td3HeadArgs {
  const float* z; int ldz; int A, B;
  uint64_t seed; const int64_t* step;
  int smooth; float noise, clip;
  void* x; int64_t ldx; int xoff;
  float* th;                           // cache of tanh z (policy side) or null
};

struct RowdotArgs {
  const void* H; int64_t ld; int K, rows;
  const void* w; const float* bias; float* q;
};

struct HeadBwdArgs {
  const float* dq; const void* w; const void* H; void* dH; int64_t ld; int K, rows;
  // When set (bf16, K % 32 == 0), the ReLU mask comes from these bits instead of H:
  // bit k % 32 of bits[(k / 32) * ldbits + b].
  const uint32_t* bits; int64_t ldbits;
  // With bits: when set, the column sums of the stored dH over each block of rows go
  // to colpart[block, K] (head_bwd_blocks(rows) blocks; reduced by a deferred reduction).
  float* colpart;
  // With bits and without colpart: when map is set, row r < *m_dyn of dH is row
  // map[r] of the product (dq, bits read there), a zero row where map[r] < 0; rows
  // from *m_dyn on are not written. Row maps come from launch_minq_split.
  const int32_t* map; const int32_t* m_dyn;
  // With colpart, when set: the output layer's weight and bias gradients over each
  // block of rows, wpart[block, k] = sum of rnd(dq[b]) H[b, k] and wpart_extra[block] =
  // sum of rnd(dq[b]) (H: the stored last hidden layer, read in the same pass).
  float* wpart; float* wpart_extra;
};

// Sampler observations -> actor operand rows: x[r, c] = obs[r, c] for r < n, c < O;
// zero for c in [O, ldx_used) and for rows [n, rows).
struct ObsArgs { const float* obs; int n, rows, O, cols; void* x; int64_t ldx; };

// Actions for samplers from the actor head output z [rows, ldz]: SAC mean action
// tanh(mu) or a policy sample tanh(mu + exp(clip(l)) eps), eps from Philox purpose
// P_ACT at counter `counter`, element index (row0 + r) * A + j; TD3 tanh(z).
struct ActHeadArgs {
  const float* z; int ldz; int A, n; int64_t row0;
  int sac, stochastic; uint64_t seed; uint32_t counter; float lmin, lmax;
  float* a;
};

// A critic's output q [Bp]. With parts > 0 the output layer was folded into the last
// hidden product (row-dot partials): q[r] = *bias + sum over p < parts in order of
// part[p * ld + r], computed by the kernel that consumes q, which also stores it to q
// (for the kernels and debug reads after it). Otherwise q[r] is read as stored.
struct QSrc {
  float* q; const float* part; int parts; int64_t ld; const float* bias;
};

struct TdArgs {
  QSrc q1, q2; const float *r, *d, *logp, *log_alpha; float* y; float gamma; int B, Bp;
};

struct CriticLossArgs {
  QSrc q1, q2; const float* y; float *dq1, *dq2; double* part; int B, Bp;
};

// TD3: has_qp2 = 0 (the loss takes critic 1 only).
struct ActorLossArgs {
  QSrc qp1, qp2; int has_qp2; const float *logp, *log_alpha; float *dqp1, *dqp2; double* part; int B, Bp;
  // With qp2, when set: cnt1[k] = the rows b < B of the k-th 256-row block whose
  // minimum critic is critic 1 (qp1[b] <= qp2[b], the loss's own choice).
  int32_t* cnt1;
};

// Rows of the SAC actor loss split by the critic that attains min(qp1, qp2) (critic 1
// on ties, as in the loss): map1 lists in ascending order the rows b < B of critic 1,
// map2 those of critic 2; list i is padded with -1 up to rows[i] = min(n_i rounded up
// to 512, Bp) entries (n_i: its row count). cnt1 as written by the actor loss.
struct MinqSplitArgs {
  const float *qp1, *qp2; const int32_t* cnt1; int B, Bp;
  int32_t *map1, *map2, *rows;
};

// dst[w * ld + r] = src[w * ld + map[r]] (0 where map[r] < 0), w < words, r < *m_dyn:
// the rows of a bit-packed ReLU mask (layout of HeadBwdArgs::bits) gathered by a map.
struct RowBitsGatherArgs {
  const uint32_t* src; uint32_t* dst; int64_t ld; int words; const int32_t* map; const int32_t* m_dyn; int rows;
};

// dst[map[r] * ld + j] = src[r * ld + j] for r < *m_dyn with map[r] >= 0, j < cols.
struct RowScatterArgs {
  const float* src; float* dst; int64_t ld; int cols; const int32_t* map; const int32_t* m_dyn; int rows;
};

struct ActorHeadBwdArgs {
  const float *da1, *da2; int ldda; const float *th, *se, *lm, *log_alpha;
  void* dz; int ldz; int A, B; int sac;
};

struct ColsumArgs {
  const void* X; int64_t ld; int N, rows, chunk; const float* weights; int extra; float* part;
  float* part_extra;   // [chunks] when extra
};

struct AdamArgs {
  float *P, *M, *V, *T; const float* G; bf16_t *Pb, *Tb;
  int64_t n, a0, a1, c0, c1, la;
  int do_actor, do_critic, do_alpha, polyak_critic, polyak_actor, td3, delay;
  float lr_a, lr_c, lr_al, b1, b2, eps, tau;
  const int64_t* step;
  int step_add;   // the step being completed is *step + step_add (1 before k_finish ran)
};

struct FinishArgs {
  const double *cpart, *apart; int nc, na, B;
  int sac, actor_step, learn_alpha; float target_entropy;
  const float* log_alpha; float* grad_alpha;
  float* rec; int64_t rec_cap; int64_t* step;
};

hipError_t launch_gather(bool bf16, const GatherArgs& g, hipStream_t s);
hipError_t launch_pack(bool bf16, const PackArgs& p, hipStream_t s);
hipError_t launch_sac_head(bool bf16, const SacHeadArgs& h, hipStream_t s);
hipError_t launch_td3_head(bool bf16, const Td3HeadArgs& h, hipStream_t s);
hipError_t launch_rowdot(bool bf16, const RowdotArgs& r, hipStream_t s);
hipError_t launch_head_bwd(bool bf16, const HeadBwdArgs& a, hipStream_t s);
hipError_t launch_obs_operand(bool bf16, const ObsArgs& a, hipStream_t s);
hipError_t launch_act_head(const ActHeadArgs& a, hipStream_t s);
hipError_t launch_td_target(const TdArgs& a, hipStream_t s);
int loss_blocks(int Bp);
hipError_t launch_critic_loss(const CriticLossArgs& a, hipStream_t s);
hipError_t launch_actor_loss(const ActorLossArgs& a, hipStream_t s);
hipError_t launch_minq_split(const MinqSplitArgs& a, hipStream_t s);
hipError_t launch_row_bits_gather(const RowBitsGatherArgs& a, hipStream_t s);
hipError_t launch_row_scatter(const RowScatterArgs& a, hipStream_t s);
hipError_t launch_actor_head_bwd(bool bf16, const ActorHeadBwdArgs& h, hipStream_t s);
int colsum_chunks(int rows);
int head_bwd_blocks(int rows);
// Column-sum partials a.part[chunks, N] (and a.part_extra[chunks]) for a deferred
// reduction (ReduceJob with colsum_groups()).
hipError_t launch_colsum_partial(bool bf16, const ColsumArgs& a, hipStream_t s);
int colsum_groups();

// Deferred reduction: out[r * ldo + c] = sum over slices z < slices of
// part[z * zstride + r * ld + c], for r < rows, c < cols. A piece of vec (4 or 1)
// output columns is summed by `groups` threads (a power of two): thread g takes
// z = g, g + groups, ... in order, then the group sums are added in g order -- a
// fixed order for a fixed job. block0: first block of the job (set by the launch).
struct ReduceJob {
  const float* part; float* out; int64_t zstride, ld, ldo;
  int rows, cols, slices, groups, vec, block0;
};
constexpr int MAX_REDUCE_JOBS = 24;
struct ReduceJobs { ReduceJob j[MAX_REDUCE_JOBS]; int n; };
// All jobs in one launch (n <= MAX_REDUCE_JOBS).
hipError_t launch_reduce_jobs(ReduceJobs& jobs, hipStream_t s);
hipError_t launch_adam(const AdamArgs& a, hipStream_t s);
hipError_t launch_finish(const FinishArgs& f, hipStream_t s);
hipError_t launch_to_bf16(const float* src, bf16_t* dst, int64_t n, hipStream_t s);

// Transposed weight images (operand type: bfloat16 or float32): job j writes
// dst[dst_off + c * ldd + r] = src[src_off + r * lds + c]
// for r < rows, c < cols (the [cols, rows] transpose of a [rows, cols] matrix); the
// jobs' 64 x 64 tiles are numbered consecutively from tile0 (ascending with j).
struct TransposeJob { int64_t src_off, dst_off, lds, ldd; int rows, cols, tile0; };
inline int transpose_tiles(int rows, int cols) { return ((rows + 63) / 64) * ((cols + 63) / 64); }
hipError_t launch_transpose(bool bf16, const void* src, void* dst, const TransposeJob* jobs, int njobs, int tiles,
                            hipStream_t s);

}  // namespace spz
