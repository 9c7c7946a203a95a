// C ABI and step orchestration of the actor-critic update.
//
// Memory layout in HBM (per context):
//   parameter arenas P (online), T (targets), G (gradients), M, V (Adam), all
//     float32 with one common layout: actor | critic1 | critic2 | log(alpha);
//     each layer stores W [out_p, in_p] then b [out_p], 256-byte aligned, with
//     feature dimensions padded to multiples of 32 and zero padding. For bf16
//     contexts Pb / Tb hold the bfloat16 images of P / T used as GEMM operands.
//   replay ring: capacity rows of [obs | act | next_obs | pad | rew | done],
//     obs/act/next_obs in the operand type, rew/done float32, 16-byte rows.
//   batch operands [Bp, Kc] (Bp = batch rounded up to 256): critic input
//     [obs | 0 | act | 0] with the action block at column Ka = pad32(obs_dim);
//     the actor reads the first Ka columns of the same tensors.
//   per-stream workspaces for activations, gradients and reduction partials.
//
// One update step (snapshot semantics: every read of step t sees the parameters
// of the start of step t; all parameter writes happen in the final Adam/Polyak
// pass after the two streams join):
//   s0: gather                          -> fork
//   critic stream: target action, target critics, TD target, online critics,
//                  critic loss, critic backward (weight and bias gradients)
//   actor stream:  actor forward on s, critics on (s, a~), actor loss, critic
//                  input-gradient to the action (SAC: each critic on the rows where
//                  it attains min(Q1, Q2)), head backward, actor backward
//   s0: join -> finish (loss record, temperature gradient, step counter) -> Adam + Polyak
// Sequential ordering (the published algorithms' order) runs everything on s0 and
// moves the critics' Adam + Polyak between the critic part and the actor part.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>

#include "kernels.h"

using namespace spz;

// Device scratch of the allocation-free sampler-action call (spz_act_noalloc): the
// observation operand, two hidden-activation buffers and the actor head output of
// one call. One copy per GPU, held until the process ends; every call on a GPU uses
// that GPU's copy. Host code never passes the array's name to a kernel: it uses the
// device address taken by hipGetSymbolAddress (g_scratch_ptr below).
constexpr size_t ACT_SCRATCH_BYTES = (size_t)64 << 20;
static __device__ __align__(256) uint8_t scratch[ACT_SCRATCH_BYTES];

namespace {

thread_local std::string tl_err;

// Device address of `scratch` per device ordinal, taken once per device (with the
// device current) by the first spz_create on it.
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

hipError_t scratch_init(int device) {
  if (device < 0 || device >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[device]) return hipSuccess;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!p) return hipErrorInvalidSymbol;
  g_scratch_ptr[device] = p;
  return hipSuccess;
}

struct Lay {
  int in_f, out_f, in_p, out_p;
  int64_t w, b;  // float offsets into an arena
};

struct Net {
  std::vector<Lay> L;
  int64_t off = 0, end = 0;
};

inline int pad32(int x) { return (x + 31) / 32 * 32; }
inline int64_t align64(int64_t x) { return (x + 63) / 64 * 64; }
inline int64_t align16(int64_t x) { return (x + 15) / 16 * 16; }

}  // namespace

struct spz_ctx {
  // configuration
  int O = 0, A = 0, B = 0, Bp = 0, Ka = 0, Ap = 0, Kc = 0;
  int Bmax = 0, Bpmax = 0;   // batch given to spz_create: sizes every batch buffer
  std::vector<int> hidden;
  spz_hparams hp{};
  uint64_t seed = 0;
  bool bf16 = false, td3 = false;
  Net net[3];
  int64_t la = 0, n_arena = 0;
  int hmax = 0;
  // parameters
  float *P = nullptr, *G = nullptr, *M = nullptr, *V = nullptr, *T = nullptr;
  bf16_t *Pb = nullptr, *Tb = nullptr;
  // bf16 contexts: transposed images of the online weights the input-gradient products
  // read (layer l >= 1 of each net, the critics' output layers aside), at the same
  // arena offsets as Pb: WT + L.w holds W^T [in_p, out_p], so that those products read
  // both operands k-contiguous (the large-tile kernel needs it). For a critic's first
  // layer WT + L.w holds the transposed action block [Ap, out_p] (columns Ka .. Ka + Ap
  // of W), the weight of the gradient to the action. Refreshed whenever P changes.
  // float32 contexts read W itself: there the per-step transpose costs about what the
  // k-contiguous reads save.
  void* WT = nullptr;
  TransposeJob* tjobs = nullptr;
  int n_tjobs = 0, t_tiles = 0;
  double t_elems = 0.0;
  // replay ring
  uint8_t* buf = nullptr;
  int64_t row_bytes = 0, cap = 0, ptr = 0, size = 0;
  int off_a = 0, off_s2 = 0, off_r = 0, off_d = 0;
  float* stage = nullptr;
  // asynchronous ingestion: pinned host slots copied to device slots on their own
  // stream, committed into the ring on the update stream
  struct IngestSlot { float* host = nullptr; float* dev = nullptr; hipEvent_t copied = nullptr, done = nullptr; bool used = false; };
  std::vector<IngestSlot> slots;
  int next_slot = 0;
  hipStream_t si = nullptr;
  hipStream_t commit_stream = nullptr;   // stream the latest ring commits were enqueued on
  bool commits_pending = false;          // ... and the next update must be ordered after them
  hipEvent_t ev_commit = nullptr;
  int64_t stage_rows = 0;
  // step state
  int64_t* d_step = nullptr;
  int64_t h_step = 0;
  float* rec = nullptr;
  int64_t rec_cap = 65536;
  // batch
  void *xsa = nullptr, *xs2 = nullptr, *xsp = nullptr;
  // Critic input of the actor part in the step being enqueued: xsp when the two parts
  // run on concurrent streams; xsa itself (action columns overwritten by the actor's
  // sample) when they run in order on one stream and the critic part is done with it.
  void* xs_act = nullptr;
  void* abuf = nullptr;   // sampled actions [Bp, A] of a one-stream step (debug read of the batch)
  float *r = nullptr, *d = nullptr;
  int32_t* idx = nullptr;
  // critic-stream workspace
  void* cs_h[2] = {nullptr, nullptr};
  void* cs_h2[2] = {nullptr, nullptr};   // target critic 2 (the twins run layer by layer)
  float *z2 = nullptr, *logp2 = nullptr, *qt1 = nullptr, *qt2 = nullptr, *y = nullptr;
  float *q1 = nullptr, *q2 = nullptr, *dq1 = nullptr, *dq2 = nullptr;
  std::vector<void*> hc[2];
  std::vector<uint32_t*> bhc[2];     // ReLU masks of hc as bits (null where not fused)
  float* c_rdot[2] = {nullptr, nullptr};   // row-dot partials of the critic stream (two heads in flight)
  void* c_dz[2] = {nullptr, nullptr};
  void* c_dz2[2] = {nullptr, nullptr};   // critic 2
  double* c_lpart = nullptr;
  // actor-stream workspace
  std::vector<void*> ha;
  float *z = nullptr, *th = nullptr, *se = nullptr, *lm = nullptr, *logp = nullptr;
  float *qp1 = nullptr, *qp2 = nullptr, *dqp1 = nullptr, *dqp2 = nullptr, *da1 = nullptr, *da2 = nullptr;
  std::vector<void*> hpc[2];
  std::vector<uint32_t*> bha, bhpc[2];
  float* a_rdot[2] = {nullptr, nullptr};
  // SAC row split of the actor's gradient through the critics: two row maps [Bp]
  // and their padded lengths (device side), the actor loss's per-block critic-1
  // counts, and one layer's mask bits gathered by a map.
  bool row_split = false;
  int32_t *rmap = nullptr, *rrows = nullptr, *rcnt = nullptr;
  uint32_t *rbits = nullptr, *rbits2 = nullptr;
  void* a_dz[2] = {nullptr, nullptr};
  void* a_dz2[2] = {nullptr, nullptr};   // critic 2's action-gradient chain
  void* dzh = nullptr;
  double* a_lpart = nullptr;
  // Deferred gradient reductions of the critic part (0) and the actor part (1): the
  // split-K and column-sum partials of every layer go to consecutive slots of the
  // part's workspace and one launch at the end of the part reduces them all.
  struct RedQueue { float* base = nullptr; int64_t cap = 0, off = 0; double bytes = 0.0; ReduceJobs jobs{}; };
  RedQueue red[2];
  // streams
  hipStream_t sc = nullptr, sa = nullptr;
  hipEvent_t ev_fork = nullptr, ev_c = nullptr, ev_a = nullptr;
  // Captured update steps (hp.graphs): one executable graph per step kind (index:
  // 1 when the step updates the actor), valid for the batch, fill level and seed it
  // was captured with (they are kernel arguments); captured on stream sg.
  struct GraphSlot { hipGraphExec_t exec = nullptr; int B = 0, Bp = 0; int64_t size = 0; uint64_t seed = 0; };
  GraphSlot gslot[2];
  hipStream_t sg = nullptr;
  hipStream_t last = nullptr;
  bool has_last = false;   // an update was enqueued on `last` (which may be the null stream)
  std::vector<void*> cs_hid, cs_hid2;   // ping-pong views of cs_h, cs_h2, one entry per hidden layer
  std::vector<void*> allocs;
  // kernel timing
  struct ProfKey { std::string name; int M, N, K; double flops, bytes; int64_t launches; double ms; };
  struct ProfEv { int key; hipEvent_t a, b; };
  bool prof = false;
  std::vector<ProfKey> pkeys;
  bool pf_on = false;           // time only launches of this family and shape
  int pf_stride = 1;            // ... in update steps t with t % pf_stride == 0
  bool pf_step = true;          // the step being enqueued is one of them
  std::string pf_name;
  int pf_M = 0, pf_N = 0, pf_K = 0;
  std::vector<ProfEv> pevs;
  std::vector<hipEvent_t> pool;
  std::string err;
};

namespace {

int set_err(spz_ctx* c, int code, const std::string& msg) {
  tl_err = msg;
  if (c) c->err = msg;
  return code;
}

int fail_hip(spz_ctx* c, hipError_t e, const char* what) {
  return set_err(c, SPZ_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define CK(x)                                          \
  do {                                                 \
    hipError_t e_ = (x);                               \
    if (e_ != hipSuccess) return fail_hip(c, e_, #x);  \
  } while (0)

#define HK(x)                               \
  do {                                      \
    hipError_t e_ = (x);                    \
    if (e_ != hipSuccess) return e_;        \
  } while (0)

hipError_t dalloc(spz_ctx* c, void** p, size_t bytes) {
  *p = nullptr;
  if (bytes == 0) bytes = 256;
  HK(hipMalloc(p, bytes));
  c->allocs.push_back(*p);
  return hipMemset(*p, 0, bytes);
}

template <typename P>
hipError_t dalloc_t(spz_ctx* c, P** p, size_t bytes) {
  void* v = nullptr;
  hipError_t e = dalloc(c, &v, bytes);
  *p = static_cast<P*>(v);
  return e;
}

// ---------------------------------------------------------------------------------- timing
int prof_key(spz_ctx* c, const char* name, int M, int N, int K, double flops, double bytes) {
  for (size_t i = 0; i < c->pkeys.size(); ++i) {
    const auto& k = c->pkeys[i];
    if (k.M == M && k.N == N && k.K == K && k.name == name) return (int)i;
  }
  c->pkeys.push_back({name, M, N, K, flops, bytes, 0, 0.0});
  return (int)c->pkeys.size() - 1;
}

hipError_t prof_take(spz_ctx* c, hipEvent_t* e) {
  if (c->pool.empty()) return hipEventCreate(e);
  *e = c->pool.back();
  c->pool.pop_back();
  return hipSuccess;
}

// Run one launch; while timing is enabled, bracket it with events on its stream.
template <class F>
hipError_t timed(spz_ctx* c, const char* name, int M, int N, int K, double flops, double bytes, hipStream_t s,
                 F&& f) {
  if (!c->prof || !c->pf_step ||
      (c->pf_on && (M != c->pf_M || N != c->pf_N || K != c->pf_K || c->pf_name != name)))
    return f();
  hipEvent_t a, b;
  HK(prof_take(c, &a));
  HK(prof_take(c, &b));
  HK(hipEventRecord(a, s));
  HK(f());
  HK(hipEventRecord(b, s));
  c->pevs.push_back({prof_key(c, name, M, N, K, flops, bytes), a, b});
  return hipSuccess;
}

// Flat (unpadded) column i of layer l of net ni -> padded column.
inline int pcol(const spz_ctx* c, int ni, int l, int i) {
  return (ni != 0 && l == 0 && i >= c->O) ? c->Ka + (i - c->O) : i;
}

int64_t flat_count(const Net& n) {
  int64_t s = 0;
  for (const Lay& L : n.L) s += (int64_t)L.in_f * L.out_f + L.out_f;
  return s;
}

// ---------------------------------------------------------------------------------- layout
void plan_layout(spz_ctx* c) {
  const int O = c->O, A = c->A;
  c->Ka = pad32(O);
  c->Ap = pad32(A);
  c->Kc = c->Ka + c->Ap;
  int64_t off = 0;
  for (int ni = 0; ni < 3; ++ni) {
    Net& n = c->net[ni];
    n.L.clear();
    n.off = off;
    std::vector<int> dims;
    dims.push_back(ni == 0 ? O : O + A);
    for (int h : c->hidden) dims.push_back(h);
    dims.push_back(ni == 0 ? (c->td3 ? A : 2 * A) : 1);
    const int nl = (int)dims.size() - 1;
    for (int l = 0; l < nl; ++l) {
      Lay L;
      L.in_f = dims[l];
      L.out_f = dims[l + 1];
      L.in_p = l == 0 ? (ni == 0 ? c->Ka : c->Kc) : pad32(dims[l]);
      L.out_p = (ni != 0 && l == nl - 1) ? 1 : pad32(dims[l + 1]);
      L.w = off;
      off = align64(off + (int64_t)L.out_p * L.in_p);
      L.b = off;
      off = align64(off + L.out_p);
      n.L.push_back(L);
    }
    n.end = off;
  }
  c->la = off;
  off = align64(off + 1);
  c->n_arena = off;
  c->hmax = 32;
  for (int h : c->hidden) c->hmax = std::max(c->hmax, pad32(h));
}

// ---------------------------------------------------------------------------------- init
// Fan-in uniform init from Philox (computed on the host, bit-exact):
// k = fl32(1/sqrt(fan_in)), u = (w >> 8) 2^-24, value = fl32((2u - 1) k).
void host_init(spz_ctx* c, std::vector<float>& img) {
  img.assign(c->n_arena, 0.0f);
  for (int ni = 0; ni < 3; ++ni) {
    for (int l = 0; l < (int)c->net[ni].L.size(); ++l) {
      const Lay& L = c->net[ni].L[l];
      const double k = (double)(float)(1.0 / std::sqrt((double)L.in_f));
      const uint32_t tw = (uint32_t)(ni * 16 + l * 2), tb = tw + 1;
      for (int o = 0; o < L.out_f; ++o)
        for (int i = 0; i < L.in_f; ++i) {
          const uint64_t e = (uint64_t)o * L.in_f + i;
          const double u = (double)(philox_word(c->seed, e, 0, P_INIT, tw) >> 8) * 0x1p-24;
          img[L.w + (int64_t)o * L.in_p + pcol(c, ni, l, i)] = (float)((2.0 * u - 1.0) * k);
        }
      for (int o = 0; o < L.out_f; ++o) {
        const double u = (double)(philox_word(c->seed, (uint64_t)o, 0, P_INIT, tb) >> 8) * 0x1p-24;
        img[L.b + o] = (float)((2.0 * u - 1.0) * k);
      }
    }
  }
  img[c->la] = c->td3 ? 0.0f : (float)std::log((double)c->hp.alpha_init);
}

// ---------------------------------------------------------------------------------- pieces
const void* wop(const spz_ctx* c, bool target, int64_t off) {
  if (c->bf16) return (target ? c->Tb : c->Pb) + off;
  return (target ? c->T : c->P) + off;
}
const float* wf(const spz_ctx* c, bool target, int64_t off) { return (target ? c->T : c->P) + off; }
size_t es(const spz_ctx* c) { return c->bf16 ? 2 : 4; }
double head_bwd_bytes(const spz_ctx* c, int K, const uint32_t* bits) {
  return (double)c->Bp * K * es(c) + (bits ? c->Bp * K / 8.0 : (double)c->Bp * K * es(c));
}
const void* elem(const spz_ctx* c, const void* base, int64_t off) {
  return static_cast<const uint8_t*>(base) + off * (int64_t)es(c);
}

// Transposed weight images (bf16 contexts) from Pb.
hipError_t refresh_wt(spz_ctx* c, hipStream_t s) {
  if (!c->WT || !c->n_tjobs) return hipSuccess;
  return timed(c, "transpose", c->n_tjobs, 0, 0, 0.0, 4.0 * c->t_elems, s,
               [&] { return launch_transpose(true, c->Pb, c->WT, c->tjobs, c->n_tjobs, c->t_tiles, s); });
}
// Transposed image of the online layer L (the B operand of its input-gradient
// product), or null (float32 contexts).
const void* wt(const spz_ctx* c, const Lay& L) { return c->WT ? elem(c, c->WT, L.w) : nullptr; }

// Deferred reductions: partial buffers come from the part's workspace in enqueue
// order (the same addresses every step, as graph replay needs); a full job list is
// reduced early (same stream, so the slots may then be reused).
float* red_alloc(spz_ctx* c, int q, int64_t n) {
  spz_ctx::RedQueue& r = c->red[q];
  const int64_t need = (n + 63) / 64 * 64;
  if (r.off + need > r.cap) return nullptr;
  float* p = r.base + r.off;
  r.off += need;
  return p;
}

hipError_t red_flush(spz_ctx* c, int q, hipStream_t s) {
  spz_ctx::RedQueue& r = c->red[q];
  if (r.jobs.n) {
    HK(timed(c, "grad_reduce", r.jobs.n, 0, 0, 0.0, r.bytes, s, [&] { return launch_reduce_jobs(r.jobs, s); }));
  }
  r.jobs.n = 0;
  r.off = 0;
  r.bytes = 0.0;
  return hipSuccess;
}

hipError_t red_job(spz_ctx* c, int q, const ReduceJob& j) {
  spz_ctx::RedQueue& r = c->red[q];
  if (r.jobs.n == MAX_REDUCE_JOBS) return hipErrorInvalidValue;   // callers flush before allocating
  r.jobs.j[r.jobs.n++] = j;
  r.bytes += 4.0 * j.rows * j.cols * (j.slices + 1.0);
  return hipSuccess;
}

// Room for `jobs` more jobs (flushing what is queued otherwise).
hipError_t red_room(spz_ctx* c, int q, int jobs, hipStream_t s) {
  return c->red[q].jobs.n + jobs > MAX_REDUCE_JOBS ? red_flush(c, q, s) : hipSuccess;
}

// Reduction of column-sum partials part[slices, N] into out[N] (and of the extra
// scalars part_extra[slices] into *out_extra), in the fixed group order of colsum_groups().
hipError_t red_colsum(spz_ctx* c, int q, const float* part, int slices, int N, float* out, const float* part_extra,
                      float* out_extra, hipStream_t s) {
  HK(red_job(c, q, ReduceJob{part, out, N, 0, 0, 1, N, slices, colsum_groups(), 4, 0}));
  if (!part_extra) return hipSuccess;
  return red_job(c, q, ReduceJob{part_extra, out_extra, 1, 0, 0, 1, 1, slices, colsum_groups(), 1, 0});
}

int colsum_rows(int Bp) {
  return std::max({colsum_chunks(Bp), Bp / 256, head_bwd_blocks(Bp)});
}

// Workspace floats a part's deferred reductions may need at padded batch Bp.
int64_t red_need(const spz_ctx* c, int q, int Bp) {
  const int chunks = colsum_rows(Bp);
  int64_t n = 0;
  for (int ni = (q == 0 ? 1 : 0); ni <= (q == 0 ? 2 : 0); ++ni)
    for (const Lay& L : c->net[ni].L) {
      n += (int64_t)wgrad_splits(c->bf16, L.out_p, L.in_p, Bp) * L.out_p * L.in_p + 64;
      n += 2 * ((int64_t)chunks * (std::max(L.out_p, L.in_p) + 1) + 64);
    }
  return n;
}

// A matrix product, or the same product of both twin critics (g1): one launch where
// gemm_pairs holds (recorded as one product of the stacked rows), else two.
hipError_t gemm2(spz_ctx* c, const char* name, GemmMode mode, const GemmArgs& g0, const GemmArgs* g1, bool flops,
                 hipStream_t s) {
  auto fl = [&](const GemmArgs& g) { return flops ? 2.0 * g.M * g.N * g.K : 0.0; };
  if (g1 && gemm_pairs(c->bf16, mode, g0, *g1))
    return timed(c, name, 2 * g0.M, g0.N, g0.K, fl(g0) + fl(*g1), 0.0, s,
                 [&] { return gemm_pair(c->bf16, mode, g0, *g1, s); });
  HK(timed(c, name, g0.M, g0.N, g0.K, fl(g0), 0.0, s, [&] { return gemm(c->bf16, mode, g0, s); }));
  if (!g1) return hipSuccess;
  return timed(c, name, g1->M, g1->N, g1->K, fl(*g1), 0.0, s, [&] { return gemm(c->bf16, mode, *g1, s); });
}

// Per-net outputs of a forward: hidden layers (and their ReLU masks as bits where
// set), the row-dot partials of a folded critic output layer, the head output (actor:
// z [Bp, out_p]; critic: q [Bp]) and, for a critic, where q comes from.
struct NetOut {
  void* const* hid;
  uint32_t* const* bits;
  float* rdot;
  float* head;
  QSrc* qs;
  const SacHeadArgs* sac = nullptr;   // actor: the SAC head fused into the output product (head unused)
};

// Whether the actor's output product takes the SAC head in its epilogue.
bool sac_head_fused(const spz_ctx* c) {
  const Lay& H = c->net[0].L.back();
  return !c->td3 && gemm_sac_head_ok(c->Bp, H.out_p, H.in_p, c->A);
}

bool fused_layer(const spz_ctx* c, const Lay& L) { return gemm_fused_ok(c->bf16, GEMM_FWD, c->Bp, L.out_p, L.in_p); }

// Forward of nets ni .. ni + nn - 1 on the same operand tensor X [Bp, ldx] (the first
// in_p(0) columns are read), net k's outputs in o[k]; nn = 2 runs both critics layer
// by layer, so that a layer's two products can share a launch. Where the large-tile
// kernel covers the last hidden layer of a critic, the output layer is folded into
// that product's epilogue (row-dot partials in o[k].rdot, which the kernel consuming q
// sums in order and stores to o[k].head); otherwise a row-dot kernel writes q to
// o[k].head. The last hidden layer is then stored only when keep_last.
hipError_t forward(spz_ctx* c, int ni, int nn, bool target, const void* X, int64_t ldx, const NetOut* o,
                   bool keep_last, hipStream_t s) {
  if (nn < 1 || nn > 2 || (ni == 0 && nn != 1) || ni + nn > 3) return hipErrorInvalidValue;
  for (int k = 0; k < nn; ++k)
    if ((ni != 0 && !o[k].qs) || (o[k].sac && ni != 0)) return hipErrorInvalidValue;
  const int nl = (int)c->net[ni].L.size();
  const void* in[2] = {X, X};
  int64_t ld = ldx;
  for (int l = 0; l < nl; ++l) {
    const Lay& L = c->net[ni].L[l];   // the twin critics have the same shapes
    if (l == nl - 1 && ni != 0) {
      for (int k = 0; k < nn; ++k) {
        const Lay& Lk = c->net[ni + k].L[l];
        *o[k].qs = QSrc{o[k].head, nullptr, 0, 0, nullptr};
        RowdotArgs r{in[k], ld, L.in_p, c->Bp, wop(c, target, Lk.w), wf(c, target, Lk.b), o[k].head};
        HK(timed(c, "rowdot", c->Bp, 1, L.in_p, 2.0 * c->Bp * L.in_p, (double)c->Bp * L.in_p * es(c) + 4.0 * c->Bp, s,
                 [&] { return launch_rowdot(c->bf16, r, s); }));
      }
      return hipSuccess;
    }
    const bool folded = ni != 0 && l == nl - 2 && fused_layer(c, L);
    GemmArgs g[2]{};
    for (int k = 0; k < nn; ++k) {
      const Lay& Lk = c->net[ni + k].L[l];
      GemmArgs& gk = g[k];
      gk.A = in[k]; gk.lda = ld;
      gk.B = wop(c, target, Lk.w); gk.ldb = L.in_p;
      gk.bias = wf(c, target, Lk.b);
      gk.M = c->Bp; gk.N = L.out_p; gk.K = L.in_p;
      if (l == nl - 1) {
        gk.C = o[k].head; gk.ldc = L.out_p; gk.relu = 0; gk.out_f32 = 1;
        continue;
      }
      gk.C = o[k].hid[l]; gk.ldc = L.out_p; gk.relu = 1; gk.out_f32 = 0;
      if (o[k].bits && o[k].bits[l]) {
        gk.bits_out = o[k].bits[l];
        gk.ldbits = c->Bp;
      }
      if (folded) {
        gk.rdot_w = wop(c, target, c->net[ni + k].L[nl - 1].w);
        gk.rdot_part = o[k].rdot;
        gk.ldrd = c->Bp;
        gk.no_store = keep_last ? 0 : 1;
      }
    }
    if (l == nl - 1 && o[0].sac) {   // the actor's output layer with the SAC head
      HK(timed(c, "gemm_fwd", g[0].M, g[0].N, g[0].K, 2.0 * g[0].M * g[0].N * g[0].K, 0.0, s,
               [&] { return gemm_fwd_sac_head(c->bf16, g[0], *o[0].sac, s); }));
      return hipSuccess;
    }
    HK(gemm2(c, "gemm_fwd", GEMM_FWD, g[0], nn > 1 ? &g[1] : nullptr, true, s));
    if (folded) {
      for (int k = 0; k < nn; ++k)
        *o[k].qs = QSrc{o[k].head, o[k].rdot, L.out_p / gemm_rdot_cols(c->Bp, L.out_p), c->Bp,
                        wf(c, target, c->net[ni + k].L[nl - 1].b)};
      return hipSuccess;
    }
    for (int k = 0; k < nn; ++k) in[k] = g[k].C;
    ld = L.out_p;
  }
  return hipSuccess;
}

// One weight-gradient product: layer l of net ni from dz [Bp, out_p] and the layer
// input X [Bp, ldx].
struct WgradIn {
  int ni, l;
  const void* dz;
  const void* X;
  int64_t ldx;
};

// Weight gradients of nn (1 or 2) layers, split-K over the batch (slices reduced in order
// by the part's deferred reduction q) and, when `bias`, the bias gradients as the column
// sums of dz. Two products of one shape (a layer of both twin critics, or two equal layers
// of one net) split K half as finely and share one launch where the large-tile kernel
// takes them: half the slices to write and reduce (which also pays where the pair leaves
// compute units idle: there the reduction outweighs the product).
hipError_t wgrad(spz_ctx* c, int q, int nn, const WgradIn* w, bool bias, hipStream_t s) {
  HK(red_room(c, q, 2 * nn, s));
  GemmArgs g[2]{};
  float* part[2] = {nullptr, nullptr};
  for (int k = 0; k < nn; ++k) {
    const Lay& L = c->net[w[k].ni].L[w[k].l];
    GemmArgs& gk = g[k];
    gk.A = w[k].dz; gk.lda = L.out_p;
    gk.B = w[k].X; gk.ldb = w[k].ldx;
    gk.M = L.out_p; gk.N = L.in_p; gk.K = c->Bp;
    gk.splits = wgrad_splits(c->bf16, gk.M, gk.N, gk.K);
    gk.ldc = L.in_p;
  }
  if (nn == 2 && g[0].splits > 1) {
    GemmArgs h0 = g[0], h1 = g[1];
    h0.splits /= 2;
    h1.splits /= 2;
    if (gemm_pairs(c->bf16, GEMM_WGRAD, h0, h1)) {
      g[0].splits = h0.splits;
      g[1].splits = h1.splits;
    }
  }
  for (int k = 0; k < nn; ++k) {
    if (!(part[k] = red_alloc(c, q, (int64_t)g[k].splits * g[k].M * g[k].N))) return hipErrorOutOfMemory;
    g[k].C = part[k];
  }
  HK(gemm2(c, "gemm_wgrad", GEMM_WGRAD, g[0], nn > 1 ? &g[1] : nullptr, true, s));
  for (int k = 0; k < nn; ++k)
    HK(red_job(c, q, ReduceJob{part[k], c->G + c->net[w[k].ni].L[w[k].l].w, (int64_t)g[k].M * g[k].ldc, g[k].ldc,
                               g[k].N, g[k].M, g[k].N, g[k].splits, splitk_groups(g[k].M, g[k].N, g[k].splits), 4,
                               0}));
  if (!bias) return hipSuccess;
  const int chunks = colsum_chunks(c->Bp);
  for (int k = 0; k < nn; ++k) {
    const int N = g[k].M;   // the layer's outputs
    float* cpart = red_alloc(c, q, (int64_t)chunks * N);
    if (!cpart) return hipErrorOutOfMemory;
    ColsumArgs cs{w[k].dz, N, N, c->Bp, COLSUM_CHUNK, nullptr, 0, cpart, nullptr};
    HK(timed(c, "colsum", c->Bp, N, 0, 0.0, (double)c->Bp * N * es(c), s,
             [&] { return launch_colsum_partial(c->bf16, cs, s); }));
    HK(red_colsum(c, q, cpart, chunks, N, c->G + c->net[w[k].ni].L[w[k].l].b, nullptr, nullptr, s));
  }
  return hipSuccess;
}

// One net's operands of an input-gradient product through a layer: dz [Bp, out_p], the
// ReLU mask of the layer below (stored tensor, or bits), the output, where the column
// sums of the output go (the bias gradient of the layer below; or null) and a
// device-side count of leading rows (or null: every row).
struct DgradIn {
  const void* dz;
  const void* mask;
  const uint32_t* bits;
  void* out;
  float* bias_out;
  const int32_t* m_dyn;
};

// Input gradients through layer l of nets ni .. ni + nn - 1: out = (dz . W) masked by
// mask > 0 (or by the mask bits), N columns of W from column col0 on (row stride ldw),
// or, with `transposed`, the transposed image of those columns (WT + L.w), which both
// GEMM kernels then read instead (bf16 contexts; float32 contexts have none and read W).
// Column sums of the stored out go to bias_out: fused into the product's epilogue where
// the large-tile kernel covers it, the partials reduced by the part's deferred reduction q.
hipError_t dgrad(spz_ctx* c, int ni, int nn, int l, const DgradIn* d, int col0, int64_t ldw, bool transposed, int N,
                 int64_t ldo, bool out_f32, int q, hipStream_t s) {
  const Lay& L = c->net[ni].L[l];
  const bool sums = d[0].bias_out != nullptr;
  for (int k = 1; k < nn; ++k)
    if ((d[k].bias_out != nullptr) != sums || (d[k].m_dyn != nullptr) != (d[0].m_dyn != nullptr))
      return hipErrorInvalidValue;
  if (sums) HK(red_room(c, q, nn, s));
  const bool fused = sums && gemm_colsum_fused(c->bf16, GEMM_DGRAD, c->Bp, N, L.out_p);
  const int chunks = fused ? c->Bp / 256 : colsum_chunks(c->Bp);
  GemmArgs g[2]{};
  float* cpart[2] = {nullptr, nullptr};
  for (int k = 0; k < nn; ++k) {
    const Lay& Lk = c->net[ni + k].L[l];
    GemmArgs& gk = g[k];
    gk.m_dyn = d[k].m_dyn;
    gk.A = d[k].dz; gk.lda = L.out_p;
    gk.B = elem(c, wop(c, false, Lk.w), col0); gk.ldb = ldw;
    gk.Bt = transposed ? wt(c, Lk) : nullptr; gk.ldbt = L.out_p;
    gk.C = d[k].out; gk.ldc = ldo; gk.out_f32 = out_f32 ? 1 : 0;
    if (d[k].bits) {
      gk.bits = d[k].bits;
      gk.ldbits = c->Bp;
    } else if (d[k].mask) {
      gk.mask = d[k].mask;
      gk.ldm = ldo;
    }
    gk.M = c->Bp; gk.N = N; gk.K = L.out_p;
    if (sums && !(cpart[k] = red_alloc(c, q, (int64_t)chunks * N))) return hipErrorOutOfMemory;
    if (fused) {
      gk.colsum = cpart[k];
      gk.ldcs = N;
    }
  }
  // Row-restricted products do a data-dependent amount of work: their records carry
  // the launch shape and no flop count.
  const bool rows = d[0].m_dyn != nullptr;
  HK(gemm2(c, rows ? "gemm_dgrad_rows" : "gemm_dgrad", GEMM_DGRAD, g[0], nn > 1 ? &g[1] : nullptr, !rows, s));
  if (!sums) return hipSuccess;
  for (int k = 0; k < nn; ++k) {
    if (!fused) {
      ColsumArgs cs{d[k].out, ldo, N, c->Bp, COLSUM_CHUNK, nullptr, 0, cpart[k], nullptr};
      HK(timed(c, "colsum", c->Bp, N, 0, 0.0, (double)c->Bp * N * es(c), s,
               [&] { return launch_colsum_partial(c->bf16, cs, s); }));
    }
    HK(red_colsum(c, q, cpart[k], chunks, N, d[k].bias_out, nullptr, nullptr, s));
  }
  return hipSuccess;
}

// Both critics: weight and bias gradients of L = sum_b dq_k[b] q_k[b] given the stored
// hidden activations hid[k] (ReLU masks bits[k]) of the forward on X, layer by layer so
// that the twins' products can share launches.
hipError_t critic_backward(spz_ctx* c, const float* const* dq, const void* X, void* const* const* hid,
                           uint32_t* const* const* bits, hipStream_t s) {
  const int nl = (int)c->net[1].L.size();
  // dz of the last hidden layer comes from the head backward. With the mask as bits,
  // that kernel also takes the column sums of dz (the last hidden layer's bias
  // gradient) and, reading the stored last hidden layer in the same pass, the output
  // layer's weight and bias gradients; otherwise those come from a column-sum pass and
  // the weight gradient. Every later dz comes from a dgrad that also produces its bias
  // gradient.
  const bool hb_sums = bits[0][nl - 2] != nullptr;
  void* dzb[2][2] = {{c->c_dz[0], c->c_dz[1]}, {c->c_dz2[0], c->c_dz2[1]}};
  for (int k = 0; k < 2; ++k) {
    const Net& n = c->net[1 + k];
    const Lay& H = n.L[nl - 1];
    HK(red_room(c, 0, 3, s));
    if (!hb_sums) {
      const int chunks = colsum_chunks(c->Bp);
      float* cpart = red_alloc(c, 0, (int64_t)chunks * H.in_p);
      float* cextra = red_alloc(c, 0, chunks);
      if (!cpart || !cextra) return hipErrorOutOfMemory;
      ColsumArgs cs{hid[k][nl - 2], H.in_p, H.in_p, c->Bp, COLSUM_CHUNK, dq[k], 1, cpart, cextra};
      HK(timed(c, "colsum", c->Bp, H.in_p, 1, 0.0, (double)c->Bp * H.in_p * es(c), s,
               [&] { return launch_colsum_partial(c->bf16, cs, s); }));
      HK(red_colsum(c, 0, cpart, chunks, H.in_p, c->G + H.w, cextra, c->G + H.b, s));
    }
    const int hblocks = head_bwd_blocks(c->Bp);
    float *hpart = nullptr, *wpart = nullptr, *wextra = nullptr;
    if (hb_sums) {
      hpart = red_alloc(c, 0, (int64_t)hblocks * H.in_p);
      wpart = red_alloc(c, 0, (int64_t)hblocks * H.in_p);
      wextra = red_alloc(c, 0, hblocks);
      if (!hpart || !wpart || !wextra) return hipErrorOutOfMemory;
    }
    HeadBwdArgs hb{dq[k], wop(c, false, H.w), hid[k][nl - 2], dzb[k][0], H.in_p, H.in_p, c->Bp, bits[k][nl - 2],
                   c->Bp, hpart, nullptr, nullptr, wpart, wextra};
    HK(timed(c, "head_bwd", c->Bp, H.in_p, 0, 0.0,
             head_bwd_bytes(c, H.in_p, bits[k][nl - 2]) + (hb_sums ? (double)c->Bp * H.in_p * es(c) : 0.0), s,
             [&] { return launch_head_bwd(c->bf16, hb, s); }));
    if (hb_sums) {
      HK(red_colsum(c, 0, hpart, hblocks, H.in_p, c->G + n.L[nl - 2].b, nullptr, nullptr, s));
      HK(red_colsum(c, 0, wpart, hblocks, H.in_p, c->G + H.w, wextra, c->G + H.b, s));
    }
  }
  int cur = 0;
  for (int l = nl - 2; l >= 0; --l) {
    const Lay& L = c->net[1].L[l];
    const void* dz[2] = {dzb[0][cur], dzb[1][cur]};
    const void* Xl[2] = {l == 0 ? X : hid[0][l - 1], l == 0 ? X : hid[1][l - 1]};
    const WgradIn w[2] = {{1, l, dz[0], Xl[0], l == 0 ? c->Kc : L.in_p}, {2, l, dz[1], Xl[1], l == 0 ? c->Kc : L.in_p}};
    HK(wgrad(c, 0, 2, w, l == nl - 2 && !hb_sums, s));
    if (l > 0) {
      DgradIn d[2];
      for (int k = 0; k < 2; ++k)
        d[k] = DgradIn{dz[k], hid[k][l - 1], bits[k][l - 1], dzb[k][cur ^ 1], c->G + c->net[1 + k].L[l - 1].b, nullptr};
      HK(dgrad(c, 1, 2, l, d, 0, L.in_p, true, L.in_p, L.in_p, false, 0, s));
      cur ^= 1;
    }
  }
  return hipSuccess;
}

// Gradient of sum_b dq[b] Q_ni(s, a)[b] with respect to the action block, into da [Bp, Ap].
hipError_t critic_action_grad(spz_ctx* c, int ni, const float* dq, void* const* hid, uint32_t* const* bits,
                              float* da, hipStream_t s) {
  const Net& n = c->net[ni];
  const int nl = (int)n.L.size();
  const Lay& H = n.L[nl - 1];
  HeadBwdArgs hb{dq, wop(c, false, H.w), hid[nl - 2], c->a_dz[0], H.in_p, H.in_p, c->Bp, bits[nl - 2], c->Bp,
                 nullptr};
  HK(timed(c, "head_bwd", c->Bp, H.in_p, 0, 0.0, head_bwd_bytes(c, H.in_p, bits[nl - 2]), s,
           [&] { return launch_head_bwd(c->bf16, hb, s); }));
  int cur = 0;
  for (int l = nl - 2; l >= 1; --l) {
    const Lay& L = n.L[l];
    const DgradIn d{c->a_dz[cur], hid[l - 1], bits[l - 1], c->a_dz[cur ^ 1], nullptr, nullptr};
    HK(dgrad(c, ni, 1, l, &d, 0, L.in_p, true, L.in_p, L.in_p, false, 1, s));
    cur ^= 1;
  }
  const DgradIn d0{c->a_dz[cur], nullptr, nullptr, da, nullptr, nullptr};
  return dgrad(c, ni, 1, 0, &d0, c->Ka, c->Kc, c->WT != nullptr, c->Ap, c->Ap, true, 1, s);
}

// The same for both critics, each restricted to the rows listed in its map (critic k:
// rmap + k Bp, padded with -1 to the device-side length rrows[k]): the head backward
// gathers those rows, every later product runs on the leading rows only (the twins'
// products layer by layer, so that they can share launches), and each action gradient
// is scattered back to da's rows (rows of da outside the maps are left as they are).
// Each row's arithmetic is that of the unrestricted chain.
hipError_t critic_action_grad_rows(spz_ctx* c, const float* const* dq, void* const* const* hid,
                                   uint32_t* const* const* bits, float* da, hipStream_t s) {
  const int nl = (int)c->net[1].L.size();
  void* dzb[2][2] = {{c->a_dz[0], c->a_dz[1]}, {c->a_dz2[0], c->a_dz2[1]}};
  uint32_t* rb[2] = {c->rbits, c->rbits2};
  for (int k = 0; k < 2; ++k) {
    const Lay& H = c->net[1 + k].L[nl - 1];
    HeadBwdArgs hb{dq[k], wop(c, false, H.w), hid[k][nl - 2], dzb[k][0], H.in_p, H.in_p, c->Bp, bits[k][nl - 2], c->Bp,
                   nullptr, c->rmap + (int64_t)k * c->Bp, c->rrows + k};
    HK(timed(c, "head_bwd_rows", c->Bp, H.in_p, 0, 0.0, 0.0, s, [&] { return launch_head_bwd(c->bf16, hb, s); }));
  }
  int cur = 0;
  for (int l = nl - 2; l >= 1; --l) {
    const Lay& L = c->net[1].L[l];
    DgradIn d[2];
    for (int k = 0; k < 2; ++k) {
      RowBitsGatherArgs gb{bits[k][l - 1], rb[k], c->Bp, L.in_p / 32, c->rmap + (int64_t)k * c->Bp, c->rrows + k, c->Bp};
      HK(timed(c, "row_bits_gather", c->Bp, L.in_p, 0, 0.0, 0.0, s, [&] { return launch_row_bits_gather(gb, s); }));
      d[k] = DgradIn{dzb[k][cur], nullptr, rb[k], dzb[k][cur ^ 1], nullptr, c->rrows + k};
    }
    HK(dgrad(c, 1, 2, l, d, 0, L.in_p, true, L.in_p, L.in_p, false, 1, s));
    cur ^= 1;
  }
  // Each action gradient of the listed rows lands in da2 (free here) and then in da.
  for (int k = 0; k < 2; ++k) {
    const DgradIn d0{dzb[k][cur], nullptr, nullptr, c->da2, nullptr, c->rrows + k};
    HK(dgrad(c, 1 + k, 1, 0, &d0, c->Ka, c->Kc, c->WT != nullptr, c->Ap, c->Ap, true, 1, s));
    RowScatterArgs sa{c->da2, da, c->Ap, c->Ap, c->rmap + (int64_t)k * c->Bp, c->rrows + k, c->Bp};
    HK(timed(c, "row_scatter", c->Bp, c->Ap, 0, 0.0, 0.0, s, [&] { return launch_row_scatter(sa, s); }));
  }
  return hipSuccess;
}

hipError_t actor_backward(spz_ctx* c, hipStream_t s) {
  const Net& n = c->net[0];
  const int nl = (int)n.L.size();
  const void* cur = c->dzh;
  int nxt = 0;
  // A hidden layer's weight gradient waits for the layer below when the two have one
  // shape, so that both can share a launch; its dz stays intact until then (the input
  // gradients alternate between two buffers).
  WgradIn held{};
  bool holding = false;
  for (int l = nl - 1; l >= 0; --l) {
    const Lay& L = n.L[l];
    const WgradIn w{0, l, cur, l == 0 ? c->xsa : c->ha[l - 1], l == 0 ? c->Kc : L.in_p};
    if (holding) {
      const WgradIn two[2] = {held, w};
      HK(wgrad(c, 1, 2, two, false, s));
      holding = false;
    } else if (l > 0 && l < nl - 1 && n.L[l - 1].out_p == L.out_p && n.L[l - 1].in_p == L.in_p) {
      held = w;
      holding = true;
    } else {
      HK(wgrad(c, 1, 1, &w, l == nl - 1, s));
    }
    if (l > 0) {
      const DgradIn d{cur, c->ha[l - 1], c->bha[l - 1], c->a_dz[nxt], c->G + n.L[l - 1].b, nullptr};
      HK(dgrad(c, 0, 1, l, &d, 0, L.in_p, true, L.in_p, L.in_p, false, 1, s));
      cur = c->a_dz[nxt];
      nxt ^= 1;
    }
  }
  return hipSuccess;
}

const float* log_alpha_ptr(const spz_ctx* c) { return c->P + c->la; }

// Critic stream: TD target from the target networks, online critic forward on (s, a),
// critic loss and critic backward.
hipError_t critic_part(spz_ctx* c, hipStream_t s) {
  const int pa = c->net[0].L.back().out_p;
  const spz_hparams& hp = c->hp;
  NetOut act{c->cs_hid.data(), nullptr, nullptr, c->z2, nullptr};
  if (!c->td3) {
    const SacHeadArgs h{c->z2, pa, c->A, c->B, c->seed, c->d_step, P_NOISE_TGT, hp.log_std_min, hp.log_std_max,
                        c->xs2, c->Kc, c->Ka, c->logp2, nullptr, nullptr, nullptr};
    if (sac_head_fused(c)) act.sac = &h;
    HK(forward(c, 0, 1, false, c->xs2, c->Kc, &act, true, s));
    if (!act.sac)
      HK(timed(c, "sac_head", c->B, c->A, 0, 0.0, 0.0, s, [&] { return launch_sac_head(c->bf16, h, s); }));
  } else {
    HK(forward(c, 0, 1, true, c->xs2, c->Kc, &act, true, s));
    Td3HeadArgs h{c->z2, pa, c->A, c->B, c->seed, c->d_step, 1, hp.policy_noise, hp.noise_clip,
                  c->xs2, c->Kc, c->Ka, nullptr};
    HK(timed(c, "td3_head", c->B, c->A, 0, 0.0, 0.0, s, [&] { return launch_td3_head(c->bf16, h, s); }));
  }
  QSrc q[2];
  const NetOut tgt[2] = {{c->cs_hid.data(), nullptr, c->c_rdot[0], c->qt1, &q[0]},
                         {c->cs_hid2.data(), nullptr, c->c_rdot[1], c->qt2, &q[1]}};
  HK(forward(c, 1, 2, true, c->xs2, c->Kc, tgt, false, s));
  TdArgs td{q[0], q[1], c->r, c->d, c->td3 ? nullptr : c->logp2, log_alpha_ptr(c), c->y, hp.gamma, c->B, c->Bp};
  HK(timed(c, "td_target", c->Bp, 0, 0, 0.0, 0.0, s, [&] { return launch_td_target(td, s); }));
  // the target critics' partials were consumed by the TD target: their buffers are free
  const NetOut onl[2] = {{c->hc[0].data(), c->bhc[0].data(), c->c_rdot[0], c->q1, &q[0]},
                         {c->hc[1].data(), c->bhc[1].data(), c->c_rdot[1], c->q2, &q[1]}};
  HK(forward(c, 1, 2, false, c->xsa, c->Kc, onl, true, s));
  CriticLossArgs cl{q[0], q[1], c->y, c->dq1, c->dq2, c->c_lpart, c->B, c->Bp};
  HK(timed(c, "critic_loss", c->Bp, 0, 0, 0.0, 0.0, s, [&] { return launch_critic_loss(cl, s); }));
  c->red[0].jobs.n = 0;
  c->red[0].off = 0;
  c->red[0].bytes = 0.0;
  const float* dq[2] = {c->dq1, c->dq2};
  void* const* hid[2] = {c->hc[0].data(), c->hc[1].data()};
  uint32_t* const* bits[2] = {c->bhc[0].data(), c->bhc[1].data()};
  HK(critic_backward(c, dq, c->xsa, hid, bits, s));
  return red_flush(c, 0, s);
}

// Actor stream: reparameterised action on s, critics at their step-start values on
// (s, a~), actor loss, gradient through the critics to the action, head and actor backward.
hipError_t actor_part(spz_ctx* c, hipStream_t s) {
  const int pa = c->net[0].L.back().out_p;
  const spz_hparams& hp = c->hp;
  NetOut act{c->ha.data(), c->bha.data(), nullptr, c->z, nullptr};
  const SacHeadArgs sh{c->z, pa, c->A, c->B, c->seed, c->d_step, P_NOISE_POL, hp.log_std_min, hp.log_std_max,
                       c->xs_act, c->Kc, c->Ka, c->logp, c->th, c->se, c->lm};
  if (sac_head_fused(c)) act.sac = &sh;
  HK(forward(c, 0, 1, false, c->xsa, c->Kc, &act, true, s));
  if (!c->td3) {
    if (!act.sac)
      HK(timed(c, "sac_head", c->B, c->A, 0, 0.0, 0.0, s, [&] { return launch_sac_head(c->bf16, sh, s); }));
  } else {
    Td3HeadArgs h{c->z, pa, c->A, c->B, c->seed, c->d_step, 0, 0.0f, 0.0f, c->xs_act, c->Kc, c->Ka, c->th};
    HK(timed(c, "td3_head", c->B, c->A, 0, 0.0, 0.0, s, [&] { return launch_td3_head(c->bf16, h, s); }));
  }
  // TD3's actor loss takes critic 1 only.
  QSrc qp[2]{};
  const NetOut cr[2] = {{c->hpc[0].data(), c->bhpc[0].data(), c->a_rdot[0], c->qp1, &qp[0]},
                        {c->hpc[1].data(), c->bhpc[1].data(), c->a_rdot[1], c->qp2, &qp[1]}};
  HK(forward(c, 1, c->td3 ? 1 : 2, false, c->xs_act, c->Kc, cr, false, s));
  ActorLossArgs al{qp[0], qp[1], c->td3 ? 0 : 1, c->logp, log_alpha_ptr(c), c->dqp1,
                   c->td3 ? nullptr : c->dqp2, c->a_lpart, c->B, c->Bp, c->row_split ? c->rcnt : nullptr};
  HK(timed(c, "actor_loss", c->Bp, 0, 0, 0.0, 0.0, s, [&] { return launch_actor_loss(al, s); }));
  if (c->row_split) {
    // The loss takes min(Q1, Q2) per row, so each row's gradient reaches one critic
    // only: each critic's chain runs on its own rows and both land in da1.
    MinqSplitArgs ms{c->qp1, c->qp2, c->rcnt, c->B, c->Bp, c->rmap, c->rmap + c->Bp, c->rrows};
    HK(timed(c, "minq_split", c->Bp, 0, 0, 0.0, 0.0, s, [&] { return launch_minq_split(ms, s); }));
    const float* dq[2] = {c->dqp1, c->dqp2};
    void* const* hid[2] = {c->hpc[0].data(), c->hpc[1].data()};
    uint32_t* const* bits[2] = {c->bhpc[0].data(), c->bhpc[1].data()};
    HK(critic_action_grad_rows(c, dq, hid, bits, c->da1, s));
  } else {
    HK(critic_action_grad(c, 1, c->dqp1, c->hpc[0].data(), c->bhpc[0].data(), c->da1, s));
    if (!c->td3) HK(critic_action_grad(c, 2, c->dqp2, c->hpc[1].data(), c->bhpc[1].data(), c->da2, s));
  }
  ActorHeadBwdArgs hb{c->da1, c->td3 || c->row_split ? nullptr : c->da2, c->Ap, c->th, c->se, c->lm,
                      log_alpha_ptr(c), c->dzh, pa, c->A, c->B, c->td3 ? 0 : 1};
  HK(timed(c, "actor_head_bwd", c->B, c->A, 0, 0.0, 0.0, s, [&] { return launch_actor_head_bwd(c->bf16, hb, s); }));
  c->red[1].jobs.n = 0;
  c->red[1].off = 0;
  c->red[1].bytes = 0.0;
  HK(actor_backward(c, s));
  return red_flush(c, 1, s);
}

// Adam (+ Polyak) over the parameter arena. critics / actor select the optimizer
// ranges of this launch; step_add is 1 when the step counter has not been advanced
// by k_finish yet.
hipError_t adam(spz_ctx* c, bool critics, bool actor_step, bool actor, int step_add, hipStream_t s) {
  const Net& an = c->net[0];
  AdamArgs a{};
  a.P = c->P; a.M = c->M; a.V = c->V; a.T = c->T; a.G = c->G; a.Pb = c->Pb; a.Tb = c->Tb;
  a.n = c->n_arena;
  a.a0 = an.off; a.a1 = an.end;
  a.c0 = c->net[1].off; a.c1 = c->net[2].end;
  a.la = c->la;
  a.do_critic = critics ? 1 : 0;
  a.do_actor = (actor && actor_step) ? 1 : 0;
  a.do_alpha = (actor && !c->td3 && c->hp.learn_alpha) ? 1 : 0;
  a.polyak_critic = (critics && (!c->td3 || actor_step)) ? 1 : 0;
  a.polyak_actor = (actor && c->td3 && actor_step) ? 1 : 0;
  a.td3 = c->td3 ? 1 : 0;
  a.delay = c->hp.policy_delay;
  a.lr_a = c->hp.lr_actor; a.lr_c = c->hp.lr_critic; a.lr_al = c->hp.lr_alpha;
  a.b1 = c->hp.beta1; a.b2 = c->hp.beta2; a.eps = c->hp.eps; a.tau = c->hp.tau;
  a.step = c->d_step;
  a.step_add = step_add;
  const double n_crit = (double)(c->net[2].end - c->net[1].off);
  const double n_act = (double)(an.end - an.off);
  const double n_adam = (critics ? n_crit : 0.0) + (a.do_actor ? n_act : 0.0) + (a.do_alpha ? 1.0 : 0.0);
  const double n_pol = (a.polyak_critic ? n_crit : 0.0) + (a.polyak_actor ? n_act : 0.0);
  const double bytes = 28.0 * n_adam + 8.0 * n_pol + (c->bf16 ? 2.0 * (n_adam + n_pol) : 0.0);
  HK(timed(c, "adam_polyak", (int)c->n_arena, 0, (critics ? 2 : 0) + (actor ? 1 : 0), 0.0, bytes, s,
           [&] { return launch_adam(a, s); }));
  return refresh_wt(c, s);
}

int enqueue_step(spz_ctx* c, hipStream_t s0) {
  const int64_t t = c->h_step + 1;
  const bool actor_step = !c->td3 || (t % c->hp.policy_delay == 0);
  const bool sequential = c->hp.ordering == SPZ_ORDER_SEQUENTIAL;
  // Kernel timing of this step (profile stride); launches outside steps are timed as before.
  struct StepTiming {
    spz_ctx* c;
    ~StepTiming() { c->pf_step = true; }
  } step_timing{c};
  c->pf_step = t % c->pf_stride == 0;
  const bool two = c->hp.n_streams == 2 && !sequential;
  c->xs_act = two ? c->xsp : c->xsa;
  GatherArgs g{c->buf, c->row_bytes, c->off_a, c->off_s2, c->off_r, c->off_d, c->O, c->A, c->Ka, c->Kc,
               c->B, c->seed, (uint32_t)c->size, c->d_step, c->xsa, c->xs2, two ? c->xsp : nullptr, c->r, c->d,
               c->idx, two ? nullptr : c->abuf};
  {
    const double e = (double)es(c);
    // s to xsa (and xsp on two streams), s' to xs2; a to xsa (and abuf on one stream)
    const double copies = two ? 3.0 : 2.0, acopies = two ? 1.0 : 2.0;
    const double bytes = (double)c->B * ((2.0 * c->O + c->A) * e + 8.0 + (copies * c->O + acopies * c->A) * e + 12.0);
    CK(timed(c, "gather", c->B, c->O, c->A, 0.0, bytes, s0, [&] { return launch_gather(c->bf16, g, s0); }));
  }
  hipStream_t sc = s0, sa = s0;
  if (two) {
    CK(hipEventRecord(c->ev_fork, s0));
    CK(hipStreamWaitEvent(c->sc, c->ev_fork, 0));
    CK(hipStreamWaitEvent(c->sa, c->ev_fork, 0));
    sc = c->sc;
    sa = c->sa;
  }
  CK(critic_part(c, sc));
  // Sequential ordering: the critics step (and their targets move) before the
  // actor's loss is taken through them.
  if (sequential) CK(adam(c, true, actor_step, false, 1, s0));
  if (actor_step) CK(actor_part(c, sa));
  if (two) {
    CK(hipEventRecord(c->ev_c, sc));
    CK(hipStreamWaitEvent(s0, c->ev_c, 0));
    if (actor_step) {
      CK(hipEventRecord(c->ev_a, sa));
      CK(hipStreamWaitEvent(s0, c->ev_a, 0));
    }
  }
  FinishArgs f{c->c_lpart, c->a_lpart, loss_blocks(c->Bp), loss_blocks(c->Bp), c->B, c->td3 ? 0 : 1,
               actor_step ? 1 : 0, c->hp.learn_alpha, c->hp.target_entropy, log_alpha_ptr(c),
               c->td3 ? nullptr : c->G + c->la, c->rec, c->rec_cap, c->d_step};
  CK(timed(c, "finish", 0, 0, 0, 0.0, 0.0, s0, [&] { return launch_finish(f, s0); }));
  CK(adam(c, !sequential, actor_step, true, 0, s0));
  c->h_step = t;
  return SPZ_OK;
}

// One update step from a captured graph (hp.graphs). Kernel arguments are fixed at
// capture: buffer addresses, shapes (batch), the replay fill level and the seed; the
// step number, which the kernels read from device memory, is not. A missing or stale
// graph for this step kind is replaced: the step runs eagerly (which also performs
// every first-launch set-up of its kernels outside the capture), then the same step
// kind is captured on sg for the next time.
int graph_step(spz_ctx* c, hipStream_t s0) {
  const int64_t t = c->h_step + 1;
  const int kind = (!c->td3 || t % c->hp.policy_delay == 0) ? 1 : 0;
  spz_ctx::GraphSlot& gs = c->gslot[kind];
  const bool fresh = gs.exec && gs.B == c->B && gs.Bp == c->Bp && gs.size == c->size && gs.seed == c->seed;
  if (fresh) {
    CK(hipGraphLaunch(gs.exec, s0));
    c->h_step = t;
    return SPZ_OK;
  }
  int rc = enqueue_step(c, s0);
  if (rc) return rc;
  if (gs.exec) {
    CK(hipGraphExecDestroy(gs.exec));
    gs.exec = nullptr;
  }
  // Capture step t's kind again (the capture enqueues nothing).
  c->h_step = t - 1;
  CK(hipStreamBeginCapture(c->sg, hipStreamCaptureModeThreadLocal));
  rc = enqueue_step(c, c->sg);
  hipGraph_t graph = nullptr;
  const hipError_t ec = hipStreamEndCapture(c->sg, &graph);
  c->h_step = t;
  if (rc) {
    if (graph) (void)hipGraphDestroy(graph);
    return rc;
  }
  if (ec != hipSuccess) return fail_hip(c, ec, "hipStreamEndCapture");
  const hipError_t ei = hipGraphInstantiate(&gs.exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  if (ei != hipSuccess) {
    gs.exec = nullptr;
    return fail_hip(c, ei, "hipGraphInstantiate");
  }
  gs.B = c->B;
  gs.Bp = c->Bp;
  gs.size = c->size;
  gs.seed = c->seed;
  return SPZ_OK;
}

int ctx_sync(spz_ctx* c) {
  if (c->has_last) CK(hipStreamSynchronize(c->last));
  if (c->si) CK(hipStreamSynchronize(c->si));
  CK(hipStreamSynchronize(c->sc));
  CK(hipStreamSynchronize(c->sa));
  return SPZ_OK;
}

int setup(spz_ctx* c) {
  const size_t e = es(c);
  const int64_t Bp = c->Bp;
  const int nh = (int)c->hidden.size();
  // replay ring
  // [obs | act | next_obs | rew done], each segment starting on a 16-byte boundary.
  c->off_a = (int)align16((int64_t)c->O * e);
  c->off_s2 = c->off_a + (int)align16((int64_t)c->A * e);
  c->off_r = c->off_s2 + (int)align16((int64_t)c->O * e);
  c->off_d = c->off_r + 4;
  c->row_bytes = align16(c->off_d + 4);
  c->cap = c->hp.capacity;
  CK(dalloc_t(c, &c->buf, (size_t)(c->row_bytes * c->cap)));
  // parameters
  const size_t ab = (size_t)c->n_arena * 4;
  CK(dalloc_t(c, &c->P, ab));
  CK(dalloc_t(c, &c->G, ab));
  CK(dalloc_t(c, &c->M, ab));
  CK(dalloc_t(c, &c->V, ab));
  CK(dalloc_t(c, &c->T, ab));
  if (c->bf16) {
    CK(dalloc_t(c, &c->Pb, (size_t)c->n_arena * 2));
    CK(dalloc_t(c, &c->Tb, (size_t)c->n_arena * 2));
    CK(dalloc(c, &c->WT, (size_t)c->n_arena * 2));
    std::vector<TransposeJob> jobs;
    int tiles = 0;
    for (int ni = 0; ni < 3; ++ni) {
      const Net& n = c->net[ni];
      const int last = (int)n.L.size() - (ni == 0 ? 1 : 2);   // critic output layers: head kernels
      for (int l = 1; l <= last; ++l) {
        const Lay& L = n.L[l];
        jobs.push_back(TransposeJob{L.w, L.w, L.in_p, L.out_p, L.out_p, L.in_p, tiles});
        tiles += transpose_tiles(L.out_p, L.in_p);
        c->t_elems += (double)L.out_p * L.in_p;
      }
      if (ni != 0) {   // a critic's first layer: the action block only, for the action gradient
        const Lay& L = n.L[0];
        jobs.push_back(TransposeJob{L.w + c->Ka, L.w, L.in_p, L.out_p, L.out_p, c->Ap, tiles});
        tiles += transpose_tiles(L.out_p, c->Ap);
        c->t_elems += (double)L.out_p * c->Ap;
      }
    }
    c->n_tjobs = (int)jobs.size();
    c->t_tiles = tiles;
    if (c->n_tjobs) {
      CK(dalloc_t(c, &c->tjobs, jobs.size() * sizeof(TransposeJob)));
      CK(hipMemcpy(c->tjobs, jobs.data(), jobs.size() * sizeof(TransposeJob), hipMemcpyHostToDevice));
    }
  }
  CK(dalloc_t(c, &c->d_step, 8));
  CK(dalloc_t(c, &c->rec, (size_t)c->rec_cap * SPZ_REC_WIDTH * 4));
  // batch
  const size_t xb = (size_t)Bp * c->Kc * e;
  CK(dalloc(c, &c->xsa, xb));
  CK(dalloc(c, &c->xs2, xb));
  CK(dalloc(c, &c->xsp, xb));
  CK(dalloc(c, &c->abuf, (size_t)Bp * c->A * e));
  CK(dalloc_t(c, &c->r, Bp * 4));
  CK(dalloc_t(c, &c->d, Bp * 4));
  CK(dalloc_t(c, &c->idx, Bp * 4));
  const size_t hb = (size_t)Bp * c->hmax * e;
  const int pa = c->net[0].L.back().out_p;
  float** f32s[] = {&c->logp2, &c->qt1, &c->qt2, &c->y, &c->q1, &c->q2, &c->dq1, &c->dq2,
                    &c->logp, &c->qp1, &c->qp2, &c->dqp1, &c->dqp2};
  for (float** p : f32s) CK(dalloc_t(c, p, Bp * 4));
  CK(dalloc_t(c, &c->z2, (size_t)Bp * pa * 4));
  CK(dalloc_t(c, &c->z, (size_t)Bp * pa * 4));
  CK(dalloc_t(c, &c->th, (size_t)Bp * c->A * 4));
  CK(dalloc_t(c, &c->se, (size_t)Bp * c->A * 4));
  CK(dalloc_t(c, &c->lm, (size_t)Bp * c->A * 4));
  CK(dalloc_t(c, &c->da1, (size_t)Bp * c->Ap * 4));
  CK(dalloc_t(c, &c->da2, (size_t)Bp * c->Ap * 4));
  CK(dalloc(c, &c->dzh, (size_t)Bp * pa * e));
  for (int i = 0; i < 2; ++i) {
    CK(dalloc(c, &c->cs_h[i], hb));
    CK(dalloc(c, &c->cs_h2[i], hb));
    CK(dalloc(c, &c->c_dz[i], hb));
    CK(dalloc(c, &c->c_dz2[i], hb));
    CK(dalloc(c, &c->a_dz[i], hb));
    CK(dalloc(c, &c->a_dz2[i], hb));
    c->hc[i].assign(nh, nullptr);
    c->hpc[i].assign(nh, nullptr);
    for (int l = 0; l < nh; ++l) {
      CK(dalloc(c, &c->hc[i][l], (size_t)Bp * pad32(c->hidden[l]) * e));
      CK(dalloc(c, &c->hpc[i][l], (size_t)Bp * pad32(c->hidden[l]) * e));
    }
  }
  c->ha.assign(nh, nullptr);
  c->cs_hid.assign(nh, nullptr);
  c->cs_hid2.assign(nh, nullptr);
  for (int l = 0; l < nh; ++l) {
    CK(dalloc(c, &c->ha[l], (size_t)Bp * pad32(c->hidden[l]) * e));
    c->cs_hid[l] = c->cs_h[l & 1];
    c->cs_hid2[l] = c->cs_h2[l & 1];
  }
  // ReLU masks as bits where the large-tile kernel produces and consumes them (the
  // same condition holds for every product that reads a layer's mask), and the
  // row-dot partials of the folded critic output layers.
  for (int i = 0; i < 2; ++i) {
    c->bhc[i].assign(nh, nullptr);
    c->bhpc[i].assign(nh, nullptr);
  }
  c->bha.assign(nh, nullptr);
  int rd_parts = 0;
  for (int l = 0; l < nh; ++l) {
    const int w = pad32(c->hidden[l]);
    if (!gemm_fused_ok(c->bf16, GEMM_FWD, (int)Bp, w, 32)) continue;
    const size_t bb = (size_t)Bp * (w / 32) * 4;
    for (int i = 0; i < 2; ++i) {
      CK(dalloc_t(c, &c->bhc[i][l], bb));
      CK(dalloc_t(c, &c->bhpc[i][l], bb));
    }
    CK(dalloc_t(c, &c->bha[l], bb));
    if (l == nh - 1) rd_parts = w / 64;   // the most partials any batch size gives (gemm_rdot_cols)
  }
  if (rd_parts) {
    for (int i = 0; i < 2; ++i) {
      CK(dalloc_t(c, &c->c_rdot[i], (size_t)rd_parts * Bp * 4));
      CK(dalloc_t(c, &c->a_rdot[i], (size_t)rd_parts * Bp * 4));
    }
  }
  // The row split needs every hidden mask of both critics as bits.
  c->row_split = !c->td3 && c->hp.actor_row_split;
  for (int l = 0; l < nh; ++l) c->row_split = c->row_split && c->bhpc[0][l] && c->bhpc[1][l];
  if (c->row_split) {
    CK(dalloc_t(c, &c->rmap, (size_t)2 * Bp * 4));
    CK(dalloc_t(c, &c->rrows, 64));
    CK(dalloc_t(c, &c->rcnt, (size_t)(Bp / 256) * 4));
    CK(dalloc_t(c, &c->rbits, (size_t)Bp * (c->hmax / 32) * 4));
    CK(dalloc_t(c, &c->rbits2, (size_t)Bp * (c->hmax / 32) * 4));
  }
  // deferred-reduction workspaces, sized for the created batch (spz_set_batch checks
  // that a smaller one fits)
  for (int q = 0; q < 2; ++q) {
    c->red[q].cap = red_need(c, q, (int)Bp);
    CK(dalloc_t(c, &c->red[q].base, (size_t)c->red[q].cap * 4));
  }
  CK(dalloc_t(c, &c->c_lpart, (size_t)loss_blocks((int)Bp) * 3 * 8));
  CK(dalloc_t(c, &c->a_lpart, (size_t)loss_blocks((int)Bp) * 2 * 8));
  // streams (default priority)
  CK(hipStreamCreateWithFlags(&c->sc, hipStreamNonBlocking));
  CK(hipStreamCreateWithFlags(&c->sa, hipStreamNonBlocking));
  if (c->hp.graphs) CK(hipStreamCreateWithFlags(&c->sg, hipStreamNonBlocking));
  CK(hipEventCreateWithFlags(&c->ev_fork, hipEventDisableTiming));
  CK(hipEventCreateWithFlags(&c->ev_c, hipEventDisableTiming));
  CK(hipEventCreateWithFlags(&c->ev_a, hipEventDisableTiming));
  CK(hipEventCreateWithFlags(&c->ev_commit, hipEventDisableTiming));
  // parameters: host init, targets = online, bf16 images
  std::vector<float> img;
  host_init(c, img);
  CK(hipMemcpy(c->P, img.data(), ab, hipMemcpyHostToDevice));
  CK(hipMemcpy(c->T, img.data(), ab, hipMemcpyHostToDevice));
  if (c->bf16) {
    CK(launch_to_bf16(c->P, c->Pb, c->n_arena, c->sc));
    CK(launch_to_bf16(c->T, c->Tb, c->n_arena, c->sc));
    CK(refresh_wt(c, c->sc));
  }
  CK(hipStreamSynchronize(c->sc));
  CK(hipDeviceSynchronize());
  return SPZ_OK;
}

void release(spz_ctx* c) {
  if (!c) return;
  (void)hipSetDevice(c->hp.device);
  if (c->sc) (void)hipStreamSynchronize(c->sc);
  if (c->sa) (void)hipStreamSynchronize(c->sa);
  if (c->has_last) (void)hipStreamSynchronize(c->last);
  if (c->si) (void)hipStreamSynchronize(c->si);
  for (auto& sl : c->slots) {
    if (sl.host) (void)hipHostFree(sl.host);
    if (sl.dev) (void)hipFree(sl.dev);
    if (sl.copied) (void)hipEventDestroy(sl.copied);
    if (sl.done) (void)hipEventDestroy(sl.done);
  }
  if (c->si) (void)hipStreamDestroy(c->si);
  for (auto& gs : c->gslot)
    if (gs.exec) (void)hipGraphExecDestroy(gs.exec);
  if (c->sg) (void)hipStreamDestroy(c->sg);
  if (c->ev_commit) (void)hipEventDestroy(c->ev_commit);
  for (void* p : c->allocs) (void)hipFree(p);
  if (c->stage) (void)hipFree(c->stage);
  for (hipEvent_t e : c->pool) (void)hipEventDestroy(e);
  for (auto& pe : c->pevs) {
    (void)hipEventDestroy(pe.a);
    (void)hipEventDestroy(pe.b);
  }
  if (c->ev_fork) (void)hipEventDestroy(c->ev_fork);
  if (c->ev_c) (void)hipEventDestroy(c->ev_c);
  if (c->ev_a) (void)hipEventDestroy(c->ev_a);
  if (c->sc) (void)hipStreamDestroy(c->sc);
  if (c->sa) (void)hipStreamDestroy(c->sa);
  delete c;
}

// Selector -> (arena, net index or -1 for log alpha).
int resolve(const spz_ctx* c, int32_t which, float** arena, int* ni) {
  switch (which) {
    case SPZ_ACTOR: *arena = c->P; *ni = 0; return 0;
    case SPZ_CRITIC1: *arena = c->P; *ni = 1; return 0;
    case SPZ_CRITIC2: *arena = c->P; *ni = 2; return 0;
    case SPZ_TCRITIC1: *arena = c->T; *ni = 1; return 0;
    case SPZ_TCRITIC2: *arena = c->T; *ni = 2; return 0;
    case SPZ_TACTOR: if (!c->td3) return -1; *arena = c->T; *ni = 0; return 0;
    case SPZ_LOG_ALPHA: *arena = c->P; *ni = -1; return 0;
    case SPZ_M_ACTOR: *arena = c->M; *ni = 0; return 0;
    case SPZ_M_CRITIC1: *arena = c->M; *ni = 1; return 0;
    case SPZ_M_CRITIC2: *arena = c->M; *ni = 2; return 0;
    case SPZ_M_LOG_ALPHA: *arena = c->M; *ni = -1; return 0;
    case SPZ_V_ACTOR: *arena = c->V; *ni = 0; return 0;
    case SPZ_V_CRITIC1: *arena = c->V; *ni = 1; return 0;
    case SPZ_V_CRITIC2: *arena = c->V; *ni = 2; return 0;
    case SPZ_V_LOG_ALPHA: *arena = c->V; *ni = -1; return 0;
    case SPZ_G_ACTOR: *arena = c->G; *ni = 0; return 0;
    case SPZ_G_CRITIC1: *arena = c->G; *ni = 1; return 0;
    case SPZ_G_CRITIC2: *arena = c->G; *ni = 2; return 0;
    case SPZ_G_LOG_ALPHA: *arena = c->G; *ni = -1; return 0;
  }
  return -1;
}

}  // namespace

// ====================================================================================== C ABI
extern "C" {

void spz_hparams_default(spz_hparams* hp) {
  if (!hp) return;
  std::memset(hp, 0, sizeof(*hp));
  hp->algo = SPZ_ALGO_SAC;
  hp->gemm_prec = SPZ_PREC_FP32;
  hp->capacity = 1000000;
  hp->gamma = 0.99f;
  hp->tau = 0.005f;
  hp->lr_actor = hp->lr_critic = hp->lr_alpha = 3e-4f;
  hp->beta1 = 0.9f;
  hp->beta2 = 0.999f;
  hp->eps = 1e-8f;
  hp->alpha_init = 1.0f;
  hp->learn_alpha = 1;
  hp->target_entropy = 0.0f;
  hp->log_std_min = -20.0f;
  hp->log_std_max = 2.0f;
  hp->policy_noise = 0.2f;
  hp->noise_clip = 0.5f;
  hp->policy_delay = 2;
  hp->device = 0;
  hp->n_streams = 2;
  hp->ordering = SPZ_ORDER_SNAPSHOT;
  hp->actor_row_split = 1;
  hp->graphs = 0;
}

spz_ctx* spz_create(int32_t obs_dim, int32_t act_dim, const int32_t* hidden, int32_t n_hidden, int32_t batch,
                    const spz_hparams* hp, uint64_t seed) {
  tl_err.clear();
  if (!hp || !hidden) { set_err(nullptr, SPZ_EINVAL, "spz_create: NULL hidden or hparams"); return nullptr; }
  if (obs_dim < 1 || act_dim < 1 || n_hidden < 1 || n_hidden > 6 || batch < 1) {
    set_err(nullptr, SPZ_EINVAL, "spz_create: dimensions out of range");
    return nullptr;
  }
  for (int i = 0; i < n_hidden; ++i)
    if (hidden[i] < 1 || hidden[i] > 65536) {
      set_err(nullptr, SPZ_EINVAL, "spz_create: hidden width out of range");
      return nullptr;
    }
  if ((hp->algo != SPZ_ALGO_SAC && hp->algo != SPZ_ALGO_TD3) ||
      (hp->gemm_prec != SPZ_PREC_FP32 && hp->gemm_prec != SPZ_PREC_BF16) || hp->capacity < 1 ||
      hp->capacity > 0xFFFFFFFFll || !(hp->tau >= 0.0f && hp->tau <= 1.0f) ||
      (hp->algo == SPZ_ALGO_SAC && !(hp->alpha_init > 0.0f)) || hp->policy_delay < 1 ||
      (hp->n_streams != 1 && hp->n_streams != 2) || !(hp->log_std_min <= hp->log_std_max) ||
      (hp->ordering != SPZ_ORDER_SNAPSHOT && hp->ordering != SPZ_ORDER_SEQUENTIAL) ||
      (hp->actor_row_split != 0 && hp->actor_row_split != 1) || (hp->graphs != 0 && hp->graphs != 1)) {
    set_err(nullptr, SPZ_EINVAL, "spz_create: invalid hyper-parameters");
    return nullptr;
  }
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || hp->device < 0 || hp->device >= ndev) {
    set_err(nullptr, SPZ_EINVAL, "spz_create: no such HIP device");
    return nullptr;
  }
  spz_ctx* c = new (std::nothrow) spz_ctx();
  if (!c) { set_err(nullptr, SPZ_ENOMEM, "spz_create: out of host memory"); return nullptr; }
  c->O = obs_dim;
  c->A = act_dim;
  c->B = batch;
  c->Bp = (batch + 255) / 256 * 256;
  c->Bmax = c->B;
  c->Bpmax = c->Bp;
  c->hidden.assign(hidden, hidden + n_hidden);
  c->hp = *hp;
  c->seed = seed;
  c->bf16 = hp->gemm_prec == SPZ_PREC_BF16;
  c->td3 = hp->algo == SPZ_ALGO_TD3;
  if (hipSetDevice(hp->device) != hipSuccess) {
    set_err(nullptr, SPZ_EHIP, "spz_create: hipSetDevice failed");
    delete c;
    return nullptr;
  }
  plan_layout(c);
  const hipError_t se = scratch_init(hp->device);
  if (se != hipSuccess) {
    set_err(nullptr, SPZ_EHIP, std::string("spz_create: hipGetSymbolAddress of the scratch array: ") +
                                   hipGetErrorString(se));
    delete c;
    return nullptr;
  }
  const int rc = setup(c);
  if (rc != SPZ_OK) {
    const std::string msg = c->err;
    release(c);
    set_err(nullptr, rc == SPZ_EHIP && msg.find("hipMalloc") != std::string::npos ? SPZ_ENOMEM : rc, msg);
    return nullptr;
  }
  return c;
}

void spz_destroy(spz_ctx* c) { release(c); }

int spz_buffer_push(spz_ctx* c, const float* obs, const float* act, const float* rew, const float* done,
                    const float* next_obs, int64_t n) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_buffer_push: NULL context");
  if (n < 0) return set_err(c, SPZ_EINVAL, "spz_buffer_push: n < 0");
  if (n == 0) return SPZ_OK;
  if (!obs || !act || !rew || !done || !next_obs) return set_err(c, SPZ_EINVAL, "spz_buffer_push: NULL array");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  const int64_t CH = 65536;
  const int64_t rowf = 2 * (int64_t)c->O + c->A + 2;
  if (!c->stage) {
    CK(hipMalloc(&c->stage, (size_t)(CH * rowf * 4)));
    c->stage_rows = CH;
  }
  // Rows overwritten within this push never need to be written.
  const int64_t skip = n > c->cap ? n - c->cap : 0;
  for (int64_t r0 = skip; r0 < n; r0 += CH) {
    const int64_t m = std::min(CH, n - r0);
    float* so = c->stage;
    float* sa_ = so + CH * c->O;
    float* sr = sa_ + CH * c->A;
    float* sd = sr + CH;
    float* sn = sd + CH;
    CK(hipMemcpy(so, obs + r0 * c->O, (size_t)(m * c->O * 4), hipMemcpyHostToDevice));
    CK(hipMemcpy(sa_, act + r0 * c->A, (size_t)(m * c->A * 4), hipMemcpyHostToDevice));
    CK(hipMemcpy(sr, rew + r0, (size_t)(m * 4), hipMemcpyHostToDevice));
    CK(hipMemcpy(sd, done + r0, (size_t)(m * 4), hipMemcpyHostToDevice));
    CK(hipMemcpy(sn, next_obs + r0 * c->O, (size_t)(m * c->O * 4), hipMemcpyHostToDevice));
    PackArgs p{c->buf, c->row_bytes, c->off_a, c->off_s2, c->off_r, c->off_d, c->O, c->A, m,
               (c->ptr + r0) % c->cap, c->cap, so, sa_, sr, sd, sn};
    CK(launch_pack(c->bf16, p, c->sc));
    CK(hipStreamSynchronize(c->sc));
  }
  c->ptr = (c->ptr + n) % c->cap;
  c->size = std::min(c->size + n, c->cap);
  return SPZ_OK;
}

int64_t spz_buffer_size(const spz_ctx* c) { return c ? c->size : SPZ_EINVAL; }

namespace {
constexpr int64_t INGEST_ROWS = 65536;   // rows per ingestion slot
constexpr int INGEST_SLOTS = 4;

static int ingest_init(spz_ctx* c) {
  if (c->si) return SPZ_OK;
  const int64_t rowf = 2 * (int64_t)c->O + c->A + 2;
  const size_t bytes = (size_t)(INGEST_ROWS * rowf * 4);
  c->slots.resize(INGEST_SLOTS);
  for (auto& sl : c->slots) {
    if (hipHostMalloc((void**)&sl.host, bytes, hipHostMallocDefault) != hipSuccess)
      return set_err(c, SPZ_ENOMEM, "spz_buffer_push_async: pinned host staging");
    if (hipMalloc((void**)&sl.dev, bytes) != hipSuccess)
      return set_err(c, SPZ_ENOMEM, "spz_buffer_push_async: device staging");
    CK(hipEventCreateWithFlags(&sl.copied, hipEventDisableTiming));
    CK(hipEventCreateWithFlags(&sl.done, hipEventDisableTiming));
  }
  CK(hipStreamCreateWithFlags(&c->si, hipStreamNonBlocking));
  return SPZ_OK;
}
}  // namespace

int spz_buffer_push_async(spz_ctx* c, const float* obs, const float* act, const float* rew, const float* done,
                          const float* next_obs, int64_t n) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_buffer_push_async: NULL context");
  if (n < 0) return set_err(c, SPZ_EINVAL, "spz_buffer_push_async: n < 0");
  if (n == 0) return SPZ_OK;
  if (!obs || !act || !rew || !done || !next_obs)
    return set_err(c, SPZ_EINVAL, "spz_buffer_push_async: NULL array");
  CK(hipSetDevice(c->hp.device));
  int rc = ingest_init(c);
  if (rc) return rc;
  // Commits go to the stream updates are enqueued on, so they take effect between
  // the steps enqueued before this call and those enqueued after it.
  hipStream_t su = c->has_last ? c->last : c->sc;
  const int64_t CH = INGEST_ROWS;
  const int64_t skip = n > c->cap ? n - c->cap : 0;
  for (int64_t r0 = skip; r0 < n; r0 += CH) {
    const int64_t m = std::min(CH, n - r0);
    auto& sl = c->slots[c->next_slot];
    c->next_slot = (c->next_slot + 1) % INGEST_SLOTS;
    if (sl.used) CK(hipEventSynchronize(sl.done));   // the slot's previous rows are in the ring
    float* ho = sl.host;
    float* ha = ho + CH * c->O;
    float* hr = ha + CH * c->A;
    float* hd = hr + CH;
    float* hn = hd + CH;
    memcpy(ho, obs + r0 * c->O, (size_t)(m * c->O * 4));
    memcpy(ha, act + r0 * c->A, (size_t)(m * c->A * 4));
    memcpy(hr, rew + r0, (size_t)(m * 4));
    memcpy(hd, done + r0, (size_t)(m * 4));
    memcpy(hn, next_obs + r0 * c->O, (size_t)(m * c->O * 4));
    float* dob = sl.dev;
    float* dac = dob + CH * c->O;
    float* drw = dac + CH * c->A;
    float* ddn = drw + CH;
    float* dnx = ddn + CH;
    CK(hipMemcpyAsync(dob, ho, (size_t)(m * c->O * 4), hipMemcpyHostToDevice, c->si));
    CK(hipMemcpyAsync(dac, ha, (size_t)(m * c->A * 4), hipMemcpyHostToDevice, c->si));
    CK(hipMemcpyAsync(drw, hr, (size_t)(m * 4), hipMemcpyHostToDevice, c->si));
    CK(hipMemcpyAsync(ddn, hd, (size_t)(m * 4), hipMemcpyHostToDevice, c->si));
    CK(hipMemcpyAsync(dnx, hn, (size_t)(m * c->O * 4), hipMemcpyHostToDevice, c->si));
    CK(hipEventRecord(sl.copied, c->si));
    CK(hipStreamWaitEvent(su, sl.copied, 0));
    PackArgs p{c->buf, c->row_bytes, c->off_a, c->off_s2, c->off_r, c->off_d, c->O, c->A, m,
               (c->ptr + r0) % c->cap, c->cap, dob, dac, drw, ddn, dnx};
    CK(launch_pack(c->bf16, p, su));
    CK(hipEventRecord(sl.done, su));
    sl.used = true;
  }
  c->commit_stream = su;
  c->commits_pending = true;
  c->ptr = (c->ptr + n) % c->cap;
  c->size = std::min(c->size + n, c->cap);
  return SPZ_OK;
}

int spz_update(spz_ctx* c, int32_t n_steps, void* hip_stream) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_update: NULL context");
  if (n_steps < 0) return set_err(c, SPZ_EINVAL, "spz_update: n_steps < 0");
  if (c->size == 0) return set_err(c, SPZ_EEMPTY, "spz_update: replay buffer is empty");
  CK(hipSetDevice(c->hp.device));
  hipStream_t s0 = static_cast<hipStream_t>(hip_stream);
  // Steps enqueued earlier on another stream, and ring commits of asynchronous
  // pushes enqueued on another stream, come first.
  hipStream_t before[2] = {c->has_last && c->last != s0 ? c->last : s0,
                           c->commits_pending && c->commit_stream != s0 ? c->commit_stream : s0};
  for (int i = 0; i < 2; ++i)
    if (before[i] != s0 && (i == 0 || before[1] != before[0])) {
      CK(hipEventRecord(c->ev_commit, before[i]));
      CK(hipStreamWaitEvent(s0, c->ev_commit, 0));
    }
  c->commits_pending = false;
  c->last = s0;
  c->has_last = true;
  for (int i = 0; i < n_steps; ++i) {
    const int rc = c->hp.graphs && !c->prof ? graph_step(c, s0) : enqueue_step(c, s0);
    if (rc) return rc;
  }
  return SPZ_OK;
}

// ---------------------------------------------------------------------------- sampler actions
int spz_act(spz_ctx* c, const float* obs, int64_t n, int32_t stochastic, uint32_t counter, float* act) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_act: NULL context");
  if (n < 0 || (n > 0 && (!obs || !act))) return set_err(c, SPZ_EINVAL, "spz_act: bad arrays");
  if (stochastic && c->td3) return set_err(c, SPZ_EINVAL, "spz_act: TD3 policies are deterministic");
  if (n == 0) return SPZ_OK;
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  if (!c->stage) {
    CK(hipMalloc(&c->stage, (size_t)(65536 * (2 * (int64_t)c->O + c->A + 2) * 4)));
    c->stage_rows = 65536;
  }
  // Chunks of at most the created batch (the actor workspaces' row count) and of the
  // observation staging area.
  const int64_t chunk = std::min<int64_t>(c->Bpmax, c->stage_rows) / 256 * 256;
  const int saveB = c->B, saveBp = c->Bp;
  const int pa = c->net[0].L.back().out_p;
  hipStream_t s = c->sc;
  for (int64_t r0 = 0; r0 < n && rc == SPZ_OK; r0 += chunk) {
    const int m = (int)std::min(chunk, n - r0);
    const int rows = (m + 255) / 256 * 256;
    hipError_t e = hipMemcpy(c->stage, obs + r0 * c->O, (size_t)m * c->O * 4, hipMemcpyHostToDevice);
    ObsArgs oa{c->stage, m, rows, c->O, c->Ka, c->xsp, c->Kc};
    if (e == hipSuccess) e = launch_obs_operand(c->bf16, oa, s);
    c->B = m;
    c->Bp = rows;
    const NetOut out{c->ha.data(), nullptr, nullptr, c->z, nullptr};
    if (e == hipSuccess) e = forward(c, 0, 1, false, c->xsp, c->Kc, &out, true, s);
    c->B = saveB;
    c->Bp = saveBp;
    ActHeadArgs ha{c->z, pa, c->A, m, r0, c->td3 ? 0 : 1, stochastic ? 1 : 0, c->seed, counter,
                   c->hp.log_std_min, c->hp.log_std_max, c->th};
    if (e == hipSuccess) e = launch_act_head(ha, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e == hipSuccess) e = hipMemcpy(act + r0 * c->A, c->th, (size_t)m * c->A * 4, hipMemcpyDeviceToHost);
    if (e != hipSuccess) rc = set_err(c, SPZ_EHIP, std::string("spz_act: ") + hipGetErrorString(e));
  }
  return rc;
}

// ---------------------------------------------------------------------------- allocation-free actions
namespace {
inline size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Scratch layout of one spz_act_noalloc call over `rows` rows: observation operand
// [rows, Ka], two hidden-activation buffers [rows, hmax] (operand type), head output
// [rows, out_p] float32, each on a 256-byte boundary. Returns the bytes used.
size_t act_scratch_layout(const spz_ctx* c, int64_t rows, size_t off[4]) {
  const size_t e = es(c);
  const int pa = c->net[0].L.back().out_p;
  off[0] = 0;
  off[1] = align256(off[0] + (size_t)rows * c->Ka * e);
  off[2] = align256(off[1] + (size_t)rows * c->hmax * e);
  off[3] = align256(off[2] + (size_t)rows * c->hmax * e);
  return off[3] + (size_t)rows * pa * 4;
}

// Largest row count (a multiple of 256) whose layout fits the scratch array.
int64_t act_scratch_rows(const spz_ctx* c) {
  size_t off[4];
  int64_t lo = 0, hi = (int64_t)(ACT_SCRATCH_BYTES / 256) + 1;   // in units of 256 rows
  while (hi - lo > 1) {
    const int64_t mid = (lo + hi) / 2;
    if (act_scratch_layout(c, mid * 256, off) <= ACT_SCRATCH_BYTES) lo = mid;
    else hi = mid;
  }
  return lo * 256;
}
}  // namespace

int spz_act_noalloc(spz_ctx* c, const float* obs, int64_t n, int32_t stochastic, uint32_t counter, float* act,
                    void* hip_stream) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_act_noalloc: NULL context");
  if (n < 0 || (n > 0 && (!obs || !act))) return set_err(c, SPZ_EINVAL, "spz_act_noalloc: bad arrays");
  if (stochastic && c->td3) return set_err(c, SPZ_EINVAL, "spz_act_noalloc: TD3 policies are deterministic");
  const int64_t max_rows = act_scratch_rows(c);
  if (n > max_rows) {
    char msg[160];
    std::snprintf(msg, sizeof(msg), "spz_act_noalloc: %lld rows exceed the %lld rows this network fits in the %zu-byte scratch",
                  (long long)n, (long long)max_rows, ACT_SCRATCH_BYTES);
    return set_err(c, SPZ_EINVAL, msg);
  }
  if (n == 0) return SPZ_OK;
  CK(hipSetDevice(c->hp.device));
  uint8_t* base = static_cast<uint8_t*>(g_scratch_ptr[c->hp.device]);
  if (!base) return set_err(c, SPZ_EHIP, "spz_act_noalloc: scratch address not initialised");
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const int rows = (int)((n + 255) / 256 * 256);
  size_t off[4];
  act_scratch_layout(c, rows, off);
  void* xop = base + off[0];
  void* hid[8];
  for (int l = 0; l < 8; ++l) hid[l] = base + off[1 + (l & 1)];
  float* z = reinterpret_cast<float*>(base + off[3]);
  // Operand rows [n, rows) and columns [obs_dim, Ka) are written as zeros here: the
  // scratch keeps the previous call's contents.
  ObsArgs oa{obs, (int)n, rows, c->O, c->Ka, xop, c->Ka};
  CK(launch_obs_operand(c->bf16, oa, s));
  const int saveB = c->B, saveBp = c->Bp;
  const bool saveProf = c->prof;
  c->B = (int)n;
  c->Bp = rows;
  c->prof = false;
  const NetOut out{hid, nullptr, nullptr, z, nullptr};
  const hipError_t e = forward(c, 0, 1, false, xop, c->Ka, &out, true, s);
  c->B = saveB;
  c->Bp = saveBp;
  c->prof = saveProf;
  CK(e);
  const int pa = c->net[0].L.back().out_p;
  ActHeadArgs ha{z, pa, c->A, (int)n, 0, c->td3 ? 0 : 1, stochastic ? 1 : 0, c->seed, counter,
                 c->hp.log_std_min, c->hp.log_std_max, act};
  CK(launch_act_head(ha, s));
  return SPZ_OK;
}

// ---------------------------------------------------------------------------- checkpoints
namespace {

struct CkptHeader {
  char magic[8];
  uint32_t version, flags;
  int32_t O, A, n_hidden, hidden[8], algo, prec, pad_;
  int64_t capacity, n_arena, row_bytes, rec_cap;
  uint64_t seed;
  int64_t step, ring_ptr, ring_size;
};
constexpr char CKPT_MAGIC[8] = {'S', 'P', 'Z', 'C', 'K', 'P', 'T', '1'};
constexpr size_t CKPT_CHUNK = (size_t)64 << 20;

// Device <-> file through a host bounce buffer, in chunks.
static int dev_to_file(spz_ctx* c, FILE* f, const void* dev, size_t bytes, std::vector<uint8_t>& tmp) {
  for (size_t o = 0; o < bytes; o += CKPT_CHUNK) {
    const size_t n = std::min(CKPT_CHUNK, bytes - o);
    CK(hipMemcpy(tmp.data(), static_cast<const uint8_t*>(dev) + o, n, hipMemcpyDeviceToHost));
    if (fwrite(tmp.data(), 1, n, f) != n) return set_err(c, SPZ_EIO, "spz_save: write failed");
  }
  return SPZ_OK;
}
static int file_to_dev(spz_ctx* c, FILE* f, void* dev, size_t bytes, std::vector<uint8_t>& tmp) {
  for (size_t o = 0; o < bytes; o += CKPT_CHUNK) {
    const size_t n = std::min(CKPT_CHUNK, bytes - o);
    if (fread(tmp.data(), 1, n, f) != n) return set_err(c, SPZ_EIO, "spz_load: file truncated");
    CK(hipMemcpy(static_cast<uint8_t*>(dev) + o, tmp.data(), n, hipMemcpyHostToDevice));
  }
  return SPZ_OK;
}

static void fill_header(const spz_ctx* c, CkptHeader& h) {
  memset(&h, 0, sizeof(h));
  memcpy(h.magic, CKPT_MAGIC, 8);
  h.version = 1;
  h.O = c->O;
  h.A = c->A;
  h.n_hidden = (int32_t)c->hidden.size();
  for (size_t i = 0; i < c->hidden.size() && i < 8; ++i) h.hidden[i] = c->hidden[i];
  h.algo = c->hp.algo;
  h.prec = c->hp.gemm_prec;
  h.capacity = c->cap;
  h.n_arena = c->n_arena;
  h.row_bytes = c->row_bytes;
  h.rec_cap = c->rec_cap;
}

struct FileCloser {
  FILE* f;
  ~FileCloser() { if (f) fclose(f); }
};

}  // namespace

int spz_save(spz_ctx* c, const char* path, int32_t flags) {
  if (!c || !path) return set_err(c, SPZ_EINVAL, "spz_save: NULL argument");
  if (flags & ~SPZ_CKPT_RING) return set_err(c, SPZ_EINVAL, "spz_save: unknown flags");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  CkptHeader h;
  fill_header(c, h);
  h.flags = (uint32_t)flags;
  h.seed = c->seed;
  h.step = c->h_step;
  h.ring_ptr = c->ptr;
  h.ring_size = c->size;
  FileCloser fc{fopen(path, "wb")};
  if (!fc.f) return set_err(c, SPZ_EIO, std::string("spz_save: cannot open ") + path);
  if (fwrite(&h, sizeof(h), 1, fc.f) != 1) return set_err(c, SPZ_EIO, "spz_save: write failed");
  std::vector<uint8_t> tmp;
  try { tmp.resize(CKPT_CHUNK); } catch (...) { return set_err(c, SPZ_ENOMEM, "spz_save: host buffer"); }
  const size_t ab = (size_t)c->n_arena * 4;
  for (const float* a : {c->P, c->T, c->M, c->V})
    if ((rc = dev_to_file(c, fc.f, a, ab, tmp))) return rc;
  if ((rc = dev_to_file(c, fc.f, c->rec, (size_t)c->rec_cap * SPZ_REC_WIDTH * 4, tmp))) return rc;
  if (flags & SPZ_CKPT_RING)
    if ((rc = dev_to_file(c, fc.f, c->buf, (size_t)(c->row_bytes * c->cap), tmp))) return rc;
  if (fflush(fc.f) != 0) return set_err(c, SPZ_EIO, "spz_save: flush failed");
  return SPZ_OK;
}

int spz_load(spz_ctx* c, const char* path) {
  if (!c || !path) return set_err(c, SPZ_EINVAL, "spz_load: NULL argument");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  FileCloser fc{fopen(path, "rb")};
  if (!fc.f) return set_err(c, SPZ_EIO, std::string("spz_load: cannot open ") + path);
  CkptHeader h, mine;
  if (fread(&h, sizeof(h), 1, fc.f) != 1 || memcmp(h.magic, CKPT_MAGIC, 8) || h.version != 1)
    return set_err(c, SPZ_EIO, "spz_load: not a checkpoint of this library");
  fill_header(c, mine);
  const bool ring = h.flags & SPZ_CKPT_RING;
  if (h.O != mine.O || h.A != mine.A || h.n_hidden != mine.n_hidden ||
      memcmp(h.hidden, mine.hidden, sizeof(h.hidden)) || h.algo != mine.algo || h.prec != mine.prec ||
      h.n_arena != mine.n_arena || h.rec_cap != mine.rec_cap ||
      (ring && (h.capacity != mine.capacity || h.row_bytes != mine.row_bytes)) || h.step < 0 ||
      h.ring_size < 0 || h.ring_size > h.capacity || h.ring_ptr < 0 || h.ring_ptr >= std::max<int64_t>(h.capacity, 1))
    return set_err(c, SPZ_EIO, "spz_load: checkpoint does not match this learner's configuration");
  std::vector<uint8_t> tmp;
  try { tmp.resize(CKPT_CHUNK); } catch (...) { return set_err(c, SPZ_ENOMEM, "spz_load: host buffer"); }
  const size_t ab = (size_t)c->n_arena * 4;
  for (float* a : {c->P, c->T, c->M, c->V})
    if ((rc = file_to_dev(c, fc.f, a, ab, tmp))) return rc;
  if ((rc = file_to_dev(c, fc.f, c->rec, (size_t)c->rec_cap * SPZ_REC_WIDTH * 4, tmp))) return rc;
  if (ring) {
    if ((rc = file_to_dev(c, fc.f, c->buf, (size_t)(c->row_bytes * c->cap), tmp))) return rc;
    c->ptr = h.ring_ptr;
    c->size = h.ring_size;
  }
  // The bf16 operand images are a pure function of the float32 parameters.
  if (c->bf16) {
    CK(launch_to_bf16(c->P, c->Pb, c->n_arena, c->sc));
    CK(launch_to_bf16(c->T, c->Tb, c->n_arena, c->sc));
    CK(refresh_wt(c, c->sc));
    CK(hipStreamSynchronize(c->sc));
  }
  c->seed = h.seed;
  CK(hipMemcpy(c->d_step, &h.step, 8, hipMemcpyHostToDevice));
  c->h_step = h.step;
  return SPZ_OK;
}

int spz_set_batch(spz_ctx* c, int32_t batch) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_set_batch: NULL context");
  if (batch < 1 || batch > c->Bmax) return set_err(c, SPZ_EINVAL, "spz_set_batch: batch out of [1, created batch]");
  const int Bp = (batch + 255) / 256 * 256;
  for (int q = 0; q < 2; ++q)
    if (red_need(c, q, Bp) > c->red[q].cap)
      return set_err(c, SPZ_EINVAL, "spz_set_batch: reduction workspace too small for this batch");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  // Rows [batch, Bp) of the batch operands and of the actor head gradient must be
  // zero (pad rows carry no gradient); a larger earlier batch may have left data there.
  if (Bp > batch) {
    const size_t e = es(c);
    const size_t pad = (size_t)(Bp - batch);
    for (void* x : {c->xsa, c->xs2, c->xsp})
      CK(hipMemset(static_cast<uint8_t*>(x) + (size_t)batch * c->Kc * e, 0, pad * c->Kc * e));
    const int pa = c->net[0].L.back().out_p;
    CK(hipMemset(static_cast<uint8_t*>(c->dzh) + (size_t)batch * pa * e, 0, pad * pa * e));
  }
  c->B = batch;
  c->Bp = Bp;
  return SPZ_OK;
}

int32_t spz_batch(const spz_ctx* c) { return c ? c->B : SPZ_EINVAL; }

int spz_autotune_batch(spz_ctx* c, int32_t b_min, int32_t probe_steps, float tolerance, void* hip_stream,
                       int32_t* chosen, int32_t* batches, float* frames_per_s, int32_t max_probes,
                       int32_t* n_probes) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_autotune_batch: NULL context");
  if (b_min < 1 || b_min > c->Bmax || probe_steps < 1 || !(tolerance >= 0.0f && tolerance < 1.0f) || !chosen ||
      max_probes < 0 || (max_probes > 0 && (!batches || !frames_per_s)))
    return set_err(c, SPZ_EINVAL, "spz_autotune_batch: invalid arguments");
  if (c->size == 0) return set_err(c, SPZ_EEMPTY, "spz_autotune_batch: replay buffer is empty");
  CK(hipSetDevice(c->hp.device));
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  CK(hipEventCreate(&e0));
  if (hipEventCreate(&e1) != hipSuccess) {
    (void)hipEventDestroy(e0);
    return set_err(c, SPZ_EHIP, "spz_autotune_batch: hipEventCreate failed");
  }
  std::vector<std::pair<int, double>> probes;
  int rc = SPZ_OK;
  double best = 0.0;
  for (int64_t b = b_min;; b *= 2) {
    const int bb = (int)std::min<int64_t>(b, c->Bmax);
    if ((rc = spz_set_batch(c, bb))) break;
    // one untimed step at the new size (first launches of new kernel shapes), then the probe
    if ((rc = spz_update(c, 1, s))) break;
    if (hipEventRecord(e0, s) != hipSuccess) { rc = set_err(c, SPZ_EHIP, "spz_autotune_batch: event"); break; }
    if ((rc = spz_update(c, probe_steps, s))) break;
    float ms = 0.0f;
    if (hipEventRecord(e1, s) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
        hipEventElapsedTime(&ms, e0, e1) != hipSuccess) {
      rc = set_err(c, SPZ_EHIP, "spz_autotune_batch: event timing failed");
      break;
    }
    const double rate = (double)bb * probe_steps / (ms * 1e-3);
    probes.emplace_back(bb, rate);
    // The frame rate is concave in the batch size: once doubling it gains less than
    // the tolerance, larger batches only lower the update frequency.
    const bool saturated = best > 0.0 && rate < best * (1.0 + tolerance);
    best = std::max(best, rate);
    if (saturated || bb == c->Bmax) break;
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (rc) return rc;
  int pick = probes.back().first;
  for (const auto& pr : probes)
    if (pr.second >= best * (1.0 - tolerance)) { pick = pr.first; break; }
  const int n = (int)probes.size();
  for (int i = 0; i < n && i < max_probes; ++i) {
    batches[i] = probes[i].first;
    frames_per_s[i] = (float)probes[i].second;
  }
  if (n_probes) *n_probes = n;
  *chosen = pick;
  return spz_set_batch(c, pick);
}

int spz_synchronize(spz_ctx* c) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_synchronize: NULL context");
  CK(hipSetDevice(c->hp.device));
  return ctx_sync(c);
}

int64_t spz_step(const spz_ctx* c) { return c ? c->h_step : SPZ_EINVAL; }

int spz_set_step(spz_ctx* c, int64_t step) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_set_step: NULL context");
  if (step < 0) return set_err(c, SPZ_EINVAL, "spz_set_step: step < 0");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  CK(hipMemcpy(c->d_step, &step, 8, hipMemcpyHostToDevice));
  c->h_step = step;
  return SPZ_OK;
}

int64_t spz_param_count(const spz_ctx* c, int32_t which) {
  if (!c) return SPZ_EINVAL;
  float* arena = nullptr;
  int ni = 0;
  if (resolve(c, which, &arena, &ni)) return SPZ_EINVAL;
  return ni < 0 ? 1 : flat_count(c->net[ni]);
}

int spz_read_params(spz_ctx* c, int32_t which, float* out, int64_t n_floats) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_read_params: NULL context");
  float* arena = nullptr;
  int ni = 0;
  if (resolve(c, which, &arena, &ni)) return set_err(c, SPZ_EINVAL, "spz_read_params: bad selector");
  const int64_t cnt = ni < 0 ? 1 : flat_count(c->net[ni]);
  if (n_floats != cnt) return set_err(c, SPZ_ESIZE, "spz_read_params: size mismatch");
  if (!out) return set_err(c, SPZ_EINVAL, "spz_read_params: NULL out");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  if (ni < 0) {
    CK(hipMemcpy(out, arena + c->la, 4, hipMemcpyDeviceToHost));
    return SPZ_OK;
  }
  const Net& n = c->net[ni];
  std::vector<float> img((size_t)(n.end - n.off));
  CK(hipMemcpy(img.data(), arena + n.off, img.size() * 4, hipMemcpyDeviceToHost));
  int64_t o = 0;
  for (int l = 0; l < (int)n.L.size(); ++l) {
    const Lay& L = n.L[l];
    for (int r = 0; r < L.out_f; ++r)
      for (int i = 0; i < L.in_f; ++i) out[o++] = img[L.w - n.off + (int64_t)r * L.in_p + pcol(c, ni, l, i)];
    for (int r = 0; r < L.out_f; ++r) out[o++] = img[L.b - n.off + r];
  }
  return SPZ_OK;
}

int spz_write_params(spz_ctx* c, int32_t which, const float* in, int64_t n_floats) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_write_params: NULL context");
  float* arena = nullptr;
  int ni = 0;
  if (which >= SPZ_G_ACTOR || resolve(c, which, &arena, &ni))
    return set_err(c, SPZ_EINVAL, "spz_write_params: bad selector");
  const int64_t cnt = ni < 0 ? 1 : flat_count(c->net[ni]);
  if (n_floats != cnt) return set_err(c, SPZ_ESIZE, "spz_write_params: size mismatch");
  if (!in) return set_err(c, SPZ_EINVAL, "spz_write_params: NULL input");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  if (ni < 0) {
    CK(hipMemcpy(arena + c->la, in, 4, hipMemcpyHostToDevice));
    return SPZ_OK;
  }
  const Net& n = c->net[ni];
  std::vector<float> img((size_t)(n.end - n.off), 0.0f);
  int64_t o = 0;
  for (int l = 0; l < (int)n.L.size(); ++l) {
    const Lay& L = n.L[l];
    for (int r = 0; r < L.out_f; ++r)
      for (int i = 0; i < L.in_f; ++i) img[L.w - n.off + (int64_t)r * L.in_p + pcol(c, ni, l, i)] = in[o++];
    for (int r = 0; r < L.out_f; ++r) img[L.b - n.off + r] = in[o++];
  }
  CK(hipMemcpy(arena + n.off, img.data(), img.size() * 4, hipMemcpyHostToDevice));
  if (c->bf16 && (arena == c->P || arena == c->T)) {
    bf16_t* sh = arena == c->P ? c->Pb : c->Tb;
    CK(launch_to_bf16(arena + n.off, sh + n.off, n.end - n.off, c->sc));
    if (arena == c->P) CK(refresh_wt(c, c->sc));
    CK(hipStreamSynchronize(c->sc));
  }
  return SPZ_OK;
}

int spz_read_losses(spz_ctx* c, float* out, int64_t first_step, int32_t n) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_read_losses: NULL context");
  if (n < 0 || first_step < 1 || first_step + n - 1 > c->h_step || first_step <= c->h_step - c->rec_cap)
    return set_err(c, SPZ_EINVAL, "spz_read_losses: steps not available");
  if (n == 0) return SPZ_OK;
  if (!out) return set_err(c, SPZ_EINVAL, "spz_read_losses: NULL out");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  for (int i = 0; i < n; ++i) {
    const int64_t slot = (first_step - 1 + i) % c->rec_cap;
    CK(hipMemcpy(out + (int64_t)i * SPZ_REC_WIDTH, c->rec + slot * SPZ_REC_WIDTH, SPZ_REC_WIDTH * 4,
                 hipMemcpyDeviceToHost));
  }
  return SPZ_OK;
}

int spz_debug_read(spz_ctx* c, int32_t what, void* out, int64_t bytes) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_debug_read: NULL context");
  const int64_t B = c->B;
  int64_t need = 0;
  switch (what) {
    case SPZ_DBG_INDICES: case SPZ_DBG_TD_TARGET: need = B * 4; break;
    case SPZ_DBG_Q: case SPZ_DBG_QPI: need = 2 * B * 4; break;
    case SPZ_DBG_LOGPI:
      if (c->td3) return set_err(c, SPZ_EINVAL, "spz_debug_read: no log pi in TD3");
      need = B * 4;
      break;
    case SPZ_DBG_DACTION: need = B * c->A * 4; break;
    case SPZ_DBG_BATCH: need = B * (2 * (int64_t)c->O + c->A + 2) * 4; break;
    default: return set_err(c, SPZ_EINVAL, "spz_debug_read: bad selector");
  }
  if (bytes != need) return set_err(c, SPZ_ESIZE, "spz_debug_read: size mismatch");
  if (!out) return set_err(c, SPZ_EINVAL, "spz_debug_read: NULL out");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  float* f = static_cast<float*>(out);
  switch (what) {
    case SPZ_DBG_INDICES: CK(hipMemcpy(out, c->idx, (size_t)bytes, hipMemcpyDeviceToHost)); break;
    case SPZ_DBG_TD_TARGET: CK(hipMemcpy(f, c->y, B * 4, hipMemcpyDeviceToHost)); break;
    case SPZ_DBG_Q:
      CK(hipMemcpy(f, c->q1, B * 4, hipMemcpyDeviceToHost));
      CK(hipMemcpy(f + B, c->q2, B * 4, hipMemcpyDeviceToHost));
      break;
    case SPZ_DBG_QPI:
      CK(hipMemcpy(f, c->qp1, B * 4, hipMemcpyDeviceToHost));
      CK(hipMemcpy(f + B, c->td3 ? c->qp1 : c->qp2, B * 4, hipMemcpyDeviceToHost));
      break;
    case SPZ_DBG_LOGPI: CK(hipMemcpy(f, c->logp, B * 4, hipMemcpyDeviceToHost)); break;
    case SPZ_DBG_BATCH: {
      // s from xsa, s' from xs2 (their first O columns), the actions from xsa's action
      // columns where the step ran on two streams (the actor part had its own operand)
      // and from the gather's copy otherwise, r and d from the arrays the TD target reads.
      const bool two = c->hp.n_streams == 2 && c->hp.ordering != SPZ_ORDER_SEQUENTIAL;
      const size_t e = es(c);
      std::vector<uint8_t> xa((size_t)B * c->Kc * e), x2((size_t)B * c->Kc * e), ab((size_t)B * c->A * e);
      std::vector<float> rr(B), dd(B);
      CK(hipMemcpy(xa.data(), c->xsa, xa.size(), hipMemcpyDeviceToHost));
      CK(hipMemcpy(x2.data(), c->xs2, x2.size(), hipMemcpyDeviceToHost));
      if (!two) CK(hipMemcpy(ab.data(), c->abuf, ab.size(), hipMemcpyDeviceToHost));
      CK(hipMemcpy(rr.data(), c->r, B * 4, hipMemcpyDeviceToHost));
      CK(hipMemcpy(dd.data(), c->d, B * 4, hipMemcpyDeviceToHost));
      auto val = [&](const std::vector<uint8_t>& v, int64_t i) {
        if (c->bf16) return bf2f(reinterpret_cast<const bf16_t*>(v.data())[i]);
        return reinterpret_cast<const float*>(v.data())[i];
      };
      const int64_t w = 2 * (int64_t)c->O + c->A + 2;
      for (int64_t b = 0; b < B; ++b) {
        float* o = f + b * w;
        for (int j = 0; j < c->O; ++j) {
          o[j] = val(xa, b * c->Kc + j);
          o[c->O + c->A + j] = val(x2, b * c->Kc + j);
        }
        for (int j = 0; j < c->A; ++j) o[c->O + j] = two ? val(xa, b * c->Kc + c->Ka + j) : val(ab, b * c->A + j);
        o[w - 2] = rr[b];
        o[w - 1] = dd[b];
      }
      break;
    }
    case SPZ_DBG_DACTION: {
      // da1 [Bp, Ap] holds the whole gradient under the SAC row split (and for TD3);
      // otherwise critic 2's part is in da2.
      const bool two = !c->td3 && !c->row_split;
      std::vector<float> d1((size_t)B * c->Ap), d2(two ? (size_t)B * c->Ap : 0);
      CK(hipMemcpy(d1.data(), c->da1, d1.size() * 4, hipMemcpyDeviceToHost));
      if (two) CK(hipMemcpy(d2.data(), c->da2, d2.size() * 4, hipMemcpyDeviceToHost));
      for (int64_t b = 0; b < B; ++b)
        for (int j = 0; j < c->A; ++j)
          f[b * c->A + j] = d1[b * c->Ap + j] + (two ? d2[b * c->Ap + j] : 0.0f);
      break;
    }
  }
  return SPZ_OK;
}

int spz_profile_enable(spz_ctx* c, int32_t on, int64_t reserve_launches) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_profile_enable: NULL context");
  if (reserve_launches < 0) return set_err(c, SPZ_EINVAL, "spz_profile_enable: reserve < 0");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  for (auto& pe : c->pevs) {
    c->pool.push_back(pe.a);
    c->pool.push_back(pe.b);
  }
  c->pevs.clear();
  c->pkeys.clear();
  c->prof = on != 0;
  if (c->prof) {
    while ((int64_t)c->pool.size() < 2 * reserve_launches) {
      hipEvent_t e;
      CK(hipEventCreate(&e));
      c->pool.push_back(e);
    }
    c->pevs.reserve((size_t)reserve_launches);
  }
  return SPZ_OK;
}

int spz_profile_stride(spz_ctx* c, int32_t stride) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_profile_stride: NULL context");
  if (stride < 1) return set_err(c, SPZ_EINVAL, "spz_profile_stride: stride < 1");
  c->pf_stride = stride;
  return SPZ_OK;
}

int spz_profile_only(spz_ctx* c, const char* name, int32_t M, int32_t N, int32_t K) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_profile_only: NULL context");
  c->pf_on = name != nullptr;
  c->pf_name = name ? name : "";
  c->pf_M = M;
  c->pf_N = N;
  c->pf_K = K;
  return SPZ_OK;
}

int spz_profile_read(spz_ctx* c, spz_kernel_stat* out, int32_t max, int32_t* n_out) {
  if (!c) return set_err(nullptr, SPZ_EINVAL, "spz_profile_read: NULL context");
  if (max < 0 || (max > 0 && !out) || !n_out) return set_err(c, SPZ_EINVAL, "spz_profile_read: bad output");
  CK(hipSetDevice(c->hp.device));
  int rc = ctx_sync(c);
  if (rc) return rc;
  for (auto& pe : c->pevs) {
    float ms = 0.0f;
    CK(hipEventElapsedTime(&ms, pe.a, pe.b));
    c->pkeys[pe.key].ms += ms;
    c->pkeys[pe.key].launches += 1;
    c->pool.push_back(pe.a);
    c->pool.push_back(pe.b);
  }
  c->pevs.clear();
  std::vector<int> order(c->pkeys.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = (int)i;
  std::sort(order.begin(), order.end(), [&](int a, int b) { return c->pkeys[a].ms > c->pkeys[b].ms; });
  const int n = std::min<int>(max, (int)order.size());
  for (int i = 0; i < n; ++i) {
    const auto& k = c->pkeys[order[i]];
    spz_kernel_stat& o = out[i];
    std::memset(&o, 0, sizeof(o));
    std::snprintf(o.name, sizeof(o.name), "%s", k.name.c_str());
    o.M = k.M;
    o.N = k.N;
    o.K = k.K;
    o.bf16 = c->bf16 ? 1 : 0;
    o.launches = k.launches;
    o.total_ms = k.ms;
    o.flops = k.flops;
    o.bytes = k.bytes;
  }
  *n_out = (int32_t)order.size();
  return SPZ_OK;
}

const char* spz_last_error(const spz_ctx* c) { return c ? c->err.c_str() : tl_err.c_str(); }

}  // extern "C"
