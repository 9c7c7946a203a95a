// Elementwise, row and reduction kernels of the update step (everything that is
// not a matrix product): replay sampling and gather, policy heads, twin-Q / TD
// target / losses, critic output head, bias-gradient column sums, the fused
// Adam + Polyak pass and the per-step finish (loss record, temperature gradient,
// step counter).
//
// Reductions are deterministic: fixed per-thread order, fixed tree inside a
// block, partials reduced in index order by a second pass. No atomics.
#include "kernels.h"

namespace spz {
namespace {

// Minimum that keeps a NaN operand (fminf would drop it), like clamp_keep_nan.
__device__ inline float min_keep_nan(float a, float b) { return (a < b || a != a) ? a : b; }

template <int NT>
__device__ inline double block_sum(double v, double* sh) {
  const int t = threadIdx.x;
  sh[t] = v;
  __syncthreads();
#pragma unroll
  for (int s = NT / 2; s > 0; s >>= 1) {
    if (t < s) sh[t] += sh[t + s];
    __syncthreads();
  }
  const double r = sh[0];
  __syncthreads();
  return r;
}

// Sum of an int over a 256-thread block (4 waves of 64 lanes).
__device__ inline int block_sum_i32(int v, int* sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
  __syncthreads();
  const int r = sh[0] + sh[1] + sh[2] + sh[3];
  __syncthreads();
  return r;
}

// ------------------------------------------------------------------------------ replay
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Elements of a segment past its whole 16-byte pieces.
template <typename T>
__device__ inline void copy_tail(uint8_t* dst, const uint8_t* src, int bytes, int lane) {
  for (int e = ((bytes >> 4) << 4) / (int)sizeof(T) + lane; e < bytes / (int)sizeof(T); e += 64)
    reinterpret_cast<T*>(dst)[e] = reinterpret_cast<const T*>(src)[e];
}

// One wave per batch row. The ring row is read once: each lane loads its 16-byte
// pieces of s, s' and a before any store, then s goes to both critic operands (and to
// the actor part's own copy when there is one). (Non-temporal loads of data the previous kernel wrote gave wrong sums in
// the column-sum kernel, so loads here stay plain.)
template <typename T>
__global__ void __launch_bounds__(256) k_gather(GatherArgs g) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= g.B) return;
  const uint32_t t = (uint32_t)(*g.step + 1);
  const uint32_t w = philox_word(g.seed, (uint64_t)b, t, P_IDX, 0u);
  const uint32_t row = mulhi32(w, g.size);
  const uint8_t* src = g.buf + (int64_t)row * g.row_bytes;
  const int64_t xrow = (int64_t)b * g.Kc * (int64_t)sizeof(T);
  uint8_t* xsa = static_cast<uint8_t*>(g.xsa) + xrow;
  uint8_t* xsp = g.xsp ? static_cast<uint8_t*>(g.xsp) + xrow : nullptr;
  uint8_t* xs2 = static_cast<uint8_t*>(g.xs2) + xrow;
  const int sb = g.O * (int)sizeof(T), ab = g.A * (int)sizeof(T);
  const int ns = sb >> 4, na = ab >> 4;
  const u32x4* __restrict__ s_in = reinterpret_cast<const u32x4*>(src);
  const u32x4* __restrict__ s2_in = reinterpret_cast<const u32x4*>(src + g.off_s2);
  const u32x4* __restrict__ a_in = reinterpret_cast<const u32x4*>(src + g.off_a);
  u32x4* __restrict__ xsa4 = reinterpret_cast<u32x4*>(xsa);
  u32x4* __restrict__ xsp4 = reinterpret_cast<u32x4*>(xsp);
  u32x4* __restrict__ xs24 = reinterpret_cast<u32x4*>(xs2);
  u32x4* __restrict__ xa4 = reinterpret_cast<u32x4*>(xsa + g.Ka * (int)sizeof(T));
  float rv = 0.0f, dv = 0.0f;
  if (lane == 0) {
    rv = *reinterpret_cast<const float*>(src + g.off_r);
    dv = *reinterpret_cast<const float*>(src + g.off_d);
  }
  const int nmax = ns > na ? ns : na;
  for (int v = lane; v < nmax; v += 64) {
    u32x4 x = {0u, 0u, 0u, 0u}, y = x, z = x;
    if (v < ns) {
      x = s_in[v];
      y = s2_in[v];
    }
    if (v < na) z = a_in[v];
    if (v < ns) {
      xsa4[v] = x;
      if (xsp4) xsp4[v] = x;
      xs24[v] = y;
    }
    if (v < na) xa4[v] = z;
  }
  copy_tail<T>(xsa, src, sb, lane);
  if (g.xsp) copy_tail<T>(xsp, src, sb, lane);
  copy_tail<T>(xs2, src + g.off_s2, sb, lane);
  copy_tail<T>(xsa + g.Ka * (int)sizeof(T), src + g.off_a, ab, lane);
  if (g.abuf) {
    const T* a_src = reinterpret_cast<const T*>(src + g.off_a);
    for (int j = lane; j < g.A; j += 64) static_cast<T*>(g.abuf)[(int64_t)b * g.A + j] = a_src[j];
  }
  if (lane == 0) {
    g.r[b] = rv;
    g.d[b] = dv;
    g.idx[b] = (int32_t)row;
  }
}

template <typename T>
__global__ void __launch_bounds__(256) k_pack_rows(PackArgs p) {
  const int lane = threadIdx.x & 63;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= p.n) return;
  const int64_t slot = (p.ptr + i) % p.capacity;
  uint8_t* dst = p.buf + slot * p.row_bytes;
  T* s = reinterpret_cast<T*>(dst);
  T* a = reinterpret_cast<T*>(dst + p.off_a);
  T* s2 = reinterpret_cast<T*>(dst + p.off_s2);
  for (int j = lane; j < p.O; j += 64) {
    s[j] = from_f<T>(p.obs[i * p.O + j]);
    s2[j] = from_f<T>(p.nobs[i * p.O + j]);
  }
  for (int j = lane; j < p.A; j += 64) a[j] = from_f<T>(p.act[i * p.A + j]);
  if (lane == 0) {
    *reinterpret_cast<float*>(dst + p.off_r) = p.rew[i];
    *reinterpret_cast<float*>(dst + p.off_d) = p.done[i];
  }
}

// ------------------------------------------------------------------------------ heads
// SAC head (sac_head_element) on a stored z, where the head product could not take it in
// its epilogue. One thread per (row, action) element, so that loads and stores of
// consecutive threads are contiguous; a block covers HEAD_ROWS rows and adds each row's
// per-action terms in action order through LDS.
constexpr int HEAD_ROWS = 64;
template <typename T>
__global__ void __launch_bounds__(256) k_sac_head(SacHeadArgs h) {
  extern __shared__ float lterm[];   // [HEAD_ROWS][A]
  const int r0 = blockIdx.x * HEAD_ROWS;
  const int rows = min(HEAD_ROWS, h.B - r0);
  const int n = rows * h.A;
  const uint32_t t = (uint32_t)(*h.step + 1);
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    const int r = e / h.A, j = e - r * h.A;
    const int b = r0 + r;
    const float* z = h.z + (int64_t)b * h.ldz;
    lterm[e] = sac_head_element<T>(h, z[j], z[h.A + j], b, j, normal_at(h.seed, (uint64_t)b * h.A + j, t, h.purpose));
  }
  __syncthreads();
  if ((int)threadIdx.x < rows) {
    float lp = 0.0f;
    for (int j = 0; j < h.A; ++j) lp += lterm[threadIdx.x * h.A + j];
    h.logp[r0 + threadIdx.x] = lp;
  }
}

// TD3 heads. Target: a' = clip(tanh z + clip(noise * eps, -c, c), -1, 1). Policy: a = tanh z.
// One thread per (row, action) element.
template <typename T>
__global__ void __launch_bounds__(256) k_td3_head(Td3HeadArgs h) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)h.B * h.A) return;
  const int b = (int)(e / h.A), j = (int)(e - (int64_t)b * h.A);
  const uint32_t t = (uint32_t)(*h.step + 1);
  float a = tanhf(h.z[(int64_t)b * h.ldz + j]);
  if (h.smooth) {
    const float eps = normal_at(h.seed, (uint64_t)e, t, P_NOISE_TGT);
    const float nz = clamp_keep_nan(h.noise * eps, -h.clip, h.clip);
    a = clamp_keep_nan(a + nz, -1.0f, 1.0f);
  }
  static_cast<T*>(h.x)[(int64_t)b * h.ldx + h.xoff + j] = from_f<T>(a);
  if (h.th) h.th[e] = a;
}

// 16-byte vector of operand values and its float image.
template <typename T> struct Vec16;
template <> struct Vec16<float> {
  static constexpr int N = 4;
  __device__ static inline void load(const float* p, float* o) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
  }
  __device__ static inline void store(float* p, const float* o) {
    *reinterpret_cast<float4*>(p) = make_float4(o[0], o[1], o[2], o[3]);
  }
};
template <> struct Vec16<bf16_t> {
  static constexpr int N = 8;
  __device__ static inline void load(const bf16_t* p, float* o) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = bf2f((bf16_t)(w[i] & 0xFFFFu));
      o[2 * i + 1] = bf2f((bf16_t)(w[i] >> 16));
    }
  }
  __device__ static inline void store(bf16_t* p, const float* o) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = (uint32_t)f2bf(o[2 * i]) | ((uint32_t)f2bf(o[2 * i + 1]) << 16);
    *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

// Critic output layer (width 1): q[b] = sum_k H[b, k] w[k] + bias. One wave per row,
// 16 bytes per lane; fixed per-lane order, then a fixed butterfly.
template <typename T>
__global__ void __launch_bounds__(256) k_rowdot(RowdotArgs r) {
  using V = Vec16<T>;
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= r.rows) return;
  const T* h = static_cast<const T*>(r.H) + (int64_t)b * r.ld;
  const T* w = static_cast<const T*>(r.w);
  float s = 0.0f;
  for (int k = lane * V::N; k < r.K; k += 64 * V::N) {
    float hv[V::N], wv[V::N];
    V::load(h + k, hv);
    V::load(w + k, wv);
#pragma unroll
    for (int i = 0; i < V::N; ++i) s = fmaf(hv[i], wv[i], s);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if (lane == 0) r.q[b] = s + *r.bias;
}

// Critic output layer backward: dH[b, k] = rnd(dq[b]) * w[k] * (H[b, k] > 0), stored
// in the operand type, 16 bytes per thread. Pad rows have dq = 0 and pad columns w = 0.
template <typename T>
__global__ void __launch_bounds__(256) k_head_bwd(HeadBwdArgs a) {
  using V = Vec16<T>;
  const int kv = a.K / V::N;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)a.rows * kv) return;
  const int b = (int)(i / kv), k = (int)(i % kv) * V::N;
  const float dq = to_f<T>(from_f<T>(a.dq[b]));
  float hv[V::N], wv[V::N], o[V::N];
  V::load(static_cast<const T*>(a.H) + (int64_t)b * a.ld + k, hv);
  V::load(static_cast<const T*>(a.w) + k, wv);
#pragma unroll
  for (int j = 0; j < V::N; ++j) o[j] = hv[j] > 0.0f ? dq * wv[j] : 0.0f;
  V::store(static_cast<T*>(a.dH) + (int64_t)b * a.ld + k, o);
}

// The same with the mask read from bits. A block covers HB_ROWS rows: their words
// (K / 32 per row, stored row-contiguously per 32-column block) are staged in LDS
// with coalesced loads; thread t writes the 16-byte pieces of column group t % kv
// (kv = K / 8) in rows t / kv, t / kv + rpi, ... (rpi = 256 / kv). With colpart,
// the column sums of the stored (rounded) values over the block's rows go to
// colpart[block, :]: per thread over its rows, then over the rpi threads of a
// column group in order. With wpart, the output layer's weight-gradient sums of the
// block's rows are taken the same way from H, read in the same pass.
constexpr int HB_ROWS = 64;
__global__ void __launch_bounds__(256) k_head_bwd_bits(HeadBwdArgs a) {
  extern __shared__ uint32_t wsh[];   // [K / 32][HB_ROWS], then [rpi][K] floats for the sums
  __shared__ int src_row[HB_ROWS];    // product row of each dH row of the block, -1: zero row
  __shared__ float dq_row[HB_ROWS];   // rnd(dq) of each row
  const int nw = a.K / 32, kv = a.K / 8, rpi = 256 / kv;
  const int r0 = blockIdx.x * HB_ROWS;
  const int rows = a.m_dyn ? min(a.rows, *a.m_dyn) : a.rows;
  if (r0 >= rows) return;
  if (threadIdx.x < HB_ROWS) {
    const int b = r0 + threadIdx.x;
    const int src = b < rows ? (a.map ? a.map[b] : b) : -1;
    src_row[threadIdx.x] = src;
    dq_row[threadIdx.x] = src >= 0 ? bf2f(f2bf(a.dq[src])) : 0.0f;
  }
  __syncthreads();
  for (int t = threadIdx.x; t < nw * HB_ROWS; t += blockDim.x) {
    const int wc = t / HB_ROWS, src = src_row[t % HB_ROWS];
    wsh[t] = src >= 0 ? a.bits[(int64_t)wc * a.ldbits + src] : 0u;
  }
  __syncthreads();
  const bf16_t* w = static_cast<const bf16_t*>(a.w);
  const int cg = threadIdx.x % kv, rs = threadIdx.x / kv, k = cg * 8;
  float cs[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  float ws[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  if (rs < rpi) {
    const uint4 w4 = *reinterpret_cast<const uint4*>(w + k);
    const uint32_t ww[4] = {w4.x, w4.y, w4.z, w4.w};
    const bf16_t* __restrict__ H = static_cast<const bf16_t*>(a.H);
    bf16_t* __restrict__ dH = static_cast<bf16_t*>(a.dH);
    // One row of the thread: the output-layer weight-gradient terms (rows in order), then
    // dz and its column sums.
    auto row = [&](int r, int b, const uint4& h4) {
      const float dq = dq_row[r];
      if (a.wpart) {
        const uint32_t hh[4] = {h4.x, h4.y, h4.z, h4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          ws[2 * e] = fmaf(dq, bf2f((bf16_t)(hh[e] & 0xFFFFu)), ws[2 * e]);
          ws[2 * e + 1] = fmaf(dq, bf2f((bf16_t)(hh[e] >> 16)), ws[2 * e + 1]);
        }
      }
      const uint32_t wd = wsh[(k >> 5) * HB_ROWS + r] >> (k & 31);
      uint32_t o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float w0 = bf2f((bf16_t)(ww[e] & 0xFFFFu)), w1 = bf2f((bf16_t)(ww[e] >> 16));
        const bf16_t h0 = f2bf((wd >> (2 * e)) & 1u ? dq * w0 : 0.0f);
        const bf16_t h1 = f2bf((wd >> (2 * e + 1)) & 1u ? dq * w1 : 0.0f);
        cs[2 * e] += bf2f(h0);
        cs[2 * e + 1] += bf2f(h1);
        o[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
      }
      *reinterpret_cast<uint4*>(dH + (int64_t)b * a.ld + k) = make_uint4(o[0], o[1], o[2], o[3]);
    };
    // Two rows per pass, both rows' loads issued before either row's store.
    for (int r = rs; r < HB_ROWS; r += 2 * rpi) {
      const int b = r0 + r, r1 = r + rpi, b1 = b + rpi;
      if (b >= rows) break;
      const bool two = r1 < HB_ROWS && b1 < rows;
      uint4 h0 = make_uint4(0u, 0u, 0u, 0u), h1 = h0;
      if (a.wpart) {
        h0 = *reinterpret_cast<const uint4*>(H + (int64_t)b * a.ld + k);
        if (two) h1 = *reinterpret_cast<const uint4*>(H + (int64_t)b1 * a.ld + k);
      }
      row(r, b, h0);
      if (two) row(r1, b1, h1);
    }
  }
  if (!a.colpart) return;
  float* ssh = reinterpret_cast<float*>(wsh + nw * HB_ROWS);
  if (rs < rpi) {
#pragma unroll
    for (int e = 0; e < 8; ++e) ssh[rs * a.K + k + e] = cs[e];
  }
  __syncthreads();
  for (int c = threadIdx.x; c < a.K; c += blockDim.x) {
    float t = 0.0f;
    for (int q = 0; q < rpi; ++q) t += ssh[q * a.K + c];
    a.colpart[(int64_t)blockIdx.x * a.K + c] = t;
  }
  if (!a.wpart) return;   // uniform per block
  __syncthreads();
  if (rs < rpi) {
#pragma unroll
    for (int e = 0; e < 8; ++e) ssh[rs * a.K + k + e] = ws[e];
  }
  __syncthreads();
  for (int c = threadIdx.x; c < a.K; c += blockDim.x) {
    float t = 0.0f;
    for (int q = 0; q < rpi; ++q) t += ssh[q * a.K + c];
    a.wpart[(int64_t)blockIdx.x * a.K + c] = t;
  }
  if (threadIdx.x == 0) {
    float t = 0.0f;
    for (int r = 0; r < HB_ROWS; ++r) t += dq_row[r];
    a.wpart_extra[blockIdx.x] = t;
  }
}

// q[r] of a critic output (QSrc); row-dot partials are summed in part order, then the
// bias is added, and the value is stored for later readers.
__device__ inline float q_value(const QSrc& s, int r) {
  if (!s.parts) return s.q[r];
  float v = 0.0f;
  for (int p = 0; p < s.parts; ++p) v += s.part[(int64_t)p * s.ld + r];
  v += *s.bias;
  s.q[r] = v;
  return v;
}

// ------------------------------------------------------------------------------ sampler actions
template <typename T>
__global__ void __launch_bounds__(256) k_obs_operand(ObsArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)a.rows * a.cols) return;
  const int r = (int)(i / a.cols), c = (int)(i - (int64_t)r * a.cols);
  const float v = (r < a.n && c < a.O) ? a.obs[(int64_t)r * a.O + c] : 0.0f;
  static_cast<T*>(a.x)[(int64_t)r * a.ldx + c] = from_f<T>(v);
}

__global__ void __launch_bounds__(256) k_act_head(ActHeadArgs h) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)h.n * h.A) return;
  const int r = (int)(e / h.A), j = (int)(e - (int64_t)r * h.A);
  const float* z = h.z + (int64_t)r * h.ldz;
  float u = z[j];
  if (h.sac && h.stochastic) {
    const float eps = normal_at(h.seed, (uint64_t)(h.row0 * h.A + e), h.counter, P_ACT);
    u += expf(clamp_keep_nan(z[h.A + j], h.lmin, h.lmax)) * eps;
  }
  h.a[e] = tanhf(u);
}

// ------------------------------------------------------------------------------ TD target, losses
__global__ void __launch_bounds__(256) k_td_target(TdArgs a) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.Bp) return;
  const float q1 = q_value(a.q1, b), q2 = q_value(a.q2, b);
  if (b >= a.B) { a.y[b] = 0.0f; return; }
  float m = min_keep_nan(q1, q2);
  if (a.logp) m -= expf(*a.log_alpha) * a.logp[b];
  a.y[b] = a.r[b] + a.gamma * (1.0f - a.d[b]) * m;
}

// dq_i = 2 (q_i - y) / B and per-block partial sums of (q1-y)^2, (q2-y)^2, q1.
__global__ void __launch_bounds__(256) k_critic_loss(CriticLossArgs a) {
  __shared__ double sh[256];
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  double e1s = 0.0, e2s = 0.0, q1s = 0.0;
  if (b < a.Bp) {
    float d1 = 0.0f, d2 = 0.0f;
    const float q1 = q_value(a.q1, b), q2 = q_value(a.q2, b);
    if (b < a.B) {
      const float e1 = q1 - a.y[b], e2 = q2 - a.y[b];
      d1 = 2.0f * e1 / (float)a.B;
      d2 = 2.0f * e2 / (float)a.B;
      e1s = (double)e1 * e1;
      e2s = (double)e2 * e2;
      q1s = q1;
    }
    a.dq1[b] = d1;
    a.dq2[b] = d2;
  }
  e1s = block_sum<256>(e1s, sh);
  e2s = block_sum<256>(e2s, sh);
  q1s = block_sum<256>(q1s, sh);
  if (threadIdx.x == 0) {
    a.part[blockIdx.x * 3 + 0] = e1s;
    a.part[blockIdx.x * 3 + 1] = e2s;
    a.part[blockIdx.x * 3 + 2] = q1s;
  }
}

// SAC: dqp_i routes -1/B to the smaller critic (critic 1 on ties); partial sums of
// alpha log pi - min(q1, q2) and log pi. TD3 (qp2 == null): dqp1 = -1/B; partial sum of q1.
__global__ void __launch_bounds__(256) k_actor_loss(ActorLossArgs a) {
  __shared__ double sh[256];
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  double l0 = 0.0, l1 = 0.0;
  bool take1 = false;
  if (b < a.Bp) {
    float g1 = 0.0f, g2 = 0.0f;
    const float q1 = q_value(a.qp1, b), q2 = a.has_qp2 ? q_value(a.qp2, b) : 0.0f;
    if (b < a.B) {
      const float inv = -1.0f / (float)a.B;
      if (a.has_qp2) {
        take1 = q1 <= q2;
        g1 = take1 ? inv : 0.0f;
        g2 = take1 ? 0.0f : inv;
        const float alpha = expf(*a.log_alpha);
        l0 = (double)alpha * a.logp[b] - (double)(take1 ? q1 : q2);
        l1 = a.logp[b];
      } else {
        g1 = inv;
        l0 = q1;
      }
    }
    a.dqp1[b] = g1;
    if (a.dqp2) a.dqp2[b] = g2;
  }
  l0 = block_sum<256>(l0, sh);
  l1 = block_sum<256>(l1, sh);
  if (threadIdx.x == 0) {
    a.part[blockIdx.x * 2 + 0] = l0;
    a.part[blockIdx.x * 2 + 1] = l1;
  }
  if (a.cnt1) {
    __shared__ int shi[4];
    const int n1 = block_sum_i32(b < a.B && take1 ? 1 : 0, shi);
    if (threadIdx.x == 0) a.cnt1[blockIdx.x] = n1;
  }
}

// Row split by the minimum critic, one row per thread over the actor loss's 256-row
// blocks. A block's first list position is the count of critic-1 rows in the blocks
// before it; within the block positions follow from a ballot prefix per wave and the
// wave totals; a critic-2 row's position is its row index less the critic-1 rows
// before it. Block 0 pads both lists and writes their padded lengths.
__global__ void __launch_bounds__(256) k_minq_split(MinqSplitArgs a) {
  __shared__ int sh[4];
  __shared__ int wtot[4];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  int p = 0;
  for (int i = t; i < (int)blockIdx.x; i += 256) p += a.cnt1[i];
  p = block_sum_i32(p, sh);
  const int b = blockIdx.x * 256 + t;
  const bool valid = b < a.B;
  const bool take1 = valid && a.qp1[b] <= a.qp2[b];
  const unsigned long long m = __ballot(take1);
  if (lane == 0) wtot[wave] = __popcll(m);
  __syncthreads();
  int pos1 = p + __popcll(m & ((1ull << lane) - 1ull));
  for (int w = 0; w < wave; ++w) pos1 += wtot[w];
  if (take1) a.map1[pos1] = b;
  else if (valid) a.map2[b - pos1] = b;
  if (blockIdx.x != 0) return;
  int n1 = 0;
  for (int i = t; i < (int)gridDim.x; i += 256) n1 += a.cnt1[i];
  n1 = block_sum_i32(n1, sh);
  const int n2 = a.B - n1;
  const int m1 = min((n1 + 511) / 512 * 512, a.Bp), m2 = min((n2 + 511) / 512 * 512, a.Bp);
  for (int i = n1 + t; i < m1; i += 256) a.map1[i] = -1;
  for (int i = n2 + t; i < m2; i += 256) a.map2[i] = -1;
  if (t == 0) {
    a.rows[0] = m1;
    a.rows[1] = m2;
  }
}

// Thread: one row, RBG_WORDS consecutive words (blockIdx.y picks the word group), so
// that each thread's loads are independent and the grid has enough blocks to keep
// the loads in flight.
constexpr int RBG_WORDS = 4;
__global__ void __launch_bounds__(256) k_row_bits_gather(RowBitsGatherArgs a) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= a.rows || r >= *a.m_dyn) return;
  const int src = a.map[r];
  const uint32_t* __restrict__ in = a.src;
  uint32_t* __restrict__ out = a.dst;
  const int w0 = blockIdx.y * RBG_WORDS;
  uint32_t v[RBG_WORDS];
#pragma unroll
  for (int i = 0; i < RBG_WORDS; ++i)
    v[i] = src >= 0 && w0 + i < a.words ? in[(int64_t)(w0 + i) * a.ld + src] : 0u;
#pragma unroll
  for (int i = 0; i < RBG_WORDS; ++i)
    if (w0 + i < a.words) out[(int64_t)(w0 + i) * a.ld + r] = v[i];
}

__global__ void __launch_bounds__(256) k_row_scatter(RowScatterArgs a) {
  const int cv = a.cols / 4;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)a.rows * cv) return;
  const int r = (int)(i / cv), j = (int)(i - (int64_t)r * cv) * 4;
  if (r >= *a.m_dyn) return;
  const int b = a.map[r];
  if (b < 0) return;
  *reinterpret_cast<float4*>(a.dst + (int64_t)b * a.ld + j) = *reinterpret_cast<const float4*>(a.src + (int64_t)r * a.ld + j);
}

// Actor head backward. SAC: g_u = da (1 - a^2) + (alpha/B) 2 a, d mu = g_u,
// d l = (g_u sigma eps - alpha/B) * [lmin <= l <= lmax]. TD3: dz = da (1 - a^2).
template <typename T>
__global__ void __launch_bounds__(256) k_actor_head_bwd(ActorHeadBwdArgs h) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // (row, action) element
  if (c >= (int64_t)h.B * h.A) return;
  const int b = (int)(c / h.A), j = (int)(c - (int64_t)b * h.A);
  T* dz = static_cast<T*>(h.dz) + (int64_t)b * h.ldz;
  const float aB = h.sac ? expf(*h.log_alpha) / (float)h.B : 0.0f;
  float da = h.da1[(int64_t)b * h.ldda + j];
  if (h.da2) da += h.da2[(int64_t)b * h.ldda + j];
  const float a = h.th[c];
  float gu = da * (1.0f - a * a);
  if (h.sac) {
    gu += aB * 2.0f * a;
    dz[h.A + j] = from_f<T>((gu * h.se[c] - aB) * h.lm[c]);
  }
  dz[j] = from_f<T>(gu);
}

// ------------------------------------------------------------------------------ column sums
// First pass: block (x, y) sums rows [y*chunk, (y+1)*chunk) of a column tile of CT
// 16-byte vectors; threads hold one vector column each and step over rows by RT,
// then the RT partial sums per column are added in row order through LDS.
// part[y, n] = sum_b wt(b) X[b, n]; wt(b) = rnd(weights[b]) or 1. With `extra`,
// part_extra[y] = sum_b wt(b) (computed by the x == 0 blocks).
template <typename T>
__global__ void __launch_bounds__(256) k_colsum(ColsumArgs a) {
  using V = Vec16<T>;
  constexpr int NT = 256;
  const int nvec = a.N / V::N;
  const int CT = nvec < 32 ? nvec : 32;
  const int RT = NT / CT;
  const int tx = threadIdx.x % CT, ty = threadIdx.x / CT;
  const int cv = blockIdx.x * CT + tx;
  const int b0 = blockIdx.y * a.chunk, b1 = min(b0 + a.chunk, a.rows);
  const T* X = static_cast<const T*>(a.X);
  float acc[V::N];
#pragma unroll
  for (int i = 0; i < V::N; ++i) acc[i] = 0.0f;
  float wsum = 0.0f;
  if (ty < RT && cv < nvec) {
#pragma unroll 4
    for (int b = b0 + ty; b < b1; b += RT) {
      const float w = a.weights ? to_f<T>(from_f<T>(a.weights[b])) : 1.0f;
      float x[V::N];
      V::load(X + (int64_t)b * a.ld + cv * V::N, x);
#pragma unroll
      for (int i = 0; i < V::N; ++i) acc[i] = fmaf(w, x[i], acc[i]);
      wsum += w;
    }
  }
  __shared__ float sh[NT * 8 + NT];
  const bool live = ty < RT;
#pragma unroll
  for (int i = 0; i < V::N; ++i) sh[threadIdx.x * V::N + i] = live ? acc[i] : 0.0f;
  __syncthreads();
  if (ty == 0 && cv < nvec) {
    float o[V::N];
#pragma unroll
    for (int i = 0; i < V::N; ++i) o[i] = 0.0f;
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int i = 0; i < V::N; ++i) o[i] += sh[(r * CT + tx) * V::N + i];
#pragma unroll
    for (int i = 0; i < V::N; ++i) a.part[(int64_t)blockIdx.y * a.N + cv * V::N + i] = o[i];
  }
  if (a.extra && blockIdx.x == 0) {   // uniform per block
    if (tx == 0 && live) sh[NT * 8 + ty] = wsum;
    __syncthreads();
    if (threadIdx.x == 0) {
      float t = 0.0f;
      for (int r = 0; r < RT; ++r) t += sh[NT * 8 + r];
      a.part_extra[blockIdx.y] = t;
    }
  }
}

// Column-sum partials are reduced by the deferred reduction (k_reduce_jobs) with
// CSF_G groups: group g adds chunks g, g + CSF_G, ... in order and the group sums are
// added in g order, a fixed order for a fixed chunk count (many groups keep each
// thread's chain of loads short: the partials are few and read once).
constexpr int CSF_G = 64;

// Deferred reductions (ReduceJob): a block belongs to the last job whose block0 it has
// reached; 256 / groups pieces per block, `groups` threads per piece.
__global__ void __launch_bounds__(256) k_reduce_jobs(ReduceJobs J) {
  __shared__ float4 sh[256];
  int k = 0;
  for (int i = 1; i < J.n; ++i)
    if ((int)blockIdx.x >= J.j[i].block0) k = i;
  const ReduceJob& jb = J.j[k];
  const int G = jb.groups, P = 256 / G;
  const int grp = threadIdx.x / P, pc = threadIdx.x % P;
  const int cv = jb.cols / jb.vec;
  const int64_t piece = (int64_t)((int)blockIdx.x - jb.block0) * P + pc;
  const bool valid = piece < (int64_t)jb.rows * cv;
  float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  int64_t r = 0;
  int col = 0;
  if (valid) {
    r = piece / cv;
    col = (int)(piece - r * cv) * jb.vec;
    const float* src = jb.part + r * jb.ld + col;
    if (jb.vec == 4) {
#pragma unroll 16
      for (int z = grp; z < jb.slices; z += G) {
        const float4 v = *reinterpret_cast<const float4*>(src + (int64_t)z * jb.zstride);
        acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
      }
    } else {
      for (int z = grp; z < jb.slices; z += G) acc.x += src[(int64_t)z * jb.zstride];
    }
  }
  if (G > 1) {   // uniform per block
    sh[threadIdx.x] = acc;
    __syncthreads();
    if (grp != 0) return;
    for (int q = 1; q < G; ++q) {
      const float4 v = sh[q * P + pc];
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
  }
  if (!valid) return;
  float* dst = jb.out + r * jb.ldo + col;
  if (jb.vec == 4) *reinterpret_cast<float4*>(dst) = acc;
  else *dst = acc.x;
}

// ------------------------------------------------------------------------------ optimizer
// Adam (bias-corrected, one counter per optimizer) on the actor range, the critic
// range and log(alpha); then Polyak tbar <- (1 - tau) tbar + tau theta on the
// target ranges; refreshes the bfloat16 shadows of what it wrote.
__global__ void __launch_bounds__(256) k_adam_polyak(AdamArgs a) {
  // Bias corrections 1 - beta^t of the step (actor: delayed-step count for TD3),
  // computed once per block in double precision.
  __shared__ float bc[4];   // beta1 / beta2 corrections at t, then at the actor's t
  const int64_t t = *a.step + a.step_add;
  const int64_t ta = a.td3 ? t / a.delay : t;
  if (threadIdx.x < 4) {
    const double beta = (threadIdx.x & 1) ? (double)a.b2 : (double)a.b1;
    bc[threadIdx.x] = (float)(1.0 - pow(beta, (double)(threadIdx.x < 2 ? t : ta)));
  }
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const bool in_actor = i >= a.a0 && i < a.a1;
  const bool in_critic = i >= a.c0 && i < a.c1 && a.do_critic;
  const bool is_alpha = i == a.la;
  float lr;
  int sel;
  if (in_actor && a.do_actor) {
    lr = a.lr_a;
    sel = 2;
  } else if (in_critic) {
    lr = a.lr_c;
    sel = 0;
  } else if (is_alpha && a.do_alpha) {
    lr = a.lr_al;
    sel = 0;
  } else {
    return;
  }
  const float bc1 = bc[sel], bc2 = bc[sel + 1];
  const float g = a.G[i];
  const float m = a.b1 * a.M[i] + (1.0f - a.b1) * g;
  const float v = a.b2 * a.V[i] + (1.0f - a.b2) * g * g;
  a.M[i] = m;
  a.V[i] = v;
  const float p = a.P[i] - lr * (m / bc1) / (sqrtf(v / bc2) + a.eps);
  a.P[i] = p;
  if (a.Pb) a.Pb[i] = f2bf(p);
  const bool pol = (in_critic && a.polyak_critic) || (in_actor && a.polyak_actor);
  if (pol) {
    const float tb = (1.0f - a.tau) * a.T[i] + a.tau * p;
    a.T[i] = tb;
    if (a.Tb) a.Tb[i] = f2bf(tb);
  }
}

// One block: reduce the step's loss partials in index order, write the loss
// record, the temperature gradient, and advance the device step counter.
__global__ void __launch_bounds__(256) k_finish(FinishArgs f) {
  __shared__ double sh[256];
  double e1 = 0.0, e2 = 0.0, q1 = 0.0, l0 = 0.0, l1 = 0.0;
  for (int i = threadIdx.x; i < f.nc; i += 256) {
    e1 += f.cpart[i * 3 + 0];
    e2 += f.cpart[i * 3 + 1];
    q1 += f.cpart[i * 3 + 2];
  }
  if (f.actor_step)
    for (int i = threadIdx.x; i < f.na; i += 256) {
      l0 += f.apart[i * 2 + 0];
      l1 += f.apart[i * 2 + 1];
    }
  e1 = block_sum<256>(e1, sh);
  e2 = block_sum<256>(e2, sh);
  q1 = block_sum<256>(q1, sh);
  l0 = block_sum<256>(l0, sh);
  l1 = block_sum<256>(l1, sh);
  if (threadIdx.x != 0) return;
  const int64_t t = *f.step + 1;
  const double invB = 1.0 / (double)f.B;
  float rec[SPZ_REC_WIDTH];
  rec[SPZ_REC_LQ] = (float)((e1 + e2) * invB);
  rec[SPZ_REC_Q1] = (float)(q1 * invB);
  rec[SPZ_REC_LPI] = 0.0f;
  rec[SPZ_REC_LALPHA] = 0.0f;
  rec[SPZ_REC_ALPHA] = 0.0f;
  rec[SPZ_REC_LOGPI] = 0.0f;
  if (f.sac) {
    const float log_alpha = *f.log_alpha;
    const double mean_lp = l1 * invB;
    rec[SPZ_REC_LPI] = (float)(l0 * invB);
    rec[SPZ_REC_LOGPI] = (float)mean_lp;
    rec[SPZ_REC_ALPHA] = expf(log_alpha);
    const double mh = mean_lp + (double)f.target_entropy;
    rec[SPZ_REC_LALPHA] = (float)(-(double)log_alpha * mh);
    if (f.grad_alpha) *f.grad_alpha = f.learn_alpha ? (float)(-mh) : 0.0f;
  } else if (f.actor_step) {
    rec[SPZ_REC_LPI] = (float)(-l0 * invB);
  }
  bool bad = false;
  for (int i = 0; i < 6; ++i) bad = bad || !isfinite(rec[i]);
  rec[SPZ_REC_NONFINITE] = bad ? 1.0f : 0.0f;
  rec[SPZ_REC_ACTOR] = f.actor_step ? 1.0f : 0.0f;
  float* dst = f.rec + ((t - 1) % f.rec_cap) * SPZ_REC_WIDTH;
  for (int i = 0; i < SPZ_REC_WIDTH; ++i) dst[i] = rec[i];
  *f.step = t;
}

__global__ void __launch_bounds__(256) k_to_bf16(const float* __restrict__ src, bf16_t* __restrict__ dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = f2bf(src[i]);
}

// One 64 x 64 tile of one transpose job per workgroup, through an LDS tile: reads of
// 64 consecutive columns per row and writes of 64 consecutive rows per column.
template <typename T>
__global__ void __launch_bounds__(256) k_transpose(const T* __restrict__ src, T* __restrict__ dst,
                                                   const TransposeJob* __restrict__ jobs, int njobs) {
  __shared__ T tile[64][65 + (sizeof(T) == 2 ? 1 : 0)];
  const int t = blockIdx.x;
  int j = 0;
  while (j + 1 < njobs && jobs[j + 1].tile0 <= t) ++j;
  const TransposeJob J = jobs[j];
  const int tc = (J.cols + 63) / 64, tl = t - J.tile0;
  const int r0 = (tl / tc) * 64, c0 = (tl % tc) * 64;
  const int x = threadIdx.x & 63, y = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int r = r0 + y + 4 * i, c = c0 + x;
    if (r < J.rows && c < J.cols) tile[y + 4 * i][x] = src[J.src_off + (int64_t)r * J.lds + c];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int c = c0 + y + 4 * i, r = r0 + x;
    if (r < J.rows && c < J.cols) dst[J.dst_off + (int64_t)c * J.ldd + r] = tile[x][y + 4 * i];
  }
}

inline unsigned blocks(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

// ------------------------------------------------------------------------------ launchers
#define SPZ_LAUNCH_T(bf16, kern, grid, block, s, arg)                 \
  do {                                                               \
    if (bf16) kern<bf16_t><<<(grid), (block), 0, (s)>>>(arg);        \
    else kern<float><<<(grid), (block), 0, (s)>>>(arg);              \
  } while (0)

hipError_t launch_gather(bool bf16, const GatherArgs& g, hipStream_t s) {
  SPZ_LAUNCH_T(bf16, k_gather, blocks(g.B, 4), 256, s, g);
  return hipGetLastError();
}
hipError_t launch_pack(bool bf16, const PackArgs& p, hipStream_t s) {
  SPZ_LAUNCH_T(bf16, k_pack_rows, blocks(p.n, 4), 256, s, p);
  return hipGetLastError();
}
hipError_t launch_sac_head(bool bf16, const SacHeadArgs& h, hipStream_t s) {
  if (h.A < 1 || h.A > 256) return hipErrorInvalidValue;
  const size_t lds = (size_t)HEAD_ROWS * h.A * sizeof(float);
  if (bf16) k_sac_head<bf16_t><<<blocks(h.B, HEAD_ROWS), 256, lds, s>>>(h);
  else k_sac_head<float><<<blocks(h.B, HEAD_ROWS), 256, lds, s>>>(h);
  return hipGetLastError();
}
hipError_t launch_td3_head(bool bf16, const Td3HeadArgs& h, hipStream_t s) {
  SPZ_LAUNCH_T(bf16, k_td3_head, blocks((int64_t)h.B * h.A, 256), 256, s, h);
  return hipGetLastError();
}
hipError_t launch_rowdot(bool bf16, const RowdotArgs& r, hipStream_t s) {
  if (r.K % (bf16 ? 8 : 4)) return hipErrorInvalidValue;
  SPZ_LAUNCH_T(bf16, k_rowdot, blocks(r.rows, 4), 256, s, r);
  return hipGetLastError();
}
hipError_t launch_head_bwd(bool bf16, const HeadBwdArgs& a, hipStream_t s) {
  const int vec = bf16 ? 8 : 4;
  if (a.K % vec || a.ld % vec) return hipErrorInvalidValue;
  if ((a.map || a.m_dyn) && (!a.bits || a.colpart)) return hipErrorInvalidValue;
  if (a.wpart && (!a.colpart || !a.wpart_extra)) return hipErrorInvalidValue;
  if (a.bits) {
    if (!bf16 || a.K % 32 || a.K / 8 > 256 || a.ldbits < a.rows) return hipErrorInvalidValue;
    const size_t lds = (size_t)(a.K / 32) * HB_ROWS * 4 + (a.colpart ? (size_t)(256 / (a.K / 8)) * a.K * 4 : 0);
    if (lds > 64 * 1024) return hipErrorInvalidValue;
    k_head_bwd_bits<<<blocks(a.rows, HB_ROWS), 256, lds, s>>>(a);
    return hipGetLastError();
  }
  if (a.colpart) return hipErrorInvalidValue;
  SPZ_LAUNCH_T(bf16, k_head_bwd, blocks((int64_t)a.rows * (a.K / vec), 256), 256, s, a);
  return hipGetLastError();
}
int head_bwd_blocks(int rows) { return (int)blocks(rows, HB_ROWS); }
hipError_t launch_obs_operand(bool bf16, const ObsArgs& a, hipStream_t s) {
  if (a.n < 0 || a.n > a.rows || a.cols < a.O || a.ldx < a.cols) return hipErrorInvalidValue;
  SPZ_LAUNCH_T(bf16, k_obs_operand, blocks((int64_t)a.rows * a.cols, 256), 256, s, a);
  return hipGetLastError();
}
hipError_t launch_act_head(const ActHeadArgs& a, hipStream_t s) {
  if (a.n < 1) return hipSuccess;
  k_act_head<<<blocks((int64_t)a.n * a.A, 256), 256, 0, s>>>(a);
  return hipGetLastError();
}
hipError_t launch_td_target(const TdArgs& a, hipStream_t s) {
  k_td_target<<<blocks(a.Bp, 256), 256, 0, s>>>(a);
  return hipGetLastError();
}
int loss_blocks(int Bp) { return (int)blocks(Bp, 256); }
hipError_t launch_critic_loss(const CriticLossArgs& a, hipStream_t s) {
  k_critic_loss<<<blocks(a.Bp, 256), 256, 0, s>>>(a);
  return hipGetLastError();
}
hipError_t launch_actor_loss(const ActorLossArgs& a, hipStream_t s) {
  if (a.cnt1 && !a.has_qp2) return hipErrorInvalidValue;
  k_actor_loss<<<blocks(a.Bp, 256), 256, 0, s>>>(a);
  return hipGetLastError();
}
hipError_t launch_minq_split(const MinqSplitArgs& a, hipStream_t s) {
  if (a.Bp % 256 || a.B < 0 || a.B > a.Bp || !a.cnt1 || !a.qp1 || !a.qp2 || !a.map1 || !a.map2 || !a.rows)
    return hipErrorInvalidValue;
  if (!a.Bp) return hipSuccess;
  k_minq_split<<<a.Bp / 256, 256, 0, s>>>(a);
  return hipGetLastError();
}
hipError_t launch_row_bits_gather(const RowBitsGatherArgs& a, hipStream_t s) {
  if (a.words < 0 || a.rows < 0 || a.ld < a.rows || !a.map || !a.m_dyn) return hipErrorInvalidValue;
  if (!a.rows || !a.words) return hipSuccess;
  k_row_bits_gather<<<dim3(blocks(a.rows, 256), blocks(a.words, RBG_WORDS)), 256, 0, s>>>(a);
  return hipGetLastError();
}
hipError_t launch_row_scatter(const RowScatterArgs& a, hipStream_t s) {
  if (a.cols % 4 || a.ld % 4 || a.cols > a.ld || a.rows < 0 || !a.map || !a.m_dyn ||
      ((uintptr_t)a.src & 15) || ((uintptr_t)a.dst & 15))
    return hipErrorInvalidValue;
  if (!a.rows || !a.cols) return hipSuccess;
  k_row_scatter<<<blocks((int64_t)a.rows * (a.cols / 4), 256), 256, 0, s>>>(a);
  return hipGetLastError();
}
hipError_t launch_actor_head_bwd(bool bf16, const ActorHeadBwdArgs& h, hipStream_t s) {
  SPZ_LAUNCH_T(bf16, k_actor_head_bwd, blocks((int64_t)h.B * h.A, 256), 256, s, h);
  return hipGetLastError();
}
int colsum_chunks(int rows) { return (int)blocks(rows, COLSUM_CHUNK); }
hipError_t launch_colsum_partial(bool bf16, const ColsumArgs& a, hipStream_t s) {
  const int vec = bf16 ? 8 : 4;
  if (a.N % vec || a.ld % vec || a.N % 4) return hipErrorInvalidValue;
  const int nvec = a.N / vec, ct = nvec < 32 ? nvec : 32;
  dim3 grid(blocks(nvec, ct), blocks(a.rows, a.chunk));
  SPZ_LAUNCH_T(bf16, k_colsum, grid, 256, s, a);
  return hipGetLastError();
}
int colsum_groups() { return CSF_G; }
hipError_t launch_reduce_jobs(ReduceJobs& J, hipStream_t s) {
  if (J.n < 1 || J.n > MAX_REDUCE_JOBS) return hipErrorInvalidValue;
  int nb = 0;
  for (int i = 0; i < J.n; ++i) {
    ReduceJob& jb = J.j[i];
    if (jb.groups < 1 || jb.groups > 256 || (jb.groups & (jb.groups - 1)) || (jb.vec != 1 && jb.vec != 4) ||
        jb.cols % jb.vec || jb.rows < 0 || jb.slices < 1)
      return hipErrorInvalidValue;
    if (jb.vec == 4 && (jb.ld % 4 || jb.ldo % 4 || jb.zstride % 4 || ((uintptr_t)jb.part & 15) ||
                        ((uintptr_t)jb.out & 15)))
      return hipErrorInvalidValue;
    jb.block0 = nb;
    const int64_t pieces = (int64_t)jb.rows * (jb.cols / jb.vec);
    nb += (int)blocks(pieces, 256 / jb.groups);
  }
  if (nb == 0) return hipSuccess;
  k_reduce_jobs<<<nb, 256, 0, s>>>(J);
  return hipGetLastError();
}
hipError_t launch_adam(const AdamArgs& a, hipStream_t s) {
  k_adam_polyak<<<blocks(a.n, 256), 256, 0, s>>>(a);
  return hipGetLastError();
}
hipError_t launch_finish(const FinishArgs& f, hipStream_t s) {
  k_finish<<<1, 256, 0, s>>>(f);
  return hipGetLastError();
}
hipError_t launch_to_bf16(const float* src, bf16_t* dst, int64_t n, hipStream_t s) {
  k_to_bf16<<<blocks(n, 256), 256, 0, s>>>(src, dst, n);
  return hipGetLastError();
}

hipError_t launch_transpose(bool bf16, const void* src, void* dst, const TransposeJob* jobs, int njobs, int tiles,
                            hipStream_t s) {
  if (njobs < 1 || tiles < 1) return hipErrorInvalidValue;
  if (bf16)
    k_transpose<bf16_t><<<tiles, 256, 0, s>>>(static_cast<const bf16_t*>(src), static_cast<bf16_t*>(dst), jobs, njobs);
  else
    k_transpose<float><<<tiles, 256, 0, s>>>(static_cast<const float*>(src), static_cast<float*>(dst), jobs, njobs);
  return hipGetLastError();
}

}  // namespace spz
