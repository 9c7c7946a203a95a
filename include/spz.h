/*
 * spz.h -- C ABI of the large-batch actor-critic update on one MI355X (gfx950).
 *
 * The library implements the network-update process of Spreeze (Section 3.2:
 * one updater drawing large uniform batches from a shared replay pool and
 * training the actor and the double-Q critics with target networks; Section
 * 3.2.2: actor and critic updated independently, here as two concurrent HIP
 * streams on one GPU). SAC is the paper's worked example; TD3 is the
 * alternative algorithm of Section 4.2.4, Fig. 8. One update step:
 *   1. Philox-sampled replay indices and a row gather from the HBM ring buffer;
 *   2. critic stream: target action (actor + tanh-Gaussian head, or TD3 target
 *      actor + smoothing), target critics, TD target, online critics, critic
 *      loss, critic backward;
 *   3. actor stream: actor forward on s, critics at their step-start parameters
 *      on (s, a~), actor loss, backward to the actor, temperature gradient;
 *   4. one fused Adam + Polyak pass over all parameters.
 *
 * Conventions
 *   - Every call returns SPZ_OK (0) or a negative SPZ_E* code; no C++ exception
 *     crosses the ABI. spz_create returns NULL on failure. The message of the
 *     last failure on the calling thread is spz_last_error(NULL); per-context
 *     messages are spz_last_error(ctx).
 *   - Pointers are HOST pointers unless stated. The caller keeps ownership of
 *     every array it passes; the library copies what it needs before returning.
 *   - A context is not thread-safe; distinct contexts are independent.
 *   - Flat parameter layout of one network (spz_read_params / spz_write_params):
 *     layer by layer, W as [out, in] row-major float32, then b [out].
 *     Actor (SAC): obs -> hidden... -> 2*act (mean | log-std); actor (TD3):
 *     obs -> hidden... -> act; critic: (obs | act) -> hidden... -> 1.
 */
#ifndef SPZ_H
#define SPZ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct spz_ctx spz_ctx;

/* Return codes. */
#define SPZ_OK 0
#define SPZ_EINVAL (-1) /* bad argument (dimension, pointer, hyper-parameter, selector) */
#define SPZ_ENOMEM (-2) /* device or host allocation failed                             */
#define SPZ_EEMPTY (-3) /* spz_update on an empty replay buffer                          */
#define SPZ_ESIZE (-4)  /* caller's array length does not match the requested object     */
#define SPZ_EHIP (-5)   /* a HIP runtime call failed (message has the HIP error string)  */
#define SPZ_EIO (-6)    /* checkpoint file not writable / readable, or not this learner's */

/* Algorithms and GEMM operand precisions. */
#define SPZ_ALGO_SAC 0
#define SPZ_ALGO_TD3 1
#define SPZ_PREC_FP32 0 /* float32 operands, float32 accumulate                        */
#define SPZ_PREC_BF16 1 /* bfloat16 operands (RNE), float32 accumulate, fp32 master    */

/* Selectors for spz_param_count / spz_read_params / spz_write_params. */
#define SPZ_ACTOR 0
#define SPZ_CRITIC1 1
#define SPZ_CRITIC2 2
#define SPZ_TCRITIC1 3
#define SPZ_TCRITIC2 4
#define SPZ_TACTOR 5 /* TD3 only */
#define SPZ_LOG_ALPHA 6
#define SPZ_M_ACTOR 7 /* Adam first moments */
#define SPZ_M_CRITIC1 8
#define SPZ_M_CRITIC2 9
#define SPZ_M_LOG_ALPHA 10
#define SPZ_V_ACTOR 11 /* Adam second moments */
#define SPZ_V_CRITIC1 12
#define SPZ_V_CRITIC2 13
#define SPZ_V_LOG_ALPHA 14
#define SPZ_G_ACTOR 15 /* gradients of the last completed step (read only) */
#define SPZ_G_CRITIC1 16
#define SPZ_G_CRITIC2 17
#define SPZ_G_LOG_ALPHA 18
#define SPZ_N_SELECTORS 19

/* Selectors for spz_debug_read (per-row values of the last step, float32 unless
 * noted; the actor-side values are those of the last step that updated the actor). */
#define SPZ_DBG_INDICES 0   /* int32 [batch]: replay rows sampled by the last step     */
#define SPZ_DBG_TD_TARGET 1 /* [batch]: TD target y                                   */
#define SPZ_DBG_Q 2         /* [2, batch]: online critics q1, q2 on (s, a)            */
#define SPZ_DBG_QPI 3       /* [2, batch]: critics 1, 2 on (s, a~) (TD3: critic 1 twice) */
#define SPZ_DBG_LOGPI 4     /* [batch]: log pi of the actor sample (SAC only)         */
#define SPZ_DBG_DACTION 5   /* [batch, act_dim]: gradient of the actor loss with respect
                               to the actor's action a~ (Section 3.2.2's twin minimum
                               for SAC, critic 1 for TD3)                              */
#define SPZ_DBG_BATCH 6     /* [batch, 2*obs_dim + act_dim + 2]: the transitions the last
                               step gathered from the replay pool (Section 3.3.2), one
                               row (s | a | s' | r | d) per batch row, as the update's
                               kernels read them (bf16 contexts: the stored bfloat16
                               values, widened to float32 exactly)                      */

/* Loss record of one step: 8 floats. */
#define SPZ_REC_LQ 0        /* mean (q1-y)^2 + mean (q2-y)^2                      */
#define SPZ_REC_LPI 1       /* actor loss (0 on TD3 steps without an actor update) */
#define SPZ_REC_LALPHA 2    /* -log(alpha) * mean(log pi + target entropy)         */
#define SPZ_REC_ALPHA 3     /* alpha used by the step                              */
#define SPZ_REC_LOGPI 4     /* mean log pi of the actor sample                     */
#define SPZ_REC_Q1 5        /* mean q1(s, a)                                       */
#define SPZ_REC_NONFINITE 6 /* 1 if any of the values above is not finite          */
#define SPZ_REC_ACTOR 7     /* 1 if the actor was updated in this step             */
#define SPZ_REC_WIDTH 8

/* Hyper-parameters. Fill with spz_hparams_default, then override. */
typedef struct spz_hparams {
  int32_t algo;      /* SPZ_ALGO_SAC | SPZ_ALGO_TD3                                */
  int32_t gemm_prec; /* SPZ_PREC_FP32 | SPZ_PREC_BF16                              */
  int64_t capacity;  /* replay ring rows (> 0)                                     */
  float gamma;       /* discount                                                   */
  float tau;         /* Polyak rate: tbar <- (1-tau) tbar + tau theta, in [0, 1]    */
  float lr_actor, lr_critic, lr_alpha;
  float beta1, beta2, eps; /* Adam                                                 */
  float alpha_init;        /* SAC temperature at step 0 (> 0)                      */
  int32_t learn_alpha;     /* SAC: 1 learns log(alpha) against target_entropy      */
  float target_entropy;
  float log_std_min, log_std_max; /* SAC log-std clamp                             */
  float policy_noise, noise_clip; /* TD3 target policy smoothing                   */
  int32_t policy_delay;           /* TD3: actor and targets every policy_delay steps */
  int32_t device;                 /* HIP device ordinal                            */
  int32_t n_streams;              /* 2: actor and critic on concurrent streams; 1: one stream */
  int32_t ordering;               /* SPZ_ORDER_SNAPSHOT | SPZ_ORDER_SEQUENTIAL (below)     */
  int32_t actor_row_split;        /* SAC: 1 takes the actor loss's gradient through each
                                     critic only on the rows where that critic attains
                                     min(Q1, Q2) (the other rows carry zero gradient
                                     there, Section 3.2.2's twin-critic minimum), with
                                     the same results as 0, which takes both critics
                                     over every row. Used where the ReLU masks are kept
                                     as bits (bf16 with 128-multiple hidden widths).  */
  int32_t graphs;                 /* 1: spz_update replays each step from a captured HIP
                                     graph (one per step kind: SAC has one, TD3 one with
                                     and one without the delayed actor update) instead of
                                     launching its kernels one by one; bit-identical
                                     results. A graph is captured the first time a step
                                     kind runs (that step itself runs eagerly) and again
                                     after the batch size, the replay fill level or the
                                     seed changed. Ignored while kernel timing is on.  */
} spz_hparams;

/* Update ordering within a step.
 * SPZ_ORDER_SNAPSHOT: every loss of step t reads the parameters of the start of
 *   step t and all Adam / Polyak writes follow both gradients: the actor and the
 *   critics are updated independently (Section 3.2.2); the two halves may run on
 *   concurrent streams.
 * SPZ_ORDER_SEQUENTIAL: the critics take their Adam step (and Polyak) first and
 *   the actor loss of the same step is taken through the updated critics, as in
 *   the published SAC and TD3 algorithms; the temperature uses the step-start
 *   actor sample and alpha. Runs on one stream whatever n_streams says. */
#define SPZ_ORDER_SNAPSHOT 0
#define SPZ_ORDER_SEQUENTIAL 1

/* Defaults: SAC, fp32, capacity 1e6, gamma 0.99, tau 0.005, lr 3e-4, Adam
 * (0.9, 0.999, 1e-8), alpha_init 1, learned alpha, target_entropy 0, log-std
 * clamp [-20, 2], TD3 noise 0.2 clipped to 0.5, delay 2, device 0, 2 streams,
 * snapshot ordering, actor row split on, no graphs. */
void spz_hparams_default(spz_hparams* hp);

/* Create a learner: the single network-update process of Section 3.2 (its actor
 * and double-Q critics with target critics, Section 3.2.2; TD3 adds a target
 * actor), on one GPU. obs_dim, act_dim >= 1; hidden[0..n_hidden) >= 1 with
 * 1 <= n_hidden <= 6; batch >= 1. Parameters are initialised on the host from
 * `seed` with the fan-in uniform rule U(-1/sqrt(fan_in), 1/sqrt(fan_in)) drawn
 * from Philox4x32-10 (counter = (i>>2, 0, 0, net*16 + layer*2 + {W:0,b:1}),
 * word i&3); targets start as exact copies; log(alpha) = ln(alpha_init).
 * `hidden` and `hp` are copied. NULL on failure (see spz_last_error(NULL)). */
spz_ctx* spz_create(int32_t obs_dim, int32_t act_dim, const int32_t* hidden, int32_t n_hidden,
                    int32_t batch, const spz_hparams* hp, uint64_t seed);

/* Release every device and host resource of ctx (NULL is ignored). Waits for
 * the context's outstanding work first. */
void spz_destroy(spz_ctx* ctx);

/* Append n transitions to the replay ring (Section 3.3.2's shared experience
 * pool). Host float32 arrays, row-major: obs [n, obs_dim], act [n, act_dim],
 * rew [n], done [n] (0 or 1), next_obs [n, obs_dim]. Row i goes to slot
 * (ptr + i) mod capacity; size = min(size + n, capacity). bf16 contexts store
 * obs, act and next_obs rounded to bfloat16 (RNE). Synchronous: the arrays may
 * be freed when the call returns. Errors: SPZ_EINVAL (n < 0, or a NULL array
 * with n > 0), SPZ_EHIP. */
int spz_buffer_push(spz_ctx* ctx, const float* obs, const float* act, const float* rew,
                    const float* done, const float* next_obs, int64_t n);

/* Asynchronous form of spz_buffer_push (Section 3.3.2: experience reaches the
 * update process without taking its time). The rows are copied into library-owned
 * pinned staging before the call returns (the caller may reuse its arrays), moved
 * to the device on the library's own ingestion stream, and written into the ring
 * on the stream of the last spz_update (or an internal stream before the first):
 * they are seen by exactly the steps enqueued after this call, and the fill level
 * and write pointer (spz_buffer_size) advance at once. The same sequence of calls
 * therefore gives the same results as with spz_buffer_push. Blocks only when all
 * four staging slots (65536 rows each) still wait for their rows to be committed.
 * Errors: SPZ_EINVAL (n < 0, or NULL with n > 0), SPZ_ENOMEM, SPZ_EHIP. */
int spz_buffer_push_async(spz_ctx* ctx, const float* obs, const float* act, const float* rew,
                          const float* done, const float* next_obs, int64_t n);

/* Rows currently held by the ring (0 .. capacity). */
int64_t spz_buffer_size(const spz_ctx* ctx);

/* Enqueue n_steps update steps on `hip_stream` (a hipStream_t; NULL = the null
 * stream) and return without waiting. One step is one large-batch update of the
 * actor and the critics from a uniform sample of the replay pool (Section 3.2.1,
 * with the two halves updated independently as in Section 3.2.2 and Fig. 3's SAC
 * computation graph). Step t (1-based, counted across calls)
 * samples idx[b] = mulhi32(Philox(seed; b>>2, t, 1, 0)[b&3], size) with
 * replacement, draws its normal deviates from purposes 2 (target) and 3
 * (policy), and ends with the Adam/Polyak pass. Non-finite values do not make
 * the call fail; they set SPZ_REC_NONFINITE in the step's loss record.
 * Errors: SPZ_EEMPTY (no rows), SPZ_EINVAL (n_steps < 0), SPZ_EHIP. */
int spz_update(spz_ctx* ctx, int32_t n_steps, void* hip_stream);

/* Wait for all work the context enqueued. */
int spz_synchronize(spz_ctx* ctx);

/* Actions for the experience-sampling processes (Section 3.1.1: the policy
 * network acts on the observations collected from N samplers; Section 3.1.2: the
 * test and visualisation processes use the policy without randomisation).
 * obs: host float32 [n, obs_dim]; act: host float32 [n, act_dim] (caller-owned).
 * SAC: stochastic = 0 gives the mean action tanh(mu); stochastic = 1 a policy
 * sample tanh(mu + exp(clip(log_std)) eps) with eps from Philox purpose 4 at
 * counter `counter` (step word), element index row * act_dim + j, so a call is
 * reproducible from (seed, counter). TD3: tanh of the actor output (stochastic must
 * be 0; samplers add their own exploration noise). Uses the current online actor
 * with the context's GEMM precision; rows are processed in chunks of the created
 * batch. Waits for the context's outstanding work; synchronous.
 * Errors: SPZ_EINVAL, SPZ_EHIP. */
int spz_act(spz_ctx* ctx, const float* obs, int64_t n, int32_t stochastic, uint32_t counter, float* act);

/* spz_act without allocation, for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * obs: DEVICE float32 [n, obs_dim]; act: DEVICE float32 [n, act_dim]; both owned by
 * the caller. Same actions as spz_act (same kernels, bit for bit), enqueued on
 * `hip_stream` (a hipStream_t; NULL = the null stream) without waiting: the actor
 * weights used are the ones current when the kernels run in that stream's order.
 * Intermediate values (observation operand, hidden activations, head output) live
 * in a 64 MiB device array of the library, one per GPU, held until the process ends
 * and shared by every call on that GPU: calls that overlap on one GPU (other streams,
 * other threads, other contexts) race, so order them on one stream or synchronize
 * between them. The call writes every scratch byte it reads, so the previous call's
 * contents do not matter. n is limited by that array: at most the largest multiple
 * of 256 rows with e * (pad32(obs_dim) + 2 * max_l pad32(hidden[l])) + 4 * pad32(out)
 * bytes per row (e = 2 for bf16 GEMM operands, 4 for fp32; out = 2*act_dim for SAC,
 * act_dim for TD3), plus alignment, within 64 MiB; larger n gives SPZ_EINVAL with
 * the limit in the message. Calls no hipMalloc / hipFree.
 * Errors: SPZ_EINVAL, SPZ_EHIP. */
int spz_act_noalloc(spz_ctx* ctx, const float* obs, int64_t n, int32_t stochastic, uint32_t counter, float* act,
                    void* hip_stream);

/* Checkpoints (the paper publishes weights through files, Section 3.3.1). A file
 * holds the whole learner state: online and target parameters, Adam moments,
 * log(alpha), the step counter, the Philox seed, the loss records and, with
 * SPZ_CKPT_RING, the replay ring with its write pointer and fill level. Loading it
 * into a context with the same dimensions, algorithm and GEMM precision (and ring
 * capacity, if the ring is in the file) continues bit-exactly where the saved one
 * stood. Hyper-parameters (rates, tau, ...) and the batch size are the loading
 * context's own. Both calls wait for the context's outstanding work.
 * Errors: SPZ_EINVAL (NULL), SPZ_EIO (file or mismatch), SPZ_EHIP, SPZ_ENOMEM. */
#define SPZ_CKPT_RING 1
int spz_save(spz_ctx* ctx, const char* path, int32_t flags);
int spz_load(spz_ctx* ctx, const char* path);

/* Batch size of subsequent updates (the paper's adaptive batch size, Sections
 * 3.2.1 and 3.4). 1 <= batch <= the batch given to spz_create, which sizes every
 * batch buffer. Waits for the context's outstanding work. A row's replay index
 * and noise depend only on (seed, step, row), so a context set to `batch`
 * computes what a context created with `batch` computes. Errors: SPZ_EINVAL. */
int spz_set_batch(spz_ctx* ctx, int32_t batch);

/* Current batch size (SPZ_EINVAL for NULL). */
int32_t spz_batch(const spz_ctx* ctx);

/* Adaptive batch size (Section 3.4: geometric enumeration, stopping where the
 * update frame rate saturates). Probes batch sizes b_min, 2 b_min, 4 b_min, ...
 * (the last one capped at the created batch): at each, one untimed update step,
 * then probe_steps timed steps on hip_stream (events); frame rate = batch x steps
 * / seconds. Stops after the first probe that is below (1 + tolerance) x the best
 * rate so far, or at the created batch, then sets the batch to the smallest probed
 * size within (1 - tolerance) of the best rate and returns it in *chosen. The
 * probes are real update steps: they advance the step counter and the networks.
 * batches / frames_per_s (host, max_probes entries, may be NULL when max_probes
 * is 0) receive the probes in order; *n_probes (may be NULL) their number.
 * Synchronous. Errors: SPZ_EINVAL (b_min outside [1, created batch],
 * probe_steps < 1, tolerance outside [0, 1)), SPZ_EEMPTY, SPZ_EHIP. */
int spz_autotune_batch(spz_ctx* ctx, int32_t b_min, int32_t probe_steps, float tolerance, void* hip_stream,
                       int32_t* chosen, int32_t* batches, float* frames_per_s, int32_t max_probes,
                       int32_t* n_probes);

/* Number of update steps enqueued so far (the step counter t of the last step). */
int64_t spz_step(const spz_ctx* ctx);

/* Set the step counter (checkpoint resume, teacher forcing). Waits first. */
int spz_set_step(spz_ctx* ctx, int64_t step);

/* Float count of the object `which` in the flat layout of the published weights
 * (Section 3.3.1; negative code on error). */
int64_t spz_param_count(const spz_ctx* ctx, int32_t which);

/* Copy object `which` to the host array out[0..n_floats): the network weights the
 * update process publishes to the other processes and to checkpoints (Section
 * 3.3.1), plus the optimizer state and gradients. Waits for the context's work first. SPZ_ESIZE if n_floats != spz_param_count(ctx, which);
 * SPZ_EINVAL for a selector the algorithm does not have. */
int spz_read_params(spz_ctx* ctx, int32_t which, float* out, int64_t n_floats);

/* Overwrite object `which` from the host array in[0..n_floats): weights read back
 * from a published copy (Section 3.3.1: checkpoints; also teacher forcing). Gradient selectors are read only (SPZ_EINVAL). */
int spz_write_params(spz_ctx* ctx, int32_t which, const float* in, int64_t n_floats);

/* Copy the loss records of steps first_step .. first_step+n-1 (1-based) into
 * out[n * SPZ_REC_WIDTH]: the critic, actor and temperature losses of each update
 * step of Section 3.2 (the training curves the test process of Section 3.1.2 is
 * there to show), with the non-finite and actor-updated flags. The library keeps the last 65536 records; older or
 * not yet enqueued steps give SPZ_EINVAL. Waits first. */
int spz_read_losses(spz_ctx* ctx, float* out, int64_t first_step, int32_t n);

/* Debug copies of internal state of the last step (see SPZ_DBG_*). `bytes`
 * must equal the object's size (SPZ_ESIZE otherwise). Waits first. */
int spz_debug_read(spz_ctx* ctx, int32_t what, void* out, int64_t bytes);

/* Kernel timing (measurement). While enabled, every kernel launch of
 * spz_update is bracketed by a pair of HIP events recorded on the stream the
 * kernel runs on; spz_profile_read aggregates them per kernel shape. Enabling
 * pre-creates events for `reserve_launches` launches (more are created on
 * demand); disabling drops the records. Waits for the context's work first. */
int spz_profile_enable(spz_ctx* ctx, int32_t on, int64_t reserve_launches);

/* Restrict kernel timing to the launches of one kernel family and shape (as
 * reported by spz_profile_read: name, M, N, K), e.g. so that a timed run carries
 * the events of only the kernel it measures; name NULL times every launch again
 * (the default). Applies to launches enqueued after the call; existing records are
 * kept. `name` is copied. Errors: SPZ_EINVAL (NULL ctx). */
int spz_profile_only(spz_ctx* ctx, const char* name, int32_t M, int32_t N, int32_t K);

/* Time launches only in the update steps whose step number t (1-based, global) is a
 * multiple of `stride` (1, the default: every step), so that a long timed run carries
 * few events; launches outside update steps are timed as before. Applies to steps
 * enqueued after the call. Errors: SPZ_EINVAL (NULL ctx, stride < 1). */
int spz_profile_stride(spz_ctx* ctx, int32_t stride);

/* One aggregated kernel shape. flops / bytes are the algorithmic work of one
 * launch (2*M*N*K for matrix products; bytes the kernel must move for the
 * memory-bound kernels, 0 when not meaningful). */
typedef struct spz_kernel_stat {
  char name[32];   /* kernel family, e.g. "gemm_fwd", "gather", "adam_polyak" */
  int32_t M, N, K; /* launch shape (0 where not applicable)                   */
  int32_t bf16;    /* operand precision of a matrix product                   */
  int64_t launches;
  double total_ms; /* sum of event-measured durations                         */
  double flops;    /* per launch                                              */
  double bytes;    /* per launch                                              */
} spz_kernel_stat;

/* Copy up to max aggregated records (sorted by total time, largest first)
 * into out and their count into *n_out; waits for the context's work first. */
int spz_profile_read(spz_ctx* ctx, spz_kernel_stat* out, int32_t max, int32_t* n_out);

/* Message of the last failure: of ctx, or of the calling thread when ctx is
 * NULL. Never NULL; empty when there was none. Valid until the next call. */
const char* spz_last_error(const spz_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* SPZ_H */
