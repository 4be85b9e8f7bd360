/* batchsim.h -- C ABI of the MI355X (gfx950) batched serving-simulator rollout library.
 *
 * Paper: "Adaptive Inference Batching using Policy Gradients". The library steps many
 * independent environments in lockstep. Each environment is the paper's discrete-event
 * inference-serving simulator (Sec. 3.1): requests arrive (Sec. 3.2 workloads), wait in
 * per-class FIFO queues capped at N with load shedding, and are dispatched in batches to
 * K simulated servers whose batch latency is alpha + beta*b. The agent's MDP (Sec. 4.1)
 * observes a state vector, chooses a (server, batch size) action and receives a reward of
 * throughput minus weighted latency. The policy is an MLP (Sec. 4.2) and the rollout feeds
 * discounted returns / GAE (Sec. 4.3).
 *
 * Conventions
 *   - Every call returns an int status: SIM_OK (0) or a negative SIM_E* code. The message
 *     of the last failure on the calling thread is returned by sim_last_error(); the
 *     string is owned by the library. No call aborts or throws across the ABI.
 *   - "d_" pointers are device pointers (HBM of the context's device), allocated and
 *     owned by the caller; "h_" pointers are host pointers. The library owns the context
 *     and the per-environment state it allocates in sim_create and frees in sim_destroy.
 *   - All device work is enqueued on the stream given to sim_create and is asynchronous;
 *     errors detected on the device (an action out of range, an event loop exceeding its
 *     bound) are latched in a device flag and reported by sim_sync().
 *   - Layouts are time-major, environment-minor: element (t, e) of a [T][E] array is at
 *     t*E + e; feature f of environment e in an [F][E] observation is at f*E + e.
 *   - Times are fp64 seconds; rates are requests per second.
 *   - Randomness is a counter-based Philox4x32-10 stream keyed by the seed, with counter
 *     (env, step, purpose<<24 | j, system); the same seed gives the same rollout.
 */
#ifndef BATCHSIM_H
#define BATCHSIM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BATCHSIM_ABI_VERSION 2u

enum sim_status {
  SIM_OK = 0,
  SIM_EINVAL = -1,       /* invalid argument or configuration */
  SIM_ENOMEM = -2,       /* device allocation failed */
  SIM_EDEVICE = -3,      /* a HIP runtime call failed */
  SIM_ESTATE = -4,       /* call out of order, or a latched device-side error */
  SIM_EUNSUPPORTED = -5  /* configuration outside the compiled shapes */
};

enum { SIM_ARR_MODULATED = 0, SIM_ARR_TRACE = 1 };
enum { SIM_DWELL_INF = 0, SIM_DWELL_EXP = 1, SIM_DWELL_PARETO = 2, SIM_DWELL_DET = 3 };
enum { SIM_ROUTE_LOWEST = 0, SIM_ROUTE_RANDOM = 1, SIM_ROUTE_ROUND_ROBIN = 2,
       SIM_ROUTE_SHORTEST = 3 };
/* policy network (Sec. 4.2) */
enum { SIM_POLICY_MLP = 0, SIM_POLICY_ATTN = 1 };
enum { SIM_SVC_DET = 0, SIM_SVC_LOGN = 1, SIM_SVC_EXP = 2 };

#define SIM_MAX_SERVERS 16
#define SIM_MAX_CLASSES 4
#define SIM_MAX_STATES 4
#define SIM_MAX_QUEUE 255

/* Simulator and policy configuration (plain data, copied by sim_create).
 *  n_envs          environments stepped in lockstep (E >= 1)
 *  n_servers       K simulated servers per environment (1..16); actions are 6K (Sec. 4.1)
 *  n_classes       request classes / model types (1..4) (Sec. 3.1 request model)
 *  queue_cap       N, waiting requests per environment over all classes (Sec. 3.1, N=100)
 *  obs_dim         F, observation width, at least the state layout's width
 *  tick_s          decision interval (the agent acts once per tick)
 *  arrival_kind    SIM_ARR_MODULATED (Poisson / MMPP / ON-OFF) or SIM_ARR_TRACE
 *  n_states        states of the modulating process (1 = plain Poisson)
 *  rate[i]         arrival rate in state i (0 = no arrivals)
 *  dwell_kind[i]   law of the time spent in state i: INF, EXP(mean dwell_mean[i]),
 *                  PARETO(pareto_alpha[i], pareto_xm[i]) or DET (exactly dwell_mean[i]; a
 *                  process whose state 0 is DET starts in state 0 at t = 0, the square
 *                  wave of the Extreme Burst workload, Sec. 3.2)
 *  class_mix[c]    probability that an arrival is of class c
 *  service_kind[c] DET: alpha + beta*n; LOGN: median*exp(sigma*Z) + beta*n;
 *                  EXP: Exp with mean alpha + beta*n (Sec. 3.1 execution model)
 *  w_thr, w_class  reward weights: w_thr * throughput - latency weighted by class
 *                  (Sec. 4.1); reward_sum = 1 sums the weighted latencies, 0 averages them
 *  obs_tw          time normaliser of ages in the observation (T_window of Sec. 4.1)
 *  lambda_ref      rate normaliser of the arrival-rate features
 *  shadow          1 runs a second system per environment on the same arrivals under the
 *                  static rule "dispatch when static_bmax requests wait or the oldest has
 *                  waited static_timeout" (Sec. 1), with its own reward and counters
 *  mlp_h1, mlp_h2  hidden widths of the policy MLP; mlp_bf16 = 1 for bf16 weights and
 *                  activations with fp32 accumulation, 0 for fp32 throughout
 *  value_head      1 adds a value output column (Sec. 4.2 value head)
 *  trace_max_len   per-environment capacity of the arrays given to sim_set_trace
 *  static_route    server that takes a batch of the static rule: SIM_ROUTE_LOWEST idle
 *                  index, SIM_ROUTE_RANDOM (uniform over the idle servers) or
 *                  SIM_ROUTE_ROUND_ROBIN (first idle server from a per-environment
 *                  pointer); the Random and Round-Robin baselines of Sec. 5.1. Or
 *                  SIM_ROUTE_SHORTEST, the Shortest-Queue baseline of Sec. 5.1: every
 *                  server holds the batch it runs and at most one queued behind it; the
 *                  rule forms a batch whenever its condition holds, whether or not a
 *                  server is idle, and sends it to the server with the fewest requests
 *                  assigned and not completed among those with room (lower index on
 *                  ties), where it starts when that server is free; with no room it waits.
 *                  At most 8 servers (SIM_EUNSUPPORTED otherwise)
 *  policy_kind     SIM_POLICY_MLP (the MLP above) or SIM_POLICY_ATTN, the attention
 *                  policy of Sec. 4.2: the obs_dim features split into attn_tokens
 *                  contiguous groups, each group's terms of the input projection summed
 *                  into one token of width attn_embed; multi-head self-attention with
 *                  attn_heads heads; the mean of the tokens feeds a policy head with
 *                  mlp_h1 GELU units and, with value_head = 1, a separate value head with
 *                  mlp_h2 GELU units. fp32 only (mlp_bf16 = 0). Built shapes:
 *                  attn_embed = 4, attn_heads in {1, 2, 4}, attn_tokens in {1, 2, 4, 8}
 *                  dividing obs_dim <= 64, n_servers in {1, 2, 4}, mlp_h1, mlp_h2 <= 256 */
typedef struct sim_cfg {
  uint32_t abi_version; /* BATCHSIM_ABI_VERSION */
  uint32_t struct_size; /* sizeof(sim_cfg) */
  int32_t n_envs, n_servers, n_classes, queue_cap, obs_dim;
  double tick_s;
  int32_t arrival_kind, n_states;
  double rate[SIM_MAX_STATES];
  int32_t dwell_kind[SIM_MAX_STATES];
  double dwell_mean[SIM_MAX_STATES], pareto_alpha[SIM_MAX_STATES], pareto_xm[SIM_MAX_STATES];
  double class_mix[SIM_MAX_CLASSES];
  int32_t service_kind[SIM_MAX_CLASSES];
  double svc_alpha[SIM_MAX_CLASSES], svc_beta[SIM_MAX_CLASSES], svc_median[SIM_MAX_CLASSES];
  double svc_sigma;
  double w_thr, w_class[SIM_MAX_CLASSES];
  int32_t reward_sum;
  double obs_tw, lambda_ref;
  int32_t shadow;
  double static_timeout;
  int32_t static_bmax;
  int32_t mlp_h1, mlp_h2, mlp_bf16, value_head;
  int32_t trace_max_len;
  int32_t static_route;
  int32_t policy_kind, attn_tokens, attn_embed, attn_heads;
} sim_cfg;

/* Byte offsets of the policy weights inside one caller-owned device buffer. Weights are
 * [in][out] row-major; W1 is [F][H1], W2 [H1][H2], W3 [H2][A'] with A' = 6K + value_head.
 * Matrices are fp32, or bf16 (raw 16-bit patterns) when mlp_bf16 = 1; biases are fp32.  */
typedef struct sim_wlayout {
  size_t w1, b1, w2, b2, w3, b3; /* offsets in bytes, 256-byte aligned (MLP policy only;
                                    zero for the attention policy) */
  size_t bytes;                  /* total size of the buffer (either policy) */
  int32_t n_out;                 /* A' */
  int32_t elem_bytes;            /* 4 (fp32) or 2 (bf16) */
} sim_wlayout;

/* Byte offsets of the attention policy's weights (policy_kind = SIM_POLICY_ATTN) in one
 * caller-owned device buffer of sim_wlayout.bytes bytes, all fp32, [in][out] row-major
 * (D = attn_embed, A = 6K): w_in [F][D] and b_in [D] (input projection), w_qkv [D][3D]
 * (columns: query, key, value) and b_qkv [3D], w_o [D][D] and b_o [D] (attention output),
 * wp1 [D][mlp_h1], bp1, wp2 [mlp_h1][A], bp2 (policy head), wv1 [D][mlp_h2], bv1,
 * wv2 [mlp_h2][1], bv2 [1] (value head). Offsets are 256-byte aligned.                  */
typedef struct sim_attn_layout {
  size_t w_in, b_in, w_qkv, b_qkv, w_o, b_o;
  size_t wp1, bp1, wp2, bp2, wv1, bv1, wv2, bv2;
  size_t bytes;
} sim_attn_layout;

/* Caller-owned device buffers filled by sim_rollout. Only `actions` is required; any
 * other pointer may be NULL to skip that output.                                       */
typedef struct sim_traj {
  uint8_t* actions;       /* [T][E] sampled actions */
  float* logp;            /* [T][E] log-probability of the sampled action */
  double* reward;         /* [T][E] learned system's reward r_k */
  double* reward_shadow;  /* [T][E] static shadow system's reward (cfg.shadow = 1) */
  float* value;           /* [T+1][E] value head (cfg.value_head = 1); row T is V(obs_T) */
  float* obs;             /* [T+1][F][E] observations obs_k, k = 0..T */
  uint64_t* rchk;         /* [T][E] learned system's running checksum after each tick */
} sim_traj;

/* Per-environment integer counters and sums, system s in {0 learned, 1 shadow}. */
#define SIM_NCNT 7 /* arrivals, accepted, dropped, dispatched, batches, completed, inflight */
#define SIM_NSUM 2 /* latency sum, weighted latency sum (seconds) */

typedef struct sim_totals {
  int64_t cnt[2][SIM_NCNT]; /* summed over environments */
  double sum[2][SIM_NSUM];
} sim_totals;

typedef struct sim_ctx sim_ctx;

/* Message of the last failed call on this thread (library-owned, never NULL). */
const char* sim_last_error(void);

/* Library ABI version (BATCHSIM_ABI_VERSION). */
uint32_t sim_abi_version(void);

/* Creates a context on the current HIP device: n_envs copies of the simulator of Sec. 3.1
 * (and of the MDP of Sec. 4.1 around it). Validates cfg (SIM_EINVAL with a message naming the
 * field), allocates the structure-of-arrays environment state and queues in HBM (SIM_ENOMEM). `hip_stream` is a hipStream_t (NULL = default stream). The context is
 * not usable until sim_reset. On failure *out is NULL and nothing stays allocated.     */
int sim_create(const sim_cfg* cfg, void* hip_stream, sim_ctx** out);

/* Waits for the context's stream and frees everything it owns. NULL is allowed.        */
int sim_destroy(sim_ctx* ctx);

/* Explicit arrivals for SIM_ARR_TRACE (Sec. 3.2 trace replay): device arrays times
 * [E][trace_max_len] (nondecreasing seconds), classes [E][trace_max_len], counts [E].
 * The arrays must stay valid until the context is destroyed or given new ones.        */
int sim_set_trace(sim_ctx* ctx, const double* d_times, const uint8_t* d_classes,
                  const int32_t* d_counts);

/* Resets every environment at t = 0 (empty queues, idle servers, zero counters, the
 * modulating state of the Sec. 3.2 arrival process drawn from its stationary law) and sets the
 * tick counter to 0: the start of an episode (Sec. 4.3).                                */
int sim_reset(sim_ctx* ctx, uint64_t seed);

/* Copies the current observation [F][E] fp32 (the state of Sec. 4.1) to d_obs.         */
int sim_obs(sim_ctx* ctx, float* d_obs);

/* One step of the MDP (Sec. 4.1): advances every environment by one tick of the simulator
 * (Sec. 3.1) under the given actions (d_actions [E], values in [0, 6K): server a/6, batch size
 * 2^(a%6)). Optional outputs: the next observation
 * [F][E], the learned and shadow rewards [E]. An action out of range latches SIM_ESTATE.*/
int sim_step(sim_ctx* ctx, const uint8_t* d_actions, float* d_obs_next, double* d_reward,
             double* d_reward_shadow);

/* Current tick index (number of ticks since the last reset). */
int sim_tick(sim_ctx* ctx, int32_t* h_tick);

/* Layout of the weights buffer for this configuration (no device work).                */
int sim_weights_layout(const sim_cfg* cfg, sim_wlayout* out);

/* Offsets of the attention policy's weights (Sec. 4.2); SIM_EINVAL unless
 * cfg->policy_kind = SIM_POLICY_ATTN with a valid attention shape.                      */
int sim_attn_weights_layout(const sim_cfg* cfg, sim_attn_layout* out);

/* Initialises the policy network of Sec. 4.2: writes Xavier-uniform weights drawn from
 * `seed` and zero biases into d_weights
 * (layout of sim_weights_layout, or of sim_attn_weights_layout for the attention policy,
 * whose seven matrices take weight-stream layers 0..6 in layout order).                 */
int sim_init_weights(sim_ctx* ctx, uint64_t seed, void* d_weights);

/* Policy on one batch of observations d_obs [F][E]: MLP (or attention) forward, then an
 * action sampled from the softmax of the logits with the ACTION uniform of (env, step).
 * Outputs (any may be NULL): d_act [E], d_logp [E], d_value [E] (value head),
 * d_logits [A'][E] fp32.                                                                */
int sim_policy(sim_ctx* ctx, const void* d_weights, const float* d_obs, uint32_t step,
               uint8_t* d_act, float* d_logp, float* d_value, float* d_logits);

/* Diagnostics for the parity tests of the policy MLP (Sec. 4.2): sim_policy, run by the same
 * kernel source instantiated with extra stores, which also writes every hidden activation as
 * the kernel hands it to the next layer: d_hidden [H1 + H2][E] fp32 (rows 0..H1-1 the first
 * hidden layer, then the second; in bf16 configurations the bf16 values, widened). Its other
 * outputs equal sim_policy's bit for bit. SIM_EUNSUPPORTED for the attention policy.       */
int sim_policy_hidden(sim_ctx* ctx, const void* d_weights, const float* d_obs, uint32_t step,
                      uint8_t* d_act, float* d_logp, float* d_value, float* d_logits,
                      float* d_hidden);

/* A rollout of the MDP (Sec. 4.1) under the policy of Sec. 4.2, the trajectory that the
 * updates of Sec. 4.3 consume: T ticks of policy + simulator from the current state
 * (obs_k -> a_k -> obs_{k+1}), writing the trajectory; with a value head, row T of
 * traj->value holds V(obs_T). Ordered on the context's stream like every other call: the
 * static shadow system's launches run on a second stream of the context, forked from the
 * context's stream when the rollout starts and joined back before it ends (one stream when
 * sim_set_timing is on). Small batches run all T ticks in one fused launch
 * (sim_set_fused_rollout), with the same outputs. Afterwards sim_obs returns obs_T.      */
int sim_rollout(sim_ctx* ctx, const void* d_weights, int32_t T, const sim_traj* traj);

/* Rollout graphs, on by default: when sim_rollout is called again with the same weights
 * buffer, T, trajectory pointers and starting tick as the call before (a training loop that
 * resets and rolls out into the same buffers), its launch sequence is captured into a HIP
 * graph on a private stream of the context, and that graph is replayed by every further
 * repeat (ordered after earlier work on the context's stream, and before later work, by
 * events). Kernels read the seed from device memory written by sim_reset, so a new seed needs
 * no new graph. Tracing (sim_set_timing) launches eagerly. sim_set_trace discards the graph.
 * on = 0 launches every rollout eagerly.                                                    */
int sim_set_graphs(sim_ctx* ctx, int32_t on);

/* Fused rollouts of small batches (Sec. 4.1-4.2: the same ticks and policy as above): with a
 * few thousand environments a tick's two launches are bound by their start-up and memory
 * latency rather than their work, so sim_rollout may instead run all T ticks in one launch,
 * each workgroup alternating the policy and the tick of its own environments (outputs
 * bit-identical to the per-tick launches). mode SIM_FUSE_AUTO (the default) fuses when the
 * policy is an MLP of a shape that has a fused kernel (the 8-64-64-6 fp32, 12-128-128-6,
 * 32-256-256-24 and 64-256-256-48 bf16 networks, any action count up to the padded width)
 * and all of the batch's workgroups of that kernel are resident on the GPU at once;
 * SIM_FUSE_ON fuses whenever the shape has a fused kernel; SIM_FUSE_OFF always launches per
 * tick. SIM_EINVAL for another mode. A change discards the rollout graph.                  */
enum { SIM_FUSE_OFF = 0, SIM_FUSE_AUTO = 1, SIM_FUSE_ON = 2 };
int sim_set_fused_rollout(sim_ctx* ctx, int32_t mode);

/* Diagnostics of the rollout graphs: graphs captured and rollouts replayed from a graph so far
 * (either pointer may be NULL).                                                          */
int sim_graph_stats(sim_ctx* ctx, int64_t* h_captures, int64_t* h_replays);

/* Discounted returns and GAE (Sec. 4.3), per environment backwards in t:
 *   delta_t = (r_t + gamma V_{t+1}) - V_t,  A_t = delta_t + (gamma*lambda) A_{t+1},
 *   A_T = 0,  R_t = A_t + V_t.
 * d_r [T][E] fp64; d_v [T+1][E] fp32 or NULL for V = 0 (with lambda = 1 this is the
 * REINFORCE return). Writes d_adv and d_ret [T][E] fp64.                                */
int returns_gae(sim_ctx* ctx, int32_t T, const double* d_r, const float* d_v, double gamma,
                double lambda, double* d_adv, double* d_ret);

/* One PPO minibatch (Sec. 4.3, clipped surrogate): M samples (t, env) drawn with
 * replacement, sample m taking u from the MINIBATCH block at counter
 * (m, 0xFFFFFFFD, MINIBATCH<<24, 0) under `seed` and index i = floor(u T E), t = i / E,
 * env = i % E. Forward through the policy (layer inputs rounded as in sim_policy, exact
 * GELU) and the loss
 *   L = -mean(min(rho A, clip(rho, 1-clip, 1+clip) A)) + c_value mean((V - R)^2)
 *       - c_entropy mean(H),   rho = exp(logp(a) - logp_old),
 * then dL/dW for every weight, the roundings passed through as the identity.
 * Inputs (device, read only): d_weights (layout of sim_weights_layout), d_obs [T][F][E]
 * fp32 (rows 0..T-1 of a rollout's observations), d_actions [T][E] u8, d_logp_old [T][E]
 * fp32, d_adv and d_ret [T][E] fp64. Outputs (device, caller-owned): d_grads fp32,
 * W1 [F][H1], b1 [H1], W2 [H1][H2], b2 [H2], W3 [H2][A'], b3 [A'] packed back to back
 * (A' = 6K + 1; sim_ppo_grad_count gives the total); d_loss [4] fp64 = total, policy,
 * value and entropy terms; d_index [M] int64 (t E + env) or NULL. Requires value_head = 1,
 * M > 0 and a multiple of 16, hidden widths that are multiples of 64, obs_dim <= 128 and
 * A' <= 128 (SIM_EUNSUPPORTED otherwise). The dense products run on the matrix cores: bf16 x bf16 -> fp32
 * for a bf16 policy (the fp32 gradient operand carried as two bf16 terms, 2^-17 relative),
 * fp32 x fp32 otherwise; the reductions over the samples are summed in a fixed order, so
 * repeated calls return identical results. Scratch of at most Mp (e (2 F + 4 H1 + 6 H2 + 4 A')
 * + 4 (H1 + H2 + A')) bytes (Mp = M rounded up to 64, e = 2 bytes for bf16 or 4 for fp32,
 * F and A' rounded up to 64) plus about 8 MiB of split-k partial sums is held by the context
 * after the first call (grown if a later call needs more). A stored action out of range latches SIM_ESTATE (reported by sim_sync);
 * that sample then contributes nothing.
 * For the attention policy (policy_kind = SIM_POLICY_ATTN) the forward is fp32 with exact
 * GELU and d_grads holds the fourteen arrays of sim_attn_layout in its order (w_in, b_in,
 * w_qkv, b_qkv, w_o, b_o, wp1, bp1, wp2, bp2, wv1, bv1, wv2, bv2), each [in][out] as in the
 * weights; per-sample gradient terms are summed over the minibatch in a fixed order (the
 * scratch then holds 4 M P + 24 M bytes, P = sim_ppo_grad_count).                        */
int ppo_minibatch_grad(sim_ctx* ctx, const void* d_weights, int32_t T, const float* d_obs,
                       const uint8_t* d_actions, const float* d_logp_old, const double* d_adv,
                       const double* d_ret, int32_t M, uint64_t seed, float clip, float c_value,
                       float c_entropy, float* d_grads, double* d_loss, int64_t* d_index);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * training loops, harnesses that forbid hipMalloc): ppo_minibatch_grad with the same arguments,
 * inputs, outputs, error behaviour and results, bit for bit, but run on a fixed scratch the
 * library holds in device memory (96 MiB per GPU, allocated when the library's code is loaded
 * on that GPU and kept until the process ends) instead of the context's on-demand buffer. It
 * calls no hipMalloc, hipFree or other allocating routine and records no tracing events.
 * SIM_EINVAL, with the sizes in the message, when the minibatch needs more scratch than that
 * (C4's shape at M = 8192 needs about 76 MiB). Every call on a GPU uses the same scratch: calls
 * whose work overlaps on one GPU (several streams or threads) race and must be serialised by
 * the caller; calls in order on one stream are safe. The scratch keeps the previous call's
 * contents; every byte a call reads is written by that call first.                        */
int ppo_minibatch_grad_noalloc(sim_ctx* ctx, const void* d_weights, int32_t T,
                               const float* d_obs, const uint8_t* d_actions,
                               const float* d_logp_old, const double* d_adv, const double* d_ret,
                               int32_t M, uint64_t seed, float clip, float c_value,
                               float c_entropy, float* d_grads, double* d_loss, int64_t* d_index);

/* Number of fp32 gradient values written by ppo_minibatch_grad (no device work), for either
 * policy network.                                                                       */
int sim_ppo_grad_count(const sim_cfg* cfg, int64_t* h_count);

/* REINFORCE with a learned baseline (Sec. 4.3) on one minibatch: as ppo_minibatch_grad, with
 * the policy term -mean(A log pi(a|s)) (A held constant) and no old log-probabilities; the
 * caller passes A = G - V and R = G (returns_gae with lambda = 1 gives both).            */
int reinforce_minibatch_grad(sim_ctx* ctx, const void* d_weights, int32_t T, const float* d_obs,
                             const uint8_t* d_actions, const double* d_adv, const double* d_ret,
                             int32_t M, uint64_t seed, float c_value, float c_entropy,
                             float* d_grads, double* d_loss, int64_t* d_index);

/* Master parameters from a weights buffer: d_params (device, sim_ppo_grad_count fp32 values
 * in the gradient layout) receives the values d_weights holds.                          */
int sim_params_from_weights(sim_ctx* ctx, const void* d_weights, float* d_params);

/* One Adam step (Kingma & Ba 2015, Algorithm 1) on the fp32 master parameters, in place:
 *   m = b1 m + (1-b1) g,  v = b2 v + (1-b2) g^2,  p -= lr (m/(1-b1^t)) / (sqrt(v/(1-b2^t)) + eps)
 * with t = step >= 1 (the step being taken); d_m, d_v are the caller's moment buffers (zero
 * before the first step). With d_weights non-NULL the policy's weights are then rewritten from
 * the parameters (matrices rounded to bf16, nearest even, in bf16 configurations; copied as
 * they are for the fp32 attention policy).                                              */
int adam_update(sim_ctx* ctx, float* d_params, const float* d_grads, float* d_m, float* d_v,
                int32_t step, float lr, float beta1, float beta2, float eps, void* d_weights);

enum sim_algo { SIM_ALGO_PPO = 0, SIM_ALGO_REINFORCE = 1 };

typedef struct sim_update_cfg {
  int32_t algo;         /* SIM_ALGO_PPO or SIM_ALGO_REINFORCE */
  int32_t epochs;       /* passes over the trajectory */
  int32_t minibatches;  /* minibatches per epoch */
  int32_t M;            /* samples per minibatch (multiple of 16) */
  uint64_t seed;        /* minibatch b of epoch e: key seed + (e*minibatches + b)*0x9E3779B97F4A7C15 */
  float clip;           /* PPO clip range epsilon */
  float c_value, c_entropy;
  float lr, beta1, beta2, eps;
} sim_update_cfg;

/* The policy update of Sec. 4.3 over one stored trajectory (d_obs [T][F][E], d_actions,
 * d_logp_old (PPO only) [T][E], d_adv, d_ret [T][E] fp64): for each epoch and minibatch,
 * the minibatch gradient and one Adam step, after which d_weights holds the new policy.
 * *h_step is Adam's step count, advanced once per minibatch. d_losses (optional, device)
 * receives [epochs*minibatches][4] fp64 loss terms, each from the weights before its step. */
int sim_update(sim_ctx* ctx, const sim_update_cfg* cfg, void* d_weights, float* d_params,
               float* d_m, float* d_v, int32_t* h_step, int32_t T, const float* d_obs,
               const uint8_t* d_actions, const float* d_logp_old, const double* d_adv,
               const double* d_ret, double* d_losses);

/* Per-environment counters [2][SIM_NCNT][E] int64 and sums [2][SIM_NSUM][E] fp64 into
 * device buffers (either may be NULL).                                                  */
int sim_counters(sim_ctx* ctx, int64_t* d_cnt, double* d_sum);

/* Per-environment integer-state checksums [2][E] (learned, shadow) into d_chk.          */
int sim_checksums(sim_ctx* ctx, uint64_t* d_chk);

/* Totals of the counters over all environments, reduced on the device, into h_out.
 * Synchronises the stream.                                                              */
int sim_stats(sim_ctx* ctx, sim_totals* h_out);

/* Waits for the stream; returns SIM_ESTATE if a device-side error was latched (and
 * clears it), with the reason in sim_last_error().                                     */
int sim_sync(sim_ctx* ctx);

/* Checkpoint and resume of the simulation: a snapshot holds every environment's state of both
 * systems (queues and timestamp rings, servers, counters, sums and checksums, arrival
 * processes, arrival-rate averages, the current observation, latched error flags) and the
 * context's tick counter and seed, behind a 256-byte header. sim_get_state with buf = NULL
 * stores the snapshot size in *bytes; otherwise *bytes must be at least that size and buf
 * (device or host memory) receives the snapshot after the work already enqueued on the
 * stream; the copy is complete when the call returns. sim_set_state restores a snapshot
 * into a context whose configuration has the same layout (n_envs, n_servers, n_classes,
 * queue_cap, obs_dim, shadow; SIM_EINVAL otherwise, or for a buffer that is not a snapshot
 * of this library version). Trace arrivals (sim_set_trace) are caller memory and not part
 * of the snapshot: set the same trace again before resuming. Continuing from a restored
 * snapshot reproduces the original continuation bit for bit (the counter-based random
 * draws depend only on the seed, the environment and the tick).                          */
int sim_get_state(sim_ctx* ctx, void* buf, size_t* bytes);
int sim_set_state(sim_ctx* ctx, const void* buf, size_t bytes);

/* Diagnostics: one of the library's device primitives evaluated elementwise on n inputs, so
 * that its bit identity with a host implementation can be checked directly (the parity of
 * whole rollouts depends on it). All arrays are device memory owned by the caller; the work
 * is enqueued on hip_stream (NULL: the default stream) and complete after it synchronizes.
 *   SIM_PRIM_PHILOX  d_in uint32 [n][4] counters, d_out uint32 [n][4]: the Philox4x32-10
 *                    block of each counter under the 64-bit key (low word first) (R13)
 *   SIM_PRIM_LOG, SIM_PRIM_EXP, SIM_PRIM_COS  fp64 [n] -> fp64 [n]: the deterministic
 *                    logarithm, exponential and cosine of the arrival and service draws (R14)
 *   SIM_PRIM_SQRT    fp64 [n] -> fp64 [n], correctly rounded square root
 *   SIM_PRIM_DIV     fp64 [n][2] -> fp64 [n], the first of each pair divided by the second
 * SIM_EINVAL for an unknown kind, n < 0 or NULL arrays with n > 0.                          */
enum { SIM_PRIM_PHILOX = 0, SIM_PRIM_LOG = 1, SIM_PRIM_EXP = 2, SIM_PRIM_COS = 3,
       SIM_PRIM_SQRT = 4, SIM_PRIM_DIV = 5 };
int sim_device_primitive(int32_t kind, int64_t n, uint64_t key, const void* d_in, void* d_out,
                         void* hip_stream);

/* Kernel classes for tracing. */
enum sim_kernel_class {
  SIM_KC_POLICY = 0,  /* policy MLP + sampler */
  SIM_KC_STEP = 1,    /* learned system, one tick */
  SIM_KC_STATIC = 2,  /* static shadow system, one tick */
  SIM_KC_GAE = 3,     /* returns / GAE */
  SIM_KC_RESET = 4,   /* reset */
  SIM_KC_OTHER = 5,   /* weight repack / init, observation packing, counters, totals */
  SIM_KC_PPO = 6,     /* policy update: minibatch gradients, Adam */
  SIM_KC_ROLLOUT = 7, /* fused rollout: every tick's policy and learned tick in one launch */
  SIM_KC_COUNT = 8
};

/* Tracing: with `on` != 0 every kernel launch of the context is bracketed by a pair of
 * HIP events recorded on the context's stream. sim_get_timing synchronises the stream
 * and adds the elapsed time of every completed pair to per-class totals, then writes the
 * totals (milliseconds) and launch counts to h_ms[SIM_KC_COUNT] and
 * h_launches[SIM_KC_COUNT]; `clear` != 0 zeroes the totals afterwards.               */
int sim_set_timing(sim_ctx* ctx, int32_t on);
int sim_get_timing(sim_ctx* ctx, double* h_ms, int64_t* h_launches, int32_t clear);

#ifdef __cplusplus
}
#endif
#endif /* BATCHSIM_H */
