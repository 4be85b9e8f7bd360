/* oracle.h -- plain sequential CPU oracle of the batched inference-serving rollout.
 *
 * TEST INFRASTRUCTURE. Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline
 * leg may load or call this library. It shares no code, header, table or constant
 * generator with the HIP path under paper_2607_05272_amd/ and include/.
 *
 * What it computes (paper: "Adaptive Inference Batching using Policy Gradients"):
 *   - the discrete-event simulator of Sec. 3.1 (arrivals, FIFO queue with a cap of N and
 *     load shedding, the batch-latency model L(b) = alpha + beta*b, K servers and a
 *     central dispatcher), driven by the workloads of Sec. 3.2;
 *   - the MDP of Sec. 4.1 (state vector, batch/routing action, reward of throughput minus
 *     weighted latency);
 *   - the policy networks of Sec. 4.2: the MLP (GELU hidden layers, categorical head,
 *     value column) and the attention policy (input projection to tokens, multi-head
 *     self-attention, mean pooling, GELU policy head and a separate GELU value head);
 *   - the static timeout rule run as a shadow system (Sec. 1) and the baseline routing rules
 *     of Sec. 5.1 (lowest idle, random and round-robin idle server, Shortest-Queue over
 *     per-server FIFOs of two batches);
 *   - discounted returns (REINFORCE) and GAE (PPO) of Sec. 4.3.
 * Every reading of a point the paper leaves open is numbered R1..R27; the comments in
 * oracle.c name the reading each step follows.
 *
 * Every function runs one environment at a time, event by event, in fp64 with no
 * implicit contraction (built with -ffp-contract=off). Parity functions:
 *   pinned:   the Philox4x32-10 block (bit for bit vs PyTorch's independent engine; its
 *             structure also vs numpy's Philox4x64), det_log/det_exp/det_cos (vs libm),
 *             samplers (KS / chi-square vs scipy), the class draw and the arrival stream's
 *             counter layout, the lognormal service law with its linear term, the
 *             stationary start, queue dynamics (M/D/1, M/M/1, M/M/1/K, M/M/c closed forms;
 *             the M/M/2 bracket of Shortest-Queue), Little's law (exact sample-path
 *             identity), conservation, hand-enumerated traces (incl. the multi-server,
 *             multi-class observation and Shortest-Queue routing), MLP (vs torch fp64),
 *             attention policy (vs torch.nn.MultiheadAttention in fp64, one-token and
 *             uniform-attention closed forms, feature-permutation invariance), GAE (closed
 *             forms).
 */
#ifndef ORACLE_H
#define ORACLE_H
#include <stdint.h>

#define ORC_MAX_K 16
#define ORC_MAX_C 4
#define ORC_MAX_S 4
#define ORC_MAX_N 255

enum { ORC_ARR_MODULATED = 0, ORC_ARR_TRACE = 1 };
enum { ORC_DWELL_INF = 0, ORC_DWELL_EXP = 1, ORC_DWELL_PARETO = 2, ORC_DWELL_DET = 3 };
enum { ORC_ROUTE_LOWEST = 0, ORC_ROUTE_RANDOM = 1, ORC_ROUTE_ROUND_ROBIN = 2, ORC_ROUTE_SHORTEST = 3 };
enum { ORC_SVC_DET = 0, ORC_SVC_LOGN = 1, ORC_SVC_EXP = 2 };
enum { ORC_POLICY_MLP = 0, ORC_POLICY_ATTN = 1 };
#define ORC_ATTN_MAX_L 16   /* tokens */
#define ORC_ATTN_MAX_D 16   /* embedding width */
enum { ORC_P_ARRIVAL = 1, ORC_P_PROCESS = 2, ORC_P_SERVICE = 3, ORC_P_ACTION = 4,
       ORC_P_WEIGHTS = 5, ORC_P_MINIBATCH = 6, ORC_P_ROUTE = 7 };
#define ORC_STEP_RESET 0xFFFFFFFFu

typedef struct orc_cfg {
  int32_t n_servers, n_classes, queue_cap, obs_dim;
  double tick_s;
  int32_t arrival_kind, n_states;
  double rate[ORC_MAX_S];
  int32_t dwell_kind[ORC_MAX_S];
  double dwell_mean[ORC_MAX_S], pareto_alpha[ORC_MAX_S], pareto_xm[ORC_MAX_S];
  double class_mix[ORC_MAX_C];
  int32_t service_kind[ORC_MAX_C];
  double svc_alpha[ORC_MAX_C], svc_beta[ORC_MAX_C], svc_median[ORC_MAX_C];
  double svc_sigma;
  double w_thr, w_class[ORC_MAX_C];
  int32_t reward_sum;
  double obs_tw, lambda_ref;
  int32_t shadow;
  double static_timeout;
  int32_t static_bmax;
  int32_t mlp_h1, mlp_h2, mlp_bf16, value_head;
  int32_t static_route;          /* ORC_ROUTE_*: server choice of the static system (R23, R27) */
  /* policy network (R16, R26): the MLP, or the attention policy of Sec. 4.2 with
   * attn_tokens tokens of width attn_embed and attn_heads heads; its policy head has
   * mlp_h1 hidden units and its value head mlp_h2 */
  int32_t policy_kind, attn_tokens, attn_embed, attn_heads;
} orc_cfg;

/* Explicit arrivals for ORC_ARR_TRACE: times [n_env][max_len] (seconds, nondecreasing),
 * classes [n_env][max_len], counts [n_env]. */
typedef struct orc_trace {
  const double* times;
  const uint8_t* classes;
  const int32_t* counts;
  int32_t max_len;
} orc_trace;

/* Policy weights in fp64 (each value already rounded to the layer's storage precision).
 * W_l is [in][out] row-major. A' = 6K + value_head.
 * MLP: w1 [F][H1], w2 [H1][H2], w3 [H2][A'].
 * Attention (R26, D = attn_embed, A = 6K): w_in [F][D], w_qkv [D][3D] (columns: query,
 * key, value), w_o [D][D], wp1 [D][mlp_h1], wp2 [mlp_h1][A], wv1 [D][mlp_h2], wv2
 * [mlp_h2][1], each with its bias. */
typedef struct orc_weights {
  const double *w1, *b1, *w2, *b2, *w3, *b3;
  const double *w_in, *b_in, *w_qkv, *b_qkv, *w_o, *b_o;
  const double *wp1, *bp1, *wp2, *bp2, *wv1, *bv1, *wv2, *bv2;
} orc_weights;

#define ORC_REC_W 10   /* n_k, dispatches, sumQ, A_k, dropped(cum), completed(cum), Q[0..3] */
#define ORC_NCNT 7     /* arrivals, accepted, dropped, dispatched, batches, completed, inflight */
#define ORC_NSUM 6     /* lat_sum, wlat_sum, wait_sum, area_n, area_q, sojourn_sum */

typedef struct orc_disp {
  int32_t env_idx, sys, k, server, cls, n;
  double t, c;
} orc_disp;

/* Output arrays; any pointer may be NULL. n = number of simulated envs. */
typedef struct orc_out {
  double* reward;          /* [T][n] learned system */
  double* reward_shadow;   /* [T][n] static shadow system */
  float* obs;              /* [T+1][n][F] learned system */
  int32_t* rec;            /* [T][n][2][ORC_REC_W] */
  uint64_t* chk;           /* [n][2] final checksums */
  uint64_t* rchk;          /* [T][n] learned running checksum after each tick */
  int64_t* counters;       /* [n][2][ORC_NCNT] */
  double* sums;            /* [n][2][ORC_NSUM] */
  orc_disp* disp;          /* dispatch log, capacity disp_cap */
  int64_t disp_cap;
  int64_t disp_count;      /* written by the oracle */
  /* policy mode */
  uint8_t* actions;        /* [T][n] */
  float* logp;             /* [T][n] */
  float* value;            /* [T+1][n] */
  double* logits;          /* [T][n][A'] fp64 logits */
  double* margin;          /* [T][n] distance of u to the nearest CDF boundary */
} orc_out;

#endif
