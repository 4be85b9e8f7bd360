// params.hpp -- kernel parameter blocks and launch entry points shared by the runtime
// (runtime.hip) and the kernel translation units of this library.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bsim {

constexpr int kMaxK = 16, kMaxC = 4, kMaxS = 4;
constexpr int kNcnt = 6;                 // arrivals, accepted, dropped, dispatched, batches, completed
constexpr uint32_t kMaxEventsPerTick = 1u << 16;
enum : uint32_t { ERR_ACTION = 1u, ERR_EVENTS = 2u, ERR_TRACE = 4u };

// Simulator constants, all derived on the host once per context.
struct SimParams {
  int E, K, C, N, F, S;
  int arrival_kind, shadow, bmax, reward_sum;
  int route;                             // server choice of the static rule (SIM_ROUTE_*;
                                         // 3 = Shortest-Queue)
  double dt;
  double rate[kMaxS], mean_gap[kMaxS], dwell_mean[kMaxS], inv_alpha[kMaxS], xm[kMaxS];
  int dwell_kind[kMaxS];
  double stat_cum[kMaxS], class_cum[kMaxC];
  int svc_kind[kMaxC];
  double svc_alpha[kMaxC], svc_beta[kMaxC], svc_median[kMaxC], svc_sigma;
  double w_thr, w_class[kMaxC];
  double inv_n, inv_tw, inv_c, inv_rs;   // observation normalisers (reciprocals)
  double static_timeout;
  const double* tr_times;
  const uint8_t* tr_cls;
  const int32_t* tr_cnt;
  int tr_len;
};

// Structure-of-arrays state of one queueing system; each array is [field][E]. Each system
// carries its own copy of the arrival process: its draws do not depend on the system, so
// both copies follow the same arrivals.
struct SysState {
  uint32_t* qpack;   // [E]     Q_c in byte c
  uint32_t* hpack;   // [E]     ring head of class c in byte c
  double* hts;       // [C][E]  arrival time of the head request of class c
  double* busy;      // [K][E]  busy-until time of server j (Shortest-Queue: its running batch)
  double* busy2;     // [K][E]  Shortest-Queue only: completion of the batch queued on server j
  uint32_t* meta;    // [K][E]  inflight | last_b << 8 | last_class << 16 (0xFF = none);
                     //         Shortest-Queue: running size | queued size << 24
  uint32_t* cnt;     // [6][E]  arrivals, accepted, dropped, dispatched, batches, completed
  double* sums;      // [2][E]  latency sum, weighted latency sum
  uint64_t* chk;     // [E]     checksum of the integer-state sequence
  double* ring;      // [E][C][N] arrival timestamps (per-class FIFO rings)
  uint32_t* proc;    // [E]     modulating state of the arrival process
  double* next_sw;   // [E]     next modulating-state switch
  double* next_arr;  // [E]     next arrival
  uint32_t* tr_idx;  // [E]     next trace arrival index
  uint32_t* rr;      // [E]     round-robin pointer (static system)
};

struct EnvState {
  SysState sys[2];   // 0 learned, 1 static shadow
  double* ewma;      // [4][E] exponentially weighted arrival counts (learned system)
  float* obs;        // [F][E] current observation
  uint32_t* obs_bf;  // [ceil(F/2)][E] its bf16 pairs, for a bf16 policy (NULL otherwise); the
                     // pairs are packed from obs at the start of a rollout, then written by
                     // its ticks (which skip obs except on the rollout's last tick)
  uint32_t* err;     // [1] latched error flags
  uint64_t* seed;    // [1] the episode seed (written by reset_k, read by every kernel that draws)
};

// Kernel launchers (asynchronous on `st`); each returns the launch's hipError_t.
hipError_t launch_reset(const SimParams& p, const EnvState& s, uint64_t seed, hipStream_t st);
// obs_mode: kObsF32 writes the current observation s.obs, kObsBf16 its bf16 pairs s.obs_bf
constexpr int kObsF32 = 1, kObsBf16 = 2;
hipError_t launch_step(const SimParams& p, const EnvState& s, uint32_t k,
                       const uint8_t* act, float* obs_out, int obs_mode, double* rew,
                       uint64_t* rchk, hipStream_t st);
// s.obs_bf from s.obs (feature pairs (2m, 2m + 1), a missing last feature as zero)
hipError_t launch_obs_pack(const SimParams& p, const EnvState& s, hipStream_t st);
// ticks k .. k + nt - 1 of the static shadow system; rew_sh [nt][E] or NULL
hipError_t launch_static(const SimParams& p, const EnvState& s, uint32_t k,
                         int nt, double* rew_sh, hipStream_t st);
hipError_t launch_counters(const SimParams& p, const EnvState& s, int64_t* cnt, double* sums,
                           hipStream_t st);
hipError_t launch_totals(const SimParams& p, const EnvState& s, int64_t* d_tot_cnt,
                         double* d_tot_sum, hipStream_t st);
hipError_t launch_gae(int T, int E, const double* r, const float* v, double gamma, double lam,
                      double* adv, double* ret, hipStream_t st);

// Policy network shapes and packed weights (MFMA-friendly, out-major, zero padded).
struct MlpParams {
  int E, F, H1, H2, A, Ap;      // A = 6K actions, Ap = A + value_head
  int bf16, value_head;
  int FP, AP;                   // padded input width and padded output width
  // repacked weights: bf16 in MFMA fragment order (see repack_frag_k), fp32 as W^T
  // [H1][FP], [H2][H1], [AP][H2]; biases zero padded to the padded output widths
  const void* w1; const float* b1;
  const void* w2; const float* b2;
  const void* w3; const float* b3;
};
hipError_t launch_repack(const MlpParams& m, const void* d_weights, const size_t off[6],
                         void* w1, float* b1, void* w2, float* b2, void* w3, float* b3,
                         hipStream_t st);
// hidden != NULL runs the diagnostic instantiation that also writes the hidden activations
// passed between layers: [H1][E] then [H2][E] fp32
// obs_bf != NULL (bf16 policies only) reads the observation as its bf16 pairs [F/2][E] instead
// of obs
hipError_t launch_policy(const MlpParams& m, const float* obs, const uint32_t* obs_bf,
                         const uint64_t* seed, uint32_t step, uint8_t* act, float* logp,
                         float* value, float* logits, float* hidden, hipStream_t st);
hipError_t launch_init_weights(int F, int H1, int H2, int Ap, int bf16, uint64_t seed,
                               void* d_weights, const size_t off[6], hipStream_t st);

// Trajectory rows written by a fused rollout: act, logp, value, rew, rchk [T][E] (value
// [T + 1][E]), obs [T + 1][F][E] from row 1; NULL entries (act excepted) are not written.
struct RolloutOut {
  uint8_t* act;
  float* logp;
  float* value;
  double* rew;
  uint64_t* rchk;
  float* obs;
};
// the number of environments whose workgroups of the fused rollout kernel are all resident on
// the current device at once (0 with hipErrorNotSupported: no fused kernel for the network)
hipError_t fused_rollout_capacity(const SimParams& p, const MlpParams& m, int* max_envs);
// T ticks from k0 of the learned system with its MLP policy in one launch (the static shadow
// system is not part of it); a bf16 policy needs s.obs_bf packed from s.obs beforehand.
// hipErrorNotSupported for other policy shapes.
hipError_t launch_rollout_fused(const SimParams& p, const EnvState& s, const MlpParams& m,
                                uint32_t k0, int T, const RolloutOut& o, hipStream_t st);
bool policy_shape_supported(const MlpParams& m);

// The attention policy (attn_kernels.hip): fp32 weights [in][out] inside the caller's
// buffer; D = 4 embedding, NH heads, L tokens over F features, heads of Hp and Hv units.
struct AttnParams {
  int E, F, L, D, NH, Hp, Hv, A, value_head;
  const float *w_in, *b_in, *w_qkv, *b_qkv, *w_o, *b_o;
  const float *wp1, *bp1, *wp2, *bp2, *wv1, *bv1, *wv2, *bv2;
};
bool attn_shape_supported(const AttnParams& p);
hipError_t launch_attn_policy(const AttnParams& p, const float* obs, const uint64_t* seed,
                              uint32_t step,
                              uint8_t* act, float* logp, float* value, float* logits,
                              hipStream_t st);
// Minibatch gradient of the attention policy (REINFORCE with baseline or PPO): indices drawn
// as for the MLP; grads in the order w_in, b_in, w_qkv, b_qkv, w_o, b_o, wp1, bp1, wp2, bp2,
// wv1, bv1, wv2, bv2 (fp32); loss_out[4] total, policy, value, entropy (fp64); scratch of
// attn_grad_scratch_bytes bytes
int attn_param_count(const AttnParams& p, int off[14]);
size_t attn_grad_scratch_bytes(const AttnParams& p, int M);
hipError_t launch_attn_grad(const AttnParams& p, int T, const float* obs, const uint8_t* act,
                            const float* logp_old, const double* adv, const double* ret, int M,
                            uint64_t seed, float clip, float c_v, float c_h, int reinforce,
                            void* scratch, double* loss_out, float* grads, int64_t* idx_out,
                            uint32_t* err, hipStream_t st);
// the attention policy's weights from / to fp32 parameters in gradient order (plain copies)
hipError_t launch_export_attn(const AttnParams& p, const float* params, void* d_weights,
                              const size_t off[14], hipStream_t st);
hipError_t launch_import_attn(const AttnParams& p, const void* d_weights, const size_t off[14],
                              float* params, hipStream_t st);
// device primitives evaluated elementwise (prim_kernels.hip); kinds as in the ABI
enum { PRIM_PHILOX = 0, PRIM_LOG = 1, PRIM_EXP = 2, PRIM_COS = 3, PRIM_SQRT = 4, PRIM_DIV = 5 };
hipError_t launch_primitive(int kind, int64_t n, uint64_t key, const void* in, void* out,
                            hipStream_t st);
// the four loss terms from per-sample [M][3] fp64 terms, summed in a fixed order
hipError_t launch_pg_loss(const double* terms, int M, float c_v, float c_h, double* out,
                          hipStream_t st);
// Xavier init of the attention policy's seven matrices (layers 0..6) and zero biases;
// off[14] are the byte offsets of w_in, b_in, ..., wv2, bv2; fin/fout the matrix shapes
hipError_t launch_init_attn(uint64_t seed, void* d_weights, const size_t off[14], const int fin[7],
                            const int fout[7], hipStream_t st);
// MLP policy-gradient minibatch (ppo_kernels.hip), value head required: the library's own MFMA
// products with fused epilogues; scratch holds ppo_scratch_bytes(m, M) bytes.
hipError_t launch_ppo(const MlpParams& m, const void* d_weights, const size_t off[6], int T,
                      const float* obs, const uint8_t* act, const float* logp_old,
                      const double* adv, const double* ret, int M, uint64_t seed, float clip,
                      float c_v, float c_h, int reinforce, void* scratch, double* loss_out,
                      float* grads, int64_t* idx_out, uint32_t* err, hipStream_t st);
bool ppo_shape_supported(const MlpParams& m);
size_t ppo_scratch_bytes(const MlpParams& m, int M);
// The fixed device scratch of ppo_minibatch_grad_noalloc: its size, and its address on the
// current device (looked up once per device with hipGetSymbolAddress; allocates nothing).
constexpr size_t kStaticScratchBytes = (size_t)96 << 20;
hipError_t static_scratch(void** ptr);
// Adam on fp32 parameters (train_kernels.hip): one step, bias corrections bc1 = 1 - b1^t and
// bc2 = 1 - b2^t computed by the caller; then the policy's weights from the parameters
hipError_t launch_adam(float* params, const float* grads, float* m, float* v, size_t n, float lr,
                       float b1, float b2, float eps, float bc1, float bc2, hipStream_t st);
hipError_t launch_export_weights(const MlpParams& m, const float* params, void* d_weights,
                                 const size_t off[6], hipStream_t st);
hipError_t launch_import_weights(const MlpParams& m, const void* d_weights, const size_t off[6],
                                 float* params, hipStream_t st);

}  // namespace bsim
