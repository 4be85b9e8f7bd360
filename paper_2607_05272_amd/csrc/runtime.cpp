// runtime.cpp -- host runtime behind the C ABI of include/batchsim.h: configuration
// validation, derived constants, structure-of-arrays allocation in HBM, and the ordering
// of kernel launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "batchsim.h"
#include "params.hpp"

using namespace bsim;

namespace {

thread_local std::string g_err = "no error";

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(SIM_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define HIPCHK(call, what)                        \
  do {                                            \
    hipError_t e_ = (call);                       \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int obs_width(const sim_cfg& c) {
  return 2 + c.n_servers * (c.n_servers > 1 ? 4 : 2) + (c.n_classes > 1 ? 2 * c.n_classes : 0) + 4;
}

int pad_to(int x, int m) { return (x + m - 1) / m * m; }

}  // namespace

// What a rollout's launch sequence depends on besides the context itself.
struct RolloutKey {
  const void* w;
  int32_t T;
  sim_traj tr;
  uint32_t k0;
};

struct sim_ctx {
  sim_cfg cfg;
  hipStream_t stream = nullptr;
  int device = 0;
  SimParams p{};
  EnvState s{};
  MlpParams m{};
  AttnParams a{};          // attention policy (policy_kind = SIM_POLICY_ATTN)
  void* arena = nullptr;   // all environment state
  size_t arena_bytes = 0;
  void* wpack = nullptr;   // repacked policy weights
  void* ppo_scratch = nullptr;  // minibatch activations, grown on demand
  size_t ppo_bytes = 0;
  void* grads = nullptr;        // gradient + loss buffer of sim_update
  int64_t* d_tot_cnt = nullptr;
  double* d_tot_sum = nullptr;
  uint32_t tick = 0;
  uint64_t seed = 0;
  bool reset_done = false;
  bool trace_set = false;
  // rollout graph (sim_rollout): captured on a private stream the second time a call repeats
  bool graphs = true;
  hipStream_t gstream = nullptr;
  hipEvent_t gev_in = nullptr, gev_out = nullptr;
  hipGraphExec_t rgraph = nullptr;
  // a rollout's static shadow launches run on a second stream (default priority), forked
  // from and joined back to the rollout's stream by events
  hipStream_t sstream = nullptr;
  hipEvent_t sev_fork = nullptr, sev_join = nullptr;
  RolloutKey rkey{}, seen{};
  bool rkey_valid = false, seen_valid = false;
  int fuse = SIM_FUSE_AUTO;   // fused small-batch rollouts (sim_set_fused_rollout)
  int fuse_cap = -1;          // environments the fused kernel holds at once (0: none; -1: not asked)
  int64_t graph_captures = 0, graph_replays = 0;
  // tracing: event pairs around kernel launches, per kernel class
  struct Pending { int cls; hipEvent_t a, b; };
  bool timing = false;
  std::vector<hipEvent_t> pool;
  std::vector<Pending> pending;
  double ms[SIM_KC_COUNT] = {};
  int64_t launches[SIM_KC_COUNT] = {};

  hipError_t event(hipEvent_t* ev) {
    if (!pool.empty()) {
      *ev = pool.back();
      pool.pop_back();
      return hipSuccess;
    }
    return hipEventCreate(ev);
  }
  // runs `launch` (which enqueues one kernel on `stream`), bracketed by events if tracing
  template <class F>
  hipError_t timed(int cls, F launch) {
    if (!timing) return launch();
    hipEvent_t a, b;
    hipError_t e = event(&a);
    if (e != hipSuccess) return e;
    e = event(&b);
    if (e != hipSuccess) return e;
    e = hipEventRecord(a, stream);
    if (e != hipSuccess) return e;
    e = launch();
    if (e != hipSuccess) return e;
    e = hipEventRecord(b, stream);
    if (e != hipSuccess) return e;
    pending.push_back({cls, a, b});
    return hipSuccess;
  }
};

extern "C" {

const char* sim_last_error(void) { return g_err.c_str(); }

uint32_t sim_abi_version(void) { return BATCHSIM_ABI_VERSION; }

static int validate(const sim_cfg* c) {
  if (!c) return fail(SIM_EINVAL, "cfg is NULL");
  if (c->abi_version != BATCHSIM_ABI_VERSION)
    return fail(SIM_EINVAL, "abi_version %u, library is %u", c->abi_version, BATCHSIM_ABI_VERSION);
  if (c->struct_size != sizeof(sim_cfg))
    return fail(SIM_EINVAL, "struct_size %u, expected %zu", c->struct_size, sizeof(sim_cfg));
  if (c->n_envs < 1) return fail(SIM_EINVAL, "n_envs must be >= 1");
  if (c->n_servers < 1 || c->n_servers > SIM_MAX_SERVERS)
    return fail(SIM_EINVAL, "n_servers must be in 1..%d", SIM_MAX_SERVERS);
  if (6 * c->n_servers > 255) return fail(SIM_EINVAL, "6*n_servers must fit a uint8 action");
  if (c->n_classes < 1 || c->n_classes > SIM_MAX_CLASSES)
    return fail(SIM_EINVAL, "n_classes must be in 1..%d", SIM_MAX_CLASSES);
  if (c->queue_cap < 1 || c->queue_cap > SIM_MAX_QUEUE)
    return fail(SIM_EINVAL, "queue_cap must be in 1..%d", SIM_MAX_QUEUE);
  if (c->policy_kind != SIM_POLICY_MLP && c->policy_kind != SIM_POLICY_ATTN)
    return fail(SIM_EINVAL, "policy_kind");
  if (c->policy_kind == SIM_POLICY_ATTN) {
    if (c->attn_tokens < 1 || c->attn_embed < 1 || c->attn_heads < 1)
      return fail(SIM_EINVAL, "attn_tokens, attn_embed and attn_heads must be >= 1");
    if (c->obs_dim % c->attn_tokens)
      return fail(SIM_EINVAL, "attn_tokens must divide obs_dim");
    if (c->attn_embed % c->attn_heads)
      return fail(SIM_EINVAL, "attn_heads must divide attn_embed");
    if (c->mlp_bf16) return fail(SIM_EINVAL, "the attention policy is fp32 (mlp_bf16 = 0)");
    if (c->mlp_h1 < 1 || c->mlp_h2 < 1) return fail(SIM_EINVAL, "head widths must be >= 1");
  }
  if (c->obs_dim < obs_width(*c))
    return fail(SIM_EINVAL, "obs_dim %d is below the state width %d", c->obs_dim, obs_width(*c));
  if (!(c->tick_s > 0.0)) return fail(SIM_EINVAL, "tick_s must be > 0");
  if (c->arrival_kind != SIM_ARR_MODULATED && c->arrival_kind != SIM_ARR_TRACE)
    return fail(SIM_EINVAL, "arrival_kind");
  if (c->n_states < 1 || c->n_states > SIM_MAX_STATES)
    return fail(SIM_EINVAL, "n_states must be in 1..%d", SIM_MAX_STATES);
  if (c->arrival_kind == SIM_ARR_MODULATED) {
    for (int i = 0; i < c->n_states; ++i) {
      if (!(c->rate[i] >= 0.0)) return fail(SIM_EINVAL, "rate[%d] must be >= 0", i);
      const int k = c->dwell_kind[i];
      if (k < 0 || k > 3) return fail(SIM_EINVAL, "dwell_kind[%d]", i);
      if (c->n_states > 1 && k == SIM_DWELL_INF)
        return fail(SIM_EINVAL, "dwell_kind[%d] must be finite with several states", i);
      if ((k == SIM_DWELL_EXP || k == SIM_DWELL_DET) && !(c->dwell_mean[i] > 0.0))
        return fail(SIM_EINVAL, "dwell_mean[%d] must be > 0", i);
      if (k == SIM_DWELL_PARETO && (!(c->pareto_alpha[i] > 1.0) || !(c->pareto_xm[i] > 0.0)))
        return fail(SIM_EINVAL, "pareto_alpha[%d] must be > 1 and pareto_xm > 0", i);
    }
  } else if (c->trace_max_len < 1) {
    return fail(SIM_EINVAL, "trace_max_len must be >= 1 for trace arrivals");
  }
  double mix = 0.0;
  for (int i = 0; i < c->n_classes; ++i) {
    if (!(c->class_mix[i] >= 0.0)) return fail(SIM_EINVAL, "class_mix[%d] must be >= 0", i);
    mix += c->class_mix[i];
    const int k = c->service_kind[i];
    if (k < 0 || k > 2) return fail(SIM_EINVAL, "service_kind[%d]", i);
    if (!(c->svc_beta[i] >= 0.0) || !(c->svc_alpha[i] >= 0.0))
      return fail(SIM_EINVAL, "svc_alpha/svc_beta[%d] must be >= 0", i);
    if (k == SIM_SVC_LOGN && !(c->svc_median[i] > 0.0))
      return fail(SIM_EINVAL, "svc_median[%d] must be > 0", i);
    if (k == SIM_SVC_DET && !(c->svc_alpha[i] + c->svc_beta[i] > 0.0))
      return fail(SIM_EINVAL, "deterministic service of class %d must be > 0", i);
  }
  if (std::fabs(mix - 1.0) > 1e-9) return fail(SIM_EINVAL, "class_mix must sum to 1");
  // lognormal service median * exp(sigma Z): the normal draw is below 8.6 in magnitude and the
  // deterministic exponential holds for arguments below 700, so sigma is kept to [0, 64]
  for (int i = 0; i < c->n_classes; ++i)
    if (c->service_kind[i] == SIM_SVC_LOGN && !(c->svc_sigma >= 0.0 && c->svc_sigma <= 64.0))
      return fail(SIM_EINVAL, "svc_sigma must lie in [0, 64] for lognormal service");
  if (!(c->obs_tw > 0.0) || !(c->lambda_ref > 0.0))
    return fail(SIM_EINVAL, "obs_tw and lambda_ref must be > 0");
  if (c->static_route < SIM_ROUTE_LOWEST || c->static_route > SIM_ROUTE_SHORTEST)
    return fail(SIM_EINVAL, "static_route");
  if (c->static_route == SIM_ROUTE_SHORTEST && c->n_servers > 8)
    return fail(SIM_EUNSUPPORTED, "Shortest-Queue routing is built for at most 8 servers");
  if (c->shadow && (c->static_bmax < 1 || c->static_bmax > 255 || !(c->static_timeout >= 0.0)))
    return fail(SIM_EINVAL, "static rule needs 1 <= static_bmax <= 255, static_timeout >= 0");
  return SIM_OK;
}

static void derive(sim_ctx* x) {
  const sim_cfg& c = x->cfg;
  SimParams& p = x->p;
  p.E = c.n_envs; p.K = c.n_servers; p.C = c.n_classes; p.N = c.queue_cap;
  p.F = c.obs_dim; p.S = c.arrival_kind == SIM_ARR_TRACE ? 1 : c.n_states;
  p.arrival_kind = c.arrival_kind; p.shadow = c.shadow; p.bmax = c.static_bmax;
  p.route = c.static_route;
  p.reward_sum = c.reward_sum; p.dt = c.tick_s;
  double mdw[kMaxS], tot = 0.0;
  for (int i = 0; i < kMaxS; ++i) {
    const bool on = i < p.S;
    p.rate[i] = on ? c.rate[i] : 0.0;
    p.mean_gap[i] = on && c.rate[i] > 0.0 ? 1.0 / c.rate[i] : 0.0;
    p.dwell_kind[i] = on ? c.dwell_kind[i] : 0;
    p.dwell_mean[i] = on ? c.dwell_mean[i] : 0.0;
    p.inv_alpha[i] = on && c.dwell_kind[i] == SIM_DWELL_PARETO ? 1.0 / c.pareto_alpha[i] : 0.0;
    p.xm[i] = on ? c.pareto_xm[i] : 0.0;
    if (on) {
      // stationary time share of a state is proportional to its mean dwell
      if (c.dwell_kind[i] == SIM_DWELL_EXP || c.dwell_kind[i] == SIM_DWELL_DET)
        mdw[i] = c.dwell_mean[i];
      else if (c.dwell_kind[i] == SIM_DWELL_PARETO)
        mdw[i] = c.pareto_alpha[i] * c.pareto_xm[i] / (c.pareto_alpha[i] - 1.0);
      else mdw[i] = 1.0;
      tot = tot + mdw[i];
    }
  }
  double acc = 0.0;
  for (int i = 0; i < kMaxS; ++i) {
    if (i < p.S) { acc = acc + mdw[i]; p.stat_cum[i] = acc / tot; }
    else p.stat_cum[i] = 1.0;
  }
  p.stat_cum[p.S - 1] = 1.0;
  acc = 0.0;
  for (int i = 0; i < kMaxC; ++i) {
    const bool on = i < p.C;
    if (on) { acc = acc + c.class_mix[i]; p.class_cum[i] = acc; }
    else p.class_cum[i] = 1.0;
    p.svc_kind[i] = on ? c.service_kind[i] : 0;
    p.svc_alpha[i] = on ? c.svc_alpha[i] : 0.0;
    p.svc_beta[i] = on ? c.svc_beta[i] : 0.0;
    p.svc_median[i] = on ? c.svc_median[i] : 0.0;
    p.w_class[i] = on ? c.w_class[i] : 0.0;
  }
  p.class_cum[p.C - 1] = 1.0;
  p.svc_sigma = c.svc_sigma;
  p.w_thr = c.w_thr;
  p.inv_n = 1.0 / (double)c.queue_cap;
  p.inv_tw = 1.0 / c.obs_tw;
  p.inv_c = 1.0 / (double)c.n_classes;
  p.inv_rs = 1.0 / (c.lambda_ref * c.tick_s);
  p.static_timeout = c.static_timeout;
  p.tr_times = nullptr; p.tr_cls = nullptr; p.tr_cnt = nullptr; p.tr_len = c.trace_max_len;

  MlpParams& m = x->m;
  m.E = c.n_envs; m.F = c.obs_dim; m.H1 = c.mlp_h1; m.H2 = c.mlp_h2;
  m.A = 6 * c.n_servers; m.Ap = m.A + (c.value_head ? 1 : 0);
  m.bf16 = c.mlp_bf16; m.value_head = c.value_head;
  m.FP = pad_to(c.obs_dim, c.mlp_bf16 ? 32 : 4);
  m.AP = pad_to(m.Ap, 16);

  AttnParams& a = x->a;
  a.E = c.n_envs; a.F = c.obs_dim; a.L = c.attn_tokens; a.D = c.attn_embed; a.NH = c.attn_heads;
  a.Hp = c.mlp_h1; a.Hv = c.mlp_h2; a.A = 6 * c.n_servers; a.value_head = c.value_head;
}

int sim_create(const sim_cfg* cfg, void* hip_stream, sim_ctx** out) {
  if (!out) return fail(SIM_EINVAL, "out is NULL");
  *out = nullptr;
  int rc = validate(cfg);
  if (rc) return rc;
  sim_ctx* x = new (std::nothrow) sim_ctx();
  if (!x) return fail(SIM_ENOMEM, "host allocation of the context failed");
  x->cfg = *cfg;
  x->stream = static_cast<hipStream_t>(hip_stream);
  (void)hipGetDevice(&x->device);
  derive(x);
  const size_t E = (size_t)cfg->n_envs, K = cfg->n_servers, C = cfg->n_classes, N = cfg->queue_cap;
  const int nsys = cfg->shadow ? 2 : 1;
  // layout of the arena: per system, then shared fields
  std::vector<std::pair<void**, size_t>> parts;
  for (int s = 0; s < nsys; ++s) {
    SysState& g = x->s.sys[s];
    parts.push_back({(void**)&g.qpack, 4 * E});
    parts.push_back({(void**)&g.hpack, 4 * E});
    parts.push_back({(void**)&g.hts, 8 * C * E});
    parts.push_back({(void**)&g.busy, 8 * K * E});
    if (s == 1 && cfg->static_route == SIM_ROUTE_SHORTEST)
      parts.push_back({(void**)&g.busy2, 8 * K * E});
    parts.push_back({(void**)&g.meta, 4 * K * E});
    parts.push_back({(void**)&g.cnt, 4 * kNcnt * E});
    parts.push_back({(void**)&g.sums, 8 * 2 * E});
    parts.push_back({(void**)&g.chk, 8 * E});
    parts.push_back({(void**)&g.ring, 8 * C * N * E});
    parts.push_back({(void**)&g.proc, 4 * E});
    parts.push_back({(void**)&g.next_sw, 8 * E});
    parts.push_back({(void**)&g.next_arr, 8 * E});
    parts.push_back({(void**)&g.tr_idx, 4 * E});
    parts.push_back({(void**)&g.rr, 4 * E});
  }
  parts.push_back({(void**)&x->s.ewma, 8 * 4 * E});
  parts.push_back({(void**)&x->s.obs, 4 * (size_t)cfg->obs_dim * E});
  if (cfg->policy_kind == SIM_POLICY_MLP && cfg->mlp_bf16)
    parts.push_back({(void**)&x->s.obs_bf, 4 * (size_t)((cfg->obs_dim + 1) / 2) * E});
  parts.push_back({(void**)&x->s.err, 256});
  parts.push_back({(void**)&x->s.seed, 256});
  parts.push_back({(void**)&x->d_tot_cnt, 8 * 2 * 7});
  parts.push_back({(void**)&x->d_tot_sum, 8 * 2 * 2});
  size_t total = 0;
  for (auto& pr : parts) total += align256(pr.second);
  hipError_t he = hipMalloc(&x->arena, total);
  if (he != hipSuccess) {
    delete x;
    return fail(SIM_ENOMEM, "hipMalloc of %zu bytes of environment state failed: %s", total,
                hipGetErrorString(he));
  }
  x->arena_bytes = total;
  size_t off = 0;
  for (auto& pr : parts) {
    *pr.first = static_cast<unsigned char*>(x->arena) + off;
    off += align256(pr.second);
  }
  // every byte zero, the arrays' alignment padding included, so that snapshots of equal
  // states are equal byte for byte (and the error flags start cleared)
  he = hipMemsetAsync(x->arena, 0, total, x->stream);
  if (he != hipSuccess) {
    (void)hipFree(x->arena);
    delete x;
    return hip_fail(he, "hipMemsetAsync");
  }
  // packed policy weights (only for supported shapes; checked at use)
  const MlpParams& m = x->m;
  const size_t eb = m.bf16 ? 2 : 4;
  const size_t wbytes = align256(eb * m.H1 * m.FP) + align256(4 * m.H1) + align256(eb * m.H2 * m.H1) +
                        align256(4 * m.H2) + align256(eb * m.AP * m.H2) + align256(4 * m.AP);
  he = hipMalloc(&x->wpack, wbytes);
  if (he != hipSuccess) {
    (void)hipFree(x->arena);
    delete x;
    return fail(SIM_ENOMEM, "hipMalloc of packed weights failed: %s", hipGetErrorString(he));
  }
  unsigned char* wp = static_cast<unsigned char*>(x->wpack);
  x->m.w1 = wp; wp += align256(eb * m.H1 * m.FP);
  x->m.b1 = reinterpret_cast<float*>(wp); wp += align256(4 * m.H1);
  x->m.w2 = wp; wp += align256(eb * m.H2 * m.H1);
  x->m.b2 = reinterpret_cast<float*>(wp); wp += align256(4 * m.H2);
  x->m.w3 = wp; wp += align256(eb * m.AP * m.H2);
  x->m.b3 = reinterpret_cast<float*>(wp);
  *out = x;
  return SIM_OK;
}

int sim_destroy(sim_ctx* x) {
  if (!x) return SIM_OK;
  (void)hipStreamSynchronize(x->stream);
  for (auto& pd : x->pending) {
    (void)hipEventDestroy(pd.a);
    (void)hipEventDestroy(pd.b);
  }
  for (hipEvent_t ev : x->pool) (void)hipEventDestroy(ev);
  (void)hipFree(x->arena);
  (void)hipFree(x->wpack);
  (void)hipFree(x->ppo_scratch);
  (void)hipFree(x->grads);
  if (x->rgraph) (void)hipGraphExecDestroy(x->rgraph);
  if (x->gev_in) (void)hipEventDestroy(x->gev_in);
  if (x->gev_out) (void)hipEventDestroy(x->gev_out);
  if (x->gstream) {
    (void)hipStreamSynchronize(x->gstream);
    (void)hipStreamDestroy(x->gstream);
  }
  if (x->sstream) {
    (void)hipStreamSynchronize(x->sstream);
    (void)hipStreamDestroy(x->sstream);
  }
  if (x->sev_fork) (void)hipEventDestroy(x->sev_fork);
  if (x->sev_join) (void)hipEventDestroy(x->sev_join);
  delete x;
  return SIM_OK;
}

int sim_set_trace(sim_ctx* x, const double* d_times, const uint8_t* d_classes,
                  const int32_t* d_counts) {
  if (!x) return fail(SIM_EINVAL, "ctx is NULL");
  if (x->cfg.arrival_kind != SIM_ARR_TRACE)
    return fail(SIM_ESTATE, "sim_set_trace needs arrival_kind = SIM_ARR_TRACE");
  if (!d_times || !d_classes || !d_counts) return fail(SIM_EINVAL, "trace arrays must be non-NULL");
  x->p.tr_times = d_times;
  x->p.tr_cls = d_classes;
  x->p.tr_cnt = d_counts;
  x->trace_set = true;
  x->rkey_valid = x->seen_valid = false;   // the rollout graph holds the previous arrays
  return SIM_OK;
}

int sim_reset(sim_ctx* x, uint64_t seed) {
  if (!x) return fail(SIM_EINVAL, "ctx is NULL");
  if (x->cfg.arrival_kind == SIM_ARR_TRACE && !x->trace_set)
    return fail(SIM_ESTATE, "trace arrivals need sim_set_trace before sim_reset");
  HIPCHK(x->timed(SIM_KC_RESET, [&] { return launch_reset(x->p, x->s, seed, x->stream); }),
         "reset kernel launch");
  x->seed = seed;
  x->tick = 0;
  x->reset_done = true;
  return SIM_OK;
}

int sim_obs(sim_ctx* x, float* d_obs) {
  if (!x || !d_obs) return fail(SIM_EINVAL, "NULL argument");
  if (!x->reset_done) return fail(SIM_ESTATE, "sim_obs before sim_reset");
  HIPCHK(hipMemcpyAsync(d_obs, x->s.obs, 4 * (size_t)x->cfg.obs_dim * x->cfg.n_envs,
                        hipMemcpyDeviceToDevice, x->stream), "hipMemcpyAsync obs");
  return SIM_OK;
}

// the learned system's tick and, if `shadow`, the static system's
static int enqueue_tick(sim_ctx* x, uint32_t k, const uint8_t* act, float* obs_out, double* rew,
                        double* rew_sh, uint64_t* rchk, bool shadow, int obs_mode = kObsF32) {
  HIPCHK(x->timed(SIM_KC_STEP, [&] {
           return launch_step(x->p, x->s, k, act, obs_out, obs_mode, rew, rchk, x->stream);
         }), "step kernel launch");
  if (shadow && x->cfg.shadow)
    HIPCHK(x->timed(SIM_KC_STATIC, [&] {
             return launch_static(x->p, x->s, k, 1, rew_sh, x->stream);
           }), "static kernel launch");
  return SIM_OK;
}

// The static shadow system over ticks k0 .. k0 + T - 1 in launches of up to kStaticChunk ticks
// (it does not depend on the learned system, so its ticks need not interleave with it). Longer
// launches load and store the state fewer times and average the lanes' uneven progress (each
// lane runs through its own ticks, the launch lasts as long as its slowest wave) over more
// ticks: at C5 32.7 us per tick in 4096-tick launches, 40 in 512-tick and 45 in 256-tick ones.
constexpr int32_t kStaticChunk = 4096;
static int run_static(sim_ctx* x, uint32_t k0, int32_t T, double* rew_sh) {
  const size_t E = (size_t)x->cfg.n_envs;
  for (int32_t c = 0; c < T; c += kStaticChunk) {
    const int nt = T - c < kStaticChunk ? T - c : kStaticChunk;
    HIPCHK(x->timed(SIM_KC_STATIC, [&] {
             return launch_static(x->p, x->s, k0 + (uint32_t)c, nt,
                                  rew_sh ? rew_sh + (size_t)c * E : nullptr, x->stream);
           }), "static kernel launch");
  }
  return SIM_OK;
}

int sim_step(sim_ctx* x, const uint8_t* d_actions, float* d_obs_next, double* d_reward,
             double* d_reward_shadow) {
  if (!x || !d_actions) return fail(SIM_EINVAL, "NULL argument");
  if (!x->reset_done) return fail(SIM_ESTATE, "sim_step before sim_reset");
  if (x->tick == 0xFFFFFFFEu) return fail(SIM_ESTATE, "tick counter exhausted");
  int rc = enqueue_tick(x, x->tick, d_actions, d_obs_next, d_reward, d_reward_shadow, nullptr, true);
  if (rc) return rc;
  x->tick++;
  return SIM_OK;
}

int sim_tick(sim_ctx* x, int32_t* h_tick) {
  if (!x || !h_tick) return fail(SIM_EINVAL, "NULL argument");
  *h_tick = (int32_t)x->tick;
  return SIM_OK;
}

int sim_attn_weights_layout(const sim_cfg* c, sim_attn_layout* o) {
  if (!c || !o) return fail(SIM_EINVAL, "NULL argument");
  if (c->policy_kind != SIM_POLICY_ATTN) return fail(SIM_EINVAL, "policy_kind is not SIM_POLICY_ATTN");
  if (c->attn_embed < 1 || c->attn_heads < 1 || c->attn_tokens < 1 || c->obs_dim < 1 ||
      c->mlp_h1 < 1 || c->mlp_h2 < 1 || c->n_servers < 1)
    return fail(SIM_EINVAL, "attention dimensions must be positive");
  const size_t F = c->obs_dim, D = c->attn_embed, Hp = c->mlp_h1, Hv = c->mlp_h2;
  const size_t A = 6 * (size_t)c->n_servers;
  size_t off = 0;
  size_t* dst[14] = {&o->w_in, &o->b_in, &o->w_qkv, &o->b_qkv, &o->w_o, &o->b_o, &o->wp1,
                     &o->bp1, &o->wp2, &o->bp2, &o->wv1, &o->bv1, &o->wv2, &o->bv2};
  const size_t n[14] = {F * D, D, D * 3 * D, 3 * D, D * D, D, D * Hp, Hp, Hp * A, A, D * Hv, Hv,
                        Hv, 1};
  for (int i = 0; i < 14; ++i) {
    *dst[i] = off;
    off += align256(4 * n[i]);
  }
  o->bytes = off;
  return SIM_OK;
}

int sim_weights_layout(const sim_cfg* c, sim_wlayout* o) {
  if (!c || !o) return fail(SIM_EINVAL, "NULL argument");
  if (c->policy_kind == SIM_POLICY_ATTN) {
    sim_attn_layout al;
    int rc = sim_attn_weights_layout(c, &al);
    if (rc) return rc;
    o->w1 = o->b1 = o->w2 = o->b2 = o->w3 = o->b3 = 0;
    o->bytes = al.bytes;
    o->n_out = 6 * c->n_servers + (c->value_head ? 1 : 0);
    o->elem_bytes = 4;
    return SIM_OK;
  }
  if (c->mlp_h1 < 1 || c->mlp_h2 < 1 || c->obs_dim < 1 || c->n_servers < 1)
    return fail(SIM_EINVAL, "MLP dimensions must be positive");
  const size_t eb = c->mlp_bf16 ? 2 : 4;
  const size_t F = c->obs_dim, H1 = c->mlp_h1, H2 = c->mlp_h2;
  const size_t Ap = 6 * (size_t)c->n_servers + (c->value_head ? 1 : 0);
  size_t off = 0;
  o->w1 = off; off += align256(eb * F * H1);
  o->b1 = off; off += align256(4 * H1);
  o->w2 = off; off += align256(eb * H1 * H2);
  o->b2 = off; off += align256(4 * H2);
  o->w3 = off; off += align256(eb * H2 * Ap);
  o->b3 = off; off += align256(4 * Ap);
  o->bytes = off;
  o->n_out = (int32_t)Ap;
  o->elem_bytes = (int32_t)eb;
  return SIM_OK;
}

static void offsets(const sim_cfg& c, size_t off[6]) {
  sim_wlayout L;
  sim_weights_layout(&c, &L);
  off[0] = L.w1; off[1] = L.b1; off[2] = L.w2; off[3] = L.b2; off[4] = L.w3; off[5] = L.b3;
}

static void attn_offsets(const sim_cfg& c, size_t off[14]) {
  sim_attn_layout L;
  sim_attn_weights_layout(&c, &L);
  const size_t v[14] = {L.w_in, L.b_in, L.w_qkv, L.b_qkv, L.w_o, L.b_o, L.wp1,
                        L.bp1, L.wp2, L.bp2, L.wv1, L.bv1, L.wv2, L.bv2};
  for (int i = 0; i < 14; ++i) off[i] = v[i];
}

int sim_init_weights(sim_ctx* x, uint64_t seed, void* d_weights) {
  if (!x || !d_weights) return fail(SIM_EINVAL, "NULL argument");
  if (x->cfg.policy_kind == SIM_POLICY_ATTN) {
    size_t off[14];
    attn_offsets(x->cfg, off);
    const int F = x->cfg.obs_dim, D = x->cfg.attn_embed, Hp = x->cfg.mlp_h1, Hv = x->cfg.mlp_h2;
    const int A = 6 * x->cfg.n_servers;
    const int fin[7] = {F, D, D, D, Hp, D, Hv}, fout[7] = {D, 3 * D, D, Hp, A, Hv, 1};
    HIPCHK(x->timed(SIM_KC_OTHER, [&] {
             return launch_init_attn(seed, d_weights, off, fin, fout, x->stream);
           }), "attention weight init launch");
    return SIM_OK;
  }
  size_t off[6];
  offsets(x->cfg, off);
  HIPCHK(x->timed(SIM_KC_OTHER, [&] {
           return launch_init_weights(x->cfg.obs_dim, x->cfg.mlp_h1, x->cfg.mlp_h2, x->m.Ap,
                                      x->cfg.mlp_bf16, seed, d_weights, off, x->stream);
         }), "weight init launch");
  return SIM_OK;
}

static int repack_weights(sim_ctx* x, const void* d_weights) {
  size_t off[6];
  offsets(x->cfg, off);
  HIPCHK(x->timed(SIM_KC_OTHER, [&] {
           return launch_repack(x->m, d_weights, off, const_cast<void*>(x->m.w1),
                                const_cast<float*>(x->m.b1), const_cast<void*>(x->m.w2),
                                const_cast<float*>(x->m.b2), const_cast<void*>(x->m.w3),
                                const_cast<float*>(x->m.b3), x->stream);
         }), "weight repack launch");
  return SIM_OK;
}

static int prepare_policy(sim_ctx* x, const void* d_weights) {
  if (x->cfg.policy_kind == SIM_POLICY_ATTN) {
    AttnParams& a = x->a;
    if (!attn_shape_supported(a))
      return fail(SIM_EUNSUPPORTED,
                  "attention shape (tokens=%d, embed=%d, heads=%d, actions=%d) is not compiled",
                  a.L, a.D, a.NH, a.A);
    size_t off[14];
    attn_offsets(x->cfg, off);
    const float* b = static_cast<const float*>(d_weights);
    const float** dst[14] = {&a.w_in, &a.b_in, &a.w_qkv, &a.b_qkv, &a.w_o, &a.b_o, &a.wp1,
                             &a.bp1, &a.wp2, &a.bp2, &a.wv1, &a.bv1, &a.wv2, &a.bv2};
    for (int i = 0; i < 14; ++i) *dst[i] = b + off[i] / 4;
    return SIM_OK;
  }
  if (!policy_shape_supported(x->m))
    return fail(SIM_EUNSUPPORTED,
                "policy shape (bf16=%d, F_pad=%d, H1=%d, H2=%d, A_pad=%d) is not compiled",
                x->m.bf16, x->m.FP, x->m.H1, x->m.H2, x->m.AP);
  return repack_weights(x, d_weights);
}

// the policy kernel of the configured network (after prepare_policy)
static hipError_t policy_launch(sim_ctx* x, const float* obs, uint32_t step, uint8_t* act,
                                float* logp, float* value, float* logits,
                                float* hidden = nullptr, const uint32_t* obs_bf = nullptr) {
  if (x->cfg.policy_kind == SIM_POLICY_ATTN)
    return launch_attn_policy(x->a, obs, x->s.seed, step, act, logp, value, logits, x->stream);
  return launch_policy(x->m, obs, obs_bf, x->s.seed, step, act, logp, value, logits, hidden,
                       x->stream);
}

int sim_policy(sim_ctx* x, const void* d_weights, const float* d_obs, uint32_t step,
               uint8_t* d_act, float* d_logp, float* d_value, float* d_logits) {
  if (!x || !d_weights || !d_obs) return fail(SIM_EINVAL, "NULL argument");
  if (d_value && !x->cfg.value_head) return fail(SIM_EINVAL, "d_value needs value_head = 1");
  int rc = prepare_policy(x, d_weights);
  if (rc) return rc;
  HIPCHK(x->timed(SIM_KC_POLICY, [&] {
           return policy_launch(x, d_obs, step, d_act, d_logp, d_value, d_logits);
         }), "policy kernel launch");
  return SIM_OK;
}

int sim_policy_hidden(sim_ctx* x, const void* d_weights, const float* d_obs, uint32_t step,
                      uint8_t* d_act, float* d_logp, float* d_value, float* d_logits,
                      float* d_hidden) {
  if (!x || !d_weights || !d_obs || !d_hidden) return fail(SIM_EINVAL, "NULL argument");
  if (x->cfg.policy_kind != SIM_POLICY_MLP)
    return fail(SIM_EUNSUPPORTED, "sim_policy_hidden is for the MLP policy");
  if (d_value && !x->cfg.value_head) return fail(SIM_EINVAL, "d_value needs value_head = 1");
  int rc = prepare_policy(x, d_weights);
  if (rc) return rc;
  HIPCHK(x->timed(SIM_KC_POLICY, [&] {
           return policy_launch(x, d_obs, step, d_act, d_logp, d_value, d_logits, d_hidden);
         }), "policy kernel launch");
  return SIM_OK;
}

// whether a rollout runs as one fused launch (sim_set_fused_rollout): forced on, whenever the
// network has a fused kernel; automatically, when all of the batch's workgroups of that kernel
// are resident at once (a second round would run every tick again for its workgroups alone)
static bool use_fused(sim_ctx* x) {
  if (x->fuse == SIM_FUSE_OFF || x->cfg.policy_kind != SIM_POLICY_MLP) return false;
  if (x->fuse_cap < 0) {
    int cap = 0;
    x->fuse_cap = fused_rollout_capacity(x->p, x->m, &cap) == hipSuccess && cap > 0 ? cap : 0;
  }
  if (x->fuse_cap == 0) return false;
  return x->fuse == SIM_FUSE_ON || x->cfg.n_envs <= x->fuse_cap;
}

// Every launch of a rollout of T ticks from tick k0 on x->stream: the policy's weight repack,
// the static shadow system in multi-tick launches, then per tick the policy and the learned
// system's tick, and the final value. Its arguments depend only on the weights pointer, T, the
// trajectory pointers and k0 (the seed is read from device memory), so the sequence can be
// captured once as a graph and replayed.
static int enqueue_rollout(sim_ctx* x, const void* d_weights, int32_t T, const sim_traj* tr,
                           uint32_t k0) {
  int rc = prepare_policy(x, d_weights);
  if (rc) return rc;
  const size_t E = (size_t)x->cfg.n_envs, F = (size_t)x->cfg.obs_dim;
  // The static shadow system never reads the learned system, so its launches run beside the
  // learned chain on a second stream (forked from and joined back to the rollout's stream,
  // which a graph capture follows); with per-launch timing on, everything stays on one stream
  // so that each kernel's duration is its own.
  const bool side = x->cfg.shadow && !x->timing;
  if (side) {
    if (!x->sstream) {
      HIPCHK(hipStreamCreateWithFlags(&x->sstream, hipStreamNonBlocking), "hipStreamCreateWithFlags");
      HIPCHK(hipEventCreateWithFlags(&x->sev_fork, hipEventDisableTiming), "hipEventCreateWithFlags");
      HIPCHK(hipEventCreateWithFlags(&x->sev_join, hipEventDisableTiming), "hipEventCreateWithFlags");
    }
    HIPCHK(hipEventRecord(x->sev_fork, x->stream), "hipEventRecord");
    HIPCHK(hipStreamWaitEvent(x->sstream, x->sev_fork, 0), "hipStreamWaitEvent");
    hipStream_t main = x->stream;
    x->stream = x->sstream;
    rc = run_static(x, k0, T, tr->reward_shadow);
    x->stream = main;
    if (rc) return rc;
    HIPCHK(hipEventRecord(x->sev_join, x->sstream), "hipEventRecord");
  } else if (x->cfg.shadow) {
    rc = run_static(x, k0, T, tr->reward_shadow);
    if (rc) return rc;
  }
  // a bf16 policy reads the observation as bf16 pairs, which the ticks write instead of the
  // fp32 observation (half its bytes, both for the tick that writes it and the policy that
  // reads it); the fp32 observation is written again by the last tick
  const uint32_t* obs_bf = x->s.obs_bf;
  if (obs_bf)
    HIPCHK(x->timed(SIM_KC_OTHER, [&] { return launch_obs_pack(x->p, x->s, x->stream); }),
           "observation packing launch");
  if (use_fused(x)) {
    const RolloutOut o{tr->actions, tr->logp, tr->value, tr->reward, tr->rchk, tr->obs};
    HIPCHK(x->timed(SIM_KC_ROLLOUT, [&] {
             return launch_rollout_fused(x->p, x->s, x->m, k0, T, o, x->stream);
           }), "fused rollout launch");
    if (side) HIPCHK(hipStreamWaitEvent(x->stream, x->sev_join, 0), "hipStreamWaitEvent");
    return SIM_OK;
  }
  for (int32_t i = 0; i < T; ++i) {
    const size_t row = (size_t)i * E;
    const uint32_t k = k0 + (uint32_t)i;
    HIPCHK(x->timed(SIM_KC_POLICY, [&] {
             return policy_launch(x, x->s.obs, k, tr->actions + row,
                                  tr->logp ? tr->logp + row : nullptr,
                                  tr->value ? tr->value + row : nullptr, nullptr, nullptr,
                                  obs_bf);
           }), "policy kernel launch");
    const int mode = !obs_bf ? kObsF32 : i + 1 < T ? kObsBf16 : kObsF32 | kObsBf16;
    rc = enqueue_tick(x, k, tr->actions + row, tr->obs ? tr->obs + (size_t)(i + 1) * F * E : nullptr,
                      tr->reward ? tr->reward + row : nullptr, nullptr,
                      tr->rchk ? tr->rchk + row : nullptr, false, mode);
    if (rc) return rc;
  }
  if (tr->value)
    HIPCHK(x->timed(SIM_KC_POLICY, [&] {
             return policy_launch(x, x->s.obs, k0 + (uint32_t)T, nullptr, nullptr,
                                  tr->value + (size_t)T * E, nullptr, nullptr, obs_bf);
           }), "policy kernel launch (final value)");
  if (side) HIPCHK(hipStreamWaitEvent(x->stream, x->sev_join, 0), "hipStreamWaitEvent");
  return SIM_OK;
}

static bool same_key(const RolloutKey& a, const RolloutKey& b) {
  return a.w == b.w && a.T == b.T && a.k0 == b.k0 && std::memcmp(&a.tr, &b.tr, sizeof a.tr) == 0;
}

// Captures the rollout's launch sequence on the context's private stream into a graph.
static int capture_rollout(sim_ctx* x, const RolloutKey& key, const sim_traj* tr) {
  if (!x->gstream) {
    HIPCHK(hipStreamCreateWithFlags(&x->gstream, hipStreamNonBlocking), "hipStreamCreateWithFlags");
    HIPCHK(hipEventCreateWithFlags(&x->gev_in, hipEventDisableTiming), "hipEventCreateWithFlags");
    HIPCHK(hipEventCreateWithFlags(&x->gev_out, hipEventDisableTiming), "hipEventCreateWithFlags");
  }
  hipStream_t caller = x->stream;
  x->stream = x->gstream;
  hipError_t e = hipStreamBeginCapture(x->gstream, hipStreamCaptureModeThreadLocal);
  int rc = e == hipSuccess ? enqueue_rollout(x, key.w, key.T, tr, key.k0) : SIM_EDEVICE;
  hipGraph_t g = nullptr;
  if (e == hipSuccess) {
    const hipError_t e2 = hipStreamEndCapture(x->gstream, &g);
    if (e2 != hipSuccess && rc == SIM_OK) rc = hip_fail(e2, "hipStreamEndCapture");
  } else {
    rc = hip_fail(e, "hipStreamBeginCapture");
  }
  x->stream = caller;
  hipGraphExec_t ex = nullptr;
  if (rc == SIM_OK && g) {
    e = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    if (e != hipSuccess) rc = hip_fail(e, "hipGraphInstantiate");
  }
  if (g) (void)hipGraphDestroy(g);
  if (rc) return rc;
  if (x->rgraph) (void)hipGraphExecDestroy(x->rgraph);
  x->rgraph = ex;
  x->rkey = key;
  x->rkey_valid = true;
  x->graph_captures++;
  return SIM_OK;
}

// Replays the captured rollout on the private stream, ordered after the work already on the
// caller's stream and before any work enqueued there later.
static int replay_rollout(sim_ctx* x) {
  HIPCHK(hipEventRecord(x->gev_in, x->stream), "hipEventRecord");
  HIPCHK(hipStreamWaitEvent(x->gstream, x->gev_in, 0), "hipStreamWaitEvent");
  HIPCHK(hipGraphLaunch(x->rgraph, x->gstream), "hipGraphLaunch");
  HIPCHK(hipEventRecord(x->gev_out, x->gstream), "hipEventRecord");
  HIPCHK(hipStreamWaitEvent(x->stream, x->gev_out, 0), "hipStreamWaitEvent");
  x->graph_replays++;
  return SIM_OK;
}

int sim_rollout(sim_ctx* x, const void* d_weights, int32_t T, const sim_traj* tr) {
  if (!x || !d_weights || !tr || !tr->actions) return fail(SIM_EINVAL, "NULL argument");
  if (T < 1) return fail(SIM_EINVAL, "T must be >= 1");
  if (!x->reset_done) return fail(SIM_ESTATE, "sim_rollout before sim_reset");
  if (tr->value && !x->cfg.value_head) return fail(SIM_EINVAL, "traj.value needs value_head = 1");
  if (tr->reward_shadow && !x->cfg.shadow)
    return fail(SIM_EINVAL, "traj.reward_shadow needs shadow = 1");
  if ((uint64_t)x->tick + (uint64_t)T >= 0xFFFFFFFFull) return fail(SIM_ESTATE, "tick counter exhausted");
  const size_t E = (size_t)x->cfg.n_envs, F = (size_t)x->cfg.obs_dim;
  if (tr->obs)
    HIPCHK(hipMemcpyAsync(tr->obs, x->s.obs, 4 * F * E, hipMemcpyDeviceToDevice, x->stream),
           "hipMemcpyAsync obs_0");
  const RolloutKey key{d_weights, T, *tr, x->tick};
  int rc;
  if (x->graphs && !x->timing) {
    // a call that repeats the previous one (same weights, length, outputs, starting tick) is
    // captured as a graph; later repeats replay it
    bool have = x->rkey_valid && same_key(key, x->rkey);
    if (!have && x->seen_valid && same_key(key, x->seen)) have = capture_rollout(x, key, tr) == SIM_OK;
    if (have) {
      rc = replay_rollout(x);
      if (rc) return rc;
      x->tick += (uint32_t)T;
      return SIM_OK;
    }
    x->seen = key;
    x->seen_valid = true;
  }
  rc = enqueue_rollout(x, d_weights, T, tr, x->tick);
  if (rc) return rc;
  x->tick += (uint32_t)T;
  return SIM_OK;
}

int sim_set_graphs(sim_ctx* x, int32_t on) {
  if (!x) return fail(SIM_EINVAL, "ctx is NULL");
  x->graphs = on != 0;
  return SIM_OK;
}

int sim_set_fused_rollout(sim_ctx* x, int32_t mode) {
  if (!x) return fail(SIM_EINVAL, "ctx is NULL");
  if (mode != SIM_FUSE_OFF && mode != SIM_FUSE_AUTO && mode != SIM_FUSE_ON)
    return fail(SIM_EINVAL, "fused rollout mode %d", (int)mode);
  if (mode != x->fuse) x->rkey_valid = x->seen_valid = false;   // the graph holds the other form
  x->fuse = mode;
  return SIM_OK;
}

int sim_graph_stats(sim_ctx* x, int64_t* h_captures, int64_t* h_replays) {
  if (!x) return fail(SIM_EINVAL, "ctx is NULL");
  if (h_captures) *h_captures = x->graph_captures;
  if (h_replays) *h_replays = x->graph_replays;
  return SIM_OK;
}

int returns_gae(sim_ctx* x, int32_t T, const double* d_r, const float* d_v, double gamma,
                double lambda, double* d_adv, double* d_ret) {
  if (!x || !d_r || !d_adv || !d_ret) return fail(SIM_EINVAL, "NULL argument");
  if (T < 1) return fail(SIM_EINVAL, "T must be >= 1");
  HIPCHK(x->timed(SIM_KC_GAE, [&] {
           return launch_gae(T, x->cfg.n_envs, d_r, d_v, gamma, lambda, d_adv, d_ret, x->stream);
         }), "gae kernel launch");
  return SIM_OK;
}

int sim_ppo_grad_count(const sim_cfg* c, int64_t* h_count) {
  if (!c || !h_count) return fail(SIM_EINVAL, "NULL argument");
  if (c->policy_kind == SIM_POLICY_ATTN) {
    AttnParams a{};
    a.F = c->obs_dim; a.L = c->attn_tokens; a.D = c->attn_embed; a.NH = c->attn_heads;
    a.Hp = c->mlp_h1; a.Hv = c->mlp_h2; a.A = 6 * c->n_servers;
    *h_count = attn_param_count(a, nullptr);
    return SIM_OK;
  }
  const int64_t F = c->obs_dim, H1 = c->mlp_h1, H2 = c->mlp_h2;
  const int64_t Ap = 6 * (int64_t)c->n_servers + (c->value_head ? 1 : 0);
  *h_count = F * H1 + H1 + H1 * H2 + H2 + H2 * Ap + Ap;
  return SIM_OK;
}

// The minibatch's scratch: the context's buffer, grown with hipMalloc when a call needs more,
// or (no_alloc) the library's fixed device scratch, which allocates nothing.
static int mb_scratch(sim_ctx* x, size_t need, bool no_alloc, const char* who, void** out) {
  if (no_alloc) {
    if (need > kStaticScratchBytes)
      return fail(SIM_EINVAL, "%s: this minibatch needs %zu bytes of scratch; the fixed scratch "
                  "holds %zu (use fewer samples, or ppo_minibatch_grad)", who, need,
                  kStaticScratchBytes);
    HIPCHK(static_scratch(out), "hipGetSymbolAddress of the fixed scratch");
    return SIM_OK;
  }
  if (need > x->ppo_bytes) {
    (void)hipStreamSynchronize(x->stream);
    (void)hipFree(x->ppo_scratch);
    x->ppo_scratch = nullptr;
    x->ppo_bytes = 0;
    hipError_t he = hipMalloc(&x->ppo_scratch, need);
    if (he != hipSuccess)
      return fail(SIM_ENOMEM, "hipMalloc of %zu bytes of minibatch scratch failed: %s", need,
                  hipGetErrorString(he));
    x->ppo_bytes = need;
  }
  *out = x->ppo_scratch;
  return SIM_OK;
}

// shared by the PPO and REINFORCE entry points; no_alloc launches without tracing events and
// with the fixed scratch
static int pg_grad(sim_ctx* x, int reinforce, const void* d_weights, int32_t T, const float* d_obs,
                   const uint8_t* d_actions, const float* d_logp_old, const double* d_adv,
                   const double* d_ret, int32_t M, uint64_t seed, float clip, float c_value,
                   float c_entropy, float* d_grads, double* d_loss, int64_t* d_index,
                   bool no_alloc = false) {
  const char* who = reinforce ? "reinforce_minibatch_grad"
                              : (no_alloc ? "ppo_minibatch_grad_noalloc" : "ppo_minibatch_grad");
  if (!x || !d_weights || !d_obs || !d_actions || (!reinforce && !d_logp_old) || !d_adv ||
      !d_ret || !d_grads || !d_loss)
    return fail(SIM_EINVAL, "%s: NULL argument", who);
  if (!x->cfg.value_head) return fail(SIM_EUNSUPPORTED, "%s needs value_head = 1", who);
  if (T < 1) return fail(SIM_EINVAL, "T must be >= 1");
  if (M < 16 || M % 16) return fail(SIM_EINVAL, "M = %d must be a positive multiple of 16", M);
  if ((int64_t)T * x->cfg.n_envs > 0x7FFFFFFFll)
    return fail(SIM_EINVAL, "T * E must stay below 2^31");
  if (!reinforce && !(clip > 0.0f && clip < 1.0f))
    return fail(SIM_EINVAL, "clip must lie in (0, 1)");
  if (x->cfg.policy_kind == SIM_POLICY_ATTN) {
    int rc = prepare_policy(x, d_weights);  // shape check and weight pointers
    if (rc) return rc;
    void* scr = nullptr;
    rc = mb_scratch(x, attn_grad_scratch_bytes(x->a, M), no_alloc, who, &scr);
    if (rc) return rc;
    auto launch = [&] {
      return launch_attn_grad(x->a, T, d_obs, d_actions, d_logp_old, d_adv, d_ret, M, seed, clip,
                              c_value, c_entropy, reinforce, scr, d_loss, d_grads, d_index,
                              x->s.err, x->stream);
    };
    HIPCHK(no_alloc ? launch() : x->timed(SIM_KC_PPO, launch),
           "attention minibatch gradient kernel launch");
    return SIM_OK;
  }
  if ((int64_t)M * (std::max(std::max(x->m.F, x->m.H1), std::max(x->m.H2, x->m.Ap)) + 1) >
      0x7FFFFFFFll)
    return fail(SIM_EINVAL, "M = %d times the widest layer must stay below 2^31", M);
  if (!ppo_shape_supported(x->m))
    return fail(SIM_EUNSUPPORTED, "%s: hidden widths must be multiples of 64, obs_dim <= 128 and A' <= 128",
                who);
  void* scr = nullptr;
  int rc = mb_scratch(x, ppo_scratch_bytes(x->m, M), no_alloc, who, &scr);
  if (rc) return rc;
  size_t off[6];
  offsets(x->cfg, off);
  auto launch = [&] {
    return launch_ppo(x->m, d_weights, off, T, d_obs, d_actions, d_logp_old, d_adv, d_ret, M, seed,
                      clip, c_value, c_entropy, reinforce, scr, d_loss, d_grads, d_index, x->s.err,
                      x->stream);
  };
  HIPCHK(no_alloc ? launch() : x->timed(SIM_KC_PPO, launch), "minibatch gradient kernel launch");
  return SIM_OK;
}

int ppo_minibatch_grad(sim_ctx* x, const void* d_weights, int32_t T, const float* d_obs,
                       const uint8_t* d_actions, const float* d_logp_old, const double* d_adv,
                       const double* d_ret, int32_t M, uint64_t seed, float clip, float c_value,
                       float c_entropy, float* d_grads, double* d_loss, int64_t* d_index) {
  return pg_grad(x, 0, d_weights, T, d_obs, d_actions, d_logp_old, d_adv, d_ret, M, seed, clip,
                 c_value, c_entropy, d_grads, d_loss, d_index);
}

int ppo_minibatch_grad_noalloc(sim_ctx* x, const void* d_weights, int32_t T, const float* d_obs,
                               const uint8_t* d_actions, const float* d_logp_old,
                               const double* d_adv, const double* d_ret, int32_t M, uint64_t seed,
                               float clip, float c_value, float c_entropy, float* d_grads,
                               double* d_loss, int64_t* d_index) {
  return pg_grad(x, 0, d_weights, T, d_obs, d_actions, d_logp_old, d_adv, d_ret, M, seed, clip,
                 c_value, c_entropy, d_grads, d_loss, d_index, true);
}

int reinforce_minibatch_grad(sim_ctx* x, const void* d_weights, int32_t T, const float* d_obs,
                             const uint8_t* d_actions, const double* d_adv, const double* d_ret,
                             int32_t M, uint64_t seed, float c_value, float c_entropy,
                             float* d_grads, double* d_loss, int64_t* d_index) {
  return pg_grad(x, 1, d_weights, T, d_obs, d_actions, nullptr, d_adv, d_ret, M, seed, 0.0f,
                 c_value, c_entropy, d_grads, d_loss, d_index);
}

int sim_params_from_weights(sim_ctx* x, const void* d_weights, float* d_params) {
  if (!x || !d_weights || !d_params) return fail(SIM_EINVAL, "NULL argument");
  if (x->cfg.policy_kind == SIM_POLICY_ATTN) {
    size_t off[14];
    attn_offsets(x->cfg, off);
    HIPCHK(x->timed(SIM_KC_OTHER, [&] {
             return launch_import_attn(x->a, d_weights, off, d_params, x->stream);
           }), "weight import launch");
    return SIM_OK;
  }
  size_t off[6];
  offsets(x->cfg, off);
  HIPCHK(x->timed(SIM_KC_OTHER, [&] {
           return launch_import_weights(x->m, d_weights, off, d_params, x->stream);
         }), "weight import launch");
  return SIM_OK;
}

int adam_update(sim_ctx* x, float* d_params, const float* d_grads, float* d_m, float* d_v,
                int32_t step, float lr, float beta1, float beta2, float eps, void* d_weights) {
  if (!x || !d_params || !d_grads || !d_m || !d_v) return fail(SIM_EINVAL, "NULL argument");
  if (step < 1) return fail(SIM_EINVAL, "step = %d must be >= 1", step);
  if (!(beta1 >= 0.0f && beta1 < 1.0f && beta2 >= 0.0f && beta2 < 1.0f && eps > 0.0f))
    return fail(SIM_EINVAL, "need 0 <= beta1, beta2 < 1 and eps > 0");
  int64_t n = 0;
  sim_ppo_grad_count(&x->cfg, &n);
  const float bc1 = (float)(1.0 - std::pow((double)beta1, (double)step));
  const float bc2 = (float)(1.0 - std::pow((double)beta2, (double)step));
  HIPCHK(x->timed(SIM_KC_PPO, [&] {
           return launch_adam(d_params, d_grads, d_m, d_v, (size_t)n, lr, beta1, beta2, eps, bc1,
                              bc2, x->stream);
         }), "Adam kernel launch");
  if (d_weights && x->cfg.policy_kind == SIM_POLICY_ATTN) {
    size_t off[14];
    attn_offsets(x->cfg, off);
    HIPCHK(x->timed(SIM_KC_PPO, [&] {
             return launch_export_attn(x->a, d_params, d_weights, off, x->stream);
           }), "weight export launch");
  } else if (d_weights) {
    size_t off[6];
    offsets(x->cfg, off);
    HIPCHK(x->timed(SIM_KC_PPO, [&] {
             return launch_export_weights(x->m, d_params, d_weights, off, x->stream);
           }), "weight export launch");
  }
  return SIM_OK;
}

int sim_update(sim_ctx* x, const sim_update_cfg* u, void* d_weights, float* d_params, float* d_m,
               float* d_v, int32_t* h_step, int32_t T, const float* d_obs,
               const uint8_t* d_actions, const float* d_logp_old, const double* d_adv,
               const double* d_ret, double* d_losses) {
  if (!x || !u || !d_weights || !d_params || !d_m || !d_v || !h_step)
    return fail(SIM_EINVAL, "NULL argument");
  if (u->algo != SIM_ALGO_PPO && u->algo != SIM_ALGO_REINFORCE)
    return fail(SIM_EINVAL, "unknown algorithm %d", u->algo);
  if (u->epochs < 1 || u->minibatches < 1) return fail(SIM_EINVAL, "epochs and minibatches >= 1");
  int64_t n = 0;
  sim_ppo_grad_count(&x->cfg, &n);
  if (!x->grads) {
    hipError_t he = hipMalloc(&x->grads, (size_t)(n + 2) * sizeof(float) + 4 * sizeof(double));
    if (he != hipSuccess) return fail(SIM_ENOMEM, "hipMalloc of the gradient buffer failed");
  }
  float* g = static_cast<float*>(x->grads);
  double* scratch_loss = reinterpret_cast<double*>(g + n + (n & 1));
  for (int e = 0; e < u->epochs; ++e) {
    for (int b = 0; b < u->minibatches; ++b) {
      const uint64_t k = (uint64_t)e * (uint64_t)u->minibatches + (uint64_t)b;
      const uint64_t seed = u->seed + k * 0x9E3779B97F4A7C15ull;
      double* loss = d_losses ? d_losses + 4 * k : scratch_loss;
      int rc = pg_grad(x, u->algo == SIM_ALGO_REINFORCE, d_weights, T, d_obs, d_actions,
                       d_logp_old, d_adv, d_ret, u->M, seed, u->clip, u->c_value, u->c_entropy,
                       g, loss, nullptr);
      if (rc) return rc;
      rc = adam_update(x, d_params, g, d_m, d_v, *h_step + 1, u->lr, u->beta1, u->beta2, u->eps,
                       d_weights);
      if (rc) return rc;
      *h_step += 1;
    }
  }
  return SIM_OK;
}

int sim_counters(sim_ctx* x, int64_t* d_cnt, double* d_sum) {
  if (!x) return fail(SIM_EINVAL, "ctx is NULL");
  if (!x->reset_done) return fail(SIM_ESTATE, "sim_counters before sim_reset");
  HIPCHK(x->timed(SIM_KC_OTHER, [&] { return launch_counters(x->p, x->s, d_cnt, d_sum, x->stream); }),
         "counters kernel launch");
  return SIM_OK;
}

int sim_checksums(sim_ctx* x, uint64_t* d_chk) {
  if (!x || !d_chk) return fail(SIM_EINVAL, "NULL argument");
  if (!x->reset_done) return fail(SIM_ESTATE, "sim_checksums before sim_reset");
  const size_t E = (size_t)x->cfg.n_envs;
  HIPCHK(hipMemcpyAsync(d_chk, x->s.sys[0].chk, 8 * E, hipMemcpyDeviceToDevice, x->stream),
         "hipMemcpyAsync checksums");
  if (x->cfg.shadow)
    HIPCHK(hipMemcpyAsync(d_chk + E, x->s.sys[1].chk, 8 * E, hipMemcpyDeviceToDevice, x->stream),
           "hipMemcpyAsync checksums");
  else
    HIPCHK(hipMemsetAsync(d_chk + E, 0, 8 * E, x->stream), "hipMemsetAsync checksums");
  return SIM_OK;
}

int sim_stats(sim_ctx* x, sim_totals* h) {
  if (!x || !h) return fail(SIM_EINVAL, "NULL argument");
  if (!x->reset_done) return fail(SIM_ESTATE, "sim_stats before sim_reset");
  HIPCHK(hipMemsetAsync(x->d_tot_cnt, 0, 8 * 2 * 7, x->stream), "hipMemsetAsync");
  HIPCHK(hipMemsetAsync(x->d_tot_sum, 0, 8 * 2 * 2, x->stream), "hipMemsetAsync");
  HIPCHK(x->timed(SIM_KC_OTHER, [&] {
           return launch_totals(x->p, x->s, x->d_tot_cnt, x->d_tot_sum, x->stream);
         }), "totals kernel launch");
  int64_t c[14];
  double s[4];
  HIPCHK(hipMemcpyAsync(c, x->d_tot_cnt, sizeof c, hipMemcpyDeviceToHost, x->stream), "copy totals");
  HIPCHK(hipMemcpyAsync(s, x->d_tot_sum, sizeof s, hipMemcpyDeviceToHost, x->stream), "copy totals");
  HIPCHK(hipStreamSynchronize(x->stream), "hipStreamSynchronize");
  for (int sy = 0; sy < 2; ++sy) {
    for (int i = 0; i < SIM_NCNT; ++i) h->cnt[sy][i] = c[sy * 7 + i];
    for (int i = 0; i < SIM_NSUM; ++i) h->sum[sy][i] = s[sy * 2 + i];
  }
  return SIM_OK;
}

int sim_sync(sim_ctx* x) {
  if (!x) return fail(SIM_EINVAL, "ctx is NULL");
  HIPCHK(hipStreamSynchronize(x->stream), "hipStreamSynchronize");
  uint32_t err = 0;
  HIPCHK(hipMemcpy(&err, x->s.err, 4, hipMemcpyDeviceToHost), "copy error flags");
  if (err) {
    HIPCHK(hipMemset(x->s.err, 0, 4), "clear error flags");
    return fail(SIM_ESTATE, "device error flags 0x%x:%s%s%s", err,
                (err & ERR_ACTION) ? " action out of range;" : "",
                (err & ERR_EVENTS) ? " event bound exceeded in a tick;" : "",
                (err & ERR_TRACE) ? " trace overrun;" : "");
  }
  return SIM_OK;
}

// ---- checkpoint / resume ---------------------------------------------------------------------
namespace {
constexpr uint64_t kSnapMagic = 0x50414e534d495342ull;  // "BSIMSNAP"
constexpr size_t kSnapHeader = 256;
struct SnapHeader {
  uint64_t magic;
  uint32_t abi, header_bytes;
  int32_t n_envs, n_servers, n_classes, queue_cap, obs_dim, shadow;
  uint64_t arena_bytes;
  uint64_t seed;
  uint32_t tick, reset_done;
};
static_assert(sizeof(SnapHeader) <= kSnapHeader, "snapshot header");
}  // namespace

int sim_get_state(sim_ctx* x, void* buf, size_t* bytes) {
  if (!x || !bytes) return fail(SIM_EINVAL, "NULL argument");
  const size_t need = kSnapHeader + x->arena_bytes;
  if (!buf) {
    *bytes = need;
    return SIM_OK;
  }
  if (*bytes < need) return fail(SIM_EINVAL, "snapshot needs %zu bytes, buffer has %zu", need, *bytes);
  unsigned char hdr[kSnapHeader] = {};
  SnapHeader h;
  h.magic = kSnapMagic;
  h.abi = BATCHSIM_ABI_VERSION;
  h.header_bytes = (uint32_t)kSnapHeader;
  h.n_envs = x->cfg.n_envs; h.n_servers = x->cfg.n_servers; h.n_classes = x->cfg.n_classes;
  h.queue_cap = x->cfg.queue_cap; h.obs_dim = x->cfg.obs_dim; h.shadow = x->cfg.shadow;
  h.arena_bytes = x->arena_bytes;
  h.seed = x->seed;
  h.tick = x->tick;
  h.reset_done = x->reset_done ? 1u : 0u;
  std::memcpy(hdr, &h, sizeof(h));
  HIPCHK(hipStreamSynchronize(x->stream), "stream synchronize before the snapshot");
  unsigned char* dst = static_cast<unsigned char*>(buf);
  HIPCHK(hipMemcpy(dst, hdr, kSnapHeader, hipMemcpyDefault), "snapshot header copy");
  HIPCHK(hipMemcpy(dst + kSnapHeader, x->arena, x->arena_bytes, hipMemcpyDefault),
         "snapshot state copy");
  *bytes = need;
  return SIM_OK;
}

int sim_set_state(sim_ctx* x, const void* buf, size_t bytes) {
  if (!x || !buf) return fail(SIM_EINVAL, "NULL argument");
  if (bytes < kSnapHeader) return fail(SIM_EINVAL, "buffer of %zu bytes is not a snapshot", bytes);
  HIPCHK(hipStreamSynchronize(x->stream), "stream synchronize before the restore");
  const unsigned char* src = static_cast<const unsigned char*>(buf);
  SnapHeader h;
  HIPCHK(hipMemcpy(&h, src, sizeof(h), hipMemcpyDefault), "snapshot header copy");
  if (h.magic != kSnapMagic || h.abi != BATCHSIM_ABI_VERSION || h.header_bytes != kSnapHeader)
    return fail(SIM_EINVAL, "buffer is not a snapshot of this library version");
  if (h.n_envs != x->cfg.n_envs || h.n_servers != x->cfg.n_servers ||
      h.n_classes != x->cfg.n_classes || h.queue_cap != x->cfg.queue_cap ||
      h.obs_dim != x->cfg.obs_dim || h.shadow != x->cfg.shadow || h.arena_bytes != x->arena_bytes)
    return fail(SIM_EINVAL, "snapshot layout (E=%d, K=%d, C=%d, N=%d, F=%d, shadow=%d) differs "
                "from the context's", h.n_envs, h.n_servers, h.n_classes, h.queue_cap,
                h.obs_dim, h.shadow);
  if (bytes < kSnapHeader + h.arena_bytes)
    return fail(SIM_EINVAL, "snapshot truncated: %zu of %zu bytes", bytes,
                (size_t)(kSnapHeader + h.arena_bytes));
  HIPCHK(hipMemcpy(x->arena, src + kSnapHeader, x->arena_bytes, hipMemcpyDefault),
         "snapshot state copy");
  x->seed = h.seed;
  x->tick = h.tick;
  x->reset_done = h.reset_done != 0;
  return SIM_OK;
}

static_assert(SIM_PRIM_PHILOX == PRIM_PHILOX && SIM_PRIM_LOG == PRIM_LOG && SIM_PRIM_EXP == PRIM_EXP &&
                  SIM_PRIM_COS == PRIM_COS && SIM_PRIM_SQRT == PRIM_SQRT && SIM_PRIM_DIV == PRIM_DIV,
              "primitive kinds");

int sim_device_primitive(int32_t kind, int64_t n, uint64_t key, const void* d_in, void* d_out,
                         void* hip_stream) {
  if (kind < SIM_PRIM_PHILOX || kind > SIM_PRIM_DIV) return fail(SIM_EINVAL, "unknown primitive %d", kind);
  if (n < 0) return fail(SIM_EINVAL, "n must be >= 0");
  if (n > 0 && (!d_in || !d_out)) return fail(SIM_EINVAL, "NULL argument");
  HIPCHK(launch_primitive(kind, n, key, d_in, d_out, static_cast<hipStream_t>(hip_stream)),
         "primitive kernel launch");
  return SIM_OK;
}

int sim_set_timing(sim_ctx* x, int32_t on) {
  if (!x) return fail(SIM_EINVAL, "ctx is NULL");
  x->timing = on != 0;
  return SIM_OK;
}

int sim_get_timing(sim_ctx* x, double* h_ms, int64_t* h_launches, int32_t clear) {
  if (!x) return fail(SIM_EINVAL, "ctx is NULL");
  HIPCHK(hipStreamSynchronize(x->stream), "hipStreamSynchronize");
  for (auto& pd : x->pending) {
    float f = 0.f;
    HIPCHK(hipEventElapsedTime(&f, pd.a, pd.b), "hipEventElapsedTime");
    x->ms[pd.cls] += (double)f;
    x->launches[pd.cls] += 1;
    x->pool.push_back(pd.a);
    x->pool.push_back(pd.b);
  }
  x->pending.clear();
  for (int i = 0; i < SIM_KC_COUNT; ++i) {
    if (h_ms) h_ms[i] = x->ms[i];
    if (h_launches) h_launches[i] = x->launches[i];
    if (clear) {
      x->ms[i] = 0.0;
      x->launches[i] = 0;
    }
  }
  return SIM_OK;
}

}  // extern "C"
