"""Workload presets C1-C5 (the five operating points of the batched rollout).

Each preset is a dict of plain parameters; nothing here is derived. Units: seconds,
requests per second. Sources (paper sections): the linear batch-latency model and the
FIFO cap of 100 (Sec. 3.1), the workload families (Sec. 3.2), the MDP state/action/
reward (Sec. 4.1), the policy network (Sec. 4.2), the discount/GAE settings
(Sec. 4.3). Values the paper does not fix are numbered readings of it (R-numbers in the
comments).
"""
import copy

# arrival kinds
ARR_MODULATED = 0   # modulated Poisson (Poisson = one state with infinite dwell)
ARR_TRACE = 1       # explicit per-env arrival list (tests / trace replay)
# dwell kinds
DWELL_INF = 0
DWELL_EXP = 1
DWELL_PARETO = 2
DWELL_DET = 3       # fixed dwell (square wave), R24
# server choice of the static shadow system (R23)
ROUTE_LOWEST = 0
ROUTE_RANDOM = 1
ROUTE_ROUND_ROBIN = 2
ROUTE_SHORTEST = 3  # Shortest-Queue over per-server FIFOs of at most two batches, R27
# policy network (R16, R26)
POLICY_MLP = 0
POLICY_ATTN = 1
# service kinds
SVC_DET = 0
SVC_LOGN = 1
SVC_EXP = 2

_BASE = dict(
    n_envs=256, T=1000, n_servers=1, n_classes=1, queue_cap=100, obs_dim=8,
    tick_s=1e-3,
    arrival_kind=ARR_MODULATED,
    # per arrival-modulation state: rate, dwell kind, dwell mean (EXP), pareto alpha / x_m
    rates=[500.0], dwell_kind=[DWELL_INF], dwell_mean=[0.0],
    pareto_alpha=[0.0], pareto_xm=[0.0],
    class_mix=[1.0],
    service_kind=[SVC_DET], svc_alpha=[5e-3], svc_beta=[0.5e-3], svc_median=[0.0],
    svc_sigma=0.0,
    w_thr=0.01, w_class=[1.0], reward_sum=0,
    obs_tw=0.010, lambda_ref=500.0,
    shadow=0, static_timeout=0.010, static_bmax=32, static_route=ROUTE_LOWEST,
    mlp_h1=64, mlp_h2=64, mlp_bf16=0, value_head=0,
    policy_kind=POLICY_MLP, attn_tokens=0, attn_embed=0, attn_heads=0,
    gamma=0.99, lam=1.0, ppo_minibatch=0,
)


def _mk(**kw):
    d = copy.deepcopy(_BASE)
    d.update(kw)
    return d


PRESETS = {
    # C1: single server, Poisson 500/s, DET 5 ms + 0.5 ms*b, obs 8, MLP 8-64-64-6 fp32,
    # 256 envs x 1000 steps, REINFORCE returns gamma=0.99.
    "C1": _mk(name="C1"),
    # C2: single server, 4096 x 2000, two-state MMPP 200/2000 req/s with Exp(0.5 s)
    # dwell, classes 80/20 with 2 ms + 0.3 ms*b and 20 ms + 2 ms*b, obs 12,
    # MLP 12-128-128-6 bf16, REINFORCE gamma=0.99.
    "C2": _mk(name="C2", n_envs=4096, T=2000, n_classes=2, obs_dim=12,
              rates=[200.0, 2000.0], dwell_kind=[DWELL_EXP, DWELL_EXP],
              dwell_mean=[0.5, 0.5], pareto_alpha=[0.0, 0.0], pareto_xm=[0.0, 0.0],
              class_mix=[0.8, 0.2], service_kind=[SVC_DET, SVC_DET],
              svc_alpha=[2e-3, 20e-3], svc_beta=[0.3e-3, 2e-3], svc_median=[0.0, 0.0],
              w_class=[200.0, 20.0], lambda_ref=2000.0,
              mlp_h1=128, mlp_h2=128, mlp_bf16=1),
    # C3: 4 servers, 16384 x 2048, Poisson 3000/s, classes 70/30 with 2 ms + 0.2 ms*b and
    # 50 ms + 5 ms*b, 24 actions, obs 32, MLP 32-256-256-24 bf16, GAE(0.99, 0.95).
    "C3": _mk(name="C3", n_envs=16384, T=2048, n_servers=4, n_classes=2, obs_dim=32,
              rates=[3000.0], class_mix=[0.7, 0.3], service_kind=[SVC_DET, SVC_DET],
              svc_alpha=[2e-3, 50e-3], svc_beta=[0.2e-3, 5e-3], svc_median=[0.0, 0.0],
              w_class=[200.0, 20.0], lambda_ref=3000.0,
              mlp_h1=256, mlp_h2=256, mlp_bf16=1, value_head=1, lam=0.95),
    # C4: 8 servers, 65536 x 1024, 3-state MMPP 500/3000/12000 (Exp(0.5 s) dwell, R11),
    # 4 classes (mix R12) with lognormal service sigma=1, medians 1/5/20/80 ms and
    # a linear per-batch term 0.1*median (R7), obs 64, MLP 64-256-256-48 bf16, GAE +
    # one PPO minibatch of 8192.
    "C4": _mk(name="C4", n_envs=65536, T=1024, n_servers=8, n_classes=4, obs_dim=64,
              rates=[500.0, 3000.0, 12000.0], dwell_kind=[DWELL_EXP] * 3,
              dwell_mean=[0.5] * 3, pareto_alpha=[0.0] * 3, pareto_xm=[0.0] * 3,
              class_mix=[0.5, 0.3, 0.15, 0.05], service_kind=[SVC_LOGN] * 4,
              svc_alpha=[0.0] * 4, svc_beta=[0.1e-3, 0.5e-3, 2e-3, 8e-3],
              svc_median=[1e-3, 5e-3, 20e-3, 80e-3], svc_sigma=1.0,
              w_class=[200.0, 100.0, 40.0, 20.0], lambda_ref=12000.0,
              mlp_h1=256, mlp_h2=256, mlp_bf16=1, value_head=1, lam=0.95,
              ppo_minibatch=8192),
    # C5: 16 servers, 262144 x 4096, heavy-tailed ON/OFF: OFF dwell Pareto(1.5, 30 ms),
    # ON dwell Exp(10 ms) with Poisson 20000/s inside bursts (R11), 4 classes 50/30/15/5,
    # lognormal service, static timeout policy (10 ms or 32 requests) as a shadow system,
    # obs 96, MLP 96-512-512-96 bf16, full GAE.
    "C5": _mk(name="C5", n_envs=262144, T=4096, n_servers=16, n_classes=4, obs_dim=96,
              rates=[0.0, 20000.0], dwell_kind=[DWELL_PARETO, DWELL_EXP],
              dwell_mean=[0.0, 0.010], pareto_alpha=[1.5, 0.0], pareto_xm=[0.030, 0.0],
              class_mix=[0.5, 0.3, 0.15, 0.05], service_kind=[SVC_LOGN] * 4,
              svc_alpha=[0.0] * 4, svc_beta=[0.1e-3, 0.5e-3, 2e-3, 8e-3],
              svc_median=[1e-3, 5e-3, 20e-3, 80e-3], svc_sigma=1.0,
              w_class=[200.0, 100.0, 40.0, 20.0], lambda_ref=20000.0,
              shadow=1, static_timeout=0.010, static_bmax=32,
              mlp_h1=512, mlp_h2=512, mlp_bf16=1, value_head=1, lam=0.95),
}


def n_actions(cfg):
    """Six power-of-two batch sizes per server (R3)."""
    return 6 * cfg["n_servers"]


def preset(name, **override):
    """A deep copy of preset `name` with fields overridden (e.g. n_envs, T)."""
    d = copy.deepcopy(PRESETS[name])
    d.update(override)
    return d


def burst_preset(**kw):
    """The paper's Extreme Burst workload (Sec. 3.2): arrivals switch squarely between
    100 req/s and 0 every 200 steps (0.2 s of 1 ms ticks), starting high (R24); one server
    and class as C1, with a static shadow system for the baseline rules."""
    d = _mk(name="burst", rates=[100.0, 0.0], dwell_kind=[DWELL_DET, DWELL_DET],
            dwell_mean=[0.2, 0.2], pareto_alpha=[0.0, 0.0], pareto_xm=[0.0, 0.0],
            lambda_ref=100.0, shadow=1)
    d.update(kw)
    return d


def baseline_preset(rule, base="C3", **kw):
    """A workload whose shadow system runs one of the paper's baselines (Sec. 5.1):
    'static8' (fixed batch 8 with the timeout of R18), 'random' or 'round_robin' routing of
    the static rule's batches to idle servers (R23), or 'shortest' (Shortest-Queue: each batch
    to the server with the fewest requests assigned and not completed, R27)."""
    extra = dict(static8=dict(static_bmax=8),
                 random=dict(static_route=ROUTE_RANDOM),
                 round_robin=dict(static_route=ROUTE_ROUND_ROBIN),
                 shortest=dict(static_route=ROUTE_SHORTEST))[rule]
    d = preset(base, shadow=1, **extra)
    d.update(kw)
    return d


def attn_preset(**kw):
    """The paper's own policy network (Sec. 4.2) on C1's single-server system: the 8 state
    features as 8 tokens through the 8 -> 4 input projection, self-attention with 2 heads of
    embedding 4, mean pooling, a GELU policy head of 64 units and a separate GELU value head
    of 64 (R26), fp32; REINFORCE with the learned baseline (lambda = 1)."""
    d = _mk(name="attn", policy_kind=POLICY_ATTN, attn_tokens=8, attn_embed=4, attn_heads=2,
            mlp_h1=64, mlp_h2=64, value_head=1)
    d.update(kw)
    return d


def trace_preset(**kw):
    """A trace-arrival configuration for hand-enumerated tests (no MLP use)."""
    d = _mk(name="trace", arrival_kind=ARR_TRACE, rates=[1000.0], lambda_ref=1000.0)
    d.update(kw)
    return d
