"""Python access to the CPU oracle (oracle.c) -- TEST INFRASTRUCTURE.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import this
package. It shares no code with the HIP path; it reads workload parameter dicts (plain
values from workloads.presets) and derives everything else itself in oracle.c.
"""
import contextlib
import ctypes as C
import os
import threading

import numpy as np

from . import build as _build

_lib = None
_lock = threading.Lock()

MAX_K, MAX_C, MAX_S = 16, 4, 4
REC_W, NCNT, NSUM = 10, 7, 6
P_ARRIVAL, P_PROCESS, P_SERVICE, P_ACTION, P_WEIGHTS, P_MINIBATCH = 1, 2, 3, 4, 5, 6
STEP_RESET = 0xFFFFFFFF
CNT_NAMES = ("arrivals", "accepted", "dropped", "dispatched", "batches", "completed", "inflight")
SUM_NAMES = ("lat_sum", "wlat_sum", "wait_sum", "area_n", "area_q", "sojourn_sum")
REC_NAMES = ("n_k", "ndisp", "sumq", "A_k", "dropped", "completed", "q0", "q1", "q2", "q3")


class OrcCfg(C.Structure):
    _fields_ = [
        ("n_servers", C.c_int32), ("n_classes", C.c_int32), ("queue_cap", C.c_int32),
        ("obs_dim", C.c_int32), ("tick_s", C.c_double),
        ("arrival_kind", C.c_int32), ("n_states", C.c_int32),
        ("rate", C.c_double * MAX_S), ("dwell_kind", C.c_int32 * MAX_S),
        ("dwell_mean", C.c_double * MAX_S), ("pareto_alpha", C.c_double * MAX_S),
        ("pareto_xm", C.c_double * MAX_S), ("class_mix", C.c_double * MAX_C),
        ("service_kind", C.c_int32 * MAX_C), ("svc_alpha", C.c_double * MAX_C),
        ("svc_beta", C.c_double * MAX_C), ("svc_median", C.c_double * MAX_C),
        ("svc_sigma", C.c_double), ("w_thr", C.c_double), ("w_class", C.c_double * MAX_C),
        ("reward_sum", C.c_int32), ("obs_tw", C.c_double), ("lambda_ref", C.c_double),
        ("shadow", C.c_int32), ("static_timeout", C.c_double), ("static_bmax", C.c_int32),
        ("mlp_h1", C.c_int32), ("mlp_h2", C.c_int32), ("mlp_bf16", C.c_int32),
        ("value_head", C.c_int32), ("static_route", C.c_int32),
        ("policy_kind", C.c_int32), ("attn_tokens", C.c_int32), ("attn_embed", C.c_int32),
        ("attn_heads", C.c_int32),
    ]


class OrcTrace(C.Structure):
    _fields_ = [("times", C.c_void_p), ("classes", C.c_void_p), ("counts", C.c_void_p),
                ("max_len", C.c_int32)]


MLP_KEYS = ("w1", "b1", "w2", "b2", "w3", "b3")
ATTN_KEYS = ("w_in", "b_in", "w_qkv", "b_qkv", "w_o", "b_o", "wp1", "bp1", "wp2", "bp2",
             "wv1", "bv1", "wv2", "bv2")
POLICY_MLP, POLICY_ATTN = 0, 1


class OrcWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in MLP_KEYS + ATTN_KEYS]


class OrcDisp(C.Structure):
    _fields_ = [("env_idx", C.c_int32), ("sys", C.c_int32), ("k", C.c_int32),
                ("server", C.c_int32), ("cls", C.c_int32), ("n", C.c_int32),
                ("t", C.c_double), ("c", C.c_double)]


class OrcOut(C.Structure):
    _fields_ = [("reward", C.c_void_p), ("reward_shadow", C.c_void_p), ("obs", C.c_void_p),
                ("rec", C.c_void_p), ("chk", C.c_void_p), ("rchk", C.c_void_p),
                ("counters", C.c_void_p), ("sums", C.c_void_p), ("disp", C.c_void_p),
                ("disp_cap", C.c_int64), ("disp_count", C.c_int64),
                ("actions", C.c_void_p), ("logp", C.c_void_p), ("value", C.c_void_p),
                ("logits", C.c_void_p), ("margin", C.c_void_p)]


def _configure(path):
    """Load an oracle library from `path` and declare its entry points."""
    L = C.CDLL(path)
    assert L.orc_sizeof_cfg() == C.sizeof(OrcCfg), "oracle cfg layout mismatch"
    assert L.orc_sizeof_out() == C.sizeof(OrcOut), "oracle out layout mismatch"
    assert L.orc_sizeof_disp() == C.sizeof(OrcDisp), "oracle disp layout mismatch"
    vp, i32, i64, u32, u64, dbl = (C.c_void_p, C.c_int32, C.c_int64, C.c_uint32,
                                   C.c_uint64, C.c_double)
    L.orc_philox4x32.argtypes = [vp, vp, vp]
    L.orc_philox4x64.argtypes = [vp, vp, vp]
    L.orc_philox4x32_batch.argtypes = [i64, vp, vp, vp]
    L.orc_philox_constants.argtypes = [vp]
    L.orc_draw.argtypes = [u64, u32, u32, u32, u32, u32, vp]
    L.orc_u01.argtypes = [u32, u32]
    L.orc_u01.restype = dbl
    for f in ("orc_det_log", "orc_det_exp", "orc_det_cos"):
        getattr(L, f).argtypes = [vp, vp, i64]
    L.orc_sample.argtypes = [i32, dbl, dbl, u64, i64, vp]
    L.orc_n_out.argtypes = [vp]
    L.orc_init_weights.argtypes = [vp, u64, vp, vp, vp, vp, vp, vp]
    L.orc_policy.argtypes = [vp, vp, u64, u32, i32, vp, vp, vp, vp, vp, vp]
    L.orc_policy.restype = i32
    L.orc_init_weights_attn.argtypes = [vp, u64, vp]
    L.orc_init_weights_attn.restype = i32
    L.orc_rollout.argtypes = [vp, u64, i32, i32, vp, vp, vp, vp, vp]
    L.orc_rollout.restype = i32
    L.orc_gae.argtypes = [i32, i32, vp, vp, dbl, dbl, vp, vp]
    L.orc_sample_logits.argtypes = [vp, i32, dbl, vp, vp]
    L.orc_sample_logits.restype = i32
    L.orc_action_u.argtypes = [u64, u32, u32]
    L.orc_action_u.restype = dbl
    L.orc_reset_probe.argtypes = [vp, u64, i32, vp, vp, vp, vp]
    L.orc_reset_probe.restype = i32
    return L


def lib():
    global _lib
    with _lock:
        if _lib is None:
            _lib = _configure(_build.build())
    return _lib


@contextlib.contextmanager
def use_library(path):
    """Run the oracle's Python entry points against another build of oracle.c (the tests'
    deliberately broken copies, built on the CPU), restoring the real one afterwards."""
    global _lib
    real = lib()
    with _lock:
        _lib = _configure(path)
    try:
        yield
    finally:
        with _lock:
            _lib = real


def _p(a):
    return None if a is None else a.ctypes.data


def make_cfg(w):
    """Fill the oracle's own config struct from a workload parameter dict."""
    c = OrcCfg()
    c.n_servers = w["n_servers"]; c.n_classes = w["n_classes"]
    c.queue_cap = w["queue_cap"]; c.obs_dim = w["obs_dim"]; c.tick_s = w["tick_s"]
    c.arrival_kind = w["arrival_kind"]; c.n_states = len(w["rates"])
    for i in range(c.n_states):
        c.rate[i] = w["rates"][i]; c.dwell_kind[i] = w["dwell_kind"][i]
        c.dwell_mean[i] = w["dwell_mean"][i]; c.pareto_alpha[i] = w["pareto_alpha"][i]
        c.pareto_xm[i] = w["pareto_xm"][i]
    for i in range(c.n_classes):
        c.class_mix[i] = w["class_mix"][i]; c.service_kind[i] = w["service_kind"][i]
        c.svc_alpha[i] = w["svc_alpha"][i]; c.svc_beta[i] = w["svc_beta"][i]
        c.svc_median[i] = w["svc_median"][i]; c.w_class[i] = w["w_class"][i]
    c.svc_sigma = w["svc_sigma"]; c.w_thr = w["w_thr"]; c.reward_sum = w["reward_sum"]
    c.obs_tw = w["obs_tw"]; c.lambda_ref = w["lambda_ref"]
    c.shadow = w["shadow"]; c.static_timeout = w["static_timeout"]
    c.static_bmax = w["static_bmax"]
    c.mlp_h1 = w["mlp_h1"]; c.mlp_h2 = w["mlp_h2"]; c.mlp_bf16 = w["mlp_bf16"]
    c.value_head = w["value_head"]
    c.static_route = w.get("static_route", 0)
    c.policy_kind = w.get("policy_kind", POLICY_MLP)
    c.attn_tokens = w.get("attn_tokens", 0)
    c.attn_embed = w.get("attn_embed", 0)
    c.attn_heads = w.get("attn_heads", 0)
    return c


# ---------------------------------------------------------------------------------------
# primitives
# ---------------------------------------------------------------------------------------
def philox4x32(ctr, key):
    c = np.ascontiguousarray(ctr, dtype=np.uint32); k = np.ascontiguousarray(key, dtype=np.uint32)
    o = np.zeros(4, np.uint32)
    lib().orc_philox4x32(_p(c), _p(k), _p(o))
    return o


def philox4x32_batch(ctr, key):
    """Philox4x32-10 blocks of counters [n][4] (uint32) under a 64-bit key (low word first)."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32).reshape(-1, 4)
    k = np.array([key & 0xFFFFFFFF, key >> 32], dtype=np.uint32)
    out = np.empty_like(c)
    lib().orc_philox4x32_batch(c.shape[0], _p(c), _p(k), _p(out))
    return out


def philox4x64(ctr, key):
    c = np.ascontiguousarray(ctr, dtype=np.uint64); k = np.ascontiguousarray(key, dtype=np.uint64)
    o = np.zeros(4, np.uint64)
    lib().orc_philox4x64(_p(c), _p(k), _p(o))
    return o


def philox_constants():
    o = np.zeros(4, np.uint32)
    lib().orc_philox_constants(_p(o))
    return o


def draw(seed, env, step, purpose, j, sys=0):
    o = np.zeros(4, np.uint32)
    lib().orc_draw(seed, env, step, purpose, j, sys, _p(o))
    return o


def u01(lo, hi):
    return lib().orc_u01(int(lo), int(hi))


def _vec(fn, x):
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    getattr(lib(), fn)(_p(x), _p(y), x.size)
    return y


def det_log(x):
    return _vec("orc_det_log", x)


def det_exp(x):
    return _vec("orc_det_exp", x)


def det_cos(x):
    return _vec("orc_det_cos", x)


SAMPLE_U01, SAMPLE_EXP, SAMPLE_PARETO, SAMPLE_NORMAL, SAMPLE_LOGN = 0, 1, 2, 3, 4


def sample(kind, p0, p1, seed, n):
    o = np.empty(n, np.float64)
    lib().orc_sample(kind, p0, p1, seed, n, _p(o))
    return o


def n_out(w):
    return 6 * w["n_servers"] + (1 if w["value_head"] else 0)


def attn_shapes(w):
    """Shapes of the attention policy's parameters (R26), in ATTN_KEYS order."""
    F, D, A = w["obs_dim"], w["attn_embed"], 6 * w["n_servers"]
    Hp, Hv = w["mlp_h1"], w["mlp_h2"]
    return dict(w_in=(F, D), b_in=(D,), w_qkv=(D, 3 * D), b_qkv=(3 * D,), w_o=(D, D), b_o=(D,),
                wp1=(D, Hp), bp1=(Hp,), wp2=(Hp, A), bp2=(A,), wv1=(D, Hv), bv1=(Hv,),
                wv2=(Hv, 1), bv2=(1,))


def init_weights(w, seed):
    """Xavier-uniform weights from the seed as fp64 arrays of the rounded values."""
    c = make_cfg(w)
    if w.get("policy_kind", POLICY_MLP) == POLICY_ATTN:
        arrs = {k: np.empty(sh) for k, sh in attn_shapes(w).items()}
        ptrs = (C.c_void_p * 14)(*[arrs[k].ctypes.data for k in ATTN_KEYS])
        if lib().orc_init_weights_attn(C.byref(c), seed, ptrs) != 0:
            raise ValueError("attention shape not supported by the oracle")
        return arrs
    F, H1, H2, A = w["obs_dim"], w["mlp_h1"], w["mlp_h2"], n_out(w)
    arrs = dict(w1=np.empty((F, H1)), b1=np.empty(H1), w2=np.empty((H1, H2)), b2=np.empty(H2),
                w3=np.empty((H2, A)), b3=np.empty(A))
    lib().orc_init_weights(C.byref(c), seed, *[_p(arrs[k]) for k in
                                              ("w1", "b1", "w2", "b2", "w3", "b3")])
    return arrs


def _weights_struct(wts):
    ws = OrcWeights()
    keep = {}
    for k in wts:
        if k not in MLP_KEYS + ATTN_KEYS:
            continue
        a = np.ascontiguousarray(wts[k], dtype=np.float64)
        keep[k] = a
        setattr(ws, k, a.ctypes.data)
    return ws, keep


def policy(w, wts, seed, k, obs, env_ids):
    """MLP forward (fp64) + inverse-CDF sampler on observations [n][F]."""
    c = make_cfg(w)
    ws, keep = _weights_struct(wts)
    obs = np.ascontiguousarray(obs, dtype=np.float32)
    n = obs.shape[0]
    ids = np.ascontiguousarray(env_ids, dtype=np.uint32)
    A = n_out(w)
    logits = np.empty((n, A)); act = np.empty(n, np.uint8)
    logp = np.empty(n); margin = np.empty(n)
    if lib().orc_policy(C.byref(c), C.byref(ws), seed, k, n, _p(ids), _p(obs), _p(logits),
                        _p(act), _p(logp), _p(margin)) != 0:
        raise ValueError("policy shape not supported by the oracle")
    return dict(logits=logits, actions=act, logp=logp, margin=margin)


def rollout(w, seed, T, env_ids, actions=None, weights=None, trace=None, want_obs=True,
            want_rec=True, want_rchk=False, disp_cap=0, want_logits=False, want_reward=True):
    """Run T ticks of each env in env_ids (sequentially). actions: [T][n] uint8 or None
    (policy mode with `weights`). trace: dict(times [n][L], classes [n][L], counts [n])."""
    c = make_cfg(w)
    ids = np.ascontiguousarray(env_ids, dtype=np.uint32)
    n = ids.size
    F = w["obs_dim"]
    res = dict(chk=np.zeros((n, 2), np.uint64), counters=np.zeros((n, 2, NCNT), np.int64),
               sums=np.zeros((n, 2, NSUM)))
    if want_reward:
        res["reward"] = np.zeros((T, n))
        res["reward_shadow"] = np.zeros((T, n))
    if want_obs:
        res["obs"] = np.zeros((T + 1, n, F), np.float32)
    if want_rec:
        res["rec"] = np.zeros((T, n, 2, REC_W), np.int32)
    if want_rchk:
        res["rchk"] = np.zeros((T, n), np.uint64)
    o = OrcOut()
    for k in ("reward", "reward_shadow", "obs", "rec", "chk", "rchk", "counters", "sums"):
        if k in res:
            setattr(o, k, res[k].ctypes.data)
    disp = None
    if disp_cap:
        disp = (OrcDisp * disp_cap)()
        o.disp = C.cast(disp, C.c_void_p)
        o.disp_cap = disp_cap
    acts = None
    keep = None
    ws = None
    if actions is not None:
        acts = np.ascontiguousarray(actions, dtype=np.uint8)
        if acts.ndim == 0 or acts.shape == ():
            raise ValueError("actions must be [T][n]")
        if acts.shape != (T, n):
            acts = np.ascontiguousarray(np.broadcast_to(acts, (T, n)))
    else:
        ws, keep = _weights_struct(weights)
        res["actions"] = np.zeros((T, n), np.uint8)
        res["logp"] = np.zeros((T, n), np.float32)
        res["value"] = np.zeros((T + 1, n), np.float32)
        res["margin"] = np.zeros((T, n))
        for k in ("actions", "logp", "value", "margin"):
            setattr(o, k, res[k].ctypes.data)
        if want_logits:
            res["logits"] = np.zeros((T, n, n_out(w)))
            o.logits = res["logits"].ctypes.data
    tr = None
    tkeep = None
    if trace is not None:
        tt = np.ascontiguousarray(trace["times"], dtype=np.float64)
        tc = np.ascontiguousarray(trace["classes"], dtype=np.uint8)
        tn = np.ascontiguousarray(trace["counts"], dtype=np.int32)
        tkeep = (tt, tc, tn)
        tr = OrcTrace(tt.ctypes.data, tc.ctypes.data, tn.ctypes.data, tt.shape[1])
    rc = lib().orc_rollout(C.byref(c), seed, T, n, _p(ids), _p(acts),
                           C.byref(tr) if tr is not None else None,
                           C.byref(ws) if ws is not None else None, C.byref(o))
    del keep, tkeep
    if rc != 0:
        raise ValueError("oracle rejected the configuration")
    if disp is not None:
        cnt = min(o.disp_count, disp_cap)
        res["disp"] = [dict(env_idx=d.env_idx, sys=d.sys, k=d.k, server=d.server, cls=d.cls,
                            n=d.n, t=d.t, c=d.c) for d in disp[:cnt]]
        res["disp_total"] = o.disp_count
    return res


def gae(r, v, gamma, lam):
    """r: [T][n] f64; v: [T+1][n] f32 or None. Returns (adv, ret) [T][n] f64."""
    r = np.ascontiguousarray(r, dtype=np.float64)
    T, n = r.shape
    vv = None if v is None else np.ascontiguousarray(v, dtype=np.float32)
    adv = np.empty_like(r); ret = np.empty_like(r)
    lib().orc_gae(T, n, _p(r), _p(vv), gamma, lam, _p(adv), _p(ret))
    return adv, ret


def sample_logits(logits, u):
    """Inverse-CDF action of one logit row for uniform u -> (action, logp, margin)."""
    l = np.ascontiguousarray(logits, dtype=np.float64)
    lp = np.zeros(1); mg = np.zeros(1)
    a = lib().orc_sample_logits(_p(l), l.size, float(u), _p(lp), _p(mg))
    return a, lp[0], mg[0]


def action_u(seed, env, k):
    return lib().orc_action_u(seed, env, k)


def reset_probe(w, seed, env_ids):
    """Arrival process state right after reset (R11): modulating state, next switch and
    first arrival, per listed env."""
    c = make_cfg(w)
    ids = np.ascontiguousarray(env_ids, dtype=np.uint32)
    n = ids.size
    proc = np.empty(n, np.int32); sw = np.empty(n); arr = np.empty(n)
    if lib().orc_reset_probe(C.byref(c), seed, n, _p(ids), _p(proc), _p(sw), _p(arr)) != 0:
        raise ValueError("reset_probe needs modulated arrivals")
    return dict(proc=proc, next_sw=sw, next_arr=arr)
