"""ctypes binding of libbatchsim.so (include/batchsim.h): argument marshalling only.

Every computation runs in the library's HIP kernels; this module only converts Python
values to the C structs of the ABI, passes device pointers of caller-owned torch tensors
and raises on a non-zero status. It never falls back to another implementation: if the
shared library is missing or fails to load, importing it raises.
"""
import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbatchsim.so")

ABI_VERSION = 2
MAX_K, MAX_C, MAX_S = 16, 4, 4
NCNT, NSUM = 7, 2
STATUS = {0: "SIM_OK", -1: "SIM_EINVAL", -2: "SIM_ENOMEM", -3: "SIM_EDEVICE", -4: "SIM_ESTATE",
          -5: "SIM_EUNSUPPORTED"}
# every symbol include/batchsim.h declares
SYMBOLS = ("sim_last_error", "sim_abi_version", "sim_create", "sim_destroy", "sim_set_trace",
           "sim_reset", "sim_obs", "sim_step", "sim_tick", "sim_weights_layout",
           "sim_init_weights", "sim_policy", "sim_rollout", "returns_gae", "sim_counters",
           "sim_checksums", "sim_stats", "sim_sync", "sim_set_timing", "sim_get_timing",
           "ppo_minibatch_grad", "sim_ppo_grad_count", "reinforce_minibatch_grad",
           "sim_params_from_weights", "adam_update", "sim_update", "sim_attn_weights_layout",
           "sim_get_state", "sim_set_state", "sim_device_primitive", "sim_policy_hidden", "sim_set_graphs", "sim_graph_stats",
           "ppo_minibatch_grad_noalloc", "sim_set_fused_rollout")
ALGO_PPO, ALGO_REINFORCE = 0, 1
KERNEL_CLASSES = ("policy", "step", "static", "gae", "reset", "other", "ppo", "rollout")
FUSE_OFF, FUSE_AUTO, FUSE_ON = 0, 1, 2


class SimCfg(C.Structure):
    _fields_ = [
        ("abi_version", C.c_uint32), ("struct_size", C.c_uint32),
        ("n_envs", C.c_int32), ("n_servers", C.c_int32), ("n_classes", C.c_int32),
        ("queue_cap", C.c_int32), ("obs_dim", C.c_int32), ("tick_s", C.c_double),
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
        ("value_head", C.c_int32), ("trace_max_len", C.c_int32), ("static_route", C.c_int32),
        ("policy_kind", C.c_int32), ("attn_tokens", C.c_int32), ("attn_embed", C.c_int32),
        ("attn_heads", C.c_int32),
    ]


class SimWLayout(C.Structure):
    _fields_ = [("w1", C.c_size_t), ("b1", C.c_size_t), ("w2", C.c_size_t), ("b2", C.c_size_t),
                ("w3", C.c_size_t), ("b3", C.c_size_t), ("bytes", C.c_size_t),
                ("n_out", C.c_int32), ("elem_bytes", C.c_int32)]


ATTN_KEYS = ("w_in", "b_in", "w_qkv", "b_qkv", "w_o", "b_o", "wp1", "bp1", "wp2", "bp2",
             "wv1", "bv1", "wv2", "bv2")
POLICY_MLP, POLICY_ATTN = 0, 1


class SimAttnLayout(C.Structure):
    _fields_ = [(k, C.c_size_t) for k in ATTN_KEYS] + [("bytes", C.c_size_t)]


class SimTraj(C.Structure):
    _fields_ = [("actions", C.c_void_p), ("logp", C.c_void_p), ("reward", C.c_void_p),
                ("reward_shadow", C.c_void_p), ("value", C.c_void_p), ("obs", C.c_void_p),
                ("rchk", C.c_void_p)]


class SimUpdateCfg(C.Structure):
    _fields_ = [("algo", C.c_int32), ("epochs", C.c_int32), ("minibatches", C.c_int32),
                ("M", C.c_int32), ("seed", C.c_uint64), ("clip", C.c_float),
                ("c_value", C.c_float), ("c_entropy", C.c_float), ("lr", C.c_float),
                ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float)]


class SimTotals(C.Structure):
    _fields_ = [("cnt", (C.c_int64 * NCNT) * 2), ("sum", (C.c_double * NSUM) * 2)]


class SimError(RuntimeError):
    pass


_lib = None


def load():
    """Load libbatchsim.so (raises ImportError if it is missing or incomplete)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    L = C.CDLL(LIB_PATH)
    missing = [s for s in SYMBOLS if not hasattr(L, s)]
    if missing:
        raise ImportError(f"libbatchsim.so lacks {missing}")
    vp, i32, u32, u64, dbl = C.c_void_p, C.c_int32, C.c_uint32, C.c_uint64, C.c_double
    L.sim_last_error.restype = C.c_char_p
    L.sim_abi_version.restype = u32
    sig = {
        "sim_create": [vp, vp, C.POINTER(vp)], "sim_destroy": [vp],
        "sim_set_trace": [vp, vp, vp, vp], "sim_reset": [vp, u64], "sim_obs": [vp, vp],
        "sim_step": [vp, vp, vp, vp, vp], "sim_tick": [vp, vp],
        "sim_weights_layout": [vp, vp], "sim_init_weights": [vp, u64, vp],
        "sim_policy": [vp, vp, vp, u32, vp, vp, vp, vp], "sim_rollout": [vp, vp, i32, vp],
        "sim_policy_hidden": [vp, vp, vp, u32, vp, vp, vp, vp, vp],
        "returns_gae": [vp, i32, vp, vp, dbl, dbl, vp, vp], "sim_counters": [vp, vp, vp],
        "sim_checksums": [vp, vp], "sim_stats": [vp, vp], "sim_sync": [vp],
        "sim_set_timing": [vp, i32], "sim_get_timing": [vp, vp, vp, i32],
        "sim_set_graphs": [vp, i32], "sim_graph_stats": [vp, vp, vp],
        "sim_set_fused_rollout": [vp, i32],
        "ppo_minibatch_grad": [vp, vp, i32, vp, vp, vp, vp, vp, i32, u64, C.c_float, C.c_float,
                               C.c_float, vp, vp, vp],
        "ppo_minibatch_grad_noalloc": [vp, vp, i32, vp, vp, vp, vp, vp, i32, u64, C.c_float,
                                       C.c_float, C.c_float, vp, vp, vp],
        "sim_ppo_grad_count": [vp, vp],
        "reinforce_minibatch_grad": [vp, vp, i32, vp, vp, vp, vp, i32, u64, C.c_float, C.c_float,
                                     vp, vp, vp],
        "sim_params_from_weights": [vp, vp, vp],
        "adam_update": [vp, vp, vp, vp, vp, i32, C.c_float, C.c_float, C.c_float, C.c_float, vp],
        "sim_update": [vp, vp, vp, vp, vp, vp, vp, i32, vp, vp, vp, vp, vp, vp],
        "sim_attn_weights_layout": [vp, vp],
        "sim_get_state": [vp, vp, vp], "sim_set_state": [vp, vp, C.c_size_t],
        "sim_device_primitive": [i32, C.c_int64, u64, vp, vp, vp],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = C.c_int
    _lib = L
    return L


def check(rc, what):
    if rc != 0:
        msg = load().sim_last_error().decode()
        raise SimError(f"{what}: {STATUS.get(rc, rc)}: {msg}")


def make_cfg(w, n_envs=None):
    """Fill the ABI's sim_cfg from a workload parameter dict."""
    c = SimCfg()
    c.abi_version = ABI_VERSION
    c.struct_size = C.sizeof(SimCfg)
    c.n_envs = w["n_envs"] if n_envs is None else n_envs
    c.n_servers = w["n_servers"]; c.n_classes = w["n_classes"]; c.queue_cap = w["queue_cap"]
    c.obs_dim = w["obs_dim"]; c.tick_s = w["tick_s"]; c.arrival_kind = w["arrival_kind"]
    c.n_states = len(w["rates"])
    for i in range(c.n_states):
        c.rate[i] = w["rates"][i]; c.dwell_kind[i] = w["dwell_kind"][i]
        c.dwell_mean[i] = w["dwell_mean"][i]; c.pareto_alpha[i] = w["pareto_alpha"][i]
        c.pareto_xm[i] = w["pareto_xm"][i]
    for i in range(c.n_classes):
        c.class_mix[i] = w["class_mix"][i]; c.service_kind[i] = w["service_kind"][i]
        c.svc_alpha[i] = w["svc_alpha"][i]; c.svc_beta[i] = w["svc_beta"][i]
        c.svc_median[i] = w["svc_median"][i]; c.w_class[i] = w["w_class"][i]
    c.svc_sigma = w["svc_sigma"]; c.w_thr = w["w_thr"]; c.reward_sum = w["reward_sum"]
    c.obs_tw = w["obs_tw"]; c.lambda_ref = w["lambda_ref"]; c.shadow = w["shadow"]
    c.static_timeout = w["static_timeout"]; c.static_bmax = w["static_bmax"]
    c.mlp_h1 = w["mlp_h1"]; c.mlp_h2 = w["mlp_h2"]; c.mlp_bf16 = w["mlp_bf16"]
    c.value_head = w["value_head"]; c.trace_max_len = w.get("trace_max_len", 0)
    c.static_route = w.get("static_route", 0)
    c.policy_kind = w.get("policy_kind", POLICY_MLP)
    c.attn_tokens = w.get("attn_tokens", 0)
    c.attn_embed = w.get("attn_embed", 0)
    c.attn_heads = w.get("attn_heads", 0)
    return c
