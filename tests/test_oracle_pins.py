"""Independent pins of the oracle parts that the closed forms and traces T1-T3 leave open,
each checked against something other than the oracle itself, and each shown to reject a
deliberately broken copy of the oracle (built on the CPU from a modified oracle.c):

* the observation layout with several servers and classes (Sec. 4.1): hand trace T4;
* the class of each arrival (Sec. 3.1 request model): class frequencies against the
  configured mixes, and the arrival stream rebuilt from raw Philox blocks as the counter
  layout prescribes (which words give the gap, which the class, how blocks are counted);
* the lognormal service law with its linear per-batch term (Sec. 3.1 execution model;
  service variance as in Sec. 5.4): Kolmogorov-Smirnov against scipy's normal law;
* the stationary start of the modulated arrival process (Sec. 3.2 workloads): state
  frequencies against the stationary law, first dwell and first gap against their laws;
* the Philox4x32-10 block itself: bit for bit against PyTorch's engine.
"""
import ctypes as C
import json
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest
from scipy import stats

from workloads import preset, trace_preset

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "hand_traces.json")))
P_ARRIVAL, STEP_RESET = 1, 0xFFFFFFFF


def _trace(g):
    arr = g["arrivals"]
    return dict(times=np.array([[a[0] for a in arr]]),
                classes=np.array([[a[1] for a in arr]], np.uint8),
                counts=np.array([len(arr)], np.int32))


# ---- T4: observation layout with K = 2 and C = 2 ------------------------------------------
def pin_t4(orc):
    g = GOLD["T4"]
    w = trace_preset(**g["cfg"])
    T = g["T"]
    acts = np.array(g["actions"], np.uint8)[:, None]
    r = orc.rollout(w, 0, T, [0], actions=acts, trace=_trace(g), disp_cap=64)
    for k, exp in g["obs"].items():
        got = r["obs"][int(k), 0]
        assert np.allclose(got, np.array(exp, np.float32), rtol=1e-6, atol=1e-9), \
            f"obs_{k}: {got} != {exp}"
    d = [(x["k"], x["server"], x["cls"], x["n"], x["t"], x["c"]) for x in r["disp"] if x["sys"] == 0]
    assert len(d) == len(g["dispatches"])
    for got, exp in zip(d, g["dispatches"]):
        assert got[:4] == tuple(exp[:4])
        assert abs(got[4] - exp[4]) < 1e-12 and abs(got[5] - exp[5]) < 1e-12
    for k in range(T):
        exp = g["rewards"].get(str(k), 0.0)
        assert abs(r["reward"][k, 0] - exp) <= 1e-9 * max(1.0, abs(exp)), (k, r["reward"][k, 0])
    rec = r["rec"][:, 0, 0]
    assert list(rec[:, 2]) == g["sumq"]
    assert list(rec[:, 0]) == g["n_k"]
    assert list(rec[:, 5]) == g["completed_cum"]


def test_hand_trace_T4_observations(orc):
    pin_t4(orc)


# ---- class of each arrival ------------------------------------------------------------------
def _instant_service(w):
    """The workload with near-zero deterministic service on every class: with the action
    'server 0, batch 1' every arrival is dispatched at its own instant as a batch of one,
    so the dispatch log is the arrival stream (time and class)."""
    C_ = w["n_classes"]
    return dict(w, service_kind=[0] * C_, svc_alpha=[1e-13] * C_, svc_beta=[0.0] * C_,
                svc_median=[0.0] * C_, shadow=0)


def _arrival_log(orc, w, seed, n_env, T):
    acts = np.zeros((T, n_env), np.uint8)
    r = orc.rollout(w, seed, T, np.arange(n_env), actions=acts, want_obs=False, want_rec=False,
                    want_reward=False, disp_cap=2_000_000)
    assert r["counters"][:, 0, 2].sum() == 0, "no drops expected with instant service"
    assert len(r["disp"]) == r["counters"][:, 0, 0].sum(), "every arrival is its own batch"
    return r["disp"]


def pin_class_mix(orc, name):
    w = _instant_service(preset(name))
    d = _arrival_log(orc, w, 0xC1A55 + len(name), 64, 1500)
    cls = np.array([x["cls"] for x in d])
    mix = np.array(w["class_mix"])
    obs = np.bincount(cls, minlength=len(mix))
    assert obs.sum() > 20000
    p = stats.chisquare(obs, mix * obs.sum()).pvalue
    assert p > 1e-5, f"{name}: class counts {obs} against mix {mix}, p = {p:.3g}"


@pytest.mark.parametrize("name", ["C2", "C3", "C4", "C5"])
def test_class_mix_frequencies(orc, name):
    pin_class_mix(orc, name)


def _u53(lo, hi):
    """Uniform in (0, 1) from two words as the counter layout defines it: the top 53 bits of
    hi:lo, centred in their cell."""
    return ((((int(hi) << 32) | int(lo)) >> 11) + 0.5) * 2.0 ** -53


def pin_arrival_stream(orc):
    """Rebuild each env's arrivals from raw Philox blocks: at reset the ARRIVAL block
    (env, RESET, 0) gives the first gap from words 0-1; the j-th arrival inside tick k takes
    the ARRIVAL block (env, k, j): its class from words 2-3 against the cumulative mix (the
    smallest c with u < P_c), the gap to the next arrival from words 0-1 (gap = -ln(u)/rate).
    Compared with the oracle's dispatch log of the same envs (instant service)."""
    base = preset("C4")
    w = _instant_service(dict(base, rates=[5000.0], dwell_kind=[0], dwell_mean=[0.0],
                              pareto_alpha=[0.0], pareto_xm=[0.0]))
    seed, n_env, T = 0xA11CE, 24, 60
    d = _arrival_log(orc, w, seed, n_env, T)
    cum = np.cumsum(w["class_mix"])
    cum[-1] = 1.0
    inv_rate = 1.0 / w["rates"][0]
    dt = w["tick_s"]
    checked = 0
    for e in range(n_env):
        got = [(x["t"], x["cls"]) for x in d if x["env_idx"] == e]
        blk = orc.draw(seed, e, STEP_RESET, P_ARRIVAL, 0)
        t = -np.log(_u53(blk[0], blk[1])) * inv_rate
        k_prev, j = -1, 0
        exp = []
        while t < T * dt:
            k = int(t // dt)
            while (k + 1) * dt <= t:
                k += 1
            while k * dt > t:
                k -= 1
            j = j + 1 if k == k_prev else 0
            k_prev = k
            blk = orc.draw(seed, e, k, P_ARRIVAL, j)
            uc = _u53(blk[2], blk[3])
            exp.append((t, int(np.argmax(uc < cum))))
            t = t + (-np.log(_u53(blk[0], blk[1])) * inv_rate)
        assert len(got) == len(exp), f"env {e}: {len(got)} arrivals, expected {len(exp)}"
        for (tg, cg), (te, ce) in zip(got, exp):
            assert abs(tg - te) <= 1e-12 * max(te, 1e-3), (e, tg, te)
            assert cg == ce, f"env {e} arrival at {te}: class {cg}, expected {ce}"
            checked += 1
    assert checked > 3000


def test_arrival_stream_follows_counter_layout(orc):
    pin_arrival_stream(orc)


# ---- lognormal service with its linear term -------------------------------------------------
def pin_lognormal_service(orc):
    """C4's classes (lognormal median_h exp(sigma Z) plus beta_h n): for every dispatched batch
    z = ln((S - beta_h n) / median_h) / sigma must be standard normal, per class."""
    from workloads.gen import seeded_actions
    w = preset("C4")
    n_env, T = 128, 1500
    acts = seeded_actions(0x5E4, T, n_env, 6 * w["n_servers"], small_bias=0.6)
    r = orc.rollout(w, 0x5E4, T, np.arange(n_env), actions=acts, want_obs=False,
                    want_rec=False, want_reward=False, disp_cap=4_000_000)
    d = r["disp"]
    cls = np.array([x["cls"] for x in d])
    n = np.array([x["n"] for x in d], np.float64)
    S = np.array([x["c"] - x["t"] for x in d])
    med = np.array(w["svc_median"])[cls]
    beta = np.array(w["svc_beta"])[cls]
    rest = S - beta * n
    assert np.all(rest > 0.0), "service time below its linear term"
    z = np.log(rest / med) / w["svc_sigma"]
    for h in range(w["n_classes"]):
        zh = z[cls == h]
        assert zh.size > 300, (h, zh.size)
        p = stats.kstest(zh, "norm").pvalue
        assert p > 1e-4, f"class {h}: KS p = {p:.3g} over {zh.size} batches"


def test_lognormal_service_law(orc):
    pin_lognormal_service(orc)


# ---- stationary start -------------------------------------------------------------------------
def _stationary(w):
    m = []
    for i, k in enumerate(w["dwell_kind"]):
        if k == 2:
            a, xm = w["pareto_alpha"][i], w["pareto_xm"][i]
            m.append(a * xm / (a - 1.0))
        else:
            m.append(w["dwell_mean"][i])
    m = np.array(m)
    return m / m.sum()


def pin_stationary_start(orc, name):
    """Initial modulating state drawn from the stationary law (time share proportional to the
    mean dwell), then a fresh dwell of that state and the first gap at its rate."""
    w = preset(name)
    n = 20000
    r = orc.reset_probe(w, 0x57A7 + len(name), np.arange(n))
    pi = _stationary(w)
    counts = np.bincount(r["proc"], minlength=len(pi))
    p = stats.chisquare(counts, pi * n).pvalue
    assert p > 1e-5, f"{name}: initial states {counts} against {pi * n}, p = {p:.3g}"
    for s in range(len(pi)):
        sel = r["proc"] == s
        dw = r["next_sw"][sel]
        k = w["dwell_kind"][s]
        if k == 1:
            p = stats.kstest(dw, "expon", args=(0.0, w["dwell_mean"][s])).pvalue
        else:
            p = stats.kstest(dw, "pareto", args=(w["pareto_alpha"][s], 0.0, w["pareto_xm"][s])).pvalue
        assert p > 1e-4, f"{name}: dwell of state {s}, KS p = {p:.3g}"
        rate = w["rates"][s]
        if rate > 0.0:
            p = stats.kstest(r["next_arr"][sel], "expon", args=(0.0, 1.0 / rate)).pvalue
            assert p > 1e-4, f"{name}: first gap in state {s}, KS p = {p:.3g}"
        else:
            assert np.all(np.isinf(r["next_arr"][sel]))


@pytest.mark.parametrize("name", ["C2", "C4", "C5"])
def test_stationary_start(orc, name):
    pin_stationary_start(orc, name)


# ---- Philox4x32-10 against PyTorch's engine ------------------------------------------------------
_TORCH_REF = None


def _torch_philox():
    global _TORCH_REF
    if _TORCH_REF is None:
        import torch
        inc = os.path.join(os.path.dirname(torch.__file__), "include")
        if not os.path.exists(os.path.join(inc, "ATen", "core", "PhiloxRNGEngine.h")):
            pytest.skip("PyTorch's Philox header is not installed")
        d = tempfile.mkdtemp(prefix="philox_ref_")
        so = os.path.join(d, "libphilox_torch.so")
        subprocess.run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-I", inc,
                        os.path.join(HERE, "philox_torch_ref.cpp"), "-o", so], check=True)
        L = C.CDLL(so)
        L.torch_philox_blocks.argtypes = [C.c_int64, C.c_void_p, C.c_void_p, C.c_void_p]
        _TORCH_REF = (L, d)
    return _TORCH_REF[0]


def pin_philox(orc):
    L = _torch_philox()
    rng = np.random.default_rng(0xF11)
    n = 50000
    ctr = rng.integers(0, 2 ** 32, size=(n, 4), dtype=np.uint64).astype(np.uint32)
    ctr[:8] = np.array([[0, 0, 0, 0], [0xFFFFFFFF] * 4, [1, 0, 0, 0], [0, 0, 0, 1],
                        [0, 0xFFFFFFFF, 0, 0], [0, 0, 0xFFFFFFFF, 0], [7, 3, 1 << 24, 1],
                        [255, 0xFFFFFFFF, (6 << 24), 0]], np.uint32)
    ctr = np.ascontiguousarray(ctr)
    for key in ([0, 0], [0xFFFFFFFF, 0xFFFFFFFF], [0xC0FFEE, 0], [0x5EED0004, 0x9E3779B9]):
        k = np.array(key, np.uint32)
        ref = np.empty_like(ctr)
        L.torch_philox_blocks(n, ctr.ctypes.data, k.ctypes.data, ref.ctypes.data)
        got = orc.philox4x32_batch(ctr, int(key[0]) | (int(key[1]) << 32))
        assert np.array_equal(got, ref), f"key {key}: {np.sum(np.any(got != ref, axis=1))} blocks differ"


def test_philox4x32_matches_pytorch_engine(orc):
    pin_philox(orc)


# ---- each pin rejects a broken oracle --------------------------------------------------------------
SRC = os.path.join(os.path.dirname(HERE), "oracle", "oracle.c")

MUTANTS = {
    # observation: last class without the +1 (a never-used server would read -1/C)
    "obs_last_class": (["(float)((double)(S->last_cls[j] + 1) * inv_c)"],
                       ["(float)((double)(S->last_cls[j]) * inv_c)"], [pin_t4]),
    # observation: remaining service and last class in the other order
    "obs_server_order": (["      obs[i++] = (float)(rem * inv_tw);\n"
                          "      obs[i++] = (float)((double)(S->last_cls[j] + 1) * inv_c);"],
                         ["      obs[i++] = (float)((double)(S->last_cls[j] + 1) * inv_c);\n"
                          "      obs[i++] = (float)(rem * inv_tw);"], [pin_t4]),
    # observation: per-class age before queue length
    "obs_class_order": (["      obs[i++] = (float)((double)S->q[cc] * inv_n);\n"
                         "      double age = S->q[cc] > 0 ? t - S->ring[cc][S->head[cc]] : 0.0;\n"
                         "      obs[i++] = (float)(age * inv_tw);"],
                        ["      double age = S->q[cc] > 0 ? t - S->ring[cc][S->head[cc]] : 0.0;\n"
                         "      obs[i++] = (float)(age * inv_tw);\n"
                         "      obs[i++] = (float)((double)S->q[cc] * inv_n);"], [pin_t4]),
    # class draw against the per-class probabilities instead of the cumulative mix
    "class_not_cumulative": (["while (!(uc < t->d->class_cum[cls])) cls++;"],
                             ["while (cls < c->n_classes - 1 && !(uc < c->class_mix[cls])) cls++;"],
                             [lambda o: pin_class_mix(o, "C4"), pin_arrival_stream]),
    # gap and class words exchanged inside the arrival block
    "arrival_words_swapped": (["double uc = u01(w[2], w[3]);",
                               "    S->next_arr = now + gap_draw(t, S->proc, u01(w[0], w[1]));"],
                              ["double uc = u01(w[0], w[1]);",
                               "    S->next_arr = now + gap_draw(t, S->proc, u01(w[2], w[3]));"],
                              [pin_arrival_stream]),
    # lognormal service without its linear per-batch term
    "logn_no_linear_term": (["return c->svc_median[h] * det_exp(c->svc_sigma * z) + c->svc_beta[h] * (double)n;"],
                            ["return c->svc_median[h] * det_exp(c->svc_sigma * z);"],
                            [pin_lognormal_service]),
    # every environment starts in state 0
    "start_state_0": (["while (!(us < d->stat_cum[s])) s++;"], ["(void)us;"],
                      [lambda o: pin_stationary_start(o, "C4")]),
    # the first dwell drawn for state 0 whatever the initial state
    "start_dwell_wrong_state": (["S->next_sw = dwell_draw(&t, s, u01(w[0], w[1]));"],
                                ["S->next_sw = dwell_draw(&t, 0, u01(w[0], w[1]));"],
                                [lambda o: pin_stationary_start(o, "C5")]),
    # a Philox round with the two multipliers' products exchanged
    "philox_round": (["uint32_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;"],
                     ["uint32_t n0 = hi0 ^ c1 ^ k0, n1 = lo0, n2 = hi1 ^ c3 ^ k1, n3 = lo1;"],
                     [pin_philox]),
}


@pytest.fixture(scope="module")
def mutant_dir():
    d = tempfile.mkdtemp(prefix="oracle_mutants_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pin_rejects_broken_oracle(orc, mutant_dir, mutant):
    from oracle import build
    olds, news, pins = MUTANTS[mutant]
    text = open(SRC).read()
    for old, new in zip(olds, news):
        assert text.count(old) == 1, f"{mutant}: the line to break is not in oracle.c"
        text = text.replace(old, new)
    lib = build.build_variant(text, os.path.join(mutant_dir, f"lib_{mutant}.so"))
    with orc.use_library(lib):
        for pin in pins:
            with pytest.raises(AssertionError):
                pin(orc)
