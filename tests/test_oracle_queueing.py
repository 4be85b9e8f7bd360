"""Pins of the oracle's simulator: textbook closed forms with the batch size fixed at 1,
Little's law as an exact sample-path identity, conservation, hand-enumerated traces,
determinism, independence of environments and the mean rates of the arrival processes."""
import json
import math
import os

import numpy as np
import pytest

from workloads import preset, trace_preset
from workloads.gen import seeded_actions
from workloads.presets import (ARR_MODULATED, DWELL_EXP, DWELL_INF, SVC_DET, SVC_EXP,
                               n_actions)

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_traces.json")))


def single_server(rate, svc_kind, alpha, beta, N=100, K=1, shadow=0, bmax=32, tout=0.010):
    return trace_preset(arrival_kind=ARR_MODULATED, rates=[rate], dwell_kind=[DWELL_INF],
                        dwell_mean=[0.0], pareto_alpha=[0.0], pareto_xm=[0.0],
                        n_servers=K, n_classes=1, queue_cap=N, service_kind=[svc_kind],
                        svc_alpha=[alpha], svc_beta=[beta], svc_median=[0.0],
                        obs_dim=2 + 4 * K + 4 if K > 1 else 8, lambda_ref=rate,
                        shadow=shadow, static_bmax=bmax, static_timeout=tout)


def run_stats(orc, w, seed, n_env, T):
    res = orc.rollout(w, seed, T, np.arange(n_env), actions=np.zeros((T, n_env), np.uint8),
                      want_obs=False, want_rec=False, want_reward=False)
    return res


def mean_se(x):
    x = np.asarray(x, dtype=np.float64)
    return x.mean(), x.std(ddof=1) / math.sqrt(len(x))


def check(val_se, expected, z=4.5, rel_bias=0.01):
    m, se = val_se
    assert abs(m - expected) <= z * se + rel_bias * abs(expected), (m, se, expected)


N_ENV, T_LONG = 48, 250000   # 48 independent replications of 250 s


def test_md1_pollaczek_khinchine(orc):
    """M/D/1, lambda=100/s, D=5 ms (alpha 4 + beta 1): L_q = rho^2/(2(1-rho)) = 0.25,
    W_q = 2.5 ms, W = 7.5 ms, L = 0.75 (batch size 1, action 0 every tick)."""
    w = single_server(100.0, SVC_DET, 0.004, 0.001)
    r = run_stats(orc, w, 1, N_ENV, T_LONG)
    H = T_LONG * 1e-3
    s, c = r["sums"][:, 0], r["counters"][:, 0]
    check(mean_se(s[:, 4] / H), 0.25)
    check(mean_se(s[:, 3] / H), 0.75)
    check(mean_se(s[:, 2] / c[:, 3]), 0.0025)
    check(mean_se(s[:, 0] / c[:, 3]), 0.0075)


def test_mm1(orc):
    """M/M/1, lambda=100/s, mean service 5 ms: L=1, L_q=0.5, W=10 ms, W_q=5 ms."""
    w = single_server(100.0, SVC_EXP, 0.005, 0.0)
    r = run_stats(orc, w, 2, N_ENV, T_LONG)
    H = T_LONG * 1e-3
    s, c = r["sums"][:, 0], r["counters"][:, 0]
    check(mean_se(s[:, 3] / H), 1.0)
    check(mean_se(s[:, 4] / H), 0.5)
    check(mean_se(s[:, 0] / c[:, 3]), 0.010)
    check(mean_se(s[:, 2] / c[:, 3]), 0.005)


def test_mm1k_blocking(orc):
    """M/M/1/K with 4 waiting places + 1 in service (K=5), lambda=90, mu=100:
    P_block = (1-rho) rho^5 / (1-rho^6), L = sum_n n p_n, W = L / (lambda (1-P_block))."""
    rho = 0.9
    p = np.array([(1 - rho) * rho**n / (1 - rho**6) for n in range(6)])
    pb = p[5]
    L = float((np.arange(6) * p).sum())
    W = L / (90.0 * (1 - pb))
    assert abs(pb - 0.126023) < 1e-6
    w = single_server(90.0, SVC_EXP, 0.010, 0.0, N=4)
    r = run_stats(orc, w, 3, N_ENV, T_LONG)
    H = T_LONG * 1e-3
    s, c = r["sums"][:, 0], r["counters"][:, 0]
    check(mean_se(c[:, 2] / c[:, 0]), pb)
    check(mean_se(s[:, 3] / H), L)
    check(mean_se(s[:, 0] / c[:, 3]), W)


def test_mmc_erlang_c_static_rule(orc):
    """M/M/4 through the static rule with B=1 and T=0 (FCFS to the lowest idle server),
    lambda=300, mu=100: Erlang C = 0.509434, W_q = C/(c mu - lambda), L_q = lambda W_q."""
    a, cc = 3.0, 4
    rho = a / cc
    top = a**cc / math.factorial(cc) / (1 - rho)
    erl = top / (sum(a**k / math.factorial(k) for k in range(cc)) + top)
    assert abs(erl - 0.509434) < 1e-6
    Wq = erl / (cc * 100.0 - 300.0)
    w = single_server(300.0, SVC_EXP, 0.010, 0.0, K=4, shadow=1, bmax=1, tout=0.0)
    r = run_stats(orc, w, 4, N_ENV, T_LONG // 2)
    H = (T_LONG // 2) * 1e-3
    s, c = r["sums"][:, 1], r["counters"][:, 1]
    check(mean_se(s[:, 2] / c[:, 3]), Wq)
    check(mean_se(s[:, 4] / H), 300.0 * Wq)
    check(mean_se(s[:, 0] / c[:, 3]), Wq + 0.010)
    # fraction of arrivals that wait at all equals Erlang C (PASTA)


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_littles_law_exact_and_conservation(orc, name):
    """Integral of N(t) over [0,H] equals the sum over accepted requests of
    min(c_r, H) - a_r (exact sample-path identity), per env and system; flow balance."""
    w = preset(name)
    T, n = 400, 6
    acts = seeded_actions(77, T, n, n_actions(w), small_bias=0.5)
    r = orc.rollout(w, 0xC0FFEE, T, np.arange(n), actions=acts)
    nsys = 2 if w["shadow"] else 1
    for s in range(nsys):
        an, soj = r["sums"][:, s, 3], r["sums"][:, s, 5]
        np.testing.assert_allclose(an, soj, rtol=1e-9, atol=1e-15)
        ct = r["counters"][:, s]
        assert np.all(ct[:, 0] == ct[:, 1] + ct[:, 2])          # arrivals = accepted + dropped
        assert np.all(ct[:, 3] == ct[:, 5] + ct[:, 6])          # dispatched = completed + inflight
        rec = r["rec"][:, :, s]
        arr = np.cumsum(rec[:, :, 3], axis=0)
        disp = np.cumsum(rec[:, :, 0], axis=0)
        acc = arr - rec[:, :, 4]
        assert np.all(acc == rec[:, :, 2] + disp)                # accepted = queued + dispatched
        assert np.all(rec[:, :, 2] <= w["queue_cap"])
        assert np.all(rec[:, :, 5] <= disp)
        assert np.all(rec[:, :, 2] == rec[:, :, 6:10].sum(axis=2))
        assert ct[:, 3].sum() > 0


def test_determinism_and_env_independence(orc):
    w = preset("C3")
    T = 300
    acts = seeded_actions(5, T, 8, n_actions(w))
    ids = np.array([3, 17, 1000, 5, 9, 123456, 2, 77], np.uint32)
    a = orc.rollout(w, 99, T, ids, actions=acts)
    b = orc.rollout(w, 99, T, ids, actions=acts)
    for k in ("reward", "obs", "rec", "chk", "sums"):
        assert np.array_equal(a[k], b[k])
    alone = orc.rollout(w, 99, T, ids[5:6], actions=acts[:, 5:6])
    assert np.array_equal(alone["reward"][:, 0], a["reward"][:, 5])
    assert np.array_equal(alone["obs"][:, 0], a["obs"][:, 5])
    assert np.array_equal(alone["chk"][0], a["chk"][5])


@pytest.mark.parametrize("name,mean_rate,tol", [("C2", 1100.0, 0.03), ("C4", 5166.6667, 0.03),
                                                ("C5", 2000.0, 0.06)])
def test_modulated_arrival_mean_rates(orc, name, mean_rate, tol):
    """Long-run arrival rate = sum_i pi_i lambda_i with pi_i proportional to the mean dwell:
    C2 (200+2000)/2, C4 (500+3000+12000)/3, C5 0.1 * 20000 (ON 10 ms, OFF Pareto mean 90 ms)."""
    base = preset(name)
    w = single_server(1.0, SVC_DET, 1e-4, 0.0)
    for k in ("rates", "dwell_kind", "dwell_mean", "pareto_alpha", "pareto_xm"):
        w[k] = base[k]
    w["lambda_ref"] = max(base["rates"])
    T = 100000
    r = run_stats(orc, w, 6, 48, T)
    rate = r["counters"][:, 0, 0].sum() / (48 * T * 1e-3)
    assert abs(rate / mean_rate - 1) < tol, rate


def _trace_cfg(g):
    w = trace_preset(**g["cfg"])
    return w


def _trace(g):
    arr = g["arrivals"]
    times = np.array([[a[0] for a in arr]])
    cls = np.array([[a[1] for a in arr]], np.uint8)
    return dict(times=times, classes=cls, counts=np.array([len(arr)], np.int32))


def test_hand_trace_T1(orc):
    g = GOLD["T1"]
    w = _trace_cfg(g)
    T = g["T"]
    r = orc.rollout(w, 0, T, [0], actions=np.full((T, 1), g["action"], np.uint8),
                    trace=_trace(g), disp_cap=64)
    rec = r["rec"][:, 0, 0]
    assert list(rec[:, 2]) == g["sumq"]
    assert list(rec[:, 0]) == g["n_k"]
    assert list(rec[:, 4]) == g["dropped_cum"]
    assert list(rec[:, 5]) == g["completed_cum"]
    for k in range(T):
        exp = g["rewards"].get(str(k), 0.0)
        assert abs(r["reward"][k, 0] - exp) <= 1e-9 * max(1.0, abs(exp))
    np.testing.assert_allclose(r["obs"][1, 0], np.array(g["obs1"], np.float32), rtol=1e-6)
    assert abs(r["sums"][0, 0, 5] - g["sojourn_sum"]) < 1e-12
    assert abs(r["sums"][0, 0, 3] - g["sojourn_sum"]) < 1e-12
    d = [(x["k"], x["server"], x["cls"], x["n"], x["t"], x["c"]) for x in r["disp"] if x["sys"] == 0]
    assert len(d) == len(g["dispatches"])
    for got, exp in zip(d, g["dispatches"]):
        assert got[:4] == tuple(exp[:4])
        assert abs(got[4] - exp[4]) < 1e-12 and abs(got[5] - exp[5]) < 1e-12


def test_hand_trace_T2(orc):
    g = GOLD["T2"]
    w = _trace_cfg(g)
    T = g["T"]
    acts = np.array(g["actions"], np.uint8)[:, None]
    r = orc.rollout(w, 0, T, [0], actions=acts, trace=_trace(g), disp_cap=64)
    d = [(x["k"], x["server"], x["cls"], x["n"], x["t"], x["c"]) for x in r["disp"] if x["sys"] == 0]
    assert len(d) == len(g["dispatches"])
    for got, exp in zip(d, g["dispatches"]):
        assert got[:4] == tuple(exp[:4])
        assert abs(got[4] - exp[4]) < 1e-12 and abs(got[5] - exp[5]) < 1e-12
    for k in range(T):
        exp = g["rewards"].get(str(k), 0.0)
        assert abs(r["reward"][k, 0] - exp) <= 1e-9 * max(1.0, abs(exp))
    for k, v in g["completed_at"].items():
        assert r["rec"][int(k), 0, 0, 5] == v
    acts2 = np.array(g["variant_actions"], np.uint8)[:, None]
    r2 = orc.rollout(w, 0, T, [0], actions=acts2, trace=_trace(g))
    assert r2["rec"][1, 0, 0, 0] == g["variant_n_k_tick1"]


def test_hand_trace_T3_static_rule(orc):
    g = GOLD["T3"]
    w = _trace_cfg(g)
    T = g["T"]
    r = orc.rollout(w, 0, T, [0], actions=np.zeros((T, 1), np.uint8), trace=_trace(g),
                    disp_cap=64)
    d = [(x["k"], x["server"], x["cls"], x["n"], x["t"], x["c"]) for x in r["disp"] if x["sys"] == 1]
    assert len(d) == len(g["shadow_dispatches"])
    for got, exp in zip(d, g["shadow_dispatches"]):
        assert got[:4] == tuple(exp[:4])
        assert abs(got[4] - exp[4]) < 1e-12 and abs(got[5] - exp[5]) < 1e-12
    assert abs(r["sums"][0, 1, 0] - g["shadow_latency_sum"]) < 1e-12
