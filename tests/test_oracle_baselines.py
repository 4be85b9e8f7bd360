"""Pins of the baseline rules and the Extreme Burst workload in the oracle (R23, R24):
the square wave's windows, the M/M/c queue under random and round-robin routing (routing
among identical idle servers leaves the Erlang-C waiting time unchanged), uniform random
routing and the exact cycle of round robin on a trace where every server is idle at every
dispatch, and a fixed batch of 8 (Static-8) on a trace. Shortest-Queue routing (R27): a
hand-enumerated trace (T5), its waiting time strictly between the central-queue M/M/2 and two
M/M/1 queues fed by a random split, Little's law and flow balance with the per-server queues."""
import math

import numpy as np
import pytest
from scipy import stats

import json
import os

from workloads import baseline_preset, burst_preset, trace_preset
from workloads.gen import seeded_actions
from workloads.presets import (ARR_MODULATED, DWELL_INF, ROUTE_RANDOM, ROUTE_ROUND_ROBIN,
                               ROUTE_SHORTEST, SVC_DET, SVC_EXP, n_actions)

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_traces.json")))


def test_extreme_burst_square_wave(orc):
    """100 req/s for 200 ticks, then none for 200 ticks, starting high: every off window is
    empty and the on windows hold Poisson(20) counts."""
    n, T = 64, 2000
    w = burst_preset(n_envs=n)
    r = orc.rollout(w, 5, T, np.arange(n), actions=np.zeros((T, n), np.uint8), want_obs=False,
                    want_reward=False)
    A = r["rec"][:, :, 0, 3].astype(np.int64)              # [T][n] arrivals per tick
    win = A.reshape(T // 200, 200, n).sum(axis=1)          # [window][env]
    assert np.all(win[1::2] == 0)
    on = win[0::2].ravel()
    assert abs(on.mean() - 20.0) <= 4.5 * math.sqrt(20.0 / on.size)
    assert abs(on.var(ddof=1) - 20.0) <= 0.2 * 20.0
    # the shadow system sees the same arrivals
    assert np.array_equal(r["rec"][:, :, 1, 3], r["rec"][:, :, 0, 3])


def mmc(route):
    return trace_preset(arrival_kind=ARR_MODULATED, rates=[300.0], dwell_kind=[DWELL_INF],
                        dwell_mean=[0.0], pareto_alpha=[0.0], pareto_xm=[0.0], n_servers=4,
                        n_classes=1, queue_cap=100, service_kind=[SVC_EXP], svc_alpha=[0.010],
                        svc_beta=[0.0], svc_median=[0.0], obs_dim=2 + 16 + 4,
                        lambda_ref=300.0, shadow=1, static_bmax=1, static_timeout=0.0,
                        static_route=route)


@pytest.mark.parametrize("route", [ROUTE_RANDOM, ROUTE_ROUND_ROBIN])
def test_mmc_waiting_time_unchanged_by_routing(orc, route):
    """M/M/4, lambda = 300, mu = 100, B = 1, T = 0: W_q = C(4, 3)/(c mu - lambda) whichever
    idle server takes the request."""
    a, cc = 3.0, 4
    top = a**cc / math.factorial(cc) / (1 - a / cc)
    erl = top / (sum(a**k / math.factorial(k) for k in range(cc)) + top)
    Wq = erl / (cc * 100.0 - 300.0)
    n_env, T = 48, 125000
    r = orc.rollout(mmc(route), 4, T, np.arange(n_env), actions=np.zeros((T, n_env), np.uint8),
                    want_obs=False, want_rec=False, want_reward=False)
    s, c = r["sums"][:, 1], r["counters"][:, 1]
    x = s[:, 2] / c[:, 3]
    m, se = x.mean(), x.std(ddof=1) / math.sqrt(len(x))
    assert abs(m - Wq) <= 4.5 * se + 0.01 * Wq, (m, se, Wq)


def sparse_trace(route, K=4, n=400, gap=0.003, svc=0.001, B=1):
    """One request every `gap` seconds with service `svc` < gap: every server is idle at
    every dispatch."""
    w = trace_preset(n_servers=K, n_classes=1, obs_dim=2 + 4 * K + 4, shadow=1,
                     static_bmax=B, static_timeout=0.0, static_route=route,
                     service_kind=[SVC_DET], svc_alpha=[svc], svc_beta=[0.0],
                     svc_median=[0.0], trace_max_len=n)
    times = (np.arange(n) + 0.5) * gap
    tr = dict(times=times[None, :], classes=np.zeros((1, n), np.uint8),
              counts=np.array([n], np.int32))
    return w, tr


def shadow_servers(orc, w, tr, T):
    r = orc.rollout(w, 9, T, [0], actions=np.zeros((T, 1), np.uint8), trace=tr,
                    disp_cap=4096, want_obs=False)
    return np.array([d["server"] for d in r["disp"] if d["sys"] == 1])


def test_round_robin_cycles_through_idle_servers(orc):
    w, tr = sparse_trace(ROUTE_ROUND_ROBIN, K=3, n=90)
    srv = shadow_servers(orc, w, tr, 300)
    assert len(srv) == 90
    assert np.array_equal(srv, np.arange(90) % 3)


def test_random_routing_is_uniform(orc):
    w, tr = sparse_trace(ROUTE_RANDOM, K=4, n=2000, gap=0.002, svc=0.0005)
    srv = shadow_servers(orc, w, tr, 4100)
    assert len(srv) == 2000
    counts = np.bincount(srv, minlength=4)
    assert stats.chisquare(counts).pvalue > 1e-4
    # successive choices are not a fixed cycle
    assert np.any(np.diff(srv) % 4 != 1)


def test_static8_dispatches_batches_of_eight(orc):
    """Eight requests 0.1 ms apart: the eighth arrival completes a batch of 8 at its own
    instant; a lone ninth request leaves only after the 10 ms timeout."""
    K = 1
    w = trace_preset(n_servers=K, n_classes=1, obs_dim=8, shadow=1, static_bmax=8,
                     static_timeout=0.010, service_kind=[SVC_DET], svc_alpha=[0.002],
                     svc_beta=[0.0], svc_median=[0.0], trace_max_len=9)
    times = np.array([0.0001 * (i + 1) for i in range(8)] + [0.0200])
    tr = dict(times=times[None, :], classes=np.zeros((1, 9), np.uint8),
              counts=np.array([9], np.int32))
    r = orc.rollout(w, 1, 40, [0], actions=np.zeros((40, 1), np.uint8), trace=tr, disp_cap=16,
                    want_obs=False)
    d = [(x["n"], x["t"]) for x in r["disp"] if x["sys"] == 1]
    assert len(d) == 2
    assert d[0][0] == 8 and d[0][1] == times[7]
    assert d[1][0] == 1 and abs(d[1][1] - (0.0200 + 0.010)) < 1e-15


def test_hand_trace_T5_shortest_queue(orc):
    g = GOLD["T5"]
    w = trace_preset(**g["cfg"])
    T = g["T"]
    arr = g["arrivals"]
    tr = dict(times=np.array([[a[0] for a in arr]]),
              classes=np.array([[a[1] for a in arr]], np.uint8),
              counts=np.array([len(arr)], np.int32))
    r = orc.rollout(w, 0, T, [0], actions=np.zeros((T, 1), np.uint8), trace=tr, disp_cap=64)
    d = [(x["k"], x["server"], x["cls"], x["n"], x["t"], x["c"]) for x in r["disp"] if x["sys"] == 1]
    assert len(d) == len(g["shadow_dispatches"])
    for got, exp in zip(d, g["shadow_dispatches"]):
        assert got[:4] == tuple(exp[:4]), (got, exp)
        assert abs(got[4] - exp[4]) < 1e-12 and abs(got[5] - exp[5]) < 1e-12, (got, exp)
    for k in range(T):
        exp = g["shadow_rewards"].get(str(k), 0.0)
        assert abs(r["reward_shadow"][k, 0] - exp) <= 1e-9 * max(1.0, abs(exp)), (k, exp)
    assert list(r["rec"][:, 0, 1, 5]) == g["shadow_completed_cum"]
    assert abs(r["sums"][0, 1, 0] - g["shadow_latency_sum"]) < 1e-12


def two_servers(route):
    return trace_preset(arrival_kind=ARR_MODULATED, rates=[150.0], dwell_kind=[DWELL_INF],
                        dwell_mean=[0.0], pareto_alpha=[0.0], pareto_xm=[0.0], n_servers=2,
                        n_classes=1, queue_cap=100, service_kind=[SVC_EXP], svc_alpha=[0.010],
                        svc_beta=[0.0], svc_median=[0.0], obs_dim=2 + 8 + 4,
                        lambda_ref=150.0, shadow=1, static_bmax=1, static_timeout=0.0,
                        static_route=route)


def test_shortest_queue_between_central_queue_and_random_split(orc):
    """Two exponential servers (mu = 100), Poisson lambda = 150, B = 1, T = 0. A central FCFS
    queue (M/M/2) has the least mean wait of any policy for identical exponential servers:
    W_q = C(2, 1.5)/(2 mu - lambda) = 12.857 ms. Shortest-Queue commits each request to one
    server's queue (a request can wait there while the other server idles), so it waits
    strictly longer; and it waits strictly less than under a blind random split, two M/M/1
    queues at lambda/2: rho/(mu - lambda/2) = 30 ms."""
    a, cc = 1.5, 2
    top = a**cc / math.factorial(cc) / (1 - a / cc)
    Wq_central = top / (sum(a**k / math.factorial(k) for k in range(cc)) + top) / (cc * 100.0 - 150.0)
    assert abs(Wq_central - 0.0128571) < 1e-6
    Wq_split = 0.75 / (100.0 - 75.0)
    n_env, T = 96, 100000
    r = orc.rollout(two_servers(ROUTE_SHORTEST), 4, T, np.arange(n_env),
                    actions=np.zeros((T, n_env), np.uint8), want_obs=False, want_rec=False,
                    want_reward=False)
    s, c = r["sums"][:, 1], r["counters"][:, 1]
    x = s[:, 2] / c[:, 3]
    m, se = x.mean(), x.std(ddof=1) / math.sqrt(len(x))
    assert m - 4.5 * se > Wq_central, (m, se, Wq_central)
    assert m + 4.5 * se < Wq_split, (m, se, Wq_split)
    # the central queue itself, through the lowest-idle rule on the same arrivals
    r0 = orc.rollout(two_servers(0), 4, T, np.arange(n_env), actions=np.zeros((T, n_env), np.uint8),
                     want_obs=False, want_rec=False, want_reward=False)
    x0 = r0["sums"][:, 1, 2] / r0["counters"][:, 1, 3]
    m0, se0 = x0.mean(), x0.std(ddof=1) / math.sqrt(len(x0))
    assert abs(m0 - Wq_central) <= 4.5 * se0 + 0.01 * Wq_central


def test_shortest_queue_littles_law_and_conservation(orc):
    """C3 with a Shortest-Queue shadow system: integral of N(t) (waiting, queued at a server or
    in service) equals the sum of min(c_r, H) - a_r exactly; every tick, arrivals = accepted +
    dropped, accepted = queued + dispatched, dispatched = completed + assigned."""
    w = baseline_preset("shortest", "C3")
    T, n = 400, 6
    acts = seeded_actions(78, T, n, n_actions(w), small_bias=0.5)
    r = orc.rollout(w, 0xC0FFEE, T, np.arange(n), actions=acts)
    an, soj = r["sums"][:, 1, 3], r["sums"][:, 1, 5]
    np.testing.assert_allclose(an, soj, rtol=1e-9, atol=1e-15)
    ct = r["counters"][:, 1]
    assert np.all(ct[:, 0] == ct[:, 1] + ct[:, 2])
    assert np.all(ct[:, 3] == ct[:, 5] + ct[:, 6])
    rec = r["rec"][:, :, 1]
    acc = np.cumsum(rec[:, :, 3], axis=0) - rec[:, :, 4]
    assert np.all(acc == rec[:, :, 2] + np.cumsum(rec[:, :, 0], axis=0))
    assert ct[:, 3].sum() > 0 and ct[:, 6].sum() >= 0
