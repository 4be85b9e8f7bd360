"""GPU parity: the HIP path through the C ABI against the CPU oracle, on the same seeded
inputs. Integer state bit-exact; fp64 floats within 1e-9 relative; fp32/bf16 policy
outputs within a tolerance derived from the rounding points (see the MLP tests)."""
import json
import os
import sys

import numpy as np
import pytest

from workloads import preset, trace_preset, burst_preset, baseline_preset, attn_preset
from workloads.gen import seeded_actions, seeded_obs, seeded_rewards_values, seeded_weights_f32
from policy_check import attn_tol, check_attn_logits, check_layers, end_to_end_bound

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_traces.json")))
NAMES = ["C1", "C2", "C3", "C4", "C5"]
RTOL = 1e-9
# the attention policy of Sec. 4.2 in the variants the kernel is built for
ATTN = {
    "attn": dict(),                                        # 8 tokens, 2 heads, 6 actions
    "attn_L1": dict(attn_tokens=1),                        # the plain input projection
    "attn_L4_H4": dict(attn_tokens=4, attn_heads=4),
    "attn_L2_H1": dict(attn_tokens=2, attn_heads=1),
    "attn_K4": dict(n_servers=4, obs_dim=2 + 16 + 6, n_classes=1, attn_tokens=8),
}


def workload(name, **kw):
    if name in ATTN:
        return attn_preset(**dict(ATTN[name], **kw))
    return preset(name, **kw)


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def bs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_05272_amd as m
    m.load()
    return m


def gpu_run_actions(bs, w, E, T, seed, acts, store_obs=True):
    """reset + T sim_step calls with the given actions [T][E] (host uint8)."""
    sim = bs.Sim(w, n_envs=E)
    sim.reset(seed)
    dev = torch.device("cuda")
    obs = [sim.obs()] if store_obs else None
    rew, rsh = [], []
    a_dev = torch.from_numpy(np.ascontiguousarray(acts)).to(dev)
    for k in range(T):
        o, r, rs = sim.step(a_dev[k], want_obs=store_obs)
        if store_obs:
            obs.append(o)
        rew.append(r)
        if rs is not None:
            rsh.append(rs)
    sim.sync()
    cnt, sums = sim.counters()
    chk = sim.checksums()
    tot = sim.stats()
    out = dict(reward=torch.stack(rew).cpu().numpy(),
               cnt=cnt.cpu().numpy(), sums=sums.cpu().numpy(),
               chk=chk.cpu().numpy().view(np.uint64), tot=tot)
    if rsh:
        out["reward_shadow"] = torch.stack(rsh).cpu().numpy()
    if store_obs:
        out["obs"] = torch.stack(obs).cpu().numpy()  # [T+1][F][E]
    sim.close()
    return out


def assert_close_rel(a, b, what):
    a = np.asarray(a); b = np.asarray(b)
    err = np.abs(a - b) / np.maximum(np.abs(b), 1e-300)
    bad = ~((err <= RTOL) | (a == b))
    assert not bad.any(), f"{what}: {bad.sum()} mismatches, first at {np.argwhere(bad)[0]}"


def compare_sim(orc_res, g, w, env_cols, nsys):
    """Oracle result for envs env_cols (in that order) vs GPU arrays indexed by env."""
    for s in range(nsys):
        assert np.array_equal(g["chk"][s, env_cols], orc_res["chk"][:, s]), f"checksum sys {s}"
        assert np.array_equal(g["cnt"][s, :, env_cols], orc_res["counters"][:, s]), f"counters sys {s}"
        assert_close_rel(g["sums"][s, :, env_cols], orc_res["sums"][:, s, :2], f"sums sys {s}")
    assert_close_rel(g["reward"][:, env_cols], orc_res["reward"], "reward")
    if nsys == 2:
        assert_close_rel(g["reward_shadow"][:, env_cols], orc_res["reward_shadow"], "reward_shadow")
    if "obs" in g:
        go = np.transpose(g["obs"][:, :, env_cols], (0, 2, 1))
        assert np.array_equal(go, orc_res["obs"]), "observations differ"


@pytest.mark.parametrize("name", NAMES)
def test_sim_step_parity_small(bs, orc, name):
    """All envs of a 300-env batch (one full block of 256 + a ragged tail), 200 ticks,
    seeded actions: checksums, counters, rewards and observations against the oracle."""
    w = preset(name)
    E, T, seed = 300, 200, 0xC0FFEE + NAMES.index(name)
    acts = seeded_actions(seed, T, E, 6 * w["n_servers"], small_bias=0.5)
    say(f"[parity-small] {name} E={E} T={T}")
    g = gpu_run_actions(bs, w, E, T, seed, acts)
    r = orc.rollout(w, seed, T, np.arange(E), actions=acts)
    nsys = 2 if w["shadow"] else 1
    compare_sim(r, g, w, np.arange(E), nsys)
    assert g["cnt"][0, 3].sum() > 0 and g["cnt"][0, 0].sum() > 0
    # device totals equal the per-env counters summed
    assert np.array_equal(g["tot"]["cnt"][0], g["cnt"][0].sum(axis=1))
    if nsys == 2:
        assert np.array_equal(g["tot"]["cnt"][1], g["cnt"][1].sum(axis=1))


def _edge(name):
    from workloads.presets import DWELL_EXP, DWELL_INF, SVC_EXP
    if name == "queue255_states4":   # capacity and modulation states at their limits, overload
        return preset("C4", queue_cap=255, rates=[200.0, 2000.0, 20000.0, 60000.0],
                      dwell_kind=[DWELL_EXP] * 4, dwell_mean=[0.05, 0.02, 0.01, 0.005],
                      pareto_alpha=[0.0] * 4, pareto_xm=[0.0] * 4, shadow=1)
    if name == "no_arrivals":        # a process that never fires
        return preset("C3", rates=[0.0], dwell_kind=[DWELL_INF], dwell_mean=[0.0],
                      pareto_alpha=[0.0], pareto_xm=[0.0])
    if name == "cap1_overload":      # one waiting slot, ten times the service capacity
        return preset("C1", queue_cap=1, rates=[5000.0])
    if name == "exp_service_K16":    # exponential service on the 16-server system
        return preset("C5", service_kind=[SVC_EXP] * 4, svc_alpha=[1e-3, 5e-3, 2e-2, 8e-2])
    raise KeyError(name)


EDGE = ["queue255_states4", "no_arrivals", "cap1_overload", "exp_service_K16"]


@pytest.mark.parametrize("name", EDGE)
def test_edge_workloads_parity(bs, orc, name):
    """Configurations at the ABI's limits and the method's degenerate cases, 300 envs (a
    ragged tail) x 150 ticks, bit-exact against the oracle; plus the expected degenerate
    behaviour (nothing counted without arrivals; drops under overload)."""
    w = _edge(name)
    E, T, seed = 300, 150, 0xED6E + EDGE.index(name)
    acts = seeded_actions(seed, T, E, 6 * w["n_servers"], small_bias=0.5)
    say(f"[edge] {name} E={E} T={T}")
    g = gpu_run_actions(bs, w, E, T, seed, acts)
    r = orc.rollout(w, seed, T, np.arange(E), actions=acts)
    nsys = 2 if w["shadow"] else 1
    compare_sim(r, g, w, np.arange(E), nsys)
    if name == "no_arrivals":
        assert not g["cnt"].any() and not g["reward"].any()
    if name in ("queue255_states4", "cap1_overload"):
        assert g["cnt"][0, 2].sum() > 0          # dropped requests (counter 2)


def _tie_traces(seed, E, L, C):
    """Trace arrivals on a 0.25 ms grid, one to three per grid instant, classes drawn
    independently and listed in random order: many instants where a lower class arrives after
    a higher one at the same time, which decides the head of line between equal head times."""
    rng = np.random.default_rng(seed)
    times = np.zeros((E, L))
    cls = np.zeros((E, L), np.uint8)
    for e in range(E):
        t, i = 0.0, 0
        while i < L:
            t += 0.25e-3 * int(rng.integers(1, 4))
            for c in rng.integers(0, C, size=int(rng.integers(1, 4))):
                if i < L:
                    times[e, i], cls[e, i] = t, c
                    i += 1
    counts = np.full(E, L, np.int32)
    counts[::7] = L // 2            # some environments run out of arrivals mid-rollout
    return times, cls, counts


def test_trace_ties_parity(bs, orc):
    """Both systems against the oracle on trace arrivals with many simultaneous arrivals of
    different classes (4 classes, 4 servers, 20 waiting slots, static batch 4 or 2 ms):
    per-tick checksums, counters, sums and rewards bit-exact over 130 envs x 60 ticks."""
    from workloads.presets import SVC_DET
    E, T, L, C = 130, 60, 180, 4
    w = trace_preset(n_servers=4, n_classes=C, queue_cap=20, obs_dim=32, shadow=1,
                     static_bmax=4, static_timeout=2e-3, class_mix=[0.25] * C,
                     service_kind=[SVC_DET] * C, svc_alpha=[0.3e-3, 1e-3, 2e-3, 4e-3],
                     svc_beta=[0.1e-3, 0.2e-3, 0.5e-3, 1e-3], svc_median=[0.0] * C,
                     w_class=[200.0, 100.0, 40.0, 20.0])
    w["trace_max_len"] = L
    times, cls, counts = _tie_traces(0x71E5, E, L, C)
    acts = seeded_actions(0x71E5, T, E, 6 * w["n_servers"], small_bias=0.5)
    say(f"[trace-ties] E={E} T={T} L={L}")
    dev = torch.device("cuda")
    sim = bs.Sim(w, n_envs=E)
    sim.set_trace(torch.from_numpy(times).to(dev), torch.from_numpy(cls).to(dev),
                  torch.from_numpy(counts).to(dev))
    sim.reset(0)
    a_dev = torch.from_numpy(acts).to(dev)
    rew, rsh, rchk = [], [], []
    for k in range(T):
        _, r, rs = sim.step(a_dev[k], want_obs=False)
        rew.append(r); rsh.append(rs)
        rchk.append(sim.checksums()[0].clone())
    sim.sync()
    cnt, sums = sim.counters()
    g = dict(reward=torch.stack(rew).cpu().numpy(), reward_shadow=torch.stack(rsh).cpu().numpy(),
             cnt=cnt.cpu().numpy(), sums=sums.cpu().numpy(),
             chk=sim.checksums().cpu().numpy().view(np.uint64))
    g_rchk = torch.stack(rchk).cpu().numpy().view(np.uint64)
    sim.close()
    r = orc.rollout(w, 0, T, np.arange(E), actions=acts, want_obs=False, want_rchk=True,
                    trace=dict(times=times, classes=cls, counts=counts))
    assert np.array_equal(g_rchk, r["rchk"]), "learned-system checksums differ at some tick"
    compare_sim(r, g, w, np.arange(E), 2)
    assert g["cnt"][1, 4].sum() > 0 and g["cnt"][0, 4].sum() > 0   # both systems dispatched
    assert g["cnt"][0, 2].sum() > 0                                  # and dropped


def test_single_tick_and_single_env(bs, orc):
    """T = 1 on one environment and on 65 (one wave and one lane), against the oracle."""
    w = preset("C4")
    for E in (1, 65):
        acts = seeded_actions(3, 1, E, 6 * w["n_servers"])
        g = gpu_run_actions(bs, w, E, 1, 5, acts)
        r = orc.rollout(w, 5, 1, np.arange(E), actions=acts)
        compare_sim(r, g, w, np.arange(E), 1)


RULES = {
    "burst": lambda: burst_preset(),
    "static8_C3": lambda: baseline_preset("static8", "C3"),
    "random_C3": lambda: baseline_preset("random", "C3"),
    "round_robin_C3": lambda: baseline_preset("round_robin", "C3"),
    "random_C5": lambda: baseline_preset("random", "C5"),
    "round_robin_C4": lambda: baseline_preset("round_robin", "C4"),
    "shortest_C3": lambda: baseline_preset("shortest", "C3"),
    "shortest_C3_K2": lambda: baseline_preset("shortest", "C3", n_servers=2),
    "shortest_C2_K1": lambda: baseline_preset("shortest", "C2"),
    "shortest_C4": lambda: baseline_preset("shortest", "C4"),
}


@pytest.mark.parametrize("name", sorted(RULES))
def test_baselines_and_burst_parity(bs, orc, name):
    """The paper's baselines on the shadow system (Static-8, random and round-robin routing,
    R23, Shortest-Queue over per-server queues, R27) and the Extreme Burst square wave (R24):
    300 envs x 600 ticks, bit-exact integer state and rewards against the oracle."""
    w = RULES[name]()
    E, T, seed = 300, 600, 0xBA5E + len(name)
    acts = seeded_actions(seed, T, E, 6 * w["n_servers"], small_bias=0.5)
    say(f"[baselines] {name} E={E} T={T}")
    g = gpu_run_actions(bs, w, E, T, seed, acts)
    r = orc.rollout(w, seed, T, np.arange(E), actions=acts)
    compare_sim(r, g, w, np.arange(E), 2)
    assert g["cnt"][1, 3].sum() > 0


def _step_actions(seed, k, E, A):
    return np.random.default_rng([seed, k]).integers(0, A, size=E, dtype=np.int64).astype(np.uint8)


@pytest.mark.parametrize("name", NAMES)
def test_sim_step_parity_full_size_sampled(bs, orc, name):
    """Full E and T of each configuration in the simulator kernels' launch shape; the
    oracle replays sampled envs (first, last, a spread and a random set) under the same
    seeded per-step actions."""
    w = preset(name)
    E, T = w["n_envs"], w["T"]
    seed = 0xC0FFEE + NAMES.index(name)
    A = 6 * w["n_servers"]
    rng = np.random.default_rng(seed)
    cols = np.unique(np.concatenate([[0, 1, 255, 256, E - 1], rng.choice(E, 27, replace=False)]))
    cols = cols[cols < E]
    say(f"[parity-full] {name} E={E} T={T} sampled={len(cols)}")
    sim = bs.Sim(w)
    sim.reset(seed)
    dev = torch.device("cuda")
    rew = np.zeros((T, len(cols)))
    rsh = np.zeros((T, len(cols)))
    acts_cols = np.zeros((T, len(cols)), np.uint8)
    cols_dev = torch.from_numpy(cols).to(dev)
    for k in range(T):
        a = _step_actions(seed, k, E, A)
        acts_cols[k] = a[cols]
        _, r, rs = sim.step(torch.from_numpy(a).to(dev), want_obs=False)
        rew[k] = r[cols_dev].cpu().numpy()
        if rs is not None:
            rsh[k] = rs[cols_dev].cpu().numpy()
        if k % 512 == 0:
            say(f"  tick {k}")
    sim.sync()
    cnt, sums = sim.counters()
    chk = sim.checksums().cpu().numpy().view(np.uint64)
    cnt = cnt.cpu().numpy(); sums = sums.cpu().numpy()
    sim.close()
    res = orc.rollout(w, seed, T, cols, actions=acts_cols, want_obs=False, want_rec=False)
    nsys = 2 if w["shadow"] else 1
    for s in range(nsys):
        assert np.array_equal(chk[s, cols], res["chk"][:, s]), f"checksum sys {s}"
        assert np.array_equal(cnt[s][:, cols].T, res["counters"][:, s])
        assert_close_rel(sums[s][:, cols].T, res["sums"][:, s, :2], "sums")
    assert_close_rel(rew, res["reward"], "reward")
    if nsys == 2:
        assert_close_rel(rsh, res["reward_shadow"], "reward_shadow")


@pytest.mark.parametrize("E,lpw", [(9001, 8), (40001, 32)])
def test_lanes_per_wave_mappings(bs, orc, E, lpw):
    """Batch sizes for which the tick kernels spread the environments over waves of 8 and of
    32 lanes (the other spreads, 4, 16 and 64, are covered by the small, C3 and full-size
    cases): C5's workload (16 servers, bursts, static shadow) for 40 ticks, sampled
    environments at wave boundaries and a ragged last wave, against the oracle."""
    w = dict(preset("C5"), n_envs=E, T=40)
    T = w["T"]
    seed = 0xC0FFEE + lpw
    A = 6 * w["n_servers"]
    rng = np.random.default_rng(seed)
    cols = np.unique(np.concatenate([[0, lpw - 1, lpw, 2 * lpw - 1, E - 2, E - 1],
                                     rng.choice(E, 20, replace=False)]))
    say(f"[lanes per wave] E={E} lpw={lpw} sampled={len(cols)}")
    sim = bs.Sim(w)
    sim.reset(seed)
    dev = torch.device("cuda")
    rew = np.zeros((T, len(cols)))
    rsh = np.zeros((T, len(cols)))
    acts_cols = np.zeros((T, len(cols)), np.uint8)
    cols_dev = torch.from_numpy(cols).to(dev)
    for k in range(T):
        a = _step_actions(seed, k, E, A)
        acts_cols[k] = a[cols]
        _, r, rs = sim.step(torch.from_numpy(a).to(dev), want_obs=False)
        rew[k] = r[cols_dev].cpu().numpy()
        rsh[k] = rs[cols_dev].cpu().numpy()
    sim.sync()
    cnt, sums = sim.counters()
    chk = sim.checksums().cpu().numpy().view(np.uint64)
    cnt = cnt.cpu().numpy(); sums = sums.cpu().numpy()
    sim.close()
    res = orc.rollout(w, seed, T, cols, actions=acts_cols, want_obs=False, want_rec=False)
    for s_ in range(2):
        assert np.array_equal(chk[s_, cols], res["chk"][:, s_]), f"checksum sys {s_}"
        assert np.array_equal(cnt[s_][:, cols].T, res["counters"][:, s_])
        assert_close_rel(sums[s_][:, cols].T, res["sums"][:, s_, :2], "sums")
    assert_close_rel(rew, res["reward"], "reward")
    assert_close_rel(rsh, res["reward_shadow"], "reward_shadow")


def _trace_tensors(g, dev):
    arr = g["arrivals"]
    L = len(arr)
    times = torch.tensor([[a[0] for a in arr]], dtype=torch.float64, device=dev)
    cls = torch.tensor([[a[1] for a in arr]], dtype=torch.uint8, device=dev)
    cnt = torch.tensor([L], dtype=torch.int32, device=dev)
    return times, cls, cnt, L


@pytest.mark.parametrize("tr", ["T1", "T2", "T3", "T4", "T5"])
def test_hand_traces_on_gpu(bs, orc, tr):
    g = GOLD[tr]
    w = trace_preset(**g["cfg"])
    dev = torch.device("cuda")
    times, cls, cnt, L = _trace_tensors(g, dev)
    w["trace_max_len"] = L
    T = g["T"]
    if tr == "T1":
        acts = np.full((T, 1), g["action"], np.uint8)
    elif tr in ("T2", "T4"):
        acts = np.array(g["actions"], np.uint8)[:, None]
    else:
        acts = np.zeros((T, 1), np.uint8)
    say(f"[trace] {tr}")
    sim = bs.Sim(w, n_envs=1)
    sim.set_trace(times, cls, cnt)
    sim.reset(0)
    rews, rshs, obs = [], [], [sim.obs()]
    a_dev = torch.from_numpy(acts).to(dev)
    for k in range(T):
        o, r, rs = sim.step(a_dev[k])
        rews.append(r); obs.append(o)
        if rs is not None:
            rshs.append(rs)
    sim.sync()
    rew = torch.stack(rews).cpu().numpy()[:, 0]
    cnt_, sums = sim.counters()
    cnt_ = cnt_.cpu().numpy(); sums = sums.cpu().numpy()
    if tr in ("T1", "T2", "T4"):
        for k, v in g["rewards"].items():
            assert abs(rew[int(k)] - v) <= 1e-9 * max(1.0, abs(v))
        nz = [k for k in range(T) if str(k) not in g["rewards"]]
        assert np.all(rew[nz] == 0.0)
    if tr == "T1":
        o1 = obs[1].cpu().numpy()[:, 0]
        np.testing.assert_allclose(o1, np.array(g["obs1"], np.float32), rtol=1e-6)
        assert cnt_[0, 2, 0] == g["dropped_cum"][-1] and cnt_[0, 5, 0] == g["completed_cum"][-1]
    if tr == "T4":
        for k, v in g["obs"].items():
            np.testing.assert_allclose(obs[int(k)].cpu().numpy()[:, 0], np.array(v, np.float32),
                                       rtol=1e-6, atol=1e-9)
        assert cnt_[0, 5, 0] == g["completed_cum"][-1]
    if tr == "T5":
        for k, v in g["shadow_rewards"].items():
            assert abs(rshs[int(k)].cpu().numpy()[0] - v) <= 1e-9 * max(1.0, abs(v))
        assert abs(sums[1, 0, 0] - g["shadow_latency_sum"]) < 1e-12
        assert cnt_[1, 4, 0] == len(g["shadow_dispatches"])
        assert cnt_[1, 5, 0] == g["shadow_completed_cum"][-1]
    if tr == "T3":
        assert abs(sums[1, 0, 0] - g["shadow_latency_sum"]) < 1e-12
        assert cnt_[1, 4, 0] == len(g["shadow_dispatches"])
    # and the oracle agrees on everything
    trace = dict(times=times.cpu().numpy(), classes=cls.cpu().numpy(), counts=cnt.cpu().numpy())
    res = orc.rollout(w, 0, T, [0], actions=acts, trace=trace)
    assert np.array_equal(sim.checksums().cpu().numpy().view(np.uint64)[:, 0][: 2 if w["shadow"] else 1],
                          res["chk"][0, : 2 if w["shadow"] else 1])
    sim.close()


@pytest.mark.parametrize("name", NAMES + ["attn", "attn_K4"])
def test_init_weights_bit_identical(bs, orc, name):
    w = workload(name)
    sim = bs.Sim(w, n_envs=64)
    buf = sim.init_weights(1234)
    torch.cuda.synchronize()
    got = bs.unpack_weights(w, buf.cpu().numpy())
    ref = orc.init_weights(w, 1234)
    assert set(got) == set(ref)
    for k in ref:
        assert np.array_equal(got[k], ref[k]), k
    sim.close()


def mlp_weights(w, seed):
    """Random MLP weights with nonzero biases (the Xavier initialisation has zero biases, which
    would leave the kernels' bias paths untested); bf16-representable matrices in bf16
    configurations."""
    dims = [w["obs_dim"], w["mlp_h1"], w["mlp_h2"], 6 * w["n_servers"] + w["value_head"]]
    W = seeded_weights_f32(seed, dims, bf16=bool(w["mlp_bf16"]))
    return {k: v.astype(np.float64) for k, v in W.items()}


def policy_weights(orc, w, seed):
    return attn_weights(orc, w, seed) if w.get("policy_kind", 0) == 1 else mlp_weights(w, seed)


def policy_tol(w, wts, obs):
    return (attn_tol if w.get("policy_kind", 0) == 1 else end_to_end_bound)(w, wts, obs)


def check_mlp_layers(sim, wb, w, wts, obs_dev, obs_rows, step, rows, out=None):
    """The diagnostic instantiation of the policy kernel on the same inputs: its outputs equal
    the production kernel's bit for bit, and its hidden activations and outputs pass the
    layer-by-layer check against fp64 arithmetic on its own layer inputs (rows `rows`)."""
    hid = sim.policy_hidden(wb, obs_dev, step)
    if out is not None:
        for k in ("logits", "actions", "logp", "value"):
            if out[k] is not None:
                assert torch.equal(out[k], hid[k]), f"{k}: diagnostic and production kernels differ"
    h1 = hid["h1"].cpu().numpy().T.astype(np.float64)[rows]
    h2 = hid["h2"].cpu().numpy().T.astype(np.float64)[rows]
    lg = hid["logits"].cpu().numpy().T.astype(np.float64)[rows]
    return check_layers(w, wts, obs_rows, h1, h2, lg)


def attn_weights(orc, w, seed):
    """Random fp32 weights of the attention policy with nonzero biases (Xavier-initialised
    weights have zero biases, which would leave the bias terms untested)."""
    rng = np.random.default_rng(seed)
    out = {}
    for k, sh in orc.attn_shapes(w).items():
        sc = 0.6 if k.startswith("w") else 0.2
        out[k] = (rng.standard_normal(sh) * sc).astype(np.float32).astype(np.float64)
    return out


def check_policy(bs, orc, w, E, ids, step=17, seed=0x5EED):
    """Policy on E seeded observations through the C ABI, random weights with nonzero biases;
    the oracle evaluates rows `ids`.
    * MLP: the hidden activations and outputs pass the layer-by-layer check (each layer
      against fp64 arithmetic on the kernel's own inputs), and the logits lie within the
      bound that check's windows give end to end; attention: the forward error bound.
    * The sampler: the oracle's inverse CDF applied to the GPU's own logits with the same
      uniform gives the GPU's action and log-probability wherever the uniform is farther
      than 1e-5 from a CDF boundary (fp32 against fp64 sums).
    * The decisions against the oracle's own logits agree outside the band 2 max|dlogit|
      + 1e-5, dlogit being the logit differences already certified above (a perturbation e
      of the logits moves each CDF value by at most about 2e)."""
    attn = w.get("policy_kind", 0) == 1
    wts = policy_weights(orc, w, 99)
    obs = seeded_obs(21, E, w["obs_dim"])
    sim = bs.Sim(w, n_envs=E)
    sim.reset(seed)
    wb = sim.upload_weights(wts)
    obs_d = torch.from_numpy(np.ascontiguousarray(obs.T)).cuda()
    out = sim.policy(wb, obs_d, step, want_logits=True)
    torch.cuda.synchronize()
    lg = out["logits"].cpu().numpy().T.astype(np.float64)[ids]
    act = out["actions"].cpu().numpy()[ids]
    logp = out["logp"].cpu().numpy().astype(np.float64)[ids]
    ref = orc.policy(w, wts, seed, step, obs[ids], ids)
    if not attn:
        amb = check_mlp_layers(sim, wb, w, wts, obs_d, obs[ids], step, ids, out)
        say(f"  hidden units with two admissible values: {amb}")
    tol = policy_tol(w, wts, obs[ids])
    err = np.abs(lg - ref["logits"])
    assert np.all(err <= tol), f"max err/tol {np.max(err / tol):.3g}"
    if attn:
        check_attn_logits(err, tol)
    A = 6 * w["n_servers"]
    near = 0
    for i, e in enumerate(ids):
        a_ref, lp_ref, mg = orc.sample_logits(lg[i, :A], orc.action_u(seed, int(e), step))
        if mg > 1e-5:
            assert act[i] == a_ref, f"env {e}: sampler"
            assert abs(logp[i] - lp_ref) <= 1e-5 * (1.0 + abs(lp_ref)), f"env {e}: logp"
        else:
            near += 1
    eps = 2 * err[:, :A].max(axis=1) + 1e-5
    sure = ref["margin"] > eps
    assert np.array_equal(act[sure], ref["actions"][sure]), "actions differ away from ties"
    say(f"  sampler near-ties {near}, decision band excludes {np.sum(~sure)} of {len(ids)}; "
        f"max logit err {err.max():.3g} (max err/bound {np.max(err / tol):.3g})")
    if w["value_head"]:
        v = out["value"].cpu().numpy()[ids]
        assert np.array_equal(v, lg[:, A].astype(np.float32))
    sim.close()


@pytest.mark.parametrize("name", NAMES)
def test_policy_parity(bs, orc, name):
    """Every environment of a batch below the large-batch tiling threshold."""
    say(f"[policy] {name}")
    check_policy(bs, orc, preset(name), 1000, np.arange(1000))


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_policy_parity_large_batch(bs, orc, name):
    """A batch above the kernels' large-batch thresholds (64 * 512 environments for the bf16
    tiling, 4096 for the fp32 one), so that the wide-tile variants run, with a ragged last
    workgroup: the first and last environments and a seeded sample in between."""
    E = 64 * 512 + 77
    rng = np.random.default_rng(7)
    ids = np.unique(np.concatenate([np.arange(96), np.arange(E - 160, E),
                                    rng.integers(0, E, 256)])).astype(np.int64)
    say(f"[policy large] {name} E={E}")
    check_policy(bs, orc, preset(name), E, ids)


@pytest.mark.parametrize("name", sorted(ATTN))
def test_attention_policy_parity(bs, orc, name):
    """The attention policy kernel on 1000 seeded observations (several workgroups and a
    ragged last one) and, for the paper's shape, on 64 * 512 + 77 with sampled rows."""
    say(f"[attn policy] {name}")
    check_policy(bs, orc, workload(name), 1000, np.arange(1000))
    if name == "attn":
        E = 64 * 512 + 77
        rng = np.random.default_rng(8)
        ids = np.unique(np.concatenate([np.arange(64), np.arange(E - 100, E),
                                        rng.integers(0, E, 256)])).astype(np.int64)
        check_policy(bs, orc, workload(name), E, ids)


def test_attention_gradient_needs_value_head(bs):
    """The minibatch gradient uses the value head's output in its loss: without a value head
    the attention policy's gradient is refused with a clear error."""
    w = workload("attn", value_head=0)
    E, T = 64, 3
    sim = bs.Sim(w, n_envs=E)
    wb = sim.init_weights(1)
    dev = torch.device("cuda")
    obs = torch.zeros((T, w["obs_dim"], E), dtype=torch.float32, device=dev)
    act = torch.zeros((T, E), dtype=torch.uint8, device=dev)
    z = torch.zeros((T, E), dtype=torch.float64, device=dev)
    with pytest.raises(bs.SimError, match="value_head"):
        sim.reinforce_minibatch_grad(wb, obs, act, z, z, 64, 1)
    sim.close()


@pytest.mark.parametrize("name", ["C1", "C3", "C5"])
def test_gae_bit_exact(bs, orc, name):
    w = preset(name)
    T, E = 300, 777
    r, v = seeded_rewards_values(5, T, E, value=bool(w["value_head"]))
    sim = bs.Sim(w, n_envs=E)
    lam = w["lam"]
    rd = torch.from_numpy(r).cuda()
    vd = torch.from_numpy(v).cuda() if v is not None else None
    adv, ret = sim.returns_gae(rd, vd, w["gamma"], lam)
    torch.cuda.synchronize()
    ra, rr = orc.gae(r, v, w["gamma"], lam)
    assert np.array_equal(adv.cpu().numpy(), ra)
    assert np.array_equal(ret.cpu().numpy(), rr)
    sim.close()


@pytest.mark.parametrize("name", NAMES + ["attn", "attn_K4"])
def test_rollout_parity_and_validity(bs, orc, name):
    """sim_rollout (policy + sampler + simulator, T ticks) checked three ways:
    (1) the oracle's own policy rollout with the same weights agrees exactly, per env, on
        every tick before the first decision whose uniform lies within the tie band of a
        CDF boundary (the band is 2*max|dlogit| + 1e-5 over logit differences certified in
        (3));
    (2) validity of the simulator part: replaying the rollout's actions in the oracle gives
        the same running checksums, rewards and observations at every tick;
    (3) validity of every decision: on the rollout's observations the policy kernel gives the
        rollout's own action, its logits pass the layer-by-layer check (MLP) or the forward
        error bound (attention), and the oracle policy picks the same action wherever its
        uniform is outside the tie band.
    Random weights with nonzero biases."""
    w = workload(name)
    E, T, seed = 300, 100, 0xC0FFEE + 10 + (NAMES + ["attn", "attn_K4"]).index(name)
    A = 6 * w["n_servers"]
    attn = w.get("policy_kind", 0) == 1
    wts = policy_weights(orc, w, 7)
    say(f"[rollout] {name}")
    sim = bs.Sim(w, n_envs=E)
    sim.reset(seed)
    wb = sim.upload_weights(wts)
    tr = sim.rollout(wb, T, store_obs=True, rchk=True)
    sim.sync()
    ga = tr.actions.cpu().numpy()
    gr = tr.reward.cpu().numpy()
    gobs = tr.obs.cpu().numpy()                      # [T+1][F][E]
    go = np.transpose(gobs, (0, 2, 1))               # [T+1][E][F]
    grchk = tr.rchk.cpu().numpy().view(np.uint64)
    # (2) replay of the rollout's actions
    rep = orc.rollout(w, seed, T, np.arange(E), actions=ga, want_rchk=True)
    assert np.array_equal(rep["rchk"], grchk), "running checksums differ"
    assert_close_rel(gr, rep["reward"], "reward")
    assert np.array_equal(rep["obs"], go), "observations differ"
    # the current observation after the rollout (its last tick writes it in fp32; the ticks
    # before it may write only the bf16 pairs a bf16 policy reads)
    assert np.array_equal(sim.obs().cpu().numpy(), gobs[T]), "current observation after the rollout"
    # (3) every decision against the oracle policy on the same observation
    lg_err = 0.0
    ties = 0
    band_te = np.zeros((T, E))
    for t in range(T):
        ob_t = tr.obs[t].contiguous()
        out = sim.policy(wb, ob_t, t, want_logits=True)
        assert np.array_equal(out["actions"].cpu().numpy(), ga[t]), f"tick {t}: not the rollout's action"
        glg = out["logits"].cpu().numpy().T.astype(np.float64)
        if not attn and t % 10 == 0:
            check_mlp_layers(sim, wb, w, wts, ob_t, go[t], t, np.arange(E), out)
        ref = orc.policy(w, wts, seed, t, go[t], np.arange(E))
        full_err = np.abs(glg - ref["logits"])
        tol_t = policy_tol(w, wts, go[t])
        assert np.all(full_err <= tol_t), f"tick {t}: logits"
        if attn:
            check_attn_logits(full_err, tol_t)
        err = full_err[:, :A].max(axis=1)
        lg_err = max(lg_err, float(err.max()))
        band_te[t] = 2 * err + 1e-5
        sure = ref["margin"] > band_te[t]
        ties += int(np.sum(~sure))
        assert np.array_equal(ga[t][sure], ref["actions"][sure]), f"tick {t}: decision differs"
    # (1) independent rollout of the oracle, compared before the first near-tie; on that
    # common prefix both sides saw the same observations, so the band measured in (3)
    # for (t, env) applies
    res = orc.rollout(w, seed, T, np.arange(E), weights=wts)
    tie = res["margin"] <= band_te
    first = np.where(tie.any(axis=0), tie.argmax(axis=0), T)
    checked = 0
    for e in range(E):
        f = first[e]
        assert np.array_equal(ga[:f, e], res["actions"][:f, e]), f"env {e} actions before tick {f}"
        assert_close_rel(gr[:f, e], res["reward"][:f, e], f"env {e} reward")
        assert np.array_equal(go[: f + 1, e], res["obs"][: f + 1, e]), f"env {e} obs"
        checked += f
    say(f"  max|dlogit| {lg_err:.3g}, decisions in tie band {ties}/{E * T}, "
        f"independent prefix covers {checked}/{E * T} env-ticks")
    assert checked > 0
    sim.close()


@pytest.mark.parametrize("name,kw", [("C3", dict(obs_dim=31)), ("C5", {}), ("C1", {})])
def test_rollout_observation_handoff(bs, orc, name, kw):
    """Inside a rollout with a bf16 policy the ticks write the observation as the bf16 feature
    pairs the policy reads, the pairs are packed from the fp32 observation when a rollout
    starts, and the rollout's last tick writes the fp32 observation again. After a reset (which
    writes only the fp32 observation): a rollout of one tick, a sim_step (fp32 only again), a
    rollout of three ticks, a sim_step. The oracle's replay of the six ticks' actions gives the
    same running checksums and, after each call, the same current observation; and the policy
    kernel on the oracle's observation of every rollout tick (the fp32 input path) gives the
    rollout's own action, which a stale or unpacked pair buffer would not. C3 with an odd
    observation width (31: the last pair holds one feature and a zero) and C1's fp32 policy,
    which keeps the fp32 observation throughout, take the same checks."""
    w = workload(name, **kw)
    E, seed = 300, 0x0B5E + len(name) + w["obs_dim"]
    A = 6 * w["n_servers"]
    wts = policy_weights(orc, w, 9)
    say(f"[observation handoff] {name} F={w['obs_dim']}")
    sim = bs.Sim(w, n_envs=E)
    sim.reset(seed)
    wb = sim.upload_weights(wts)
    steps = seeded_actions(seed, 2, E, A, small_bias=0.5)
    acts, cur, rollout_ticks, rchk = [], [], [], {}
    tick = 0
    for part, T in enumerate((1, 3)):
        tr = sim.rollout(wb, T, rchk=True)
        sim.sync()
        acts.append(tr.actions.cpu().numpy())
        for t in range(T):
            rchk[tick + t] = tr.rchk.cpu().numpy().view(np.uint64)[t]
            rollout_ticks.append(tick + t)
        tick += T
        cur.append((tick, sim.obs().cpu().numpy()))
        sim.step(torch.from_numpy(steps[part]).cuda(), want_obs=False)
        sim.sync()
        acts.append(steps[part:part + 1])
        tick += 1
        cur.append((tick, sim.obs().cpu().numpy()))
    ga = np.concatenate(acts)
    rep = orc.rollout(w, seed, tick, np.arange(E), actions=ga, want_rchk=True)
    for t, c in rchk.items():
        assert np.array_equal(rep["rchk"][t], c), f"tick {t}: running checksums differ"
    for t, o in cur:
        assert np.array_equal(rep["obs"][t], o.T), f"current observation after tick {t}"
    for t in rollout_ticks:
        ob_t = torch.from_numpy(np.ascontiguousarray(rep["obs"][t].T)).cuda()
        out = sim.policy(wb, ob_t, t)
        assert np.array_equal(out["actions"].cpu().numpy(), ga[t]), f"tick {t}: not the rollout's action"
    sim.close()


SHADOWED = {
    "C5": lambda: preset("C5"),
    "burst": lambda: burst_preset(),
    "static8_C3": lambda: baseline_preset("static8", "C3"),
    "random_C5": lambda: baseline_preset("random", "C5"),
    "round_robin_C4": lambda: baseline_preset("round_robin", "C4"),
    "shortest_C3": lambda: baseline_preset("shortest", "C3"),
}


@pytest.mark.parametrize("name,E,T", [(n, 300, 600) for n in sorted(SHADOWED)] +
                         [("burst", 6, 4100)])
def test_rollout_static_chunks_then_steps(bs, orc, name, E, T):
    """sim_rollout runs the static shadow system in launches of up to 4096 ticks with its
    state in registers; 600 ticks in one launch followed by 20 sim_step calls (the per-tick
    kernel, which resumes from the state the long launch stored) must equal the oracle's replay
    of the same ticks, bit for bit in the integer state and checksums. A longer rollout over a
    few environments (4100 ticks: launches of 4096 and 4) crosses a boundary inside the
    rollout as well."""
    w = SHADOWED[name]()
    T2 = 20
    seed = 0x5EED5 + len(name)
    say(f"[static chunks] {name} E={E} T={T}")
    sim = bs.Sim(w, n_envs=E)
    sim.reset(seed)
    wb = sim.init_weights(3)
    tr = sim.rollout(wb, T)
    acts2 = seeded_actions(seed, T2, E, 6 * w["n_servers"], small_bias=0.5)
    a2 = torch.from_numpy(np.ascontiguousarray(acts2)).cuda()
    rsh2 = []
    for k in range(T2):
        _, _, rs = sim.step(a2[k], want_obs=False)
        rsh2.append(rs)
    sim.sync()
    acts = np.concatenate([tr.actions.cpu().numpy(), acts2], axis=0)
    rsh = np.concatenate([tr.reward_shadow.cpu().numpy(), torch.stack(rsh2).cpu().numpy()])
    cnt, sums = sim.counters()
    chk = sim.checksums().cpu().numpy().view(np.uint64)
    ref = orc.rollout(w, seed, T + T2, np.arange(E), actions=acts, want_obs=False, want_rec=False)
    assert_close_rel(rsh, ref["reward_shadow"], "reward_shadow")
    for s_ in (0, 1):
        assert np.array_equal(chk[s_], ref["chk"][:, s_]), f"checksum sys {s_}"
        assert np.array_equal(cnt.cpu().numpy()[s_].T, ref["counters"][:, s_]), f"counters sys {s_}"
        assert_close_rel(sums.cpu().numpy()[s_].T, ref["sums"][:, s_, :2], f"sums sys {s_}")
    assert ref["counters"][:, 1, 4].sum() > 0
    sim.close()


FULL_ROLLOUT = {"C5": lambda: preset("C5"), "attn": lambda: attn_preset(n_envs=262144)}


@pytest.mark.parametrize("name", sorted(FULL_ROLLOUT))
def test_rollout_full_size_sampled(bs, orc, name):
    """sim_rollout at the full environment count in the launch configuration the bench times
    (large-batch policy kernel, learned tick, static shadow system in one launch of up to 4096
    ticks), 300 ticks. For sampled environments the
    oracle replays the rollout's actions: running checksums, rewards (both systems), final
    checksums and counters agree exactly; and every sampled decision equals the oracle
    policy's on the replayed observation outside the tie band (logits from the same GPU
    policy kernel on those observations)."""
    w = FULL_ROLLOUT[name]()
    E, T = w["n_envs"], 300
    seed = 0xF011 + len(name)
    rng = np.random.default_rng(seed)
    cols = np.unique(np.concatenate([[0, 1, 63, 64, E - 1], rng.choice(E, 28, replace=False)]))
    say(f"[rollout-full] {name} E={E} T={T} sampled={len(cols)}")
    sim = bs.Sim(w)
    sim.reset(seed)
    wb = sim.upload_weights(policy_weights(orc, w, seed + 1))
    tr = sim.rollout(wb, T, rchk=True)
    sim.sync()
    c = torch.from_numpy(cols).cuda()
    ga = tr.actions[:, c].cpu().numpy()
    gr = tr.reward[:, c].cpu().numpy()
    grs = tr.reward_shadow[:, c].cpu().numpy() if w["shadow"] else None
    grchk = tr.rchk[:, c].cpu().numpy().view(np.uint64)
    cnt, sums = sim.counters()
    chk = sim.checksums().cpu().numpy().view(np.uint64)[:, cols]
    cnt = cnt.cpu().numpy()[:, :, cols]
    wts = bs.unpack_weights(w, wb.cpu().numpy())
    sim.close()
    del tr
    rep = orc.rollout(w, seed, T, cols, actions=ga, want_rchk=True, want_rec=False)
    assert np.array_equal(rep["rchk"], grchk), "running checksums differ"
    assert_close_rel(gr, rep["reward"], "reward")
    nsys = 2 if w["shadow"] else 1
    if nsys == 2:
        assert_close_rel(grs, rep["reward_shadow"], "reward_shadow")
    for s_ in range(nsys):
        assert np.array_equal(chk[s_], rep["chk"][:, s_]), f"checksum sys {s_}"
        assert np.array_equal(cnt[s_].T, rep["counters"][:, s_]), f"counters sys {s_}"
    # decisions: GPU logits of the replayed observations from the same policy kernel (a
    # context of 64 * 512 environments selects the large-batch variant; the sampled rows are
    # its first columns, and logits do not depend on the environment index) against the
    # oracle policy with the true env ids
    A = 6 * w["n_servers"]
    n = len(cols)
    Ec = 64 * 512
    small = bs.Sim(w, n_envs=Ec)
    small.reset(1)
    wsm = small.upload_weights(wts)
    ob = torch.zeros((w["obs_dim"], Ec), dtype=torch.float32, device="cuda")
    ties = near = 0
    for t in range(T):
        ob[:, :n] = torch.from_numpy(np.ascontiguousarray(rep["obs"][t].T)).cuda()
        out = small.policy(wsm, ob, t, want_logits=True)
        glg = out["logits"][:, :n].cpu().numpy().T.astype(np.float64)
        if w.get("policy_kind", 0) == 0 and t % 25 == 0:
            check_mlp_layers(small, wsm, w, wts, ob, rep["obs"][t], t, np.arange(n), out)
        ref = orc.policy(w, wts, seed, t, rep["obs"][t], cols)
        tol = policy_tol(w, wts, rep["obs"][t])
        assert np.all(np.abs(glg - ref["logits"]) <= tol), f"tick {t}: logits"
        if w.get("policy_kind", 0) == 1:
            check_attn_logits(np.abs(glg - ref["logits"]), tol)
        err = np.abs(glg - ref["logits"])[:, :A].max(axis=1)
        sure = ref["margin"] > 2 * err + 1e-5
        ties += int(np.sum(~sure))
        assert np.array_equal(ga[t][sure], ref["actions"][sure]), f"tick {t}: decision differs"
        # the sampler alone: the oracle's inverse CDF on the GPU's own logits with the same
        # uniform; only fp32-versus-fp64 rounding of the sums separates the two
        for i, e in enumerate(cols):
            a_ref, _, mg = orc.sample_logits(glg[i, :A], orc.action_u(seed, int(e), t))
            if mg > 1e-5:
                assert ga[t][i] == a_ref, f"tick {t} env {e}: sampler"
            else:
                near += 1
    small.close()
    say(f"  decisions in the tie band {ties}/{n * T}; sampler-only near-ties {near}")


def test_action_out_of_range_is_latched(bs):
    w = preset("C1")
    sim = bs.Sim(w, n_envs=70)
    sim.reset(1)
    a = torch.zeros(70, dtype=torch.uint8, device="cuda")
    a[69] = 6
    sim.step(a)
    with pytest.raises(bs.SimError, match="action out of range"):
        sim.sync()
    sim.sync()  # the flag was cleared
    sim.close()
