"""GPU: the fused small-batch rollout (one launch for all ticks, each workgroup alternating the
policy and the learned tick of its own environments) against the per-tick launches, through
the C ABI. Both run the same device code, so every trajectory output, the current
observation, the environments' state, the counters and the checksums must be bit-identical.
The oracle parity of the rollout itself (test_gpu_parity.py) covers the fused kernel too: at
those batch sizes sim_rollout fuses by default."""
import sys

import numpy as np
import pytest

from workloads import preset
from workloads.gen import seeded_weights_f32

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def bs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_05272_amd as m
    m.load()
    return m


def weights(w, seed):
    """Random MLP weights with nonzero biases, bf16-representable in bf16 configurations."""
    dims = [w["obs_dim"], w["mlp_h1"], w["mlp_h2"], 6 * w["n_servers"] + w["value_head"]]
    W = seeded_weights_f32(seed, dims, bf16=bool(w["mlp_bf16"]))
    return {k: v.astype(np.float64) for k, v in W.items()}


def snapshot(sim, tr):
    sim.sync()
    out = {k: getattr(tr, k).cpu().numpy() for k in
           ("actions", "logp", "reward", "reward_shadow", "value", "obs", "rchk")
           if getattr(tr, k) is not None}
    out["cur_obs"] = sim.obs().cpu().numpy()
    out["state"] = sim.get_state(device=False).numpy()
    cnt, sums = sim.counters()
    out["cnt"], out["sums"] = cnt.cpu().numpy(), sums.cpu().numpy()
    out["chk"] = sim.checksums().cpu().numpy()
    return out


def assert_same(a, b, what):
    assert a.keys() == b.keys()
    for k in a:
        x, y = a[k], b[k]
        assert x.shape == y.shape, f"{what}: {k} shapes {x.shape} vs {y.shape}"
        if not np.array_equal(x.view(np.uint8), y.view(np.uint8)):
            bad = np.argwhere(x.view(np.uint8) != y.view(np.uint8))
            raise AssertionError(f"{what}: {k} differs at {len(bad)} bytes, first {bad[0]}")


# name, workload overrides, environments, ticks per rollout
CASES = [
    ("C1", {}, 256, 40),                       # one 16-environment tile per workgroup, 16 tiles
    ("C1", {}, 250, 7),                        # ragged last tile
    ("C1", dict(shadow=1), 300, 12),           # static shadow system on its own stream beside
    ("C2", {}, 4096, 24),
    ("C2", dict(value_head=1), 333, 5),        # value rows, including row T
    ("C2", dict(obs_dim=13), 517, 6),          # odd observation width: a half-filled last pair
    ("C2", dict(queue_cap=3), 200, 9),         # drops every tick
    ("C3", {}, 1000, 6),                       # 64-environment tiles, 16 lanes per wave, ragged
    ("C3", dict(n_servers=3), 300, 5),         # 18 actions: the sampler's run-time bound
    ("C3", dict(obs_dim=31), 200, 4),
    ("C4", {}, 700, 4),                        # 8 servers, 4 classes, lognormal service
]


@pytest.mark.parametrize("name,kw,E,T", CASES)
def test_fused_rollout_matches_per_tick(bs, name, kw, E, T):
    """Two rollouts in a row (the second from tick T) on two contexts from the same reset, one
    fused and one per tick, then a sim_step on both: identical outputs after each call."""
    w = preset(name, **kw)
    seed = 0xF05E + E + T
    say(f"[fused vs per-tick] {name} {kw} E={E} T={T}")
    sims = []
    for mode in (bs.FUSE_OFF, bs.FUSE_ON):
        sim = bs.Sim(w, n_envs=E)
        sim.set_fused_rollout(mode)
        sim.set_graphs(False)
        sim.reset(seed)
        sims.append(sim)
    wts = weights(w, 21)
    res = []
    for sim in sims:
        wb = sim.upload_weights(wts)
        snaps = []
        for _ in range(2):
            tr = sim.rollout(wb, T, store_obs=True, rchk=True)
            snaps.append(snapshot(sim, tr))
        acts = torch.from_numpy(snaps[-1]["actions"][-1]).cuda()
        sim.step(acts, want_obs=False)
        sim.sync()
        snaps.append({"cur_obs": sim.obs().cpu().numpy(),
                      "state": sim.get_state(device=False).numpy()})
        res.append(snaps)
    for i, (a, b) in enumerate(zip(*res)):
        assert_same(a, b, f"call {i}")
    for sim in sims:
        sim.close()


def test_fused_rollout_beyond_one_round(bs):
    """More workgroups than the chip holds at once (they run in rounds; none waits for
    another): C2's network over 40000 environments, fused on request, against per tick."""
    w = preset("C2")
    E, T, seed = 40000, 4, 0xB16
    say(f"[fused, many rounds] C2 E={E} T={T}")
    out = []
    for mode in (bs.FUSE_OFF, bs.FUSE_ON):
        sim = bs.Sim(w, n_envs=E)
        sim.set_fused_rollout(mode)
        sim.reset(seed)
        wb = sim.upload_weights(weights(w, 5))
        tr = sim.rollout(wb, T, store_obs=True, rchk=True)
        out.append(snapshot(sim, tr))
        sim.close()
    assert_same(out[0], out[1], "C2 40000 envs")


def test_fused_rollout_graph_and_tracing(bs):
    """The fused launch under the rollout graph (captured and replayed on the second identical
    call, replayed again on the third) and under tracing (one launch of class 'rollout' per rollout, none
    of the per-tick classes), each against the per-tick rollout from the same reset."""
    w = preset("C1")
    E, T, seed = 256, 30, 0x6A
    say(f"[fused graph + tracing] C1 E={E} T={T}")
    ref = bs.Sim(w, n_envs=E)
    ref.set_fused_rollout(bs.FUSE_OFF)
    ref.set_graphs(False)
    ref.reset(seed)
    wb_r = ref.upload_weights(weights(w, 3))
    want = snapshot(ref, ref.rollout(wb_r, T, store_obs=True, rchk=True))
    ref.close()

    sim = bs.Sim(w, n_envs=E)
    wb = sim.upload_weights(weights(w, 3))
    tr = None
    for i in range(3):
        sim.reset(seed)
        tr = sim.rollout(wb, T, store_obs=True, rchk=True, traj=tr)
        assert_same(snapshot(sim, tr), want, f"graph call {i}")
    assert sim.graph_stats() == (1, 2)
    sim.set_timing(True)
    sim.reset(seed)
    tr = sim.rollout(wb, T, store_obs=True, rchk=True, traj=tr)
    got = snapshot(sim, tr)
    timing = sim.get_timing(clear=True)
    sim.set_timing(False)
    assert_same(got, want, "traced")
    assert timing["rollout"][1] == 1, timing
    assert timing["policy"][1] == 0 and timing["step"][1] == 0, timing
    sim.close()


def test_fused_rollout_modes(bs):
    """sim_set_fused_rollout takes the three modes and rejects others. Automatic fusing takes a
    batch whose workgroups are all resident at once (C3's 16384 environments: one 64-environment
    workgroup per CU) and leaves a larger one (C4's 65536) to the per-tick launches; a network
    without a fused kernel (C5's) keeps the per-tick launches even when fusing is forced."""
    sim = bs.Sim(preset("C1"), n_envs=64)
    for mode in (bs.FUSE_OFF, bs.FUSE_AUTO, bs.FUSE_ON):
        sim.set_fused_rollout(mode)
    for bad in (-1, 3):
        with pytest.raises(bs.SimError):
            sim.set_fused_rollout(bad)
    sim.close()
    for name, E, mode, fused in (("C3", 16384, bs.FUSE_AUTO, True),
                                 ("C4", 65536, bs.FUSE_AUTO, False),
                                 ("C5", 64, bs.FUSE_ON, False)):
        say(f"[fused mode] {name} E={E} mode={mode}")
        w = preset(name)
        sim = bs.Sim(w, n_envs=E)
        sim.set_fused_rollout(mode)
        sim.set_timing(True)
        sim.reset(1)
        wb = sim.upload_weights(weights(w, 2))
        sim.rollout(wb, 3)
        timing = sim.get_timing(clear=True)
        want = (1, 0) if fused else (0, 3)
        assert (timing["rollout"][1], timing["step"][1]) == want, (name, timing)
        sim.close()


def test_fused_rollout_trace_arrivals(bs):
    """Trace arrivals (several per instant, classes in random order, some environments running
    out of arrivals mid-rollout) with a Static-8 shadow system beside: fused against per tick,
    C3's network over 4 servers and 4 classes."""
    from workloads import trace_preset
    from workloads.presets import SVC_DET
    E, T, L, C = 200, 40, 120, 4
    w = trace_preset(n_servers=4, n_classes=C, queue_cap=20, obs_dim=32, shadow=1,
                     mlp_h1=256, mlp_h2=256, mlp_bf16=1, value_head=1,
                     static_bmax=4, static_timeout=2e-3, class_mix=[0.25] * C,
                     service_kind=[SVC_DET] * C, svc_alpha=[0.3e-3, 1e-3, 2e-3, 4e-3],
                     svc_beta=[0.1e-3, 0.2e-3, 0.5e-3, 1e-3], svc_median=[0.0] * C,
                     w_class=[200.0, 100.0, 40.0, 20.0])
    w["trace_max_len"] = L
    rng = np.random.default_rng(0x7ACE)
    times = np.cumsum(0.25e-3 * rng.integers(0, 3, size=(E, L)), axis=1) + 0.25e-3
    cls = rng.integers(0, C, size=(E, L)).astype(np.uint8)
    counts = np.full(E, L, np.int32)
    counts[::5] = L // 3
    dev = torch.device("cuda")
    say(f"[fused, trace arrivals] E={E} T={T} L={L}")
    out = []
    for mode in (bs.FUSE_OFF, bs.FUSE_ON):
        sim = bs.Sim(w, n_envs=E)
        sim.set_fused_rollout(mode)
        sim.set_trace(torch.from_numpy(times).to(dev), torch.from_numpy(cls).to(dev),
                      torch.from_numpy(counts).to(dev))
        sim.reset(3)
        wb = sim.upload_weights(weights(w, 8))
        tr = sim.rollout(wb, T, store_obs=True, rchk=True)
        out.append(snapshot(sim, tr))
        sim.close()
    assert_same(out[0], out[1], "trace arrivals")
