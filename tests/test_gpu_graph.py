"""Rollout graphs (sim_rollout replayed from a captured HIP graph) against eager launches
through the C ABI: a context with graphs off gives the reference trajectories for two seeds;
a context with graphs on rolls out the same episodes (eagerly the first time, captured the
second, replayed afterwards, with other device work and host synchronisations between the
replays, and with a new seed that only device memory carries) and must match every output
bit for bit each time."""
import numpy as np
import pytest

from workloads import preset

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CASES = {"C1": dict(n_envs=256, T=120), "C3": dict(n_envs=300, T=100),
         "C5": dict(n_envs=300, T=300)}


@pytest.fixture(scope="module")
def bs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_05272_amd as m
    m.load()
    return m


def outputs(tr):
    out = {}
    for k in ("actions", "logp", "reward", "reward_shadow", "value", "obs", "rchk"):
        v = getattr(tr, k, None)
        if v is not None:
            out[k] = v.clone()
    return out


@pytest.mark.parametrize("name", sorted(CASES))
def test_rollout_graph_replays_match_eager(bs, name):
    w = preset(name, **CASES[name])
    T = w["T"]
    print(f"[graph] {name} E={w['n_envs']} T={T}", flush=True)
    ref = bs.Sim(w)
    ref.set_graphs(False)
    wb = ref.init_weights(5)
    seeds = (0x6A1, 0x6A2)
    trr = None
    expect = {}
    for sd in seeds:
        ref.reset(sd)
        trr = ref.rollout(wb, T, store_obs=True, rchk=True, traj=trr)
        ref.sync()
        expect[sd] = outputs(trr)
    assert ref.graph_stats() == (0, 0)
    ref.close()

    sim = bs.Sim(w)
    wg = sim.upload_weights(bs.unpack_weights(w, wb.cpu().numpy()))
    tr = None
    order = (seeds[0], seeds[0], seeds[1], seeds[0], seeds[1])
    for i, sd in enumerate(order):
        sim.reset(sd)
        tr = sim.rollout(wg, T, store_obs=True, rchk=True, traj=tr)
        # eager device work and a host synchronisation between the replays
        junk = sim.policy(wg, tr.obs[T // 2].contiguous(), 7)
        torch.cuda.synchronize()
        del junk
        sim.sync()
        got = outputs(tr)
        for k, v in expect[sd].items():
            assert torch.equal(got[k], v), f"rollout {i} (seed {sd:#x}): {k} differs from eager"
    captures, replays = sim.graph_stats()
    assert captures == 1 and replays == len(order) - 1, (captures, replays)
    sim.close()
