"""Checkpoint and resume through the C ABI (sim_get_state / sim_set_state): a run continued
from a restored snapshot reproduces the original continuation bit for bit, in the same
context and in a fresh one, from device and from host memory; mismatched layouts and
truncated or foreign buffers are refused."""
import sys

import numpy as np
import pytest

from workloads import preset, baseline_preset

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


def continuation(sim, wb, T):
    tr = sim.rollout(wb, T, rchk=True)
    sim.sync()
    cnt, sums = sim.counters()
    out = dict(actions=tr.actions.cpu().numpy(), reward=tr.reward.cpu().numpy(),
               rchk=tr.rchk.cpu().numpy(), chk=sim.checksums().cpu().numpy(),
               cnt=cnt.cpu().numpy(), sums=sums.cpu().numpy(), tick=sim.tick())
    if tr.reward_shadow is not None:
        out["reward_shadow"] = tr.reward_shadow.cpu().numpy()
    return out


def same(a, b):
    assert a.keys() == b.keys()
    for k in a:
        assert np.array_equal(np.asarray(a[k]), np.asarray(b[k])), k


@pytest.mark.parametrize("name", ["C4", "C5"])
def test_resume_reproduces_the_continuation(bs, name):
    w = preset(name) if name != "C5" else baseline_preset("random", "C5")
    E = 3000
    say(f"[state] {name}")
    sim = bs.Sim(w, n_envs=E)
    sim.reset(77)
    wb = sim.init_weights(5)
    sim.rollout(wb, 40)
    snap_dev = sim.get_state(device=True)
    snap_host = sim.get_state(device=False)
    assert torch.equal(snap_dev.cpu(), snap_host)
    first = continuation(sim, wb, 300)          # one static launch of 300 ticks
    sim.set_state(snap_dev)
    same(first, continuation(sim, wb, 300))
    sim.set_state(snap_host)
    same(first, continuation(sim, wb, 300))
    fresh = bs.Sim(w, n_envs=E)                 # never reset: the snapshot carries everything
    fresh.set_state(snap_host)
    same(first, continuation(fresh, fresh.upload_weights(bs.unpack_weights(w, wb.cpu().numpy())), 300))
    fresh.close()
    sim.close()


def test_state_errors(bs):
    w = preset("C3")
    a = bs.Sim(w, n_envs=500)
    a.reset(1)
    snap = a.get_state()
    b = bs.Sim(w, n_envs=501)
    with pytest.raises(bs.SimError, match="layout"):
        b.set_state(snap)
    with pytest.raises(bs.SimError, match="truncated"):
        a.set_state(snap[:-8].clone())
    junk = torch.zeros_like(snap)
    with pytest.raises(bs.SimError, match="not a snapshot"):
        a.set_state(junk)
    with pytest.raises(bs.SimError, match="not a snapshot"):
        a.set_state(snap[:100].clone())
    # a too-small destination is refused before anything is written
    import ctypes as C
    from paper_2607_05272_amd import _lib as L
    n = C.c_size_t(10)
    small = torch.zeros(10, dtype=torch.uint8, device="cuda")
    assert a.lib.sim_get_state(a._ctx, C.c_void_p(small.data_ptr()), C.byref(n)) == -1
    assert "needs" in L.load().sim_last_error().decode()
    a.close()
    b.close()
