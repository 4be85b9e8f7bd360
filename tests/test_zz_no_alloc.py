"""ppo_minibatch_grad_noalloc -- the minibatch gradient (paper Sec. 4.3) on the library's fixed
device scratch, for callers that cannot allocate -- against ppo_minibatch_grad on the same
inputs through the C ABI: two calls in a row, the second with a smaller input (fewer ticks and
samples), each equal bit for bit to the allocating call (same kernels, sums in a fixed order);
and a minibatch too large for the fixed scratch is refused with a clear error."""
import numpy as np
import pytest

from workloads import preset

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def bs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_05272_amd as m
    m.load()
    return m


def inputs(w, T, E, seed):
    rng = np.random.default_rng(seed)
    F, A = w["obs_dim"], 6 * w["n_servers"]
    obs = rng.random((T, F, E), dtype=np.float32)
    act = rng.integers(0, A, size=(T, E)).astype(np.uint8)
    logp = (np.log(1.0 / A) + rng.uniform(-0.3, 0.3, size=(T, E))).astype(np.float32)
    adv = rng.standard_normal((T, E))
    ret = rng.standard_normal((T, E))
    return [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in (obs, act, logp, adv, ret)]


def test_noalloc_minibatch_matches_allocating_call(bs):
    w = preset("C4", n_envs=512)
    sim = bs.Sim(w)
    sim.reset(1)
    wb = sim.init_weights(3)
    for T, M, seed in ((6, 4096, 11), (3, 512, 12)):
        print(f"[no-alloc] C4 E=512 T={T} M={M}", flush=True)
        obs, act, logp, adv, ret = inputs(w, T, w["n_envs"], seed)
        ref = sim.ppo_minibatch_grad(wb, obs, act, logp, adv, ret, M, seed, want_index=True)
        got = sim.ppo_minibatch_grad(wb, obs, act, logp, adv, ret, M, seed, want_index=True,
                                     noalloc=True)
        sim.sync()
        for a, b, what in zip(got, ref, ("gradients", "loss", "indices")):
            assert torch.equal(a, b), f"T={T} M={M}: {what} differ"
    # more scratch than the fixed buffer holds: refused before any device work
    obs, act, logp, adv, ret = inputs(w, 2, w["n_envs"], 13)
    with pytest.raises(bs.SimError, match="fixed scratch"):
        sim.ppo_minibatch_grad(wb, obs, act, logp, adv, ret, 16384, 13, noalloc=True)
    sim.sync()
    sim.close()
