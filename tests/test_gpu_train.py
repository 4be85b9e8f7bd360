"""GPU parity of the policy update (Sec. 4.3) through the C ABI against oracle/train.py:
the REINFORCE-with-baseline minibatch gradient, Adam steps with the re-export of the policy's
weights, the weight import, and the full epoch x minibatch update loop of both algorithms.

Tolerances: gradients as for PPO (tests/test_gpu_ppo.py: 2^-9 of the norm and 2^-8 of the
largest entry in bf16 mode, 2^-13 in fp32 mode). Adam on the GPU runs in fp32 against the
oracle's fp64: one step moves a parameter by lr * m_hat / (sqrt(v_hat) + eps), computed to
a few fp32 ulps, so after s steps the parameters agree within s * lr * 2^-18 plus 2^-22 of
their magnitude; the exported weights are the GPU parameters rounded to the element type,
exactly. Through the update loop
the minibatch gradients carry their own tolerance into Adam; with eps = 1e-2 (so that a
step depends smoothly on its gradient) each step's difference stays below lr * 2^-6."""
import sys

import numpy as np
import pytest

from oracle import ppo as orc_ppo
from oracle import train as orc_train
from workloads import preset
from workloads.gen import ppo_inputs_at, seeded_obs, seeded_weights_f32

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

KEYS = orc_train.PARAM_KEYS


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def bs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_05272_amd as m
    m.load()
    return m


def workload(name):
    w = preset(name)
    w["value_head"] = 1
    return w


def weights_for(w, seed):
    Ap = 6 * w["n_servers"] + 1
    return seeded_weights_f32(seed, [w["obs_dim"], w["mlp_h1"], w["mlp_h2"], Ap],
                              bf16=bool(w["mlp_bf16"]))


def flat(d):
    return np.concatenate([np.asarray(d[k], np.float64).ravel() for k in KEYS])


def trajectory(w, T, E, seed=11):
    F = w["obs_dim"]
    A = 6 * w["n_servers"]
    x = seeded_obs(seed, T * E, F)
    obs_t = np.ascontiguousarray(x.reshape(T, E, F).transpose(0, 2, 1))
    tt, ee = np.meshgrid(np.arange(T), np.arange(E), indexing="ij")
    act, adv, ret = ppo_inputs_at(7, tt.astype(np.int64), ee.astype(np.int64), A)
    return obs_t, act.astype(np.uint8), adv, ret


def grad_close(w, got, ref, what):
    bf = bool(w["mlp_bf16"])
    tn, te = (2.0 ** -9, 2.0 ** -8) if bf else (2.0 ** -13, 2.0 ** -13)
    for k in KEYS:
        G, g = ref[k], got[k].astype(np.float64)
        d, nG = np.linalg.norm(g - G), np.linalg.norm(G)
        say(f"  {what} {k}: |dG|/|G| {d / max(nG, 1e-300):.3g}")
        assert d <= tn * nG + 1e-30, k
        assert np.max(np.abs(g - G)) <= te * np.max(np.abs(G)) + 1e-30, k


@pytest.mark.parametrize("name,T,E,M", [("C1", 7, 300, 1024), ("C4", 9, 500, 2048)])
def test_reinforce_minibatch_parity(bs, name, T, E, M):
    w = workload(name)
    say(f"[reinforce] {name} T={T} E={E} M={M}")
    obs_t, act, adv, ret = trajectory(w, T, E)
    wts = weights_for(w, 5)
    W64 = {k: v.astype(np.float64) for k, v in wts.items()}
    seed = 0xBEEF + T
    ref_loss, ref_g = orc_train.minibatch_grad(w, W64, seed, obs_t, act, None, adv, ret, M,
                                               orc_train.ALGO_REINFORCE)
    dev = torch.device("cuda")
    sim = bs.Sim(w, n_envs=E)
    g, loss, idx = sim.reinforce_minibatch_grad(
        sim.upload_weights(wts), torch.from_numpy(obs_t).to(dev), torch.from_numpy(act).to(dev),
        torch.from_numpy(adv).to(dev), torch.from_numpy(ret).to(dev), M, seed, want_index=True)
    sim.sync()
    ti, ei = orc_ppo.sample_indices(seed, M, T, E)
    assert np.array_equal(idx.cpu().numpy(), ti * E + ei)
    grad_close(w, sim.unflatten_grads(g.cpu().numpy()), ref_g, name)
    got = loss.cpu().numpy()
    scale = abs(ref_loss["policy"]) + abs(ref_loss["value"]) + abs(ref_loss["entropy"])
    for i, k in enumerate(("loss", "policy", "value", "entropy")):
        assert abs(got[i] - ref_loss[k]) <= 2.0 ** -9 * scale, k
    sim.close()


@pytest.mark.parametrize("name", ["C1", "C4"])
def test_params_import_and_adam_steps(bs, name):
    w = workload(name)
    sim = bs.Sim(w, n_envs=64)
    wts = weights_for(w, 21)
    wb = sim.upload_weights(wts)
    p = sim.params_from_weights(wb)
    sim.sync()
    assert np.array_equal(p.cpu().numpy().astype(np.float64), flat(wts))  # exact import
    n = p.numel()
    rng = np.random.default_rng(3)
    grads = [rng.standard_normal(n).astype(np.float32) * np.float32(0.05) for _ in range(4)]
    master = flat(wts)
    m = np.zeros(n)
    v = np.zeros(n)
    md = torch.zeros(n, dtype=torch.float32, device="cuda")
    vd = torch.zeros(n, dtype=torch.float32, device="cuda")
    lr = 2e-3
    for t, g in enumerate(grads, start=1):
        orc_train.adam_step(master, g.astype(np.float64), m, v, t, lr)
        sim.adam_update(p, torch.from_numpy(g).cuda(), md, vd, t, lr, weights=wb)
    sim.sync()
    got = p.cpu().numpy().astype(np.float64)
    tol = len(grads) * lr * 2.0 ** -18 + 2.0 ** -22 * np.abs(master)
    assert np.all(np.abs(got - master) <= tol), np.max(np.abs(got - master) / tol)
    # the policy's weights were rewritten from the GPU parameters: matrices rounded to the
    # element type (bf16 nearest even), biases as they are
    back = bs.unpack_weights(w, wb.cpu().numpy())
    off = 0
    for k in KEYS:
        pk = got[off:off + back[k].size].reshape(back[k].shape)
        off += back[k].size
        exp = orc_ppo.bf16r(pk) if (w["mlp_bf16"] and k.startswith("w")) else pk
        assert np.array_equal(back[k], exp), k
    sim.close()


@pytest.mark.parametrize("name,algo", [("C1", 0), ("C1", 1), ("C4", 0), ("C4", 1)])
def test_update_loop_parity(bs, name, algo):
    w = workload(name)
    T, E = 6, 256
    epochs, nmb, M, lr, eps = 2, 3, 512, 1e-3, 1e-2
    say(f"[update] {name} algo={algo}")
    obs_t, act, adv, ret = trajectory(w, T, E, seed=31)
    wts = weights_for(w, 9)
    W64 = {k: v.astype(np.float64) for k, v in wts.items()}
    # old log-probabilities from the oracle's forward of the starting weights
    lp = np.zeros((T, E), np.float32)
    A = 6 * w["n_servers"]
    for t in range(T):
        out = orc_ppo.forward(w, W64, obs_t[t].T.astype(np.float64))["out"][:, :A]
        lse = np.log(np.exp(out - out.max(1, keepdims=True)).sum(1)) + out.max(1)
        lp[t] = (out[np.arange(E), act[t]] - lse - 0.05).astype(np.float32)
    master = {k: v.copy() for k, v in W64.items()}
    adam = dict(m={k: np.zeros_like(v) for k, v in master.items()},
                v={k: np.zeros_like(v) for k, v in master.items()}, t=0)
    ref_losses = orc_train.update(w, master, adam, 0x5151, obs_t, act, lp, adv, ret, algo, epochs,
                                  nmb, M, lr, eps=eps)
    dev = torch.device("cuda")
    sim = bs.Sim(w, n_envs=E)
    wb = sim.upload_weights(wts)
    p = sim.params_from_weights(wb)
    md = torch.zeros_like(p)
    vd = torch.zeros_like(p)
    step, losses = sim.update(wb, p, md, vd, 0, torch.from_numpy(obs_t).to(dev),
                              torch.from_numpy(act).to(dev), torch.from_numpy(lp).to(dev),
                              torch.from_numpy(adv).to(dev), torch.from_numpy(ret).to(dev), algo,
                              epochs, nmb, M, 0x5151, lr, eps=eps)
    sim.sync()
    assert step == epochs * nmb == adam["t"]
    got = p.cpu().numpy().astype(np.float64)
    ref = flat(master)
    diff = np.abs(got - ref)
    say(f"  max |dp| {diff.max():.3g} (lr {lr}, steps {step})")
    assert np.all(diff <= step * lr * 2.0 ** -6 + 2.0 ** -22 * np.abs(ref))
    gl = losses.cpu().numpy()
    scale = np.abs(ref_losses[:, 1:]).sum(axis=1)
    assert np.all(np.abs(gl - ref_losses) <= 2.0 ** -8 * scale[:, None])
    sim.close()
