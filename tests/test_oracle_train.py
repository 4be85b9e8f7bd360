"""Pins of the update oracle (oracle/train.py): the REINFORCE gradient against central finite
differences and closed forms, its identity with the PPO gradient at ratio 1, Adam against its
first-step closed form and against torch.optim.Adam, and descent of the full update loop."""
import math

import numpy as np
import pytest

from workloads import preset


def tiny(bf16=0):
    return preset("C4", n_servers=1, n_classes=1, obs_dim=8, mlp_h1=5, mlp_h2=4, mlp_bf16=bf16,
                  value_head=1)


DIMS = [8, 5, 4, 7]


def rand_wts(rng):
    return {f"w{l + 1}": rng.standard_normal((DIMS[l], DIMS[l + 1])) * 0.7 for l in range(3)} | \
           {f"b{l + 1}": rng.standard_normal(DIMS[l + 1]) * 0.1 for l in range(3)}


def test_reinforce_gradient_matches_central_differences(orc):
    from oracle import ppo, train
    w = tiny()
    rng = np.random.default_rng(10)
    wts = rand_wts(rng)
    M = 40
    x = rng.random((M, 8))
    act = rng.integers(0, 6, M)
    adv = rng.standard_normal(M)
    ret = rng.standard_normal(M)

    def L(wd):
        return train.reinforce_loss_and_dout(w, ppo.forward(w, wd, x)["out"], act, adv, ret)[0]["loss"]

    fw = ppo.forward(w, wts, x)
    g = ppo.backward(w, wts, fw, train.reinforce_loss_and_dout(w, fw["out"], act, adv, ret)[1])
    h = 1e-6
    for k in g:
        for idx in np.ndindex(wts[k].shape):
            wp = {kk: v.copy() for kk, v in wts.items()}
            wm = {kk: v.copy() for kk, v in wts.items()}
            wp[k][idx] += h
            wm[k][idx] -= h
            fd = (L(wp) - L(wm)) / (2 * h)
            assert abs(fd - g[k][idx]) <= 1e-6 * max(1.0, abs(fd)), (k, idx, fd, g[k][idx])


def test_reinforce_uniform_policy_closed_forms(orc):
    """Zero weights: p = 1/6, so L_pi = mean(A) log 6 and dL/dl_j = (A/M)(1/6 - 1[j = a])."""
    from oracle import ppo, train
    w = tiny()
    wts = {f"w{l + 1}": np.zeros((DIMS[l], DIMS[l + 1])) for l in range(3)} | \
          {f"b{l + 1}": np.zeros(DIMS[l + 1]) for l in range(3)}
    rng = np.random.default_rng(11)
    M = 64
    x = rng.random((M, 8))
    act = rng.integers(0, 6, M)
    adv = rng.standard_normal(M)
    ret = rng.standard_normal(M)
    losses, dout = train.reinforce_loss_and_dout(w, ppo.forward(w, wts, x)["out"], act, adv, ret)
    assert abs(losses["policy"] - adv.mean() * math.log(6.0)) < 1e-12
    exp = np.tile((adv / M)[:, None] / 6.0, (1, 6))
    exp[np.arange(M), act] -= adv / M
    assert np.allclose(dout[:, :6], exp, atol=1e-15)


def test_reinforce_equals_ppo_at_ratio_one(orc):
    """d(rho A)/dtheta = A dlog pi/dtheta at rho = 1: with logp_old = logp the PPO gradient
    (inside the clip range) is the REINFORCE gradient."""
    from oracle import ppo, train
    w = tiny()
    rng = np.random.default_rng(12)
    wts = rand_wts(rng)
    M = 50
    x = rng.random((M, 8))
    act = rng.integers(0, 6, M)
    adv = rng.standard_normal(M)
    ret = rng.standard_normal(M)
    fw = ppo.forward(w, wts, x)
    l = fw["out"][:, :6]
    lse = np.log(np.exp(l - l.max(1, keepdims=True)).sum(1)) + l.max(1)
    logp = l[np.arange(M), act] - lse
    _, d_ppo = ppo.loss_and_dout(w, fw["out"], act, logp, adv, ret)
    _, d_rf = train.reinforce_loss_and_dout(w, fw["out"], act, adv, ret)
    assert np.allclose(d_ppo, d_rf, atol=1e-14, rtol=1e-12)


def test_adam_first_step_closed_form(orc):
    """After one step m_hat = g and v_hat = g^2, so the step is lr g / (|g| + eps)."""
    from oracle import train
    rng = np.random.default_rng(13)
    p0 = rng.standard_normal(100)
    g = rng.standard_normal(100) * 10.0 ** rng.uniform(-4, 2, 100)
    p = p0.copy()
    m = np.zeros(100)
    v = np.zeros(100)
    train.adam_step(p, g, m, v, 1, 1e-3, 0.9, 0.999, 1e-8)
    assert np.allclose(p0 - p, 1e-3 * g / (np.abs(g) + 1e-8), rtol=1e-12, atol=0)


def test_adam_matches_torch(orc):
    torch = pytest.importorskip("torch")
    from oracle import train
    rng = np.random.default_rng(14)
    p0 = rng.standard_normal(64)
    grads = [rng.standard_normal(64) for _ in range(7)]
    p = p0.copy()
    m = np.zeros(64)
    v = np.zeros(64)
    for t, g in enumerate(grads, start=1):
        train.adam_step(p, g, m, v, t, 3e-3, 0.9, 0.999, 1e-8)
    tp = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([tp], lr=3e-3, betas=(0.9, 0.999), eps=1e-8)
    for g in grads:
        opt.zero_grad()
        tp.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    assert np.allclose(p, tp.detach().numpy(), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("algo", [0, 1])
def test_update_loop_descends(orc, algo):
    """A small learning rate lowers the loss of the first minibatch over the epochs (first-
    order descent), Adam's step counter advances once per minibatch, and each minibatch of an
    epoch draws different indices."""
    from oracle import ppo, train
    w = tiny()
    rng = np.random.default_rng(15 + algo)
    master = rand_wts(rng)
    T, E = 6, 30
    obs_t = rng.random((T, 8, E)).astype(np.float32)
    act = rng.integers(0, 6, (T, E)).astype(np.uint8)
    adv = rng.standard_normal((T, E))
    ret = rng.standard_normal((T, E))
    wts0 = train.policy_weights(w, master)
    lp = np.zeros((T, E), np.float32)
    for t in range(T):
        out = ppo.forward(w, wts0, obs_t[t].T.astype(np.float64))["out"][:, :6]
        lse = np.log(np.exp(out - out.max(1, keepdims=True)).sum(1)) + out.max(1)
        lp[t] = (out[np.arange(E), act[t]] - lse).astype(np.float32)
    adam = dict(m={k: np.zeros_like(v) for k, v in master.items()},
                v={k: np.zeros_like(v) for k, v in master.items()}, t=0)
    losses = train.update(w, master, adam, 99, obs_t, act, lp, adv, ret, algo, epochs=4,
                          n_minibatches=3, M=32, lr=1e-3)
    assert adam["t"] == 12 and losses.shape == (12, 4)
    # same minibatch (b = 0) in epochs 0 and 3 under the same seed schedule: loss went down
    first = train.minibatch_seed(99, 0, 3, 0)
    assert first == train.minibatch_seed(99, 0, 3, 0) != train.minibatch_seed(99, 0, 3, 1)
    l_before = train.minibatch_grad(w, wts0, first, obs_t, act, lp, adv, ret, 32, algo)[0]["loss"]
    l_after = train.minibatch_grad(w, train.policy_weights(w, master), first, obs_t, act, lp,
                                   adv, ret, 32, algo)[0]["loss"]
    assert l_after < l_before
    t0, e0 = ppo.sample_indices(train.minibatch_seed(99, 0, 3, 0), 32, T, E)
    t1, e1 = ppo.sample_indices(train.minibatch_seed(99, 0, 3, 1), 32, T, E)
    assert not (np.array_equal(t0, t1) and np.array_equal(e0, e1))
