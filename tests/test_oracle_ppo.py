"""Pins of the PPO minibatch oracle: the analytic gradient against central finite
differences of the loss, closed-form loss values, the clipped regime, index sampling."""
import math

import numpy as np
from scipy import stats

from workloads import preset


def tiny(bf16=0):
    return preset("C4", n_servers=1, n_classes=1, obs_dim=8, mlp_h1=5, mlp_h2=4, mlp_bf16=bf16,
                  value_head=1)


def rand_wts(rng, dims):
    return {f"w{l + 1}": rng.standard_normal((dims[l], dims[l + 1])) * 0.7 for l in range(3)} | \
           {f"b{l + 1}": rng.standard_normal(dims[l + 1]) * 0.1 for l in range(3)}


def test_gradient_matches_central_differences(orc):
    from oracle import ppo
    w = tiny()
    rng = np.random.default_rng(0)
    dims = [8, 5, 4, 7]
    wts = rand_wts(rng, dims)
    M = 40
    x = rng.random((M, 8))
    act = rng.integers(0, 6, M)
    logp_old = np.log(rng.uniform(0.05, 0.4, M))
    adv = rng.standard_normal(M)
    ret = rng.standard_normal(M)

    def L(wd):
        fw = ppo.forward(w, wd, x)
        return ppo.loss_and_dout(w, fw["out"], act, logp_old, adv, ret)[0]["loss"]

    fw = ppo.forward(w, wts, x)
    _, dout = ppo.loss_and_dout(w, fw["out"], act, logp_old, adv, ret)
    g = ppo.backward(w, wts, fw, dout)
    h = 1e-6
    checked = 0
    for k in g:
        for idx in np.ndindex(wts[k].shape):
            wp = {kk: v.copy() for kk, v in wts.items()}
            wm = {kk: v.copy() for kk, v in wts.items()}
            wp[k][idx] += h
            wm[k][idx] -= h
            fd = (L(wp) - L(wm)) / (2 * h)
            assert abs(fd - g[k][idx]) <= 1e-6 * max(1.0, abs(fd)), (k, idx, fd, g[k][idx])
            checked += 1
    assert checked == sum(v.size for v in wts.values())


def test_uniform_policy_closed_forms(orc):
    """Zero weights: logits 0 -> p = 1/6, entropy log 6; with logp_old = -log 6 the ratio is
    1, so the surrogate is mean(A); the value is b3[A]."""
    from oracle import ppo
    w = tiny()
    dims = [8, 5, 4, 7]
    wts = {f"w{l + 1}": np.zeros((dims[l], dims[l + 1])) for l in range(3)} | \
          {f"b{l + 1}": np.zeros(dims[l + 1]) for l in range(3)}
    wts["b3"][6] = 0.25
    rng = np.random.default_rng(1)
    M = 64
    x = rng.random((M, 8))
    act = rng.integers(0, 6, M)
    adv = rng.standard_normal(M)
    ret = rng.standard_normal(M)
    fw = ppo.forward(w, wts, x)
    losses, dout = ppo.loss_and_dout(w, fw["out"], act, np.full(M, -math.log(6.0)), adv, ret)
    assert abs(losses["policy"] + adv.mean()) < 1e-12
    assert abs(losses["entropy"] + 0.01 * math.log(6.0)) < 1e-12
    assert abs(losses["value"] - 0.5 * ((0.25 - ret) ** 2).mean()) < 1e-12
    # entropy gradient vanishes at the uniform distribution; policy gradient is A (1[a] - 1/6)/M
    exp = np.zeros((M, 6))
    exp[np.arange(M), act] = -adv / M
    exp += (adv / M)[:, None] / 6.0
    assert np.allclose(dout[:, :6], exp, atol=1e-15)


def test_clipped_regime_has_no_policy_gradient(orc):
    from oracle import ppo
    w = tiny()
    rng = np.random.default_rng(2)
    dims = [8, 5, 4, 7]
    wts = rand_wts(rng, dims)
    M = 32
    x = rng.random((M, 8))
    fw = ppo.forward(w, wts, x)
    act = rng.integers(0, 6, M)
    l = fw["out"][:, :6]
    logp = (l - l.max(1, keepdims=True)) - np.log(np.exp(l - l.max(1, keepdims=True)).sum(1, keepdims=True))
    lp = logp[np.arange(M), act]
    # rho = e^1 > 1.2 with A > 0: the clipped term is the minimum, its gradient is zero
    losses, dout = ppo.loss_and_dout(w, fw["out"], act, lp - 1.0, np.ones(M), np.zeros(M),
                                     c_h=0.0)
    assert abs(losses["policy"] + 1.2) < 1e-12
    assert np.allclose(dout[:, :6], 0.0)


def test_sample_indices_uniform(orc):
    from oracle import ppo
    t, e = ppo.sample_indices(17, 20000, 40, 50)
    assert t.min() >= 0 and t.max() < 40 and e.min() >= 0 and e.max() < 50
    assert stats.chisquare(np.bincount(t, minlength=40)).pvalue > 1e-4
    assert stats.chisquare(np.bincount(e, minlength=50)).pvalue > 1e-4
