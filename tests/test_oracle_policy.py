"""Pins of the oracle's policy: the MLP against torch's fp64 Linear/GELU with the same
bf16 rounding points (torch's own bf16 conversion), the inverse-CDF sampler against the
softmax it samples, and the Xavier initialisation against its definition's bounds and
moments."""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from workloads import preset
from workloads.gen import seeded_obs, seeded_weights_f32


def torch_mlp(obs, wts, bf16):
    def rnd(t):
        return t.to(torch.float32).to(torch.bfloat16).to(torch.float64) if bf16 else t
    x = rnd(torch.tensor(obs, dtype=torch.float64))
    W = {k: torch.tensor(v, dtype=torch.float64) for k, v in wts.items()}
    h1 = rnd(Fn.gelu(x @ W["w1"] + W["b1"]))
    h2 = rnd(Fn.gelu(h1 @ W["w2"] + W["b2"]))
    return (h2 @ W["w3"] + W["b3"]).numpy()


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C5"])
def test_mlp_matches_torch_fp64(orc, name):
    w = preset(name)
    A = orc.n_out(w)
    dims = [w["obs_dim"], w["mlp_h1"], w["mlp_h2"], A]
    wts = seeded_weights_f32(3, dims, bf16=bool(w["mlp_bf16"]))
    obs = seeded_obs(4, 64, w["obs_dim"])
    got = orc.policy(w, {k: v.astype(np.float64) for k, v in wts.items()}, 1, 0, obs,
                     np.arange(64))["logits"]
    ref = torch_mlp(obs, {k: v.astype(np.float64) for k, v in wts.items()}, bool(w["mlp_bf16"]))
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)


def test_sampler_boundaries(orc):
    p = np.array([0.1, 0.2, 0.3, 0.4])
    l = np.log(p) + 3.0
    cdf = np.cumsum(p)
    for i, c in enumerate(cdf[:-1]):
        a, lp, mg = orc.sample_logits(l, c - 1e-9)
        assert a == i and abs(lp - np.log(p[i])) < 1e-12 and mg < 2e-9
        a, lp, mg = orc.sample_logits(l, c + 1e-9)
        assert a == i + 1 and abs(lp - np.log(p[i + 1])) < 1e-12
    a, _, mg = orc.sample_logits(l, 0.05)
    assert a == 0 and abs(mg - 0.05) < 1e-12
    # a -inf-like logit is never chosen
    l2 = np.array([0.0, -1e30, 0.0])
    assert orc.sample_logits(l2, 0.5 + 1e-9)[0] == 2


def test_sampler_frequencies_follow_softmax(orc):
    from scipy import stats
    rng = np.random.default_rng(8)
    l = rng.standard_normal(6) * 1.5
    p = np.exp(l - l.max()); p /= p.sum()
    n = 60000
    acts = np.array([orc.sample_logits(l, orc.action_u(123, e, 7))[0] for e in range(n)])
    cnt = np.bincount(acts, minlength=6)
    assert stats.chisquare(cnt, p * n).pvalue > 1e-4


def test_action_uniform_is_centered_23_bit(orc):
    us = np.array([orc.action_u(5, e, 0) for e in range(2000)])
    assert np.all((us > 0) & (us < 1))
    assert np.all(np.abs(us * 2**23 - np.floor(us * 2**23) - 0.5) < 1e-9)


@pytest.mark.parametrize("name", ["C1", "C5"])
def test_xavier_init(orc, name):
    w = preset(name)
    a = orc.init_weights(w, 42)
    b = orc.init_weights(w, 42)
    c = orc.init_weights(w, 43)
    dims = [w["obs_dim"], w["mlp_h1"], w["mlp_h2"], orc.n_out(w)]
    for l in range(3):
        W = a[f"w{l + 1}"]
        assert np.array_equal(W, b[f"w{l + 1}"]) and not np.array_equal(W, c[f"w{l + 1}"])
        lim = np.sqrt(6.0 / (dims[l] + dims[l + 1]))
        assert np.all(np.abs(W) <= lim * (1 + 2**-7))
        assert abs(W.mean()) < 4 * lim / np.sqrt(3 * W.size)
        assert abs(W.var() / (lim**2 / 3) - 1) < 0.1
        assert np.all(a[f"b{l + 1}"] == 0)
        f32 = W.astype(np.float32)
        assert np.array_equal(f32.astype(np.float64), W)
        if w["mlp_bf16"]:
            assert np.all((f32.view(np.uint32) & 0xFFFF) == 0)
