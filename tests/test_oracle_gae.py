"""Pins of the oracle's returns/GAE: closed forms, the lambda=1 and lambda=0 special
cases, and the non-recursive definition A_t = sum_l (gamma lambda)^l delta_{t+l}."""
import numpy as np

from workloads.gen import seeded_rewards_values


def test_constant_reward_closed_form(orc):
    T, n, g = 1000, 3, 0.99
    r = np.ones((T, n))
    adv, ret = orc.gae(r, None, g, 1.0)
    assert abs(ret[0, 0] - (1 - g**1000) / (1 - g)) < 1e-10
    assert abs(ret[0, 0] - 99.99568287) < 1e-6
    t = np.arange(T)
    np.testing.assert_allclose(ret[:, 1], (1 - g ** (T - t)) / (1 - g), rtol=1e-12)
    assert np.array_equal(adv, ret)


def _direct(r, v, g, lam):
    T = r.shape[0]
    vv = v.astype(np.float64)
    delta = r + g * vv[1:] - vv[:-1]
    i = np.arange(T)
    D = np.where(i[None, :] >= i[:, None], (g * lam) ** (i[None, :] - i[:, None]), 0.0)
    return D @ delta


def test_gae_matches_direct_sum(orc):
    r, v = seeded_rewards_values(9, 300, 7)
    for lam in (0.95, 0.5):
        adv, ret = orc.gae(r, v, 0.99, lam)
        ref = _direct(r, v, 0.99, lam)
        np.testing.assert_allclose(adv, ref, rtol=1e-9, atol=1e-9)
        np.testing.assert_allclose(ret, adv + v[:-1].astype(np.float64), rtol=0, atol=0)


def test_gae_lambda_one_is_return_minus_value(orc):
    r, v = seeded_rewards_values(10, 200, 5)
    g = 0.99
    adv, _ = orc.gae(r, v, g, 1.0)
    T = r.shape[0]
    i = np.arange(T)
    D = np.where(i[None, :] >= i[:, None], g ** (i[None, :] - i[:, None]), 0.0)
    G = D @ r + (g ** (T - i))[:, None] * v[T].astype(np.float64)[None, :]
    np.testing.assert_allclose(adv, G - v[:-1].astype(np.float64), rtol=1e-9, atol=1e-8)


def test_gae_lambda_zero_is_td_error(orc):
    r, v = seeded_rewards_values(11, 50, 4)
    adv, _ = orc.gae(r, v, 0.9, 0.0)
    vv = v.astype(np.float64)
    np.testing.assert_allclose(adv, r + 0.9 * vv[1:] - vv[:-1], rtol=1e-14, atol=1e-12)
