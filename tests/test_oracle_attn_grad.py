"""Pins of the attention-policy gradient oracle (oracle/attn.py): its forward against the C
oracle's attention policy, the analytic gradient of the REINFORCE and PPO losses against central
finite differences for every parameter, against torch autograd through
torch.nn.MultiheadAttention in fp64, and the magnitude sums as upper bounds."""
import numpy as np
import pytest

from workloads import attn_preset

torch = pytest.importorskip("torch")


def tiny(L=4, NH=2, value_head=1):
    return attn_preset(attn_tokens=L, attn_heads=NH, mlp_h1=5, mlp_h2=3, value_head=value_head)


def rand_w(orc, w, rng, scale=0.7):
    return {k: rng.standard_normal(sh) * (scale if k.startswith("w") else 0.2)
            for k, sh in orc.attn_shapes(w).items()}


def batch(rng, M, F=8):
    x = rng.standard_normal((M, F))
    act = rng.integers(0, 6, M)
    adv = rng.standard_normal(M)
    ret = rng.standard_normal(M)
    return x, act, adv, ret


def test_forward_matches_c_oracle(orc):
    from oracle import attn
    for L, NH in ((8, 2), (4, 2), (1, 2), (2, 1)):
        w = tiny(L, NH)
        rng = np.random.default_rng(L + NH)
        W = rand_w(orc, w, rng)
        x = rng.standard_normal((16, 8)).astype(np.float32)
        ref = orc.policy(w, W, 1, 0, x, np.arange(16))["logits"]
        got = attn.forward(w, W, x.astype(np.float64))["out"]
        assert np.allclose(got, ref, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("algo", [0, 1])
@pytest.mark.parametrize("L,NH", [(4, 2), (8, 1)])
def test_gradient_matches_central_differences(orc, algo, L, NH):
    from oracle import attn, ppo, train
    w = tiny(L, NH)
    rng = np.random.default_rng(20 + algo + L)
    W = rand_w(orc, w, rng)
    M = 12
    x, act, adv, ret = batch(rng, M)
    fw0 = attn.forward(w, W, x)
    lp = fw0["out"][:, :6]
    lse = np.log(np.exp(lp - lp.max(1, keepdims=True)).sum(1)) + lp.max(1)
    logp_old = lp[np.arange(M), act] - lse - rng.uniform(-0.1, 0.1, M)   # inside the clip range

    def loss(Wd):
        out = attn.forward(w, Wd, x)["out"]
        if algo == 0:
            return ppo.loss_and_dout(w, out, act, logp_old, adv, ret)[0]["loss"]
        return train.reinforce_loss_and_dout(w, out, act, adv, ret)[0]["loss"]

    if algo == 0:
        dout = ppo.loss_and_dout(w, fw0["out"], act, logp_old, adv, ret)[1]
    else:
        dout = train.reinforce_loss_and_dout(w, fw0["out"], act, adv, ret)[1]
    g = attn.backward(w, W, fw0, dout)
    h = 1e-6
    for k in W:
        for idx in np.ndindex(W[k].shape):
            Wp = {kk: v.copy() for kk, v in W.items()}
            Wm = {kk: v.copy() for kk, v in W.items()}
            Wp[k][idx] += h
            Wm[k][idx] -= h
            fd = (loss(Wp) - loss(Wm)) / (2 * h)
            assert abs(fd - g[k][idx]) <= 2e-6 * max(1.0, abs(fd)), (k, idx, fd, g[k][idx])


def test_gradient_matches_torch_autograd(orc):
    """The REINFORCE-with-baseline loss written with torch modules (nn.MultiheadAttention,
    batch_first) in fp64, differentiated by autograd."""
    import torch.nn.functional as Fn
    from oracle import attn, train
    w = attn_preset(mlp_h1=16, mlp_h2=8)
    L, D, NH, G = 8, 4, 2, 1
    rng = np.random.default_rng(31)
    W = rand_w(orc, w, rng)
    M = 40
    x, act, adv, ret = batch(rng, M)
    fw = attn.forward(w, W, x)
    _, dout = train.reinforce_loss_and_dout(w, fw["out"], act, adv, ret)
    g = attn.backward(w, W, fw, dout)

    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in W.items()}
    xt = torch.tensor(x)
    tok = (xt.reshape(M, L, G, 1) * t["w_in"].reshape(1, L, G, D)).sum(dim=2) + t["b_in"]
    # torch's multi-head attention (the function behind nn.MultiheadAttention), sequence-first
    y, _ = torch.nn.functional.multi_head_attention_forward(
        tok.transpose(0, 1), tok.transpose(0, 1), tok.transpose(0, 1), D, NH,
        t["w_qkv"].T, t["b_qkv"], None, None, False, 0.0, t["w_o"].T, t["b_o"],
        training=False, need_weights=False)
    p = y.transpose(0, 1).mean(dim=1)
    logits = Fn.gelu(p @ t["wp1"] + t["bp1"]) @ t["wp2"] + t["bp2"]
    V = (Fn.gelu(p @ t["wv1"] + t["bv1"]) @ t["wv2"] + t["bv2"])[:, 0]
    logp_all = torch.log_softmax(logits, dim=1)
    prob = logp_all.exp()
    A_t = torch.tensor(adv)
    lp = logp_all[torch.arange(M), torch.tensor(act)]
    H = -(prob * logp_all).sum(dim=1)
    Lt = -(A_t * lp).mean() + 0.5 * ((V - torch.tensor(ret)) ** 2).mean() - 0.01 * H.mean()
    Lt.backward()
    for k in W:
        assert np.allclose(g[k], t[k].grad.numpy(), rtol=1e-10, atol=1e-12), k


def test_magnitude_sums_bound_the_gradient(orc):
    from oracle import attn, train
    w = tiny(8, 2)
    rng = np.random.default_rng(41)
    W = rand_w(orc, w, rng)
    x, act, adv, ret = batch(rng, 30)
    fw = attn.forward(w, W, x)
    _, dout = train.reinforce_loss_and_dout(w, fw["out"], act, adv, ret)
    g = attn.backward(w, W, fw, dout)
    ga = attn.backward(w, W, fw, dout, absolute=True)
    for k in W:
        assert np.all(ga[k] >= np.abs(g[k]) - 1e-15), k
        assert np.all(ga[k] >= 0)


def test_update_loop_descends(orc):
    """A few Adam steps with a small learning rate lower the loss of a fixed minibatch."""
    from oracle import attn
    w = tiny(4, 2)
    rng = np.random.default_rng(51)
    master = rand_w(orc, w, rng)
    T, E = 5, 20
    obs_t = rng.random((T, 8, E)).astype(np.float32)
    act = rng.integers(0, 6, (T, E)).astype(np.uint8)
    adv = rng.standard_normal((T, E))
    ret = rng.standard_normal((T, E))
    W0 = attn.policy_weights(master)
    l0 = attn.minibatch_grad(w, W0, 7, obs_t, act, None, adv, ret, 32, attn.ALGO_REINFORCE)[0]
    adam = dict(m={k: np.zeros_like(v) for k, v in master.items()},
                v={k: np.zeros_like(v) for k, v in master.items()}, t=0)
    # every minibatch of the loop under the same key, so each step descends the same loss
    for _ in range(6):
        attn.update(w, master, adam, 7, obs_t, act, None, adv, ret, attn.ALGO_REINFORCE, 1, 1, 32,
                    1e-3)
    l1 = attn.minibatch_grad(w, attn.policy_weights(master), 7, obs_t, act, None, adv, ret, 32,
                             attn.ALGO_REINFORCE)[0]
    assert adam["t"] == 6
    assert l1["loss"] < l0["loss"]
