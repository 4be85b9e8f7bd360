"""Pins of the oracle's attention policy (paper Sec. 4.2, reading R26): against
torch.nn.MultiheadAttention in fp64 (an independent implementation of scaled dot-product
multi-head attention), the closed form of a single token (a softmax over one key is 1), the
permutation invariance of one-token-per-feature attention with mean pooling, the closed form
of uniform attention when the queries carry no information, and the Xavier initialisation."""
import math

import numpy as np
import pytest

from workloads import attn_preset

torch = pytest.importorskip("torch")


def rand_wts(orc, w, rng, scale=0.8):
    return {k: rng.standard_normal(sh) * scale for k, sh in orc.attn_shapes(w).items()}


def torch_forward(w, W, x):
    """The attention policy written with torch modules in fp64: tokens from the input
    projection's per-feature terms, nn.MultiheadAttention (batch_first), mean pooling, two
    GELU heads."""
    import torch.nn.functional as Fn
    n, F = x.shape
    L, D, NH = w["attn_tokens"], w["attn_embed"], w["attn_heads"]
    G = F // L
    t = {k: torch.tensor(v, dtype=torch.float64) for k, v in W.items()}
    xt = torch.tensor(x, dtype=torch.float64)
    # token g: sum over its features of x_i * W_in[i, :], plus the bias
    tok = (xt.reshape(n, L, G, 1) * t["w_in"].reshape(1, L, G, D)).sum(dim=2) + t["b_in"]
    mha = torch.nn.MultiheadAttention(D, NH, batch_first=True, dtype=torch.float64)
    with torch.no_grad():
        mha.in_proj_weight.copy_(t["w_qkv"].T)
        mha.in_proj_bias.copy_(t["b_qkv"])
        mha.out_proj.weight.copy_(t["w_o"].T)
        mha.out_proj.bias.copy_(t["b_o"])
        y, _ = mha(tok, tok, tok, need_weights=False)
    p = y.mean(dim=1)
    logits = Fn.gelu(p @ t["wp1"] + t["bp1"]) @ t["wp2"] + t["bp2"]
    v = Fn.gelu(p @ t["wv1"] + t["bv1"]) @ t["wv2"] + t["bv2"]
    return torch.cat([logits, v], dim=1).numpy()


@pytest.mark.parametrize("L,NH", [(8, 2), (4, 2), (2, 1), (1, 2), (8, 4)])
def test_attention_matches_torch_mha(orc, L, NH):
    w = attn_preset(attn_tokens=L, attn_heads=NH)
    rng = np.random.default_rng(100 + 10 * L + NH)
    W = rand_wts(orc, w, rng)
    x = rng.standard_normal((64, w["obs_dim"])).astype(np.float32)
    got = orc.policy(w, W, 1, 0, x, np.arange(64))["logits"]
    ref = torch_forward(w, W, x.astype(np.float64))
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12), np.abs(got - ref).max()


def test_single_token_is_the_value_path(orc):
    """L = 1: the one token is the whole input projection, its attention weight is exactly 1,
    so the pooled vector is (x W_in + b_in) W_v + b_v then W_o + b_o."""
    w = attn_preset(attn_tokens=1)
    rng = np.random.default_rng(3)
    W = rand_wts(orc, w, rng)
    x = rng.standard_normal((20, 8)).astype(np.float32)
    D = w["attn_embed"]
    e = x.astype(np.float64) @ W["w_in"] + W["b_in"]
    vv = e @ W["w_qkv"][:, 2 * D:] + W["b_qkv"][2 * D:]
    p = vv @ W["w_o"] + W["b_o"]
    gelu = lambda z: 0.5 * z * (1.0 + np.vectorize(math.erf)(z / math.sqrt(2.0)))
    logits = gelu(p @ W["wp1"] + W["bp1"]) @ W["wp2"] + W["bp2"]
    val = gelu(p @ W["wv1"] + W["bv1"]) @ W["wv2"] + W["bv2"]
    got = orc.policy(w, W, 1, 0, x, np.arange(20))["logits"]
    assert np.allclose(got[:, :6], logits, rtol=1e-12, atol=1e-13)
    assert np.allclose(got[:, 6], val[:, 0], rtol=1e-12, atol=1e-13)


def test_feature_permutation_invariance(orc):
    """One token per feature: permuting the features together with the rows of W_in permutes
    the tokens; self-attention is permutation-equivariant and the mean pool invariant."""
    w = attn_preset(attn_tokens=8)
    rng = np.random.default_rng(4)
    W = rand_wts(orc, w, rng)
    x = rng.standard_normal((30, 8)).astype(np.float32)
    perm = rng.permutation(8)
    W2 = dict(W, w_in=W["w_in"][perm])
    a = orc.policy(w, W, 1, 0, x, np.arange(30))["logits"]
    b = orc.policy(w, W2, 1, 0, np.ascontiguousarray(x[:, perm]), np.arange(30))["logits"]
    assert np.allclose(a, b, rtol=1e-11, atol=1e-13)
    # while a permutation of the features alone changes the output
    c = orc.policy(w, W, 1, 0, np.ascontiguousarray(x[:, perm]), np.arange(30))["logits"]
    assert np.abs(a - c).max() > 1e-3


def test_uninformative_queries_give_uniform_attention(orc):
    """W_q = 0 and b_q = 0: every score is 0, each head averages the values, and every token's
    output equals mean_j v_j W_o + b_o (so does the pool)."""
    w = attn_preset(attn_tokens=8)
    D = w["attn_embed"]
    rng = np.random.default_rng(5)
    W = rand_wts(orc, w, rng)
    W["w_qkv"][:, :D] = 0.0
    W["b_qkv"][:D] = 0.0
    x = rng.standard_normal((25, 8)).astype(np.float32)
    tok = x.astype(np.float64)[:, :, None] * W["w_in"][None, :, :] + W["b_in"]     # [n][8][D]
    vv = tok @ W["w_qkv"][:, 2 * D:] + W["b_qkv"][2 * D:]
    p = vv.mean(axis=1) @ W["w_o"] + W["b_o"]
    gelu = lambda z: 0.5 * z * (1.0 + np.vectorize(math.erf)(z / math.sqrt(2.0)))
    logits = gelu(p @ W["wp1"] + W["bp1"]) @ W["wp2"] + W["bp2"]
    got = orc.policy(w, W, 1, 0, x, np.arange(25))["logits"]
    assert np.allclose(got[:, :6], logits, rtol=1e-12, atol=1e-13)


def test_attention_init_xavier(orc):
    w = attn_preset()
    W = orc.init_weights(w, 77)
    F, D, A, Hp, Hv = 8, w["attn_embed"], 6, w["mlp_h1"], w["mlp_h2"]
    fans = dict(w_in=(F, D), w_qkv=(D, 3 * D), w_o=(D, D), wp1=(D, Hp), wp2=(Hp, A),
                wv1=(D, Hv), wv2=(Hv, 1))
    for k, (fi, fo) in fans.items():
        lim = math.sqrt(6.0 / (fi + fo))
        a = W[k]
        assert a.shape == (fi, fo)
        assert np.all(np.abs(a) <= lim) and np.all(a == a.astype(np.float32))
        if a.size >= 200:
            # uniform on [-lim, lim]: mean 0, variance lim^2 / 3
            assert abs(a.mean()) < 4 * lim / math.sqrt(3 * a.size)
            assert abs(a.var() / (lim * lim / 3.0) - 1.0) < 0.25
    for k in ("b_in", "b_qkv", "b_o", "bp1", "bp2", "bv1", "bv2"):
        assert not W[k].any()
    assert not np.array_equal(W["wp1"], W["wv1"])      # separate streams per matrix
    W2 = orc.init_weights(w, 77)
    assert all(np.array_equal(W[k], W2[k]) for k in W)


def test_attention_rollout_runs_and_is_valid(orc):
    """The oracle's own rollout under the attention policy: actions in range, replaying them
    reproduces the same simulation, and V is the value head on each observation."""
    w = attn_preset(n_envs=8)
    W = orc.init_weights(w, 3)
    T = 50
    r = orc.rollout(w, 11, T, np.arange(8), weights=W)
    assert r["actions"].max() < 6
    rep = orc.rollout(w, 11, T, np.arange(8), actions=r["actions"])
    assert np.array_equal(rep["obs"], r["obs"])
    assert np.array_equal(rep["chk"], r["chk"])
    for t in (0, 17, T):
        out = orc.policy(w, W, 11, t, r["obs"][t], np.arange(8))
        assert np.array_equal(r["value"][t], out["logits"][:, 6].astype(np.float32))
