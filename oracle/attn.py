"""Attention-policy gradient oracle (paper Sec. 4.2 network, Sec. 4.3 losses) -- TEST
INFRASTRUCTURE.

The network of reading R26 in fp64 over a minibatch of M observations, its forward written
out step by step with every intermediate kept, and the exact gradient of the REINFORCE or PPO
loss with respect to all fourteen parameter arrays by the chain rule taken backwards through
the same steps:

    tokens     e_g = b_in + sum_{i in g} x_i W_in[i, :]
    attention  [q | k | v] = e W_qkv + b_qkv; per head h, s = q_h k_h^T / sqrt(dh),
               a = softmax(s) over keys, o_h = a v_h
    output     y = o W_o + b_o;  p = mean_g y_g
    heads      logits = GELU(p W_p1 + b_p1) W_p2 + b_p2,  V = GELU(p W_v1 + b_v1) W_v2 + b_v2

Softmax backward: ds = a (da - sum_j a_j da_j). The same backward evaluated on absolute values
(|W|, |activations|, |dL/dout|, |GELU'|, and a (|da| + sum_j a_j |da_j|) for the softmax) gives,
for every parameter, the sum over samples and tokens of the magnitudes of its gradient terms;
tests derive the fp32 tolerance from it.
"""
import math

import numpy as np

from . import ppo, train, attn_shapes, ATTN_KEYS

ALGO_PPO, ALGO_REINFORCE = train.ALGO_PPO, train.ALGO_REINFORCE


def forward(w, W, x):
    """x [M][F] -> dict of every intermediate and out [M][A'] (logits, then V)."""
    x = np.asarray(x, np.float64)
    M, F = x.shape
    L, D, NH = w["attn_tokens"], w["attn_embed"], w["attn_heads"]
    G, dh = F // L, D // NH
    xg = x.reshape(M, L, G)
    e = np.einsum("mlg,lgd->mld", xg, W["w_in"].reshape(L, G, D)) + W["b_in"]
    qkv = e @ W["w_qkv"] + W["b_qkv"]
    q, k, v = qkv[..., :D], qkv[..., D:2 * D], qkv[..., 2 * D:]
    a = np.zeros((M, NH, L, L))
    o = np.zeros((M, L, D))
    for h in range(NH):
        c = slice(h * dh, (h + 1) * dh)
        s = np.einsum("mgt,mjt->mgj", q[..., c], k[..., c]) / math.sqrt(dh)
        ex = np.exp(s - s.max(axis=2, keepdims=True))
        a[:, h] = ex / ex.sum(axis=2, keepdims=True)
        o[..., c] = np.einsum("mgj,mjt->mgt", a[:, h], v[..., c])
    y = o @ W["w_o"] + W["b_o"]
    p = y.mean(axis=1)
    z1 = p @ W["wp1"] + W["bp1"]
    h1 = ppo.gelu(z1)
    logits = h1 @ W["wp2"] + W["bp2"]
    cols = [logits]
    z2 = h2 = None
    if w["value_head"]:
        z2 = p @ W["wv1"] + W["bv1"]
        h2 = ppo.gelu(z2)
        cols.append(h2 @ W["wv2"] + W["bv2"])
    return dict(x=x, xg=xg, e=e, q=q, k=k, v=v, a=a, o=o, y=y, p=p, z1=z1, h1=h1, z2=z2, h2=h2,
                out=np.concatenate(cols, axis=1))


def backward(w, W, fw, dout, absolute=False):
    """Gradients (dict keyed like the parameters) of a loss whose derivative with respect to
    out is dout [M][A']; with absolute=True the magnitude sums described above."""
    M, F = fw["x"].shape
    L, D, NH = w["attn_tokens"], w["attn_embed"], w["attn_heads"]
    G, dh = F // L, D // NH
    A = 6 * w["n_servers"]
    f = np.abs if absolute else (lambda t: t)
    Wt = {k: f(v) for k, v in W.items()}
    g = {}
    dl = f(dout[:, :A])
    g["wp2"] = f(fw["h1"]).T @ dl
    g["bp2"] = dl.sum(axis=0)
    dz1 = (dl @ Wt["wp2"].T) * f(ppo.gelu_grad(fw["z1"]))
    g["wp1"] = f(fw["p"]).T @ dz1
    g["bp1"] = dz1.sum(axis=0)
    dp = dz1 @ Wt["wp1"].T
    if w["value_head"]:
        dV = f(dout[:, A:A + 1])
        g["wv2"] = f(fw["h2"]).T @ dV
        g["bv2"] = dV.sum(axis=0)
        dz2 = (dV @ Wt["wv2"].T) * f(ppo.gelu_grad(fw["z2"]))
        g["wv1"] = f(fw["p"]).T @ dz2
        g["bv1"] = dz2.sum(axis=0)
        dp = dp + dz2 @ Wt["wv1"].T
    else:
        for kk in ("wv1", "bv1", "wv2", "bv2"):
            g[kk] = np.zeros_like(W[kk])
    dy = np.repeat(dp[:, None, :] / L, L, axis=1)
    g["w_o"] = np.einsum("mli,mld->id", f(fw["o"]), dy)
    g["b_o"] = dy.sum(axis=(0, 1))
    do = dy @ Wt["w_o"].T
    dq = np.zeros((M, L, D))
    dk = np.zeros((M, L, D))
    dv = np.zeros((M, L, D))
    q, k, v = f(fw["q"]), f(fw["k"]), f(fw["v"])
    for h in range(NH):
        c = slice(h * dh, (h + 1) * dh)
        a = fw["a"][:, h]
        da = np.einsum("mgt,mjt->mgj", do[..., c], v[..., c])
        dv[..., c] = np.einsum("mgj,mgt->mjt", a, do[..., c])
        if absolute:
            ds = a * (da + (a * da).sum(axis=2, keepdims=True))
        else:
            ds = a * (da - (a * da).sum(axis=2, keepdims=True))
        dq[..., c] = np.einsum("mgj,mjt->mgt", ds, k[..., c]) / math.sqrt(dh)
        dk[..., c] = np.einsum("mgj,mgt->mjt", ds, q[..., c]) / math.sqrt(dh)
    dqkv = np.concatenate([dq, dk, dv], axis=2)
    g["w_qkv"] = np.einsum("mli,mlj->ij", f(fw["e"]), dqkv)
    g["b_qkv"] = dqkv.sum(axis=(0, 1))
    de = dqkv @ Wt["w_qkv"].T
    g["w_in"] = np.einsum("mlg,mld->lgd", f(fw["xg"]), de).reshape(F, D)
    g["b_in"] = de.sum(axis=(0, 1))
    return g


def minibatch_grad(w, W, seed, obs_t, act_t, logp_t, adv_t, ret_t, M, algo, clip=0.2, c_v=0.5,
                   c_h=0.01):
    """One minibatch: indices as the MLP's (ppo.sample_indices), gather, forward, loss terms,
    gradients and their magnitude sums. obs_t [T][F][E]."""
    T, E = act_t.shape
    ti, ei = ppo.sample_indices(seed, M, T, E)
    x = obs_t[ti, :, ei].astype(np.float64)
    fw = forward(w, W, x)
    act = act_t[ti, ei].astype(np.int64)
    if algo == ALGO_PPO:
        losses, dout = ppo.loss_and_dout(w, fw["out"], act, logp_t[ti, ei].astype(np.float64),
                                         adv_t[ti, ei], ret_t[ti, ei], clip, c_v, c_h)
    else:
        losses, dout = train.reinforce_loss_and_dout(w, fw["out"], act, adv_t[ti, ei],
                                                     ret_t[ti, ei], c_v, c_h)
    return losses, backward(w, W, fw, dout), backward(w, W, fw, dout, absolute=True), (ti, ei)


def policy_weights(master):
    """The attention policy's fp32 weights from fp64 master parameters."""
    return {k: np.asarray(master[k], np.float64).astype(np.float32).astype(np.float64)
            for k in ATTN_KEYS}


def update(w, master, adam, seed, obs_t, act_t, logp_t, adv_t, ret_t, algo, epochs,
           n_minibatches, M, lr, clip=0.2, c_v=0.5, c_h=0.01, b1=0.9, b2=0.999, eps=1e-8):
    """The update loop of train.update for the attention policy (same minibatch keys, Adam on
    fp64 masters, fp32 re-export)."""
    losses = []
    for e in range(epochs):
        for b in range(n_minibatches):
            Wp = policy_weights(master)
            lo, g, _, _ = minibatch_grad(w, Wp, train.minibatch_seed(seed, e, n_minibatches, b),
                                         obs_t, act_t, logp_t, adv_t, ret_t, M, algo, clip, c_v,
                                         c_h)
            adam["t"] += 1
            for k in ATTN_KEYS:
                train.adam_step(master[k], g[k], adam["m"][k], adam["v"][k], adam["t"], lr, b1,
                                b2, eps)
            losses.append([lo["loss"], lo["policy"], lo["value"], lo["entropy"]])
    return np.array(losses)


__all__ = ["forward", "backward", "minibatch_grad", "policy_weights", "update", "attn_shapes"]
