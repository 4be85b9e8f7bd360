"""Policy-gradient update oracle (paper Sec. 4.3) -- TEST INFRASTRUCTURE.

REINFORCE with a learned baseline and PPO, each as an on-device-style update: E epochs of
B minibatches of M samples over a stored trajectory, each minibatch's gradient followed by
one Adam step (Kingma & Ba, "Adam: a method for stochastic optimization", ICLR 2015,
Algorithm 1) on fp64 master parameters; the policy's own weights are the master parameters
rounded to the policy's element type (bf16 or fp32) after every step. Plain numpy, one step
after another; the minibatch forward and backward are oracle/ppo.py's.

REINFORCE loss over a minibatch (advantage A = G - V(s), G the Monte-Carlo return):
    L = -mean(A log pi(a|s)) + c_v mean((V - G)^2) - c_h mean(H)
with A held constant (the baseline does not receive the policy term's gradient).
Minibatch b of epoch e draws its indices under the key seed + (e * B + b) * GOLDEN.
"""
import numpy as np

from . import ppo

GOLDEN = 0x9E3779B97F4A7C15
ALGO_PPO, ALGO_REINFORCE = 0, 1
PARAM_KEYS = ("w1", "b1", "w2", "b2", "w3", "b3")


def minibatch_seed(seed, epoch, n_minibatches, b):
    return (seed + (epoch * n_minibatches + b) * GOLDEN) % (1 << 64)


def reinforce_loss_and_dout(w, out, act, adv, ret, c_v=0.5, c_h=0.01):
    """Loss terms and dL/d(out) of the REINFORCE-with-baseline loss for outputs out [M][A']."""
    M = out.shape[0]
    A = 6 * w["n_servers"]
    l = out[:, :A]
    v = out[:, A] if w["value_head"] else np.zeros(M)
    m = l.max(axis=1, keepdims=True)
    ex = np.exp(l - m)
    S = ex.sum(axis=1, keepdims=True)
    p = ex / S
    logp_all = (l - m) - np.log(S)
    logp = logp_all[np.arange(M), act]
    H = -(p * logp_all).sum(axis=1)
    L_pi = -(adv * logp).mean()
    L_v = c_v * ((v - ret) ** 2).mean()
    L_h = -c_h * H.mean()
    # d(-A log p_a)/dl_j = -A (1[j=a] - p_j)
    dl = (adv / M)[:, None] * p
    dl[np.arange(M), act] -= adv / M
    dl += (c_h / M) * p * (logp_all + H[:, None])
    dout = np.zeros_like(out)
    dout[:, :A] = dl
    if w["value_head"]:
        dout[:, A] = 2.0 * c_v * (v - ret) / M
    return dict(loss=L_pi + L_v + L_h, policy=L_pi, value=L_v, entropy=L_h), dout


def minibatch_grad(w, wts, seed, obs_t, act_t, logp_t, adv_t, ret_t, M, algo, clip=0.2,
                   c_v=0.5, c_h=0.01):
    """One minibatch's loss terms and gradients for either algorithm."""
    if algo == ALGO_PPO:
        losses, g, _ = ppo.minibatch_grad(w, wts, seed, obs_t, act_t, logp_t, adv_t, ret_t, M,
                                          clip, c_v, c_h)
        return losses, g
    T, E = act_t.shape
    ti, ei = ppo.sample_indices(seed, M, T, E)
    x = obs_t[ti, :, ei].astype(np.float64)
    fw = ppo.forward(w, wts, x)
    losses, dout = reinforce_loss_and_dout(w, fw["out"], act_t[ti, ei].astype(np.int64),
                                           adv_t[ti, ei], ret_t[ti, ei], c_v, c_h)
    return losses, ppo.backward(w, wts, fw, dout)


def adam_step(p, g, m, v, t, lr, b1=0.9, b2=0.999, eps=1e-8):
    """In place on fp64 arrays; t is the 1-based step count after this step."""
    m *= b1
    m += (1.0 - b1) * g
    v *= b2
    v += (1.0 - b2) * g * g
    mhat = m / (1.0 - b1 ** t)
    vhat = v / (1.0 - b2 ** t)
    p -= lr * mhat / (np.sqrt(vhat) + eps)


def policy_weights(w, master):
    """The policy's weights from fp64 master parameters: matrices rounded to the element type
    through fp32 (bf16 by round-to-nearest-even), biases to fp32."""
    out = {}
    for k in PARAM_KEYS:
        a = np.asarray(master[k], np.float64)
        if k.startswith("w") and w["mlp_bf16"]:
            out[k] = ppo.bf16r(a)
        else:
            out[k] = a.astype(np.float32).astype(np.float64)
    return out


def update(w, master, adam, seed, obs_t, act_t, logp_t, adv_t, ret_t, algo, epochs,
           n_minibatches, M, lr, clip=0.2, c_v=0.5, c_h=0.01, b1=0.9, b2=0.999, eps=1e-8):
    """epochs x n_minibatches gradient + Adam steps. master: dict of fp64 arrays (updated in
    place); adam: dict with 'm', 'v' (dicts like master) and 't' (int, updated in place).
    Returns the per-minibatch loss terms [steps][4] (total, policy, value, entropy)."""
    losses = []
    for e in range(epochs):
        for b in range(n_minibatches):
            wts = policy_weights(w, master)
            lo, g = minibatch_grad(w, wts, minibatch_seed(seed, e, n_minibatches, b), obs_t,
                                   act_t, logp_t, adv_t, ret_t, M, algo, clip, c_v, c_h)
            adam["t"] += 1
            for k in PARAM_KEYS:
                adam_step(master[k], g[k], adam["m"][k], adam["v"][k], adam["t"], lr, b1, b2,
                          eps)
            losses.append([lo["loss"], lo["policy"], lo["value"], lo["entropy"]])
    return np.array(losses)
