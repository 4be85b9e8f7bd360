"""PPO minibatch oracle (paper Sec. 4.3, clipped surrogate) -- TEST INFRASTRUCTURE.

One minibatch of M (t, env) samples drawn with replacement from a rollout; forward through
the policy MLP (bf16 rounding points as in the rollout), loss

    L = -mean(min(rho A, clip(rho, 1-eps, 1+eps) A)) + c_v mean((V - R)^2) - c_h mean(H),
    rho = exp(logp_new(a) - logp_old),  H = entropy of the action distribution,

and its exact gradient with respect to every weight and bias in fp64 (the bf16 rounding
of layer inputs is treated as the identity for gradients). Plain numpy, written out step by
step; the sample indices come from the oracle's own Philox draws.
"""
import math

import numpy as np

from . import lib, draw, u01, P_MINIBATCH, _vec  # noqa: F401

STEP_MINIBATCH = 0xFFFFFFFD


def bf16r(x):
    """fp64 -> fp32 -> bf16 (round to nearest even), returned as fp64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def sample_indices(seed, M, T, E):
    """Sample m takes u from the MINIBATCH block at counter (m, STEP_MINIBATCH,
    MINIBATCH<<24, 0); index = floor(u * T * E), so t = index // E, env = index % E."""
    idx = np.empty(M, np.int64)
    n = T * E
    for m in range(M):
        w = draw(seed, m, STEP_MINIBATCH, P_MINIBATCH, 0, 0)
        u = u01(int(w[0]), int(w[1]))
        i = int(u * float(n))
        idx[m] = min(i, n - 1)
    return idx // E, idx % E


def _erf(x):
    return np.vectorize(math.erf)(x)


def gelu(z):
    return 0.5 * z * (1.0 + _erf(z / math.sqrt(2.0)))


def gelu_grad(z):
    """d/dz z Phi(z) = Phi(z) + z phi(z)."""
    return 0.5 * (1.0 + _erf(z / math.sqrt(2.0))) + z * np.exp(-0.5 * z * z) / math.sqrt(2.0 * math.pi)


def forward(w, wts, x):
    """x [M][F] fp32 observations -> dict of pre-activations, activations and outputs."""
    bf = bool(w["mlp_bf16"])
    r = bf16r if bf else (lambda v: np.asarray(v, np.float64))
    x0 = r(x)
    z1 = x0 @ wts["w1"] + wts["b1"]
    h1 = r(gelu(z1))
    z2 = h1 @ wts["w2"] + wts["b2"]
    h2 = r(gelu(z2))
    out = h2 @ wts["w3"] + wts["b3"]
    return dict(x=x0, z1=z1, h1=h1, z2=z2, h2=h2, out=out)


def loss_and_dout(w, out, act, logp_old, adv, ret, clip=0.2, c_v=0.5, c_h=0.01):
    """Loss terms and dL/d(out) for outputs out [M][A'] (logits then value)."""
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
    rho = np.exp(logp - logp_old)
    clipped = np.clip(rho, 1.0 - clip, 1.0 + clip)
    s1, s2 = rho * adv, clipped * adv
    surr = np.minimum(s1, s2)
    H = -(p * logp_all).sum(axis=1)
    L_pi = -surr.mean()
    L_v = c_v * ((v - ret) ** 2).mean()
    L_h = -c_h * H.mean()
    # d surr / d rho: A where the unclipped term is the minimum, A * 1[inside] otherwise
    inside = (rho > 1.0 - clip) & (rho < 1.0 + clip)
    g_rho = np.where(s1 <= s2, adv, adv * inside)
    d_logp = -g_rho * rho / M
    dl = -d_logp[:, None] * p
    dl[np.arange(M), act] += d_logp
    # entropy: dH/dl_j = -p_j (log p_j + H); L has -c_h H / M
    dl += (c_h / M) * p * (logp_all + H[:, None])
    dout = np.zeros_like(out)
    dout[:, :A] = dl
    if w["value_head"]:
        dout[:, A] = 2.0 * c_v * (v - ret) / M
    return dict(loss=L_pi + L_v + L_h, policy=L_pi, value=L_v, entropy=L_h), dout


def backward(w, wts, fw, dout):
    """Gradients of the loss with respect to W1,b1,W2,b2,W3,b3 ([in][out] like the weights)."""
    g = {}
    g["w3"] = fw["h2"].T @ dout
    g["b3"] = dout.sum(axis=0)
    dz2 = (dout @ wts["w3"].T) * gelu_grad(fw["z2"])
    g["w2"] = fw["h1"].T @ dz2
    g["b2"] = dz2.sum(axis=0)
    dz1 = (dz2 @ wts["w2"].T) * gelu_grad(fw["z1"])
    g["w1"] = fw["x"].T @ dz1
    g["b1"] = dz1.sum(axis=0)
    return g


def minibatch_grad(w, wts, seed, obs_t, act_t, logp_t, adv_t, ret_t, M, clip=0.2, c_v=0.5,
                   c_h=0.01, obs_of=None):
    """Full minibatch: indices, gather, forward, loss, gradients.
    obs_t [T][F][E] (or obs_of(t, e) -> [F]), act_t/logp_t/adv_t/ret_t [T][E]."""
    T, E = act_t.shape
    ti, ei = sample_indices(seed, M, T, E)
    if obs_of is None:
        x = obs_t[ti, :, ei].astype(np.float64)
    else:
        x = np.stack([obs_of(t, e) for t, e in zip(ti, ei)])
    fw = forward(w, wts, x)
    losses, dout = loss_and_dout(w, fw["out"], act_t[ti, ei].astype(np.int64),
                                 logp_t[ti, ei].astype(np.float64), adv_t[ti, ei], ret_t[ti, ei],
                                 clip, c_v, c_h)
    return losses, backward(w, wts, fw, dout), (ti, ei)
