"""The layer-by-layer policy check (tests/policy_check.py) on the CPU: it accepts a numpy
emulation of what the policy kernels compute (fp32 sums, the kernels' GELU forms, bf16
round-to-nearest-even) and rejects plausible kernel mistakes at every configuration's shape:
a sigmoid-form GELU, hidden activations left unrounded, a dropped hidden unit, a bias read one
unit off. It also pins the bf16 kernel's fitted GELU to the error bound the check assumes.
The attention policy's check accepts an fp32 evaluation of the network and rejects one with
the tanh form of GELU."""
import numpy as np
import pytest

import math

import policy_check as pc
from workloads import attn_preset, preset
from workloads.gen import seeded_obs, seeded_weights_f32

NAMES = ["C1", "C2", "C3", "C4", "C5"]


def f32(x):
    return np.asarray(x, np.float64).astype(np.float32)


def fitted_gelu_f32(x):
    """The bf16 kernel's GELU, max(x, 0) - |x| 2^q(|x|) with q a fitted degree-5 polynomial
    (q(t) ~ log2 Phi(-t)), evaluated step by step in fp32 (each fma and the exp2 rounded once
    to fp32)."""
    x = f32(x)
    t = np.abs(np.float64(x))
    c = [np.float64(np.float32(v)) for v in (-0.00047566284774802625, 0.007099142298102379,
                                              -0.051859911531209946, -0.45996034145355225,
                                              -1.150801420211792, -1.0000358819961548)]
    q = f32(c[0] * t + c[1])
    for ck in c[2:]:
        q = f32(np.float64(q) * t + ck)
    e = f32(np.exp2(np.float64(q)))
    return f32(-t * np.float64(e) + np.maximum(np.float64(x), 0.0))


def erf_gelu_f32(x):
    from scipy.special import erf
    x = f32(x)
    return f32(np.float32(0.5) * x * f32(np.float32(1.0) + f32(erf(np.float64(f32(x * np.float32(0.70710678)))))))


def sigmoid_gelu_f32(x):
    x = f32(x)
    return f32(x / f32(1.0 + np.exp(-1.702 * np.float64(x))))


def weights(w, seed):
    dims = [w["obs_dim"], w["mlp_h1"], w["mlp_h2"], 6 * w["n_servers"] + w["value_head"]]
    W = seeded_weights_f32(seed, dims, bf16=bool(w["mlp_bf16"]))
    return {k: v.astype(np.float64) for k, v in W.items()}


def emulate(w, W, obs, act="kernel", round_hidden=True, drop_unit=None, bias_shift=False):
    """What a policy kernel returns: (h1, h2, outputs) as fp64 copies."""
    bf = bool(w["mlp_bf16"])
    g = {"kernel": fitted_gelu_f32 if bf else erf_gelu_f32, "sigmoid": sigmoid_gelu_f32}[act]
    a = f32(obs)
    if bf:
        a = f32(pc.bf16_rne(a))
    hs = []
    for l in (1, 2):
        b = W[f"b{l}"]
        if bias_shift:
            b = np.roll(b, 1)
        z = a @ f32(W[f"w{l}"]) + f32(b)
        h = g(z)
        if bf and round_hidden:
            h = f32(pc.bf16_rne(h))
        hs.append(np.float64(h))
        a = h
    W3 = W["w3"].copy()
    if drop_unit is not None:
        W3[drop_unit] = 0.0
    out = a @ f32(W3) + f32(W["b3"])
    return hs[0], hs[1], np.float64(out)


def test_fitted_gelu_within_bound():
    """Every fp32 input in [-16, 16] on a grid of 2^-12, 10^6 random ones and magnitudes up to
    10^30: the kernel's fitted GELU is within the bound the check assumes (EPS_GELU_BF16 plus
    two fp32 ulps of the result: the kernel's evaluation in fp32 rounds the final value)."""
    rng = np.random.default_rng(3)
    big = np.geomspace(16.0, 1e30, 10 ** 4)
    x = np.concatenate([np.arange(-16.0, 16.0, 2.0 ** -12), rng.standard_normal(10 ** 6) * 3.0,
                        big, -big])
    x = np.float64(f32(x))
    g = pc.gelu(x)
    err = np.abs(np.float64(fitted_gelu_f32(x)) - g)
    assert np.all(err <= pc.EPS_GELU_BF16 + 2.0 * pc.U * np.abs(g)), (err.max(), x[err.argmax()])


def test_fitted_gelu_bound_rejects_the_previous_fit():
    """The bound is tight enough to reject a GELU that is good to 2.6e-5 (the logistic form
    x / (1 + 2^(x p(x^2))) with a fitted quadratic p)."""
    x = f32(np.arange(-8.0, 8.0, 2.0 ** -10))
    x2 = np.minimum(f32(x * x), np.float32(64.0))
    p = f32(np.float64(np.float32(0.001014263)) * x2 + np.float64(np.float32(-0.10677572)))
    p = f32(np.float64(p) * x2 + np.float64(np.float32(-2.3011212)))
    e = f32(np.exp2(np.float64(f32(x * p))))
    old = np.float64(f32(x * f32(1.0 / np.float64(f32(np.float32(1.0) + e)))))
    g = pc.gelu(np.float64(x))
    assert np.any(np.abs(old - g) > pc.EPS_GELU_BF16 + 2.0 * pc.U * np.abs(g))


@pytest.mark.parametrize("name", NAMES)
def test_check_accepts_the_kernel_arithmetic(orc, name):
    w = preset(name)
    W = weights(w, 11)
    obs = seeded_obs(5, 400, w["obs_dim"])
    h1, h2, out = emulate(w, W, obs)
    amb = pc.check_layers(w, W, obs, h1, h2, out)
    ref = orc.policy(w, W, 1, 0, obs, np.arange(400))
    tol = pc.end_to_end_bound(w, W, obs)
    assert np.all(np.abs(out - ref["logits"]) <= tol)
    units = 400 * (w["mlp_h1"] + w["mlp_h2"])
    assert amb < 0.75 * units, f"{amb} of {units} units admit two values"


MUTANTS = {
    "sigmoid_gelu": dict(act="sigmoid"),
    "hidden_unrounded": dict(round_hidden=False),
    "dropped_unit": dict(drop_unit=5),
    "bias_off_by_one": dict(bias_shift=True),
}


@pytest.mark.parametrize("name", NAMES)
@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_check_rejects_kernel_mistakes(name, mutant):
    w = preset(name)
    if mutant == "hidden_unrounded" and not w["mlp_bf16"]:
        pytest.skip("fp32 configurations do not round hidden activations")
    W = weights(w, 11)
    obs = seeded_obs(5, 400, w["obs_dim"])
    h1, h2, out = emulate(w, W, obs, **MUTANTS[mutant])
    with pytest.raises(AssertionError):
        pc.check_layers(w, W, obs, h1, h2, out)


ATTN = {
    "attn": dict(),
    "attn_L1": dict(attn_tokens=1),
    "attn_L4_H4": dict(attn_tokens=4, attn_heads=4),
    "attn_L2_H1": dict(attn_tokens=2, attn_heads=1),
    "attn_K4": dict(n_servers=4, obs_dim=2 + 16 + 6, n_classes=1, attn_tokens=8),
}


def attn_weights(orc, w, seed):
    rng = np.random.default_rng(seed)
    return {k: (rng.standard_normal(sh) * (0.6 if k.startswith("w") else 0.2)).astype(np.float32)
            .astype(np.float64) for k, sh in orc.attn_shapes(w).items()}


def attn_forward_f32(w, W, x, tanh_gelu=False):
    """The attention policy evaluated in fp32 throughout (numpy float32 arithmetic)."""
    from scipy.special import erf
    f = np.float32
    x = np.asarray(x, f)
    W = {k: np.asarray(v, f) for k, v in W.items()}
    M, F = x.shape
    L, D, NH = w["attn_tokens"], w["attn_embed"], w["attn_heads"]
    G, dh = F // L, D // NH
    e = np.einsum("mlg,lgd->mld", x.reshape(M, L, G), W["w_in"].reshape(L, G, D)) + W["b_in"]
    qkv = e @ W["w_qkv"] + W["b_qkv"]
    q, k, v = qkv[..., :D], qkv[..., D:2 * D], qkv[..., 2 * D:]
    o = np.zeros((M, L, D), f)
    for h in range(NH):
        c = slice(h * dh, (h + 1) * dh)
        s = np.einsum("mgt,mjt->mgj", q[..., c], k[..., c]) / f(math.sqrt(dh))
        ex = np.exp(s - s.max(axis=2, keepdims=True))
        o[..., c] = np.einsum("mgj,mjt->mgt", ex / ex.sum(axis=2, keepdims=True), v[..., c])
    p = (o @ W["w_o"] + W["b_o"]).mean(axis=1)

    def g(z):
        if tanh_gelu:
            return f(0.5) * z * (f(1) + np.tanh(f(0.7978845608) * (z + f(0.044715) * z * z * z)))
        return f(0.5) * z * (f(1) + erf(z.astype(np.float64) / math.sqrt(2.0)).astype(f))
    cols = [g(p @ W["wp1"] + W["bp1"]) @ W["wp2"] + W["bp2"]]
    if w["value_head"]:
        cols.append(g(p @ W["wv1"] + W["bv1"]) @ W["wv2"] + W["bv2"])
    return np.concatenate(cols, axis=1).astype(np.float64)


@pytest.mark.parametrize("name", sorted(ATTN))
def test_attention_check_accepts_fp32_and_rejects_tanh_gelu(orc, name):
    from oracle import attn as oa
    w = attn_preset(**ATTN[name])
    W = attn_weights(orc, w, 99)
    obs = seeded_obs(21, 1000, w["obs_dim"])
    ref = oa.forward(w, W, obs)["out"]
    tol = pc.attn_tol(w, W, obs)
    pc.check_attn_logits(np.abs(attn_forward_f32(w, W, obs) - ref), tol)
    with pytest.raises(AssertionError):
        pc.check_attn_logits(np.abs(attn_forward_f32(w, W, obs, tanh_gelu=True) - ref), tol)
