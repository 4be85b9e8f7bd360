"""Layer-by-layer parity check of the policy MLP kernels (paper Sec. 4.2) -- test helper.

The kernel hands each hidden layer's activations to the next layer; its diagnostic variant
(sim_policy_hidden) also writes them out. Given the kernel's own input to a layer, the layer's
exact result is fixed by fp64 arithmetic on the same values; what a correct kernel may return
differs from it only by

* fp32 accumulation: a sum of n terms taken in any order with fp32 roundings (or with a
  truncating adder) is within 2 n u sum|terms| of the exact sum, u = 2^-24;
* the kernel's GELU: within EPS_GELU_BF16 plus two fp32 ulps of the result (the bf16 kernel's
  fitted form) or within a few fp32 ulps of the exact value (the fp32 kernel's erff form);
* for bf16 configurations, the round-to-nearest-even to bf16 that follows, which is monotone:
  every value in [lo, hi] rounds into [bf16(lo), bf16(hi)].

So each unit admits one bf16 value, or two or three adjacent ones when the exact value lies
within the error window of a rounding boundary. A kernel that skips the rounding, evaluates
a different GELU, mis-indexes a bias or drops a unit produces values outside these sets. The
last layer (logits, value) is checked the same way with no GELU and no rounding.

`end_to_end_bound` propagates the same windows from the oracle's exact inputs through all
layers: a bound on |kernel logit - oracle logit| for sizing the band in which sampled actions
may legitimately differ.

The attention policy (fp32) is checked on its outputs: a forward error analysis bounds every
output (`attn_tol`), and `check_attn_logits` also bounds the average error-to-bound ratio.
"""
import numpy as np
from scipy.special import erf

U = 2.0 ** -24
EPS_GELU_BF16 = 2.0 ** -20   # the bf16 kernel's fitted GELU: absolute part of its bound
GELU_SLOPE = 1.13            # max |GELU'| (1.1289 at x = sqrt(2))


def gelu(z):
    return 0.5 * z * (1.0 + erf(z / np.sqrt(2.0)))


def f32(x):
    return np.asarray(x, np.float64).astype(np.float32).astype(np.float64)


def bf16_rne(x):
    """fp64 -> fp32 (nearest) -> bf16 (nearest even), returned as fp64."""
    f = np.asarray(x, np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def is_bf16(x):
    return np.all((np.asarray(x, np.float32).view(np.uint32) & 0xFFFF) == 0)


def _acc_err(a, W, b):
    """Bound on the fp32 accumulation error of a @ W + b, per output."""
    n = a.shape[1] + 1
    return 2.0 * n * U * (np.abs(a) @ np.abs(W) + np.abs(b))


def _gelu_err(z, g, bf16):
    if bf16:
        return EPS_GELU_BF16 + 2.0 * U * np.abs(g)
    # fp32 0.5 x (1 + erff(x / sqrt 2)): a few roundings of the product and the argument
    return 8.0 * U * (np.abs(z) + z * z + np.abs(g)) + 1e-38


def hidden_window(a_in, W, b, bf16):
    """Lowest and highest value a correct kernel may write for each unit of GELU(a W + b),
    given the layer input a_in [n][K] exactly as the kernel used it."""
    z = a_in @ W + b
    g = gelu(z)
    d = GELU_SLOPE * _acc_err(a_in, W, b) + _gelu_err(z, g, bf16)
    lo, hi = g - d, g + d
    if bf16:
        return bf16_rne(lo), bf16_rne(hi)
    # fp32 result: one more rounding of the final value
    return lo - np.abs(lo) * U - 1e-38, hi + np.abs(hi) * U + 1e-38


def check_layers(w, W, obs, h1, h2, logits):
    """Assert the kernel's activations h1 [n][H1], h2 [n][H2] and outputs logits [n][A'] (all
    fp64 copies of the kernel's values) against the windows above. Returns the number of
    units that admitted more than one value (for reporting)."""
    bf = bool(w["mlp_bf16"])
    x = np.asarray(obs, np.float32).astype(np.float64)
    x = bf16_rne(x) if bf else x
    amb = 0
    for name, a_in, Wk, bk, h in (("h1", x, W["w1"], W["b1"], h1), ("h2", h1, W["w2"], W["b2"], h2)):
        if bf:
            assert is_bf16(h), f"{name}: values that are not bf16 (rounding skipped)"
        lo, hi = hidden_window(a_in, Wk, bk, bf)
        bad = (h < lo) | (h > hi)
        assert not bad.any(), (f"{name}: {int(bad.sum())} of {bad.size} units outside their "
                               f"window, first at {np.argwhere(bad)[0]}: {h[bad][0]} not in "
                               f"[{lo[bad][0]}, {hi[bad][0]}]")
        amb += int(np.sum(lo != hi)) if bf else 0
    z = h2 @ W["w3"] + W["b3"]
    d = _acc_err(h2, W["w3"], W["b3"]) + np.abs(z) * U + 1e-38
    err = np.abs(logits - z)
    bad = err > d
    assert not bad.any(), (f"outputs: {int(bad.sum())} of {bad.size} off by more than the "
                           f"accumulation bound, worst {np.max(err / d):.3g}x")
    return amb


def end_to_end_bound(w, W, obs):
    """Bound on |kernel output - exact output| per output for the oracle's own (exact) forward:
    the hidden windows carried through the layers (every admitted value of a unit differs from
    the oracle's by at most the window width plus the oracle's own rounding offset)."""
    bf = bool(w["mlp_bf16"])
    rnd = bf16_rne if bf else (lambda v: v)
    x = np.asarray(obs, np.float32).astype(np.float64)
    x = bf16_rne(x) if bf else x
    a, da = x, np.zeros_like(x)
    for Wk, bk in ((W["w1"], W["b1"]), (W["w2"], W["b2"])):
        z = a @ Wk + bk
        dz = da @ np.abs(Wk)
        g = gelu(z)
        d = GELU_SLOPE * (dz + _acc_err(a, Wk, bk)) + _gelu_err(z, g, bf)
        lo, hi = rnd(g - d), rnd(g + d)
        if not bf:
            lo, hi = lo - np.abs(lo) * U, hi + np.abs(hi) * U
        h = rnd(g)
        da = np.maximum(h - lo, hi - h)
        a = h
    z = a @ W["w3"] + W["b3"]
    return da @ np.abs(W["w3"]) + _acc_err(a, W["w3"], W["b3"]) + np.abs(z) * U


# ---- attention policy (fp32) ---------------------------------------------------------------
def attn_tol(w, W, obs):
    """Per-output tolerance of the fp32 attention kernel against the fp64 oracle, from a
    forward error analysis in fp64 over the exact intermediates (u = 2^-24):
    * a fp32 dot product with fma over n terms plus a bias is off by at most (n + 1) u times
      the sum of its terms' magnitudes (local rounding), and an input error e propagates
      as |W|^T e;
    * a score error ds changes the softmax weights by at most 2 max|ds| in L1 (exp, sum and
      the division add (L + 2) u), so the weighted values move by that times max|v| plus the
      weights' average of the values' errors;
    * the mean pool adds L u of the mean magnitude; GELU has slope at most 1.13 and erff is
      good to a few ulps (8 u |z|).
    The tolerance is four times the bound (margin for the first-order treatment); the check
    that uses it (check_attn_logits) also bounds the average ratio of error to tolerance."""
    u = 2.0 ** -24
    x = np.asarray(obs, np.float64)
    n, F = x.shape
    L, D, NH = w["attn_tokens"], w["attn_embed"], w["attn_heads"]
    G, dh = F // L, D // NH
    Wa = {k: np.abs(v) for k, v in W.items()}

    def lin(inp, err, k_w, k_b):
        """value, error of inp @ W + b given inp's error."""
        val = inp @ W[k_w] + W[k_b]
        nt = W[k_w].shape[0]
        e = err @ Wa[k_w] + (nt + 1) * u * (np.abs(inp) @ Wa[k_w] + Wa[k_b])
        return val, e

    xt = x.reshape(n, L, G)
    win = W["w_in"].reshape(L, G, D)
    tok = np.einsum("nlg,lgd->nld", xt, win) + W["b_in"]
    e_tok = (G + 1) * u * (np.einsum("nlg,lgd->nld", np.abs(xt), np.abs(win)) + Wa["b_in"])
    qkv, e_qkv = lin(tok, e_tok, "w_qkv", "b_qkv")
    q, k, v = qkv[..., :D], qkv[..., D:2 * D], qkv[..., 2 * D:]
    eq, ek, ev = e_qkv[..., :D], e_qkv[..., D:2 * D], e_qkv[..., 2 * D:]
    o = np.zeros((n, L, D))
    eo = np.zeros((n, L, D))
    for h in range(NH):
        c = slice(h * dh, (h + 1) * dh)
        sc = np.einsum("ngt,njt->ngj", q[..., c], k[..., c]) / np.sqrt(dh)
        esc = (np.einsum("ngt,njt->ngj", eq[..., c], np.abs(k[..., c])) +
               np.einsum("ngt,njt->ngj", np.abs(q[..., c]), ek[..., c]) +
               (dh + 1) * u * np.einsum("ngt,njt->ngj", np.abs(q[..., c]), np.abs(k[..., c])))
        esc = esc / np.sqrt(dh)
        a = np.exp(sc - sc.max(axis=2, keepdims=True))
        a = a / a.sum(axis=2, keepdims=True)
        ea = 2.0 * esc.max(axis=2) + (L + 2) * u                        # [n][g], L1 over j
        vmax = np.abs(v[..., c]).max(axis=1)                            # [n][t]
        o[..., c] = np.einsum("ngj,njt->ngt", a, v[..., c])
        eo[..., c] = (ea[..., None] * vmax[:, None, :] + np.einsum("ngj,njt->ngt", a, ev[..., c])
                      + L * u * np.einsum("ngj,njt->ngt", a, np.abs(v[..., c])))
    y, ey = lin(o, eo, "w_o", "b_o")
    p = y.mean(axis=1)
    ep = ey.mean(axis=1) + L * u * np.abs(y).mean(axis=1)

    def head(k1, b1, k2, b2):
        z, ez = lin(p, ep, k1, b1)
        hz = 0.5 * z * (1.0 + np.vectorize(__import__("math").erf)(z / np.sqrt(2.0)))
        eh = 1.13 * ez + 8 * u * np.abs(z)
        return lin(hz, eh, k2, b2)[1]

    cols = [head("wp1", "bp1", "wp2", "bp2")]
    if w["value_head"]:
        cols.append(head("wv1", "bv1", "wv2", "bv2"))
    return 4.0 * np.concatenate(cols, axis=1)


ATTN_MEAN_RATIO = 2.0 ** -10


def check_attn_logits(err, tol):
    """Every |kernel - oracle| output difference within its worst-case tolerance, and their
    average ratio to it below ATTN_MEAN_RATIO. The worst-case analysis adds the magnitudes of
    all n terms of every fp32 sum (n u each), while rounding errors of independent steps
    largely cancel (about sqrt(n) u), and it bounds the softmax weights' change by 2 max|ds|;
    an fp32 evaluation of the network therefore lands near 10^-4 of the tolerance on average
    (measured on an emulation, tests/test_policy_check.py). An average far above that is a
    systematic deviation, such as another GELU, rather than rounding."""
    r = np.asarray(err) / np.asarray(tol)
    assert np.all(r <= 1.0), f"max err/tol {r.max():.3g}"
    assert r.mean() <= ATTN_MEAN_RATIO, f"mean err/tol {r.mean():.3g} above {ATTN_MEAN_RATIO:.3g}"
