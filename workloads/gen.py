"""Seeded synthetic input generators (numpy PCG64). No method arithmetic lives here."""
import numpy as np


def seeded_actions(seed, T, n_envs, n_actions, small_bias=0.0):
    """Actions [T][E] uint8 uniform over [0, n_actions). With small_bias > 0, that
    fraction of draws is instead restricted to batch sizes 1..4 (keeps queues moving)."""
    rng = np.random.default_rng(seed)
    a = rng.integers(0, n_actions, size=(T, n_envs), dtype=np.int64)
    if small_bias > 0.0:
        servers = n_actions // 6
        m = rng.random((T, n_envs)) < small_bias
        small = rng.integers(0, servers, size=(T, n_envs)) * 6 + rng.integers(0, 3, size=(T, n_envs))
        a = np.where(m, small, a)
    return a.astype(np.uint8)


def seeded_obs(seed, n, F):
    """Observation-like fp32 rows [n][F]: fractions in [0,1], a few ages up to ~3,
    binary flags, zero tail padding is not imposed."""
    rng = np.random.default_rng(seed)
    x = rng.random((n, F)).astype(np.float64)
    x[:, 1::5] *= 3.0
    x[:, 2::7] = (x[:, 2::7] > 0.5)
    return x.astype(np.float32)


def seeded_rewards_values(seed, T, n, value=True):
    """Rewards [T][n] f64 (throughput-like positive mass minus latency-like terms) and
    values [T+1][n] f32."""
    rng = np.random.default_rng(seed)
    r = np.where(rng.random((T, n)) < 0.4, 10.0 * rng.integers(1, 33, size=(T, n)), 0.0)
    r = r - rng.exponential(0.5, size=(T, n))
    v = (rng.standard_normal((T + 1, n)) * 50.0).astype(np.float32) if value else None
    return r, v


def seeded_weights_f32(seed, dims, bf16=False):
    """Random fp32 weights/biases for layer dims [F, H1, H2, A']; bf16=True rounds weights
    to bf16-representable values (truncation of the low 16 bits)."""
    rng = np.random.default_rng(seed)
    out = {}
    for l in range(3):
        fi, fo = dims[l], dims[l + 1]
        w = (rng.standard_normal((fi, fo)) / np.sqrt(fi)).astype(np.float32)
        if bf16:
            w = (w.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)
        out[f"w{l + 1}"] = w
        out[f"b{l + 1}"] = (rng.standard_normal(fo) * 0.1).astype(np.float32)
    return out


def hashed_u24(salt, t, f, e):
    """24-bit integers from a multiplicative hash of (salt, t, f, e); works on numpy int64
    arrays and on torch int64 tensors alike (only +, *, &, >> on values below 2^63), so a
    device-side fill and a host-side lookup of single entries give the same numbers."""
    s = (t * 1000003 + f * 7919 + e * 104729 + salt * 15485863) & 0xFFFFFFFF
    return ((s * 0x5BD1E995) >> 7) & 0xFFFFFF


def ppo_inputs_at(salt, t, e, n_actions):
    """Stored-rollout stand-ins at positions (t, e): action (uint8), advantage and return
    (fp64, exact dyadic values). Same formulas on numpy or torch int64 inputs."""
    def f64(h):
        return h.double() if hasattr(h, "double") else np.asarray(h, dtype=np.float64)
    act = hashed_u24(salt, t, 0, e) % n_actions
    adv = (f64(hashed_u24(salt + 1, t, 0, e)) * 2.0 ** -24 - 0.5) * 8.0
    ret = (f64(hashed_u24(salt + 2, t, 0, e)) * 2.0 ** -24 - 0.5) * 4.0
    return act, adv, ret


def ratio_offsets(seed, n, lo=-0.5, hi=0.5, avoid=(), gap=0.01):
    """Log-ratio offsets d in [lo, hi] (fp64) kept at least `gap` away from every value in
    `avoid` (values that fall inside a gap are moved to its upper edge plus `gap`)."""
    rng = np.random.default_rng(seed)
    d = rng.uniform(lo, hi, size=n)
    for a in avoid:
        near = np.abs(d - a) < gap
        d[near] = a + 2.0 * gap
    return d
