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
