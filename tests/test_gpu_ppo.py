"""GPU parity of the PPO minibatch (Sec. 4.3) through the C ABI against oracle/ppo.py.

Sample indices are compared bit for bit. Loss and gradients are compared within a
tolerance derived from the rounding points: the GPU forward runs in fp32 with the layer
inputs rounded to bf16 (bf16 mode), the oracle in fp64 with the same rounding points, so
an activation whose two pre-rounding images straddle a bf16 rounding boundary rounds one
bf16 ulp (2^-8 relative) apart. Such flips hit about (fp32 relative error ~ 2^-16) /
(bf16 spacing 2^-8) = 2^-8 of the activations, so the activations of a sample move by
about sqrt(2^-8) * 2^-8 = 2^-12 relative in norm and the gradients, sums of per-sample
products, by about as much: the norm bound is 2^-9 (a factor of 8 margin) and the
elementwise bound 2^-8 of the tensor's largest entry. fp32 mode differs only in fp32
rounding (sums of at most 64 terms over three layers, erf/exp to an ulp or two: about
2^-16 relative per sample), summed over the M <= 4096 samples of the parity cases in fp32
GEMMs (sign-mixed sums whose rounding error grows about as sqrt(M) u, about 2^-18): 2^-13 for
both bounds (a factor of 8 margin). The clip decision of the surrogate is taken away from its
boundaries by construction: logp_old = logp_new - d with |d - ln(1 +- clip)| >= 0.01, far
beyond any logit difference the tolerances allow."""
import sys

import numpy as np
import pytest

from oracle import ppo as orc_ppo
from workloads import preset
from workloads.gen import hashed_u24, ppo_inputs_at, ratio_offsets, seeded_obs, seeded_weights_f32

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CLIP, C_V, C_H = 0.2, 0.5, 0.01
AVOID = (np.log(1.0 - CLIP), np.log(1.0 + CLIP))


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def bs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_05272_amd as m
    m.load()
    return m


def workload(name, **kw):
    w = preset(name, **kw)
    w["value_head"] = 1
    return w


def weights_for(w, seed):
    Ap = 6 * w["n_servers"] + 1
    return seeded_weights_f32(seed, [w["obs_dim"], w["mlp_h1"], w["mlp_h2"], Ap],
                              bf16=bool(w["mlp_bf16"]))


def oracle_logp(w, wts, x, act):
    """log pi(act | x) from the oracle forward (fp64)."""
    out = orc_ppo.forward(w, {k: v.astype(np.float64) for k, v in wts.items()}, x)["out"]
    A = 6 * w["n_servers"]
    l = out[:, :A]
    m = l.max(axis=1, keepdims=True)
    lse = np.log(np.exp(l - m).sum(axis=1)) + m[:, 0]
    return l[np.arange(len(act)), act] - lse


def check_grads(w, got_g, got_loss, ref_loss, ref_g, what):
    bf = bool(w["mlp_bf16"])
    tn, te = (2.0 ** -9, 2.0 ** -8) if bf else (2.0 ** -13, 2.0 ** -13)
    worst = 0.0
    for k in ("w1", "b1", "w2", "b2", "w3", "b3"):
        G = ref_g[k]
        g = got_g[k].astype(np.float64)
        assert g.shape == G.shape, (k, g.shape, G.shape)
        nG = np.linalg.norm(G)
        d = np.linalg.norm(g - G)
        e = np.max(np.abs(g - G))
        mx = np.max(np.abs(G))
        say(f"  {what} {k}: |dG|/|G| {d / max(nG, 1e-300):.3g}  max|dG|/max|G| {e / max(mx, 1e-300):.3g}")
        worst = max(worst, d / max(nG, 1e-300))
        assert d <= tn * nG + 1e-30, f"{k}: norm error {d:.3g} > {tn} * {nG:.3g}"
        assert e <= te * mx + 1e-30, f"{k}: max error {e:.3g} > {te} * {mx:.3g}"
    scale = abs(ref_loss["policy"]) + abs(ref_loss["value"]) + abs(ref_loss["entropy"])
    tl = tn * scale
    for i, k in enumerate(("loss", "policy", "value", "entropy")):
        assert abs(got_loss[i] - ref_loss[k]) <= tl, (k, got_loss[i], ref_loss[k])
    return worst


def run_small(bs, w, T, E, M, seed, wseed=7, obs_seed=11):
    """Host-built inputs at a size the oracle handles entirely."""
    F = w["obs_dim"]
    A = 6 * w["n_servers"]
    x = seeded_obs(obs_seed, T * E, F)                       # row t*E + e
    obs_t = np.ascontiguousarray(x.reshape(T, E, F).transpose(0, 2, 1))   # [T][F][E]
    tt, ee = np.meshgrid(np.arange(T), np.arange(E), indexing="ij")
    act, adv, ret = ppo_inputs_at(5, tt.astype(np.int64), ee.astype(np.int64), A)
    act = act.astype(np.uint8)
    wts = weights_for(w, wseed)
    lp_new = oracle_logp(w, wts, x.astype(np.float64), act.reshape(-1).astype(np.int64))
    d = ratio_offsets(seed + 1, T * E, avoid=AVOID)
    logp_old = (lp_new - d).astype(np.float32).reshape(T, E)
    ref_loss, ref_g, (ti, ei) = orc_ppo.minibatch_grad(
        w, {k: v.astype(np.float64) for k, v in wts.items()}, seed, obs_t, act, logp_old,
        adv, ret, M, CLIP, C_V, C_H)
    sim = bs.Sim(w, n_envs=E)
    dev = torch.device("cuda")
    wb = sim.upload_weights(wts)
    g, loss, idx = sim.ppo_minibatch_grad(
        wb, torch.from_numpy(obs_t).to(dev), torch.from_numpy(act).to(dev),
        torch.from_numpy(logp_old).to(dev), torch.from_numpy(adv).to(dev),
        torch.from_numpy(ret).to(dev), M, seed, CLIP, C_V, C_H, want_index=True)
    sim.sync()
    got_g = sim.unflatten_grads(g.cpu().numpy())
    got_loss = loss.cpu().numpy()
    got_idx = idx.cpu().numpy()
    sim.close()
    assert np.array_equal(got_idx, ti * E + ei), "sample indices differ"
    return check_grads(w, got_g, got_loss, ref_loss, ref_g, f"T={T} E={E} M={M}")


# shapes of every compiled policy size, fp32 (8-64-64) and bf16 (32/64/96 inputs, 128/256/512
# wide)
SMALL = [("C1", 7, 300, 1024), ("C2", 9, 257, 2048), ("C3", 5, 611, 2048), ("C4", 13, 640, 4096),
         ("C5", 3, 700, 2048)]


@pytest.mark.parametrize("name,T,E,M", SMALL)
def test_ppo_minibatch_parity(bs, name, T, E, M):
    say(f"[ppo] {name} T={T} E={E} M={M}")
    run_small(bs, workload(name), T, E, M, seed=0xC0FFEE + T)


def test_ppo_edge_single_position(bs):
    """T = E = 1: every sample is the same (t, env); one workgroup (M = 16)."""
    say("[ppo] edge T=E=1 M=16")
    run_small(bs, workload("C1"), 1, 1, 16, seed=3)


def test_ppo_full_size_c4_sampled(bs):
    """C4 at its full size (65536 environments x 1024 steps, 8192 samples): inputs filled
    on the device from the hashed generator; the oracle evaluates the sampled positions."""
    w = workload("C4")
    T, E, M, F = w["T"], w["n_envs"], w["ppo_minibatch"], w["obs_dim"]
    A = 6 * w["n_servers"]
    seed = 0xA13
    say(f"[ppo] full size C4 T={T} E={E} M={M}")
    dev = torch.device("cuda")
    ti, ei = orc_ppo.sample_indices(seed, M, T, E)
    # observations [T][F][E]: u24 * 2^-24, filled one time step at a time
    obs = torch.empty((T, F, E), dtype=torch.float32, device=dev)
    fr = torch.arange(F, dtype=torch.int64, device=dev)[:, None]
    er = torch.arange(E, dtype=torch.int64, device=dev)[None, :]
    for t in range(T):
        obs[t] = (hashed_u24(17, torch.tensor(t, dtype=torch.int64, device=dev), fr, er)
                  .to(torch.float64) * 2.0 ** -24).to(torch.float32)
    tr = torch.arange(T, dtype=torch.int64, device=dev)[:, None]
    act_d, adv_d, ret_d = ppo_inputs_at(5, tr, er, A)
    act_d = act_d.to(torch.uint8)
    x = (hashed_u24(17, ti[:, None], np.arange(F)[None, :], ei[:, None]).astype(np.float64)
         * 2.0 ** -24).astype(np.float32)                   # sampled rows [M][F]
    act_s, adv_s, ret_s = ppo_inputs_at(5, ti, ei, A)
    wts = weights_for(w, 8)
    W64 = {k: v.astype(np.float64) for k, v in wts.items()}
    lp_new = oracle_logp(w, wts, x.astype(np.float64), act_s)
    # one offset per distinct position (samples repeat), keyed by the flat index
    flat = ti * E + ei
    uniq, inv = np.unique(flat, return_inverse=True)
    d = ratio_offsets(seed, len(uniq), avoid=AVOID)[inv]
    lp_old_s = (lp_new - d).astype(np.float32)
    logp_old = torch.full((T, E), -4.0, dtype=torch.float32, device=dev)
    logp_old.view(-1)[torch.from_numpy(flat).to(dev)] = torch.from_numpy(lp_old_s).to(dev)
    ref_loss, dout = orc_ppo.loss_and_dout(w, orc_ppo.forward(w, W64, x)["out"], act_s,
                                           lp_old_s.astype(np.float64), adv_s, ret_s, CLIP, C_V, C_H)
    ref_g = orc_ppo.backward(w, W64, orc_ppo.forward(w, W64, x), dout)
    sim = bs.Sim(w, n_envs=E)
    wb = sim.upload_weights(wts)
    g, loss, idx = sim.ppo_minibatch_grad(wb, obs, act_d, logp_old, adv_d, ret_d, M, seed,
                                          CLIP, C_V, C_H, want_index=True)
    sim.sync()
    assert np.array_equal(idx.cpu().numpy(), flat), "sample indices differ"
    check_grads(w, sim.unflatten_grads(g.cpu().numpy()), loss.cpu().numpy(), ref_loss, ref_g,
                "C4 full")
    sim.close()
    del obs


def test_ppo_gradient_is_deterministic(bs):
    """Two calls on the same inputs return bit-identical gradients and losses (the GEMM library
    runs with atomics disabled, every other sum has a fixed order); M = 2064 leaves a partial
    workgroup in the gather."""
    w = workload("C3")
    T, E, M = 5, 611, 2064
    A = 6 * w["n_servers"]
    say(f"[ppo] determinism C3 M={M}")
    dev = torch.device("cuda")
    x = seeded_obs(11, T * E, w["obs_dim"])
    obs = torch.from_numpy(np.ascontiguousarray(x.reshape(T, E, -1).transpose(0, 2, 1))).to(dev)
    tt, ee = np.meshgrid(np.arange(T), np.arange(E), indexing="ij")
    act, adv, ret = ppo_inputs_at(5, tt.astype(np.int64), ee.astype(np.int64), A)
    act, adv, ret = (torch.from_numpy(v).to(dev) for v in (act.astype(np.uint8), adv, ret))
    lp = torch.full((T, E), -3.0, dtype=torch.float32, device=dev)
    sim = bs.Sim(w, n_envs=E)
    wb = sim.upload_weights(weights_for(w, 4))
    g1, l1, _ = sim.ppo_minibatch_grad(wb, obs, act, lp, adv, ret, M, 99)
    g1, l1 = g1.clone(), l1.clone()
    g2, l2, _ = sim.ppo_minibatch_grad(wb, obs, act, lp, adv, ret, M, 99)
    sim.sync()
    assert torch.equal(g1, g2) and torch.equal(l1, l2)
    assert bool(torch.isfinite(g1).all()) and float(g1.abs().sum()) > 0
    sim.close()


def test_ppo_bad_action_is_latched(bs):
    w = workload("C2")
    T, E, M = 2, 64, 64
    A = 6 * w["n_servers"]
    dev = torch.device("cuda")
    sim = bs.Sim(w, n_envs=E)
    wb = sim.upload_weights(weights_for(w, 1))
    obs = torch.zeros((T, w["obs_dim"], E), dtype=torch.float32, device=dev)
    act = torch.full((T, E), A, dtype=torch.uint8, device=dev)
    z32 = torch.zeros((T, E), dtype=torch.float32, device=dev)
    z64 = torch.zeros((T, E), dtype=torch.float64, device=dev)
    g, loss, _ = sim.ppo_minibatch_grad(wb, obs, act, z32, z64, z64, M, 1)
    with pytest.raises(RuntimeError, match="action out of range"):
        sim.sync()
    assert torch.count_nonzero(g).item() == 0
    sim.close()


def test_ppo_argument_errors(bs):
    w = workload("C2")
    T, E = 2, 64
    dev = torch.device("cuda")
    sim = bs.Sim(w, n_envs=E)
    wb = sim.upload_weights(weights_for(w, 1))
    obs = torch.zeros((T, w["obs_dim"], E), dtype=torch.float32, device=dev)
    act = torch.zeros((T, E), dtype=torch.uint8, device=dev)
    z32 = torch.zeros((T, E), dtype=torch.float32, device=dev)
    z64 = torch.zeros((T, E), dtype=torch.float64, device=dev)
    with pytest.raises(RuntimeError, match="multiple of 16"):
        sim.ppo_minibatch_grad(wb, obs, act, z32, z64, z64, 40, 1)
    with pytest.raises(RuntimeError, match="clip"):
        sim.ppo_minibatch_grad(wb, obs, act, z32, z64, z64, 64, 1, clip=1.5)
    sim.close()
