#!/usr/bin/env python3
"""Throughput of the batched serving-simulator rollout on one MI355X.

One step = one pass of the whole hot path over one synthetic batch: reset every
environment, then T ticks of (policy MLP + action sampling on MFMA, simulator tick of the
learned system and, where configured, of the static shadow system), then returns/GAE
over the trajectory, for workloads with a PPO minibatch (C4) one minibatch gradient over
the stored trajectory, and the device-side reduction of the per-environment counters.
value = environments x ticks per second of wall time (inputs resident in HBM).

Prints one JSON line. Kernel durations come from HIP events recorded by the library on
its own stream around every launch during the timed region.
"""
import argparse
import hashlib
import json
import os
import statistics
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3       # dense fp32 matrix
PEAK_FP32_VALU_TFLOPS = 157.3  # fp32 vector FMA: 256 CUs x 4 SIMD x 2 x 64 lanes x 2.4 GHz

DESCR = {
    "C1": "C1: 256 envs x 1000 ticks, 1 server, Poisson 500/s, DET 5ms+0.5ms*b, obs 8, MLP 8-64-64-6 fp32, REINFORCE returns",
    "C2": "C2: 4096 envs x 2000 ticks, 1 server, MMPP 200/2000 req/s, 2 classes 80/20, obs 12, MLP 12-128-128-6 bf16, REINFORCE returns",
    "C3": "C3: 16384 envs x 2048 ticks, 4 servers, Poisson 3000/s, 2 classes 70/30, obs 32, MLP 32-256-256-24 bf16, GAE",
    "C4": "C4: 65536 envs x 1024 ticks, 8 servers, 3-state MMPP, 4 classes lognormal, obs 64, MLP 64-256-256-48 bf16, GAE",
    "C5": "C5: 262144 envs x 4096 ticks, 16 servers, Pareto ON/OFF bursts 20000/s, 4 classes 50/30/15/5 lognormal, static shadow, obs 96, MLP 96-512-512-96 bf16, GAE",
    "burst": "Extreme Burst: 65536 envs x 1000 ticks, square wave 100 <-> 0 req/s every 200 ticks, 1 server, DET 5ms+0.5ms*b, static shadow (B=32, T=10ms), MLP 8-64-64-6 fp32",
    "C3-static8": "C3 with a Static-8 shadow (fixed batch 8, 10 ms timeout, lowest idle server)",
    "C3-random": "C3 with a static shadow routing each batch to a uniformly random idle server",
    "C3-round_robin": "C3 with a static shadow routing batches round-robin over the idle servers",
    "C5-random": "C5 with the static shadow routing each batch to a uniformly random idle server",
    "C3-shortest": "C3 with a Shortest-Queue shadow: each static-rule batch to the server with the fewest requests assigned (one batch running and at most one queued per server)",
    "attn": "attention policy (Sec. 4.2): 262144 envs x 1000 ticks, C1's system (1 server, Poisson 500/s, DET 5ms+0.5ms*b), 8 features as 8 tokens, 8->4 projection, 2-head self-attention, mean pool, GELU heads of 64 (policy) and 64 (value), fp32, REINFORCE with baseline returns",
}


def workload_of(name):
    """The workload dict of a bench configuration name."""
    from workloads import preset, burst_preset, baseline_preset, attn_preset
    if name == "attn":
        return attn_preset(n_envs=262144, T=1000)
    if name == "burst":
        return burst_preset(n_envs=65536, T=1000)
    if "-" in name:
        base, rule = name.split("-", 1)
        return baseline_preset(rule, base)
    return preset(name)


def mlp_flops(w):
    A1 = 6 * w["n_servers"] + (1 if w["value_head"] else 0)
    return 2 * (w["obs_dim"] * w["mlp_h1"] + w["mlp_h1"] * w["mlp_h2"] + w["mlp_h2"] * A1)


def attn_flops(w):
    """Multiply-adds (x2) of one attention-policy forward (Sec. 4.2): tokens, q/k/v,
    scores and weighted values per head, output projection, both heads."""
    F, L, D, NH = w["obs_dim"], w["attn_tokens"], w["attn_embed"], w["attn_heads"]
    A, Hp, Hv = 6 * w["n_servers"], w["mlp_h1"], w["mlp_h2"]
    dh = D // NH
    mac = (F * D + L * D * 3 * D + 2 * NH * L * L * dh + L * D * D + D * Hp + Hp * A
           + (D * Hv + Hv if w["value_head"] else 0))
    return 2 * mac


def ppo_flops(w):
    """One PPO minibatch: forward, backward through the activations (all but the input
    layer) and the three weight gradients, 2 flops per multiply-add."""
    M = w["ppo_minibatch"]
    F, H1, H2 = w["obs_dim"], w["mlp_h1"], w["mlp_h2"]
    Ap = 6 * w["n_servers"] + 1
    fwd = F * H1 + H1 * H2 + H2 * Ap
    return 2 * M * (fwd + (H1 * H2 + H2 * Ap) + fwd)


def step_bytes(w, tot, E, T):
    """Algorithmic HBM bytes per env-tick of the learned-system kernel: the structure-of-
    arrays state it must read and write, the action, reward and observation, the ring
    entries touched by accepted arrivals and dispatched requests, and the server entries
    rewritten by dispatches (busy + meta) and completions (meta). Inside a rollout with a
    bf16 MLP policy the tick writes the observation as bf16 feature pairs (2 bytes per
    feature; the fp32 observation only on the rollout's last tick), otherwise as fp32."""
    K, C, F = w["n_servers"], w["n_classes"], w["obs_dim"]
    from workloads.presets import POLICY_MLP
    obs_b = 4 * ((F + 1) // 2) if (w["mlp_bf16"] and w["policy_kind"] == POLICY_MLP) else 4 * F
    state_rw = 4 + 4 + 8 * C + 4 * 6 + 16 + 8 + 4 + 8 + 8 + 32   # queues, counters, arrivals, ewma
    fixed = 1 + 2 * state_rw + 12 * K + obs_b + 8                 # + action, servers read, obs, reward
    n = E * T
    c = tot["cnt"][0]
    var = 8.0 * (c[1] + c[3]) / n + 12.0 * c[4] / n + 4.0 * c[4] / n
    return fixed + var


def static_bytes(w, tot, E, T, ticks_per_launch):
    """Algorithmic HBM bytes per environment of one launch of the static shadow kernel,
    which runs `ticks_per_launch` ticks with the state in registers: the state read and
    written once (queues, counters, arrival process, servers), then per tick the reward and
    the ring entries of accepted arrivals and dispatched requests, and per dispatch the
    server's meta word and busy time."""
    K, C = w["n_servers"], w["n_classes"]
    state_rw = 4 + 4 + 8 * C + 4 * 6 + 16 + 8 + 4 + 8 + 8
    n = E * T
    c = tot["cnt"][1]
    per_tick = 8 + 8.0 * (c[1] + c[3]) / n + 12.0 * c[4] / n
    return 2 * state_rw + 12 * K + ticks_per_launch * per_tick


# the source of each kernel class (with the shared device headers)
KERNEL_SOURCE = {"policy": ["mlp_kernels.hip", "policy_dev.hpp"],
                 "step": ["sim_kernels.hip", "sim_dev.hpp"],
                 "static": ["sim_kernels.hip", "sim_dev.hpp"], "gae": ["gae_kernels.hip"],
                 "ppo": ["ppo_kernels.hip"],
                 "rollout": ["rollout_kernels.hip", "policy_dev.hpp", "sim_dev.hpp"]}


def kernel_hash(cls=None):
    """Hash of the sources a kernel class is built from (all kernel sources without a class)."""
    d = os.path.join(ROOT, "paper_2607_05272_amd", "csrc")
    files = (KERNEL_SOURCE[cls] + ["devmath.hpp", "params.hpp"] if cls in KERNEL_SOURCE else
             sorted(f for f in os.listdir(d) if f.endswith((".hip", ".hpp"))))
    h = hashlib.sha256()
    for f in files:
        h.update(open(os.path.join(d, f), "rb").read())
    return h.hexdigest()[:16]


def traffic_for(kernel, cfg_name):
    """HBM bytes per launch measured by rocprofv3 PMC counters (profiles/traffic.json),
    or None if absent or taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        d = json.load(open(path))
    except (OSError, ValueError):
        return None
    ent = d.get(f"{cfg_name}:{kernel}")
    if not ent or ent.get("kernel_hash") != kernel_hash(kernel):
        return None
    return ent.get("bytes_per_launch")


# kernel classes whose HBM traffic is taken from counters (the minibatch gradient, a sequence of
# library GEMMs and small kernels, has no single kernel to attribute it to)
KERNEL_OF = {"policy": "policy_", "step": "learned_k", "static": "static_k", "gae": "gae_k"}


def _pmc_rows(d):
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        rows += list(csv.DictReader(open(f)))
    return rows


def _per_dispatch(rows, counter, match):
    """Counter total over the kernels that `match`, per dispatch of them."""
    tot, disp = 0.0, set()
    for r in rows:
        if r["Counter_Name"] != counter or not match(r["Kernel_Name"]):
            continue
        tot += float(r["Counter_Value"])
        disp.add(r.get("Dispatch_Id") or r.get("Correlation_Id"))
    return (tot / len(disp), len(disp)) if disp else (None, 0)


def write_traffic(d, cfg_name):
    """HBM bytes per launch of each kernel class from FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch), each scaled so that the calibration copy reads and writes its known size."""
    calib = 1024 << 20
    cf, _ = _per_dispatch(_pmc_rows(os.path.join(d, "cfetch")), "FETCH_SIZE",
                          lambda k: "elementwise" in k and "Mul" in k)
    cw, _ = _per_dispatch(_pmc_rows(os.path.join(d, "cwrite")), "WRITE_SIZE",
                          lambda k: "elementwise" in k and "Mul" in k)
    f_fac = calib / (cf * 1024.0)
    w_fac = calib / (cw * 1024.0)
    fr, wr = _pmc_rows(os.path.join(d, "fetch")), _pmc_rows(os.path.join(d, "write"))
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        out = json.load(open(path))
    except (OSError, ValueError):
        out = {}
    for cls, pat in KERNEL_OF.items():
        fk, nf = _per_dispatch(fr, "FETCH_SIZE", lambda k, p=pat: p in k)
        wk, nw = _per_dispatch(wr, "WRITE_SIZE", lambda k, p=pat: p in k)
        if fk is None or wk is None:
            continue
        out[f"{cfg_name}:{cls}"] = {
            "bytes_per_launch": fk * 1024.0 * f_fac + wk * 1024.0 * w_fac,
            "fetch_kib_raw": fk, "write_kib_raw": wk, "dispatches": [nf, nw],
            "fetch_factor": f_fac, "write_factor": w_fac, "kernel_hash": kernel_hash(cls)}
    json.dump(out, open(path, "w"), indent=1, sort_keys=True)
    print(json.dumps(out, indent=1, sort_keys=True))


def copy_ceiling(mib=1024, reps=5):
    """Measured HBM ceiling: a device-to-device copy of `mib` MiB (read + write bytes per
    second, best of `reps`)."""
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    best = 0.0
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src)
        b.record()
        b.synchronize()
        best = max(best, 2.0 * n / (a.elapsed_time(b) * 1e-3) / 1e9)
    del src, dst
    return best


def host_info():
    """The host the CPU baseline runs on."""
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        aff = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        aff = os.cpu_count() or 1
    return {"host_cpus": os.cpu_count(), "affinity_cpus": aff, "cpu_model": model}


# worker threads of the CPU baseline: the host's CPUs available to this process, at most 16
# (the host-CPU share of one GPU on the machines this runs on)
MAX_CPU_THREADS = 16


def sample_ids(n_envs, n, seed):
    """Environment ids of a CPU-baseline sample: the first n/2 ids, then ids drawn without
    replacement from the rest by numpy's Philox generator."""
    import numpy as np
    a = min(n // 2, n_envs)
    rest = np.arange(a, n_envs)
    k = min(n - a, rest.size)
    pick = np.random.Generator(np.random.Philox(seed)).choice(rest, size=k, replace=False)
    return np.sort(np.concatenate([np.arange(a), pick])).astype(np.uint32)


def _threaded(fn, chunks):
    th = [threading.Thread(target=fn, args=(c,)) for c in chunks]
    t0 = time.perf_counter()
    for t in th:
        t.start()
    for t in th:
        t.join()
    return time.perf_counter() - t0


def cpu_baseline(w, name, budget_s, seed, sim_only=False):
    """The oracle on the host cores over a bounded sample of the same workload, env-steps per
    second: the sequential fp64 simulator + fp64 policy + sampler, or (sim_only) the simulator
    alone replaying uniform random actions. Run once on the worker threads and once, on a
    proportionally smaller sample, on one thread."""
    import numpy as np
    import oracle
    info = host_info()
    threads = max(1, min(MAX_CPU_THREADS, info["affinity_cpus"]))
    T = min(w["T"], 256)
    A = 6 * w["n_servers"]
    wts = None if sim_only else oracle.init_weights(w, seed)

    def run(ids, n_ticks):
        if sim_only:
            acts = np.random.default_rng(seed).integers(0, A, (n_ticks, ids.size)).astype(np.uint8)
            oracle.rollout(w, seed, n_ticks, ids, actions=acts, want_obs=False, want_rec=False)
        else:
            oracle.rollout(w, seed, n_ticks, ids, weights=wts, want_obs=False, want_rec=False)

    cal = sample_ids(w["n_envs"], 8, seed)
    run(cal[:2], 8)
    t0 = time.perf_counter()
    run(cal, 32)
    per_step = (time.perf_counter() - t0) / (32 * cal.size)
    n_env = min(w["n_envs"], max(threads, int(budget_s * threads / (per_step * T))))
    ids = sample_ids(w["n_envs"], n_env, seed)
    dt = _threaded(lambda c: run(ids[c], T) if len(c) else None,
                   np.array_split(np.arange(n_env), threads))
    n1 = max(1, n_env // threads)
    dt1 = _threaded(lambda c: run(ids[c], T), [np.arange(n1)])
    what = ("simulator only (uniform random actions replayed)" if sim_only else
            f"fp64 {'attention policy' if w.get('policy_kind', 0) == 1 else 'policy MLP'} + "
            "sampler + simulator")
    return dict({"value": n_env * T / dt, "unit": "env-steps/s", "cores": threads,
                 "threads": threads, "kind": "oracle",
                 "single_thread": {"value": n1 * T / dt1, "envs": int(n1), "wall_s": dt1},
                 "sample": f"{n_env} envs (ids 0..{n_env // 2 - 1} and the rest drawn by a "
                           f"Philox generator) x {T} ticks of {name}, {what}; {dt:.1f} s wall "
                           f"on {threads} worker threads (the host's {info['affinity_cpus']} "
                           f"available CPUs, at most {MAX_CPU_THREADS}); single thread: "
                           f"{n1} envs"}, **info)


def kernel_table(timing, steps):
    return {k: {"total_ms_per_step": ms / steps, "launches_per_step": n // steps,
                "avg_us": 1000.0 * ms / n} for k, (ms, n) in timing.items() if n}


def rooflines(w, kern, tot, E, T, train, args, cfg_name):
    """Achieved work rate of each hot kernel class against its MI355X peak."""
    rl = {}
    if "policy" in kern and w.get("policy_kind", 0) == 1:
        fl = attn_flops(w) * E
        ach = fl / (kern["policy"]["avg_us"] * 1e-6) / 1e12
        rl["policy"] = {"bound": "alu", "achieved": ach, "peak": PEAK_FP32_VALU_TFLOPS,
                        "unit": "TFLOP/s", "frac": ach / PEAK_FP32_VALU_TFLOPS,
                        "traffic": traffic_for("policy", cfg_name), "work_per_launch": fl}
    elif "policy" in kern:
        fl = mlp_flops(w) * E
        ach = fl / (kern["policy"]["avg_us"] * 1e-6) / 1e12
        peak = PEAK_BF16_TFLOPS if w["mlp_bf16"] else PEAK_FP32_TFLOPS
        rl["policy"] = {"bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s",
                        "frac": ach / peak, "traffic": traffic_for("policy", cfg_name),
                        "work_per_launch": fl}
    if "step" in kern:
        by = step_bytes(w, tot, E, T) * E
        ach = by / (kern["step"]["avg_us"] * 1e-6) / 1e9
        rl["step"] = {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                      "frac": ach / PEAK_HBM_GBS, "traffic": traffic_for("step", cfg_name),
                      "work_per_launch": by}
    if "static" in kern:
        by = static_bytes(w, tot, E, T, T / kern["static"]["launches_per_step"]) * E
        ach = by / (kern["static"]["avg_us"] * 1e-6) / 1e9
        rl["static"] = {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": ach / PEAK_HBM_GBS, "traffic": traffic_for("static", cfg_name),
                        "work_per_launch": by}
    if "rollout" in kern:
        # the fused small-batch rollout: every tick's policy and learned tick in one launch,
        # against both ceilings (a launch this small is bound by latency, far below either)
        n_pol = T + (1 if w["value_head"] else 0)
        fl = mlp_flops(w) * E * n_pol
        by = step_bytes(w, tot, E, T) * E * T
        sec = kern["rollout"]["avg_us"] * 1e-6
        peak = PEAK_BF16_TFLOPS if w["mlp_bf16"] else PEAK_FP32_TFLOPS
        rl["rollout"] = {"bound": "mfma", "achieved": fl / sec / 1e12, "peak": peak,
                         "unit": "TFLOP/s", "frac": fl / sec / 1e12 / peak, "traffic": None,
                         "work_per_launch": fl,
                         "simulator": {"achieved": by / sec / 1e9, "peak": PEAK_HBM_GBS,
                                       "unit": "GB/s", "frac": by / sec / 1e9 / PEAK_HBM_GBS,
                                       "bytes_per_launch": by},
                         "us_per_tick": kern["rollout"]["avg_us"] / T}
    if "gae" in kern:
        by = 28.0 * E * T
        ach = by / (kern["gae"]["avg_us"] * 1e-6) / 1e9
        rl["gae"] = {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": ach / PEAK_HBM_GBS, "traffic": traffic_for("gae", cfg_name),
                     "work_per_launch": by}
    if "ppo" in kern:
        # minibatch gradients per step (one, or epochs x minibatches when training), each with
        # its share of Adam; the MLP's products run on the matrix cores (bf16, or fp32 for an
        # fp32 policy), the attention network's on the vector units
        n_grad = args.epochs * args.minibatches if train else 1
        if w.get("policy_kind", 0) == 1:
            fl = 3 * attn_flops(w) * (w.get("ppo_minibatch", 0) or 8192) * n_grad
            bound, peak = "alu", PEAK_FP32_VALU_TFLOPS
        else:
            fl = ppo_flops(dict(w, ppo_minibatch=w.get("ppo_minibatch", 0) or 8192)) * n_grad
            bound, peak = "mfma", (PEAK_BF16_TFLOPS if w["mlp_bf16"] else PEAK_FP32_TFLOPS)
        ach = fl / (kern["ppo"]["total_ms_per_step"] * 1e-3) / 1e12
        rl["ppo"] = {"bound": bound, "achieved": ach, "peak": peak, "unit": "TFLOP/s",
                     "frac": ach / peak, "traffic": None, "work_per_launch": fl}
    return rl


def measure(name, args, steps, warmup, timing_steps, ticks=0):
    """One configuration: `warmup` untimed steps, a graph-priming step, `steps` timed steps
    (rollouts replayed from the captured graph, no per-launch events), then `timing_steps`
    steps launched eagerly with HIP events around every launch for the kernels' durations."""
    import torch
    import paper_2607_05272_amd as bs
    w = workload_of(name)
    if ticks:
        w["T"] = ticks
    E, T, F = w["n_envs"], w["T"], w["obs_dim"]
    dev = torch.device("cuda")
    seed = 0x5EED0000 + (int(name[1]) if name[0] == "C" and name[1].isdigit() else 9)
    sim = bs.Sim(w)
    if args.no_graphs:
        sim.set_graphs(False)
    weights = sim.init_weights(seed)
    ppo = w.get("ppo_minibatch", 0) > 0 and args.train == "none"
    train = args.train != "none"
    traj = bs.Trajectory(T, E, F, dev, value=bool(w["value_head"]), shadow=bool(w["shadow"]),
                         obs=ppo or train)
    st = {}
    if train:
        st["params"] = sim.params_from_weights(weights)
        st["m"] = torch.zeros_like(st["params"])
        st["v"] = torch.zeros_like(st["params"])
        st["t"] = 0
        st["mb"] = w.get("ppo_minibatch", 0) or 8192
        st["algo"] = bs.ALGO_PPO if args.train == "ppo" else bs.ALGO_REINFORCE
    grads = torch.empty(sim.ppo_grad_count(), dtype=torch.float32, device=dev) if ppo else None
    ploss = torch.empty(4, dtype=torch.float64, device=dev) if ppo else None
    adv = torch.empty((T, E), dtype=torch.float64, device=dev)
    ret = torch.empty((T, E), dtype=torch.float64, device=dev)
    gae = bool(w["value_head"])
    lam = 1.0 if args.train == "reinforce" or not gae else w["lam"]

    def one_step(i, ev=None):
        if ev:
            ev[0].record(sim.stream)
        sim.reset(seed + i)
        if ev:
            ev[1].record(sim.stream)
        sim.rollout(weights, T, traj=traj)
        if ev:
            ev[2].record(sim.stream)
        sim.returns_gae(traj.reward, traj.value if gae else None, w["gamma"], lam, adv, ret)
        if ppo:
            sim.ppo_minibatch_grad(weights, traj.obs, traj.actions, traj.logp, adv, ret,
                                   w["ppo_minibatch"], seed + i, grads=grads, loss=ploss)
        if train:
            st["t"], _ = sim.update(weights, st["params"], st["m"], st["v"], st["t"], traj.obs,
                                    traj.actions, traj.logp, adv, ret, st["algo"], args.epochs,
                                    args.minibatches, st["mb"], seed + i, 3e-4, want_losses=False)
        if ev:
            ev[3].record(sim.stream)
        return sim.stats()

    def progress(what):
        print(f"[bench] {name}: {what}", file=sys.stderr, flush=True)

    for i in range(warmup):
        one_step(i)
        progress(f"warmup step {i + 1} of {warmup}")
    one_step(warmup)           # captures the rollout's graph (it repeats the previous call)
    sim.sync()
    torch.cuda.synchronize()
    progress("graph-priming step")
    marks = []
    t0 = time.perf_counter()
    tot = None
    for i in range(steps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        marks.append(ev)
        tot = one_step(1000 + i, ev)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    progress(f"{steps} timed steps")
    sim.sync()
    captures, replays = sim.graph_stats()
    ms_per_step = (t1 - t0) * 1000.0 / steps
    step_ms = [ev[0].elapsed_time(ev[3]) for ev in marks]
    rollout_ms = [ev[1].elapsed_time(ev[2]) for ev in marks]
    # kernel durations: eager launches bracketed by HIP events on the library's stream
    sim.get_timing(clear=True)
    sim.set_timing(True)
    t2 = time.perf_counter()
    for i in range(timing_steps):
        one_step(2000 + i)
        progress(f"event-timed step {i + 1} of {timing_steps}")
    sim.sync()
    t3 = time.perf_counter()
    timing = sim.get_timing(clear=True)
    sim.set_timing(False)
    kern = kernel_table(timing, timing_steps)
    rl = rooflines(w, kern, tot, E, T, train, args, name)
    kernel_ms = sum(v["total_ms_per_step"] for v in kern.values())
    res = {
        "workload": (DESCR[name] if not ticks else DESCR[name] + f" [T={T}]")
        + ("" if not train else f"; + {args.train} update, {args.epochs} epochs x "
           f"{args.minibatches} minibatches of {st['mb']} samples, Adam"),
        "envs": E, "ticks": T, "env_steps_per_step": E * T,
        "value": E * T / (ms_per_step / 1000.0), "ms_per_step": ms_per_step,
        "step_ms": {"median": statistics.median(step_ms), "min": min(step_ms),
                    "max": max(step_ms)},
        "rollout_only": {"median_ms": statistics.median(rollout_ms),
                         "env_steps_per_s": E * T / (statistics.median(rollout_ms) / 1000.0)},
        "graph": {"captures": captures, "replays": replays},
        "eager_timed_ms_per_step": (t3 - t2) * 1000.0 / max(timing_steps, 1),
        "kernel_ms_per_step": kernel_ms,
        "launch_gap_frac": max(0.0, 1.0 - kernel_ms / ms_per_step),
        "kernels": {k: dict(v, **{kk: vv for kk, vv in rl.get(k, {}).items()
                                  if kk in ("achieved", "unit", "frac")}) for k, v in kern.items()},
        "totals": {"arrivals": int(tot["cnt"][0][0]), "dropped": int(tot["cnt"][0][2]),
                   "dispatched": int(tot["cnt"][0][3]), "batches": int(tot["cnt"][0][4])},
    }
    sim.close()
    del traj, adv, ret, grads
    torch.cuda.empty_cache()
    return w, res, rl, kern


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="C5", choices=sorted(DESCR))
    ap.add_argument("--ticks", type=int, default=0, help="override T (diagnostics only)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--timing-steps", type=int, default=2,
                    help="eager steps with per-launch HIP events for the kernels' durations")
    ap.add_argument("--train", default="none", choices=("none", "ppo", "reinforce"),
                    help="add the policy update (epochs x minibatches of gradient + Adam over "
                         "the stored trajectory) to every step")
    ap.add_argument("--epochs", type=int, default=4)
    ap.add_argument("--minibatches", type=int, default=8)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graphs", action="store_true",
                    help="launch every rollout eagerly (for counter collection, which serializes "
                         "each dispatch)")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the sub-measurements of C1-C4 that follow the headline line's")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="only copy this many MiB device-to-device (HBM counter calibration)")
    ap.add_argument("--write-traffic", default="",
                    help="directory of rocprofv3 --pmc runs (fetch/, write/, cfetch/, cwrite/): "
                         "write profiles/traffic.json and exit")
    args = ap.parse_args()
    if args.calib_copy_mib:
        # a plain elementwise copy of known size (reads n bytes, writes n bytes), for
        # scaling the HBM byte counters of the profiler
        import torch
        n = args.calib_copy_mib << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"calib_copy_bytes": n, "copies": 3}))
        return
    if args.write_traffic:
        write_traffic(args.write_traffic, args.config)
        return
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only (environments are independent; the "
              "path would shard by environment, but only the one-GPU path is built). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)
    w, res, rl, kern = measure(args.config, args, args.steps, args.warmup, args.timing_steps,
                               args.ticks)
    dom = max(kern, key=lambda k: kern[k]["total_ms_per_step"])
    roof = dict(rl.get(dom, {}))
    roof["kernel"] = dom
    work = roof.pop("work_per_launch", None)
    # the simulator kernels together against HBM (algorithmic bytes over their time)
    sim_by = sum(rl[k]["work_per_launch"] * kern[k]["launches_per_step"] for k in ("step", "static")
                 if k in rl)
    sim_ms = sum(kern[k]["total_ms_per_step"] for k in ("step", "static") if k in kern)
    line = {
        "metric": "simulated env-steps/sec on 1 MI355X + % of HBM roofline (MLP: % MFMA peak)",
        "value": res["value"], "unit": "env-steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": res["ms_per_step"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None,
        "dtype": "f64 simulator + bf16 MLP (fp32 accumulate)" if w["mlp_bf16"] else "f64 simulator + f32 MLP",
        "data": "synthetic (seeded workload generator; untrained Xavier policy)",
        "config": {"workload": res["workload"], "envs": res["envs"], "ticks": res["ticks"],
                   "env_steps_per_step": res["env_steps_per_step"]},
        "roofline": roof,
        "simulator_hbm": ({"achieved": sim_by / (sim_ms * 1e-3) / 1e9, "peak": PEAK_HBM_GBS,
                           "unit": "GB/s", "frac": sim_by / (sim_ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                           "kernels": [k for k in ("step", "static") if k in kern]}
                          if sim_ms > 0 else None),
        "work_per_launch": work,
        "graph_priming_steps": 1,
    }
    for k in ("step_ms", "rollout_only", "graph", "eager_timed_ms_per_step", "kernel_ms_per_step",
              "launch_gap_frac", "kernels", "totals"):
        line[k] = res[k]
    line["hbm_copy_ceiling_GBs"] = copy_ceiling()
    if not args.no_other_configs and args.config == "C5" and not args.ticks and args.train == "none":
        # every other configuration, measured the same way (fewer steps)
        line["configs"] = {}
        for name in ("C1", "C2", "C3", "C4"):
            _, r2, rl2, _ = measure(name, args, 3, 1, 2)
            r2["roofline"] = {k: {kk: v[kk] for kk in ("bound", "achieved", "peak", "unit", "frac",
                                                     "simulator", "us_per_tick") if kk in v}
                              for k, v in rl2.items()}
            line["configs"][name] = r2
    if not args.no_cpu_baseline:
        seed = 0x5EED0000 + (int(args.config[1]) if args.config[0] == "C" and args.config[1].isdigit() else 9)
        line["cpu_baseline"] = cpu_baseline(w, args.config, args.cpu_seconds, seed)
        line["cpu_baseline_sim_only"] = cpu_baseline(w, args.config, args.cpu_seconds / 3, seed,
                                                     sim_only=True)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
