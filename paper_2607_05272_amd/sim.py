"""Python face of the C ABI in include/batchsim.h (argument marshalling only).

Tensors passed in or returned are CUDA (HIP) tensors owned by torch; the library writes
into them on the context's stream. Layouts follow the ABI: [T][E] time-major arrays and
[F][E] observations.
"""
import ctypes as C

import numpy as np
import torch

from . import _lib as L


def _p(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def weights_layout(w):
    """Byte offsets of the policy weight buffer for workload `w` (sim_weights_layout)."""
    lib = L.load()
    cfg = L.make_cfg(w, n_envs=max(1, w.get("n_envs", 1)))
    lay = L.SimWLayout()
    L.check(lib.sim_weights_layout(C.byref(cfg), C.byref(lay)), "sim_weights_layout")
    return dict(w1=lay.w1, b1=lay.b1, w2=lay.w2, b2=lay.b2, w3=lay.w3, b3=lay.b3,
                bytes=lay.bytes, n_out=lay.n_out, elem_bytes=lay.elem_bytes)


def attn_layout(w):
    """Byte offsets of the attention policy's weights (sim_attn_weights_layout) and their
    shapes ([in][out] matrices, vectors)."""
    lib = L.load()
    cfg = L.make_cfg(w, n_envs=max(1, w.get("n_envs", 1)))
    lay = L.SimAttnLayout()
    L.check(lib.sim_attn_weights_layout(C.byref(cfg), C.byref(lay)), "sim_attn_weights_layout")
    F, D, A = w["obs_dim"], w["attn_embed"], 6 * w["n_servers"]
    Hp, Hv = w["mlp_h1"], w["mlp_h2"]
    shapes = dict(w_in=(F, D), b_in=(D,), w_qkv=(D, 3 * D), b_qkv=(3 * D,), w_o=(D, D),
                  b_o=(D,), wp1=(D, Hp), bp1=(Hp,), wp2=(Hp, A), bp2=(A,), wv1=(D, Hv),
                  bv1=(Hv,), wv2=(Hv, 1), bv2=(1,))
    return {k: getattr(lay, k) for k in L.ATTN_KEYS}, shapes, lay.bytes


def _is_attn(w):
    return w.get("policy_kind", L.POLICY_MLP) == L.POLICY_ATTN


def _dims(w, n_out):
    return [w["obs_dim"], w["mlp_h1"], w["mlp_h2"], n_out]


def pack_weights(w, arrays):
    """Host bytes of the ABI weight buffer from arrays w1,b1,w2,b2,w3,b3 ([in][out]).
    Matrices must hold fp32 values (bf16-representable ones in bf16 mode). For the attention
    policy: the fp32 arrays named by sim_attn_weights_layout."""
    if _is_attn(w):
        off, shapes, nbytes = attn_layout(w)
        buf = np.zeros(nbytes, np.uint8)
        for k in L.ATTN_KEYS:
            a = np.ascontiguousarray(arrays[k], dtype=np.float64).reshape(shapes[k])
            f32 = a.astype(np.float32)
            if not np.array_equal(f32.astype(np.float64), a):
                raise ValueError(f"{k} is not fp32-representable")
            raw = f32.tobytes()
            buf[off[k]:off[k] + len(raw)] = np.frombuffer(raw, np.uint8)
        return buf
    lay = weights_layout(w)
    buf = np.zeros(lay["bytes"], np.uint8)
    dims = _dims(w, lay["n_out"])
    for l in range(3):
        W = np.ascontiguousarray(arrays[f"w{l + 1}"], dtype=np.float64).reshape(dims[l], dims[l + 1])
        f32 = W.astype(np.float32)
        if not np.array_equal(f32.astype(np.float64), W):
            raise ValueError(f"w{l + 1} is not fp32-representable")
        if lay["elem_bytes"] == 2:
            bits = f32.view(np.uint32)
            if np.any(bits & 0xFFFF):
                raise ValueError(f"w{l + 1} is not bf16-representable")
            raw = (bits >> 16).astype(np.uint16).tobytes()
        else:
            raw = f32.tobytes()
        o = lay[f"w{l + 1}"]
        buf[o:o + len(raw)] = np.frombuffer(raw, np.uint8)
        b = np.ascontiguousarray(arrays[f"b{l + 1}"], dtype=np.float32).reshape(dims[l + 1])
        o = lay[f"b{l + 1}"]
        buf[o:o + b.nbytes] = np.frombuffer(b.tobytes(), np.uint8)
    return buf


def unpack_weights(w, buf):
    """fp64 arrays of the values held in an ABI weight buffer (host bytes)."""
    if _is_attn(w):
        off, shapes, _ = attn_layout(w)
        buf = np.asarray(buf, dtype=np.uint8)
        out = {}
        for k in L.ATTN_KEYS:
            n = int(np.prod(shapes[k]))
            out[k] = np.frombuffer(buf[off[k]:off[k] + 4 * n].tobytes(),
                                   np.float32).astype(np.float64).reshape(shapes[k])
        return out
    lay = weights_layout(w)
    buf = np.asarray(buf, dtype=np.uint8)
    dims = _dims(w, lay["n_out"])
    out = {}
    for l in range(3):
        n = dims[l] * dims[l + 1]
        o = lay[f"w{l + 1}"]
        if lay["elem_bytes"] == 2:
            bits = np.frombuffer(buf[o:o + 2 * n].tobytes(), np.uint16).astype(np.uint32) << 16
            W = bits.view(np.float32)
        else:
            W = np.frombuffer(buf[o:o + 4 * n].tobytes(), np.float32)
        out[f"w{l + 1}"] = W.astype(np.float64).reshape(dims[l], dims[l + 1])
        o = lay[f"b{l + 1}"]
        out[f"b{l + 1}"] = np.frombuffer(buf[o:o + 4 * dims[l + 1]].tobytes(),
                                         np.float32).astype(np.float64)
    return out


class Trajectory:
    """Caller-owned device buffers of one rollout (sim_traj)."""

    def __init__(self, T, E, F, device, value=False, shadow=False, obs=False, rchk=False,
                 logp=True, reward=True):
        self.T, self.E = T, E
        self.actions = torch.empty((T, E), dtype=torch.uint8, device=device)
        self.logp = torch.empty((T, E), dtype=torch.float32, device=device) if logp else None
        self.reward = torch.empty((T, E), dtype=torch.float64, device=device) if reward else None
        self.reward_shadow = (torch.empty((T, E), dtype=torch.float64, device=device)
                              if shadow else None)
        self.value = torch.empty((T + 1, E), dtype=torch.float32, device=device) if value else None
        self.obs = torch.empty((T + 1, F, E), dtype=torch.float32, device=device) if obs else None
        self.rchk = torch.empty((T, E), dtype=torch.int64, device=device) if rchk else None

    def struct(self):
        return L.SimTraj(*(None if t is None else t.data_ptr() for t in
                           (self.actions, self.logp, self.reward, self.reward_shadow,
                            self.value, self.obs, self.rchk)))


class Sim:
    """One simulator context (sim_create ... sim_destroy) on the current HIP device."""

    def __init__(self, w, n_envs=None, device="cuda", stream=None):
        self.lib = L.load()
        self.w = w
        self.cfg = L.make_cfg(w, n_envs)
        self.E = self.cfg.n_envs
        self.F = w["obs_dim"]
        self.K = w["n_servers"]
        self.A = 6 * self.K
        self.Ap = self.A + (1 if w["value_head"] else 0)
        self.device = torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self._ctx = C.c_void_p()
        self._keep = []
        L.check(self.lib.sim_create(C.byref(self.cfg), C.c_void_p(self.stream.cuda_stream),
                                    C.byref(self._ctx)), "sim_create")

    def close(self):
        if self._ctx:
            L.check(self.lib.sim_destroy(self._ctx), "sim_destroy")
            self._ctx = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    # -- environment ------------------------------------------------------------------
    def set_trace(self, times, classes, counts):
        """Device tensors times [E][L] f64, classes [E][L] u8, counts [E] i32."""
        self._keep = [times, classes, counts]
        L.check(self.lib.sim_set_trace(self._ctx, _p(times), _p(classes), _p(counts)),
                "sim_set_trace")

    def reset(self, seed):
        L.check(self.lib.sim_reset(self._ctx, C.c_uint64(seed)), "sim_reset")

    def obs(self):
        o = torch.empty((self.F, self.E), dtype=torch.float32, device=self.device)
        L.check(self.lib.sim_obs(self._ctx, _p(o)), "sim_obs")
        return o

    def step(self, actions, want_obs=True, want_reward=True):
        obs = (torch.empty((self.F, self.E), dtype=torch.float32, device=self.device)
               if want_obs else None)
        r = torch.empty(self.E, dtype=torch.float64, device=self.device) if want_reward else None
        rs = (torch.empty(self.E, dtype=torch.float64, device=self.device)
              if want_reward and self.w["shadow"] else None)
        L.check(self.lib.sim_step(self._ctx, _p(actions), _p(obs), _p(r), _p(rs)), "sim_step")
        return obs, r, rs

    def tick(self):
        t = C.c_int32()
        L.check(self.lib.sim_tick(self._ctx, C.byref(t)), "sim_tick")
        return t.value

    # -- policy -----------------------------------------------------------------------
    def init_weights(self, seed):
        lay = weights_layout(self.w)
        buf = torch.zeros(lay["bytes"], dtype=torch.uint8, device=self.device)
        L.check(self.lib.sim_init_weights(self._ctx, C.c_uint64(seed), _p(buf)), "sim_init_weights")
        return buf

    def upload_weights(self, arrays):
        return torch.from_numpy(pack_weights(self.w, arrays)).to(self.device)

    def policy(self, weights, obs, step, want_logits=False):
        E = obs.shape[1]
        assert E == self.E and obs.shape[0] == self.F
        act = torch.empty(E, dtype=torch.uint8, device=self.device)
        logp = torch.empty(E, dtype=torch.float32, device=self.device)
        val = torch.empty(E, dtype=torch.float32, device=self.device) if self.w["value_head"] else None
        lg = torch.empty((self.Ap, E), dtype=torch.float32, device=self.device) if want_logits else None
        L.check(self.lib.sim_policy(self._ctx, _p(weights), _p(obs), C.c_uint32(step), _p(act),
                                    _p(logp), _p(val), _p(lg)), "sim_policy")
        return dict(actions=act, logp=logp, value=val, logits=lg)

    def policy_hidden(self, weights, obs, step):
        """sim_policy_hidden: the policy's outputs plus the hidden activations h1 [H1][E] and
        h2 [H2][E] that the kernel passes between layers."""
        E = obs.shape[1]
        assert E == self.E and obs.shape[0] == self.F
        H1, H2 = self.w["mlp_h1"], self.w["mlp_h2"]
        act = torch.empty(E, dtype=torch.uint8, device=self.device)
        logp = torch.empty(E, dtype=torch.float32, device=self.device)
        val = torch.empty(E, dtype=torch.float32, device=self.device) if self.w["value_head"] else None
        lg = torch.empty((self.Ap, E), dtype=torch.float32, device=self.device)
        hid = torch.empty((H1 + H2, E), dtype=torch.float32, device=self.device)
        L.check(self.lib.sim_policy_hidden(self._ctx, _p(weights), _p(obs), C.c_uint32(step),
                                           _p(act), _p(logp), _p(val), _p(lg), _p(hid)),
                "sim_policy_hidden")
        return dict(actions=act, logp=logp, value=val, logits=lg, h1=hid[:H1], h2=hid[H1:])

    def rollout(self, weights, T, store_obs=False, rchk=False, traj=None):
        if traj is None:
            traj = Trajectory(T, self.E, self.F, self.device, value=bool(self.w["value_head"]),
                              shadow=bool(self.w["shadow"]), obs=store_obs, rchk=rchk)
        st = traj.struct()
        L.check(self.lib.sim_rollout(self._ctx, _p(weights), T, C.byref(st)), "sim_rollout")
        return traj

    def returns_gae(self, r, v, gamma, lam, adv=None, ret=None):
        T = r.shape[0]
        adv = torch.empty_like(r) if adv is None else adv
        ret = torch.empty_like(r) if ret is None else ret
        L.check(self.lib.returns_gae(self._ctx, T, _p(r), _p(v), C.c_double(gamma),
                                     C.c_double(lam), _p(adv), _p(ret)), "returns_gae")
        return adv, ret

    def ppo_grad_count(self):
        n = C.c_int64()
        L.check(self.lib.sim_ppo_grad_count(C.byref(self.cfg), C.byref(n)), "sim_ppo_grad_count")
        return n.value

    def ppo_minibatch_grad(self, weights, obs, actions, logp_old, adv, ret, M, seed, clip=0.2,
                           c_value=0.5, c_entropy=0.01, want_index=False, grads=None, loss=None,
                           noalloc=False):
        """One PPO minibatch: obs [T(+1)][F][E] (rows 0..T-1 used), actions/logp_old/adv/ret
        [T][E]. Returns (grads fp32 flat W1,b1,W2,b2,W3,b3; loss [4] fp64; index or None).
        noalloc=True calls ppo_minibatch_grad_noalloc (the library's fixed scratch)."""
        T = actions.shape[0]
        assert actions.shape[1] == self.E and obs.shape[1] == self.F and obs.shape[0] >= T
        grads = (torch.empty(self.ppo_grad_count(), dtype=torch.float32, device=self.device)
                 if grads is None else grads)
        loss = torch.empty(4, dtype=torch.float64, device=self.device) if loss is None else loss
        idx = torch.empty(M, dtype=torch.int64, device=self.device) if want_index else None
        name = "ppo_minibatch_grad_noalloc" if noalloc else "ppo_minibatch_grad"
        L.check(getattr(self.lib, name)(self._ctx, _p(weights), T, _p(obs), _p(actions),
                                        _p(logp_old), _p(adv), _p(ret), M, C.c_uint64(seed),
                                        clip, c_value, c_entropy, _p(grads), _p(loss), _p(idx)),
                name)
        return grads, loss, idx

    def reinforce_minibatch_grad(self, weights, obs, actions, adv, ret, M, seed, c_value=0.5,
                                 c_entropy=0.01, want_index=False, grads=None, loss=None):
        """REINFORCE with baseline on one minibatch (adv = G - V, ret = G)."""
        T = actions.shape[0]
        assert actions.shape[1] == self.E and obs.shape[1] == self.F and obs.shape[0] >= T
        grads = (torch.empty(self.ppo_grad_count(), dtype=torch.float32, device=self.device)
                 if grads is None else grads)
        loss = torch.empty(4, dtype=torch.float64, device=self.device) if loss is None else loss
        idx = torch.empty(M, dtype=torch.int64, device=self.device) if want_index else None
        L.check(self.lib.reinforce_minibatch_grad(self._ctx, _p(weights), T, _p(obs), _p(actions),
                                                  _p(adv), _p(ret), M, C.c_uint64(seed), c_value,
                                                  c_entropy, _p(grads), _p(loss), _p(idx)),
                "reinforce_minibatch_grad")
        return grads, loss, idx

    def params_from_weights(self, weights):
        p = torch.empty(self.ppo_grad_count(), dtype=torch.float32, device=self.device)
        L.check(self.lib.sim_params_from_weights(self._ctx, _p(weights), _p(p)),
                "sim_params_from_weights")
        return p

    def adam_update(self, params, grads, m, v, step, lr, beta1=0.9, beta2=0.999, eps=1e-8,
                    weights=None):
        L.check(self.lib.adam_update(self._ctx, _p(params), _p(grads), _p(m), _p(v), step, lr,
                                     beta1, beta2, eps, _p(weights)), "adam_update")

    def update(self, weights, params, m, v, step, obs, actions, logp_old, adv, ret, algo,
               epochs, minibatches, M, seed, lr, clip=0.2, c_value=0.5, c_entropy=0.01,
               beta1=0.9, beta2=0.999, eps=1e-8, want_losses=True):
        """sim_update: epochs x minibatches of gradient + Adam; returns (new step, losses)."""
        T = actions.shape[0]
        cfg = L.SimUpdateCfg(algo, epochs, minibatches, M, seed, clip, c_value, c_entropy, lr,
                             beta1, beta2, eps)
        st = C.c_int32(step)
        losses = (torch.empty((epochs * minibatches, 4), dtype=torch.float64, device=self.device)
                  if want_losses else None)
        L.check(self.lib.sim_update(self._ctx, C.byref(cfg), _p(weights), _p(params), _p(m),
                                    _p(v), C.byref(st), T, _p(obs), _p(actions), _p(logp_old),
                                    _p(adv), _p(ret), _p(losses)), "sim_update")
        return st.value, losses

    def unflatten_grads(self, g):
        """Split a flat gradient vector (host numpy) into the policy's arrays (W1,b1,W2,b2,W3,b3,
        or the attention policy's fourteen in sim_attn_layout order)."""
        if _is_attn(self.w):
            _, sh, _ = attn_layout(self.w)
            shapes = [(k, sh[k]) for k in L.ATTN_KEYS]
        else:
            F, H1, H2, Ap = self.F, self.w["mlp_h1"], self.w["mlp_h2"], self.Ap
            shapes = [("w1", (F, H1)), ("b1", (H1,)), ("w2", (H1, H2)), ("b2", (H2,)),
                      ("w3", (H2, Ap)), ("b3", (Ap,))]
        out, o = {}, 0
        for k, sh in shapes:
            n = int(np.prod(sh))
            out[k] = np.asarray(g[o:o + n]).reshape(sh)
            o += n
        return out

    # -- checkpoint / resume ------------------------------------------------------------
    def get_state(self, device=True):
        """Snapshot of every environment's state, the tick counter and the seed, as a uint8
        tensor on the device (or in host memory)."""
        n = C.c_size_t()
        L.check(self.lib.sim_get_state(self._ctx, None, C.byref(n)), "sim_get_state")
        buf = torch.empty(n.value, dtype=torch.uint8, device=self.device if device else "cpu")
        L.check(self.lib.sim_get_state(self._ctx, _p(buf), C.byref(n)), "sim_get_state")
        return buf

    def set_state(self, buf):
        L.check(self.lib.sim_set_state(self._ctx, _p(buf), buf.numel()), "sim_set_state")

    # -- statistics -------------------------------------------------------------------
    def counters(self):
        cnt = torch.empty((2, L.NCNT, self.E), dtype=torch.int64, device=self.device)
        sums = torch.empty((2, L.NSUM, self.E), dtype=torch.float64, device=self.device)
        L.check(self.lib.sim_counters(self._ctx, _p(cnt), _p(sums)), "sim_counters")
        return cnt, sums

    def checksums(self):
        chk = torch.empty((2, self.E), dtype=torch.int64, device=self.device)
        L.check(self.lib.sim_checksums(self._ctx, _p(chk)), "sim_checksums")
        return chk

    def stats(self):
        t = L.SimTotals()
        L.check(self.lib.sim_stats(self._ctx, C.byref(t)), "sim_stats")
        return dict(cnt=np.array([[t.cnt[s][i] for i in range(L.NCNT)] for s in range(2)]),
                    sum=np.array([[t.sum[s][i] for i in range(L.NSUM)] for s in range(2)]))

    def sync(self):
        L.check(self.lib.sim_sync(self._ctx), "sim_sync")

    # -- tracing ----------------------------------------------------------------------
    def set_timing(self, on):
        L.check(self.lib.sim_set_timing(self._ctx, 1 if on else 0), "sim_set_timing")

    def set_graphs(self, on):
        """Rollout graphs on (default) or off (every rollout launched eagerly)."""
        L.check(self.lib.sim_set_graphs(self._ctx, 1 if on else 0), "sim_set_graphs")

    def set_fused_rollout(self, mode):
        """Fused small-batch rollouts: FUSE_AUTO (default), FUSE_ON or FUSE_OFF (per-tick
        launches); see sim_set_fused_rollout."""
        L.check(self.lib.sim_set_fused_rollout(self._ctx, int(mode)), "sim_set_fused_rollout")

    def graph_stats(self):
        """(graphs captured, rollouts replayed from a graph)."""
        c, r = C.c_int64(0), C.c_int64(0)
        L.check(self.lib.sim_graph_stats(self._ctx, C.byref(c), C.byref(r)), "sim_graph_stats")
        return c.value, r.value

    def get_timing(self, clear=True):
        """Per kernel class: (total ms, launches) from HIP events on the context's stream."""
        ms = (C.c_double * len(L.KERNEL_CLASSES))()
        n = (C.c_int64 * len(L.KERNEL_CLASSES))()
        L.check(self.lib.sim_get_timing(self._ctx, ms, n, 1 if clear else 0), "sim_get_timing")
        return {k: (ms[i], n[i]) for i, k in enumerate(L.KERNEL_CLASSES)}
