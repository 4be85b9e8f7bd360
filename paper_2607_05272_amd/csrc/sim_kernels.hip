// sim_kernels.hip -- reset, the learned system's one-tick kernel and the static shadow
// system's multi-tick kernel of the batched discrete-event simulator (device code and model in
// sim_dev.hpp), observation packing and per-environment statistics.
#include "sim_dev.hpp"

namespace bsim {
namespace {

// ---- learned system: one tick per launch ----------------------------------------------------
template <int CM, bool PF>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(PF ? 1 : 4))) void learned_k(
    SimParams p, EnvState g, uint32_t k, int lpw, const uint8_t* __restrict__ act,
    float* __restrict__ obs_out, int obs_mode, double* __restrict__ rew,
    uint64_t* __restrict__ rchk) {
  __shared__ Stage<kStageLearned> stage[4];
  // wave w owns environments w * lpw .. + lpw - 1 in its first lpw lanes (lanes_per_wave);
  // the episode seed was written by reset_k
  learned_tick<CM, PF>(p, g, *g.seed, k, (blockIdx.x * 4 + (threadIdx.x >> 6)) * lpw, lpw,
                       stage[threadIdx.x >> 6], act, obs_out, obs_mode, rew, rchk);
}

// ---- static shadow system: one tick ---------------------------------------------------------
// The set of idle servers {j : busy_j <= now} and the next completion min{busy_j > now} only
// change at a completion instant or a dispatch, so they are kept as a bit mask and a time and
// recomputed by one scan of the servers at those points (not at every arrival).
// Busy-until times of the static system's servers: the first kBusyRegs in registers, the rest
// in the wave's slab of LDS, one double per lane, so that a 16-server system does not spill
// them inside the event loop (four workgroups of four waves fill the CU's 160 KiB exactly:
// 20 KiB of arrival stages and 20 KiB of busy times each). Loops over j with a compile-time bound resolve each
// access to a register or an LDS word at a fixed offset.
constexpr int kBusyRegs = 6;
template <int KM>
struct BusyTimes {
  static constexpr int KR = KM > 8 ? kBusyRegs : KM;
  double r[KR];
  double* slab;   // [KM - KR][64] in LDS (unused when KM <= 8)
  int lane;
  __device__ __forceinline__ double get(int j) const {
    return j < KR ? r[j < KR ? j : 0] : slab[(j - KR) * 64 + lane];
  }
  __device__ __forceinline__ void set(int j, double v) {
    if (KM <= KR || j < KR) put<KR>(r, j, v);
    else slab[(j - KR) * 64 + lane] = v;
  }
};

template <int KM>
__device__ __forceinline__ void server_scan(const BusyTimes<KM>& busy, int K, double now,
                                            uint32_t& idle, double& next_done) {
  idle = 0u;
  next_done = kInf;
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    if (j < K) {
      const double b = busy.get(j);
      if (b <= now) idle |= 1u << j;
      else if (b < next_done) next_done = b;
    }
  }
}

// one byte per server (at most 16) in two 64-bit registers
struct ServerBytes {
  uint64_t lo = 0, hi = 0;
  __device__ __forceinline__ uint32_t get(int j) const {
    return (uint32_t)(((j < 8 ? lo : hi) >> (8 * (j & 7))) & 0xffu);
  }
  __device__ __forceinline__ void set(int j, uint32_t v) {
    const int sh = 8 * (j & 7);
    const uint64_t keep = ~(0xffull << sh), x = (uint64_t)(v & 0xffu) << sh;
    lo = j < 8 ? (lo & keep) | x : lo;
    hi = j < 8 ? hi : (hi & keep) | x;
  }
};
static_assert(kMaxK <= 16, "ServerBytes holds 16 servers");

// Server for the static rule's next batch among the idle ones: the lowest index; uniformly
// at random (the idx-th idle server in index order, idx = floor(u * n_idle), u from ROUTE
// block jroute of (env, tick, system 1)); or round robin (the first idle server at or after
// the pointer rr, cyclically).
__device__ __forceinline__ int route_pick(uint32_t idle, int route, uint32_t rr, uint64_t seed,
                                          int e, uint32_t k, uint32_t& jroute) {
  if (route == 1) {
    const int n_idle = __popc(idle);
    const u32x4 w = draw(seed, (uint32_t)e, k, P_ROUTE, jroute++, 1);
    int idx = (int)(unit(w.x, w.y) * (double)n_idle);
    if (idx > n_idle - 1) idx = n_idle - 1;
    uint32_t m = idle;
    for (int i = 0; i < idx; ++i) m &= m - 1u;  // drop the idx lowest idle servers
    return __builtin_ctz(m);
  }
  if (route == 2) {
    const uint32_t at_or_after = idle & ~((1u << rr) - 1u);
    return __builtin_ctz(at_or_after ? at_or_after : idle);
  }
  return __builtin_ctz(idle);
}

// Shortest-Queue routing (Sec. 5.1 baselines): each server holds the batch it runs (completion
// busy_j, size infl_j) and at most one batch queued behind it (completion c2_j, size n2_j),
// served in order. At a scan instant `now` the batches that have completed (c <= now) leave
// their server and count as completed; the slot mask marks servers with room for a batch
// (nothing queued) and next_done is the next completion.
template <int KM>
struct SqState {
  double c2[KM];
  ServerBytes n2;
};

template <int KM>
__device__ __forceinline__ void sq_scan(BusyTimes<KM>& busy, ServerBytes& infl, SqState<KM>& sq,
                                        int K, double now, uint32_t& done, uint32_t& slots,
                                        double& next_done) {
  slots = 0u;
  next_done = kInf;
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    if (j < K) {
      double b = busy.get(j);
      uint32_t n1 = infl.get(j);
      if (n1 > 0 && b <= now) {
        done += n1;
        n1 = sq.n2.get(j);
        if (n1 > 0) b = sq.c2[j];
        sq.n2.set(j, 0u);
        if (n1 > 0 && b <= now) {
          done += n1;
          n1 = 0;
        }
        busy.set(j, b);
        infl.set(j, n1);
      }
      if (sq.n2.get(j) == 0u) slots |= 1u << j;
      if (n1 > 0 && b > now && b < next_done) next_done = b;
    }
  }
}

// Ticks k0 .. k0 + nt - 1 of the static system of one environment whose state is held in
// registers: per tick, arrivals, the static rule's dispatches to the routed server,
// completions, and the tick's reward (into rew [nt][E] when given).
//
// Each lane runs through its own ticks, in one of four modes:
//   EVT    it takes its next event (switch, arrival, completion or timeout instant) in the
//          tick, or finds that none is left (-> READY);
//   PEND   the static rule has a batch to dispatch at the lane's current instant;
//   READY  its tick has no event left and waits to be closed;
//   OFF    all nt ticks are done (or the lane has no environment).
// The wave takes every lane's events one at a time, but serves dispatches and tick closes in
// passes shared by many lanes: a dispatch (service draw, batch pop over the request ring,
// checksum) and a close (a walk over every server) cost the wave the same whether one lane or
// forty take them; so does a refill of the arrival stage (wave_refill). A pending lane waits
// until a quarter of the wave's active lanes are pending too, or no lane has an event to take;
// a lane that needs arrival draws staged waits until a quarter of the active lanes do, or no
// lane takes an event; lanes whose tick is over wait until half of the active lanes are.
// Waiting changes no result: a lane's state is frozen while it waits, and each lane still
// processes its own events, dispatches and closes in the order of its timeline.
// The event counts of bursty environments differ widely from tick to tick; stepping the lanes
// tick by tick would take, at every tick, as many passes as the busiest lane.
//
// A dispatch stores its server's meta word at once; a completion clears the in-flight byte
// only in registers and marks the server in `clear`, and `dirty` marks servers whose
// busy-until time changed; the caller writes both back. With SQ (Shortest-Queue routing) the
// idle mask holds the servers with a free slot instead, and completions are retired at every
// scan (sq_scan).
// shares of the wave's active lanes that trigger a dispatch pass, a close pass and a refill
// pass (1 / share of the lanes; measured at C5 and on the baseline workloads)
constexpr int kDispatchShare = 4, kCloseShare = 2, kRefillShare = 4;
template <int KM, int CM, bool SQ>
__device__ __forceinline__ void static_run(const SimParams& p, const SysState& G, uint32_t* err,
                                           uint64_t seed, uint32_t k0, int nt, bool live, int e,
                                           int ee, int e_lane0, int lane, Stage<kStageStatic>& st,
                                           Queue<CM>& Q, Count& C, Arrivals& A,
                                           BusyTimes<KM>& busy, ServerBytes& infl,
                                           SqState<KM>& sq, uint32_t& dirty, uint32_t& clear,
                                           uint32_t& rr, double* __restrict__ rew) {
  enum { OFF = 0, EVT = 1, PEND = 2, READY = 3 };
  const size_t E = (size_t)p.E;
  // the lane's current tick: index i in the launch, k = k0 + i, interval [t0, t1)
  int i = 0;
  uint32_t k = k0;
  double t0 = 0.0, t1 = 0.0, now = 0.0, next_done = kInf;
  uint32_t idle = 0u, jroute = 0u, staged_hi = 0u, it = 0u;
  int A_k = 0;
  int mode = OFF;
  // the static rule's condition at `now`: a server (slot) free, and B requests of the head-of-
  // line class waiting or its head waiting for T
  auto due = [&]() -> bool {
    if (idle == 0u || Q.qsum <= 0) return false;
    return Q.q(Q.hh) >= p.bmax || now >= Q.hts_h + p.static_timeout;
  };
  auto begin_tick = [&]() {
    C.n_k = 0;
    C.Lw = 0.0;
    C.jsvc = 0;
    A.jarr = 0;
    A.jproc = 0;
    jroute = 0;
    A_k = 0;
    staged_hi = 0;
    it = 0;
    t0 = (double)k * p.dt;
    t1 = (double)(k + 1) * p.dt;
    now = t0;
    if constexpr (SQ) sq_scan(busy, infl, sq, p.K, now, C.c[C_DONE], idle, next_done);
    else server_scan(busy, p.K, now, idle, next_done);
    mode = due() ? PEND : EVT;
  };
  if (live && nt > 0) begin_tick();
  for (;;) {
    bool go = false, need = false;
    double te = now;
    if (mode == EVT) {
      te = A.next_sw < A.next_arr ? A.next_sw : A.next_arr;
      if (next_done < te) te = next_done;
      if (Q.qsum > 0 && idle != 0u) {
        const double tout = Q.hts_h + p.static_timeout;
        if (tout > now && tout < te) te = tout;
      }
      if (!(te < t1)) {
        mode = READY;
      } else if (it > kMaxEventsPerTick) {
        atomicOr(err, ERR_EVENTS);
        mode = READY;
      } else {
        need = p.arrival_kind != 1 && (A.next_sw == te || A.next_arr == te) &&
               A.jarr + 2u > staged_hi;
        go = !need;
      }
    }
    const uint64_t need_m = __ballot(need);
    if (need_m != 0ull && (kRefillShare * __popcll(need_m) >= __popcll(__ballot(mode != OFF)) ||
                           __ballot(go) == 0ull))
      refill_arrivals<CM>(st, p, need, A.jarr, staged_hi, seed, e_lane0, k, lane);
    if (go) {
      ++it;
      now = te;
      if (next_done == now) {
        if constexpr (SQ) sq_scan(busy, infl, sq, p.K, now, C.c[C_DONE], idle, next_done);
        else server_scan(busy, p.K, now, idle, next_done);
      }
      const int cls = advance_staged<CM>(A, p, st, lane, seed, ee, k, now);
      if (cls >= 0) {
        ++A_k;
        enqueue(Q, C, p, cls, now);
      }
      if (due()) mode = PEND;
    }
    const int n_act = __popcll(__ballot(mode != OFF));
    const int n_pend = __popcll(__ballot(mode == PEND));
    const int n_work = __popcll(__ballot(mode == EVT));
    if (n_pend > 0 && (kDispatchShare * n_pend >= n_act || n_work == 0) && mode == PEND) {
      // one batch: min(B, Q_h) requests of the head-of-line class to the routed server
      const int h = Q.hh;
      const int qh = Q.q(h);
      const int n = qh < p.bmax ? qh : p.bmax;
      if constexpr (SQ) {
        // the server with the fewest requests assigned among those with a free slot (nothing
        // queued: the load is its running batch), ties to the lower index; the batch starts
        // when that server has finished its running batch
        int j = -1;
        uint32_t best = 0u;
#pragma unroll
        for (int jj = 0; jj < KM; ++jj) {
          const uint32_t L = infl.get(jj);
          if (jj < p.K && ((idle >> jj) & 1u) && (j < 0 || L < best)) {
            j = jj;
            best = L;
          }
        }
        const uint32_t n1 = infl.get(j);
        const double start = n1 > 0u ? busy.get(j) : now;
        const double sv = service<CM>(C, p, seed, ee, k, 1, h, n);
        const double cdone = pop_batch(Q, C, p, k, j, h, n, start, sv);
        if (n1 == 0u) {
          busy.set(j, cdone);
          infl.set(j, (uint32_t)n);
          if (cdone > now && cdone < next_done) next_done = cdone;
        } else {
          put<KM>(sq.c2, j, cdone);
          sq.n2.set(j, (uint32_t)n);
          idle &= ~(1u << j);
        }
      } else {
        const int j = route_pick(idle, p.route, rr, seed, ee, k, jroute);
        if (p.route == 2) rr = (uint32_t)((j + 1) % p.K);
        C.c[C_DONE] += infl.get(j);  // the previous batch on j finished at busy_j <= now
        infl.set(j, (uint32_t)n);
        const double sv = service<CM>(C, p, seed, ee, k, 1, h, n);
        const double cdone = pop_batch(Q, C, p, k, j, h, n, now, sv);
        busy.set(j, cdone);
        G.meta[(size_t)j * E + ee] = (uint32_t)n | ((uint32_t)n << 8) | ((uint32_t)h << 16);
        dirty |= 1u << j;
        if (cdone > now) {
          idle &= ~(1u << j);
          if (cdone < next_done) next_done = cdone;
        }
      }
      if (!due()) mode = EVT;
    }
    const int n_ready = __popcll(__ballot(mode == READY));
    if (kCloseShare * n_ready >= n_act && mode == READY) {
      // completions before t1, the tick's reward, then the lane's next tick
      if constexpr (SQ) {
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          if (j < p.K) {
            uint32_t n1 = infl.get(j);
            if (n1 > 0 && busy.get(j) < t1) {
              C.c[C_DONE] += n1;
              n1 = sq.n2.get(j);
              if (n1 > 0) busy.set(j, sq.c2[j]);
              sq.n2.set(j, 0u);
              if (n1 > 0 && busy.get(j) < t1) {
                C.c[C_DONE] += n1;
                n1 = 0;
              }
              infl.set(j, n1);
            }
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          const uint32_t n = infl.get(j);
          if (j < p.K && n > 0 && busy.get(j) < t1) {
            C.c[C_DONE] += n;
            clear |= 1u << j;
            infl.set(j, 0u);
          }
        }
      }
      const double r = close_tick(Q, C, p, A.proc, A_k);
      if (rew) rew[(size_t)i * E + e] = r;
      ++i;
      ++k;
      if (i < nt) begin_tick();
      else mode = OFF;
    }
    if (__ballot(mode != OFF) == 0ull) break;
  }
}

// Ticks k0 .. k0 + nt - 1 of the static shadow system. The static rule never looks at the
// learned system, so one launch may cover many ticks: the state is loaded once, kept in
// registers from tick to tick, and stored once; each lane advances at its own pace instead of
// waiting at every tick for the slowest lane of its wave. rew [nt][E] (optional) receives the
// rewards; nt = 1 is the per-tick kernel of the step interface.
template <int KM, int CM, bool SQ>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void static_k(
    SimParams p, EnvState g, uint32_t k0, int nt, int lpw, double* __restrict__ rew) {
  const uint64_t seed = *g.seed;   // the episode seed, written by reset_k
  __shared__ Stage<kStageStatic> stage[4];
  __shared__ double busy_lds[4][KM > 8 ? KM - kBusyRegs : 1][64];
  const int lane = threadIdx.x & 63;
  Stage<kStageStatic>& st = stage[threadIdx.x >> 6];
  // wave w owns environments w * lpw .. + lpw - 1 in its first lpw lanes (lanes_per_wave)
  const int e_lane0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * lpw;
  const int e = e_lane0 + lane;
  const bool live = lane < lpw && e < p.E;
  if (__ballot(live) == 0ull) return;
  const int ee = live ? e : 0;
  const size_t E = (size_t)p.E;
  const SysState& G = g.sys[1];
  Queue<CM> Q;
  load_queue(Q, G, p, ee);
  Count C;
  load_count(C, G, p, ee);
  Arrivals A;
  load_arrivals(A, G, p, ee);
  // busy-until times in registers; of each server's meta word only the in-flight count
  // (low byte) is kept, eight servers to a 64-bit register (the word is stored at dispatch)
  BusyTimes<KM> busy;
  busy.slab = &busy_lds[threadIdx.x >> 6][0][0];
  busy.lane = lane;
  ServerBytes infl;
  SqState<KM> sq;
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    busy.set(j, j < p.K ? G.busy[(size_t)j * E + ee] : kInf);
    if (j < p.K) {
      const uint32_t m = G.meta[(size_t)j * E + ee];
      infl.set(j, m & 0xffu);
      if constexpr (SQ) {
        sq.n2.set(j, m >> 24);
        sq.c2[j] = G.busy2[(size_t)j * E + ee];
      }
    }
  }
  uint32_t dirty = 0, clear = 0;
  uint32_t rr = p.route == 2 ? G.rr[ee] : 0u;
  static_run<KM, CM, SQ>(p, G, g.err, seed, k0, nt, live, e, ee, e_lane0, lane, st, Q, C, A,
                         busy, infl, sq, dirty, clear, rr, rew);
  if (!live) return;
  if constexpr (SQ) {
    // every server's running and queued batch: completion times and the meta word (running
    // size in the low byte, queued size in the high byte)
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      if (j < p.K) {
        G.busy[(size_t)j * E + e] = busy.get(j);
        G.busy2[(size_t)j * E + e] = sq.c2[j];
        G.meta[(size_t)j * E + e] = infl.get(j) | (sq.n2.get(j) << 24);
      }
    }
    store_queue(Q, G, p, e);
    store_count(C, G, p, e);
    store_arrivals(A, G, p, e);
    return;
  }
  // servers whose last batch completed: clear the in-flight byte of the stored meta word
  uint32_t m[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j)
    m[j] = ((clear >> j) & 1u) && infl.get(j) == 0u ? G.meta[(size_t)j * E + e] : 0u;
#pragma unroll
  for (int j = 0; j < KM; ++j)
    if (((clear >> j) & 1u) && infl.get(j) == 0u) G.meta[(size_t)j * E + e] = m[j] & ~0xffu;
#pragma unroll
  for (int j = 0; j < KM; ++j)
    if (dirty & (1u << j)) G.busy[(size_t)j * E + e] = busy.get(j);
  if (p.route == 2) G.rr[e] = rr;
  store_queue(Q, G, p, e);
  store_count(C, G, p, e);
  store_arrivals(A, G, p, e);
}

// ---- reset ------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void reset_k(SimParams p, EnvState g, uint64_t seed) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e == 0) *g.seed = seed;   // read by every later kernel of the episode
  if (e >= p.E) return;
  const size_t E = (size_t)p.E;
  // modulating state from its stationary law, its dwell, then the first arrival
  uint32_t proc = 0;
  double next_sw = kInf, next_arr = kInf;
  if (p.arrival_kind == 1) {
    // validate the caller's trace: count within capacity, classes within range
    const int cnt = p.tr_cnt[e];
    bool bad = cnt < 0 || cnt > p.tr_len;
    const int n = cnt < 0 ? 0 : (cnt > p.tr_len ? p.tr_len : cnt);
    for (int i = 0; i < n; ++i) bad = bad || p.tr_cls[(size_t)e * p.tr_len + i] >= p.C;
    if (bad) atomicOr(g.err, ERR_TRACE);
    next_arr = n > 0 ? p.tr_times[(size_t)e * p.tr_len] : kInf;
  } else {
    if (p.S > 1 && p.dwell_kind[0] == 3) {
      // a square wave starts in state 0 with its full dwell: the same phase everywhere
      proc = 0;
      next_sw = p.dwell_mean[0];
    } else if (p.S > 1) {
      const u32x4 w = draw(seed, (uint32_t)e, STEP_RESET, P_PROCESS, 0, 0);
      const double us = unit(w.z, w.w);
      int st = p.S - 1;
#pragma unroll
      for (int i = kMaxS - 2; i >= 0; --i)
        if (i < p.S - 1 && us < p.stat_cum[i]) st = i;
      proc = (uint32_t)st;
      next_sw = dwell(p, st, unit(w.x, w.y));
    }
    if (pick<kMaxS>(p.rate, (int)proc) > 0.0) {
      const u32x4 w = draw(seed, (uint32_t)e, STEP_RESET, P_ARRIVAL, 0, 0);
      next_arr = -dlog(unit(w.x, w.y)) * pick<kMaxS>(p.mean_gap, (int)proc);
    }
  }
  const int nsys = p.shadow ? 2 : 1;
  for (int sy = 0; sy < nsys; ++sy) {
    const SysState& s = g.sys[sy];
    s.qpack[e] = 0u;
    s.hpack[e] = 0u;
    for (int c = 0; c < p.C; ++c) s.hts[(size_t)c * E + e] = 0.0;
    for (int j = 0; j < p.K; ++j) {
      s.busy[(size_t)j * E + e] = 0.0;
      s.meta[(size_t)j * E + e] = 0xffu << 16;
      if (s.busy2) s.busy2[(size_t)j * E + e] = kInf;
    }
    for (int i = 0; i < kNcnt; ++i) s.cnt[(size_t)i * E + e] = 0u;
    s.sums[e] = 0.0;
    s.sums[E + e] = 0.0;
    s.chk[e] = kFnvInit;
    s.proc[e] = proc;
    s.next_sw[e] = next_sw;
    s.next_arr[e] = next_arr;
    s.tr_idx[e] = 0u;
    s.rr[e] = 0u;
  }
  for (int r = 0; r < 4; ++r) g.ewma[(size_t)r * E + e] = 0.0;
  // obs_0 is all zeros: empty queues, idle servers, no last batch (class feature
  // (none + 1)/C = 0), zero rates
  for (int i = 0; i < p.F; ++i) g.obs[(size_t)i * E + e] = 0.0f;
}

// per-env counters out: [2][7][E] int64 (7th = inflight), sums [2][2][E]
// bf16 pairs of the current observation: pair m of environment e packs features 2m and 2m + 1
// (zero past the last feature), rounded as a bf16 policy rounds its input
__global__ __launch_bounds__(256) void obs_pack_k(SimParams p, EnvState g) {
  const int e = blockIdx.x * 256 + threadIdx.x, m = blockIdx.y;
  if (e >= p.E) return;
  const size_t E = (size_t)p.E;
  const float a = g.obs[(size_t)(2 * m) * E + e];
  const float b = 2 * m + 1 < p.F ? g.obs[(size_t)(2 * m + 1) * E + e] : 0.0f;
  g.obs_bf[(size_t)m * E + e] = pack_bf16_pair(a, b);
}

__global__ void counters_k(SimParams p, EnvState g, int64_t* cnt, double* sums) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= p.E) return;
  const size_t E = (size_t)p.E;
  for (int sy = 0; sy < 2; ++sy) {
    const bool on = sy == 0 || p.shadow;
    const SysState& s = g.sys[sy];
    if (cnt) {
      int64_t* o = cnt + (size_t)sy * 7 * E;
      int64_t infl = 0;
      for (int i = 0; i < kNcnt; ++i)
        o[(size_t)i * E + e] = on ? (int64_t)s.cnt[(size_t)i * E + e] : 0;
      if (on)
        for (int j = 0; j < p.K; ++j) {
          const uint32_t m = s.meta[(size_t)j * E + e];
          infl += (m & 0xffu) + (m >> 24);   // running batch, batch queued (Shortest-Queue)
        }
      o[(size_t)6 * E + e] = infl;
    }
    if (sums) {
      double* o = sums + (size_t)sy * 2 * E;
      o[e] = on ? s.sums[e] : 0.0;
      o[E + e] = on ? s.sums[E + e] : 0.0;
    }
  }
}

// totals over environments: wave shuffle reduction, then one atomic per wave
__global__ __launch_bounds__(256) void totals_k(SimParams p, EnvState g, int64_t* tc, double* ts) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  const size_t E = (size_t)p.E;
  const int lane = threadIdx.x & 63;
  for (int sy = 0; sy < 2; ++sy) {
    const bool on = (sy == 0 || p.shadow) && e < p.E;
    const SysState& s = g.sys[sy];
    for (int i = 0; i < 7; ++i) {
      long long v = 0;
      if (on) {
        if (i < kNcnt) {
          v = s.cnt[(size_t)i * E + e];
        } else {
          for (int j = 0; j < p.K; ++j) {
            const uint32_t m = s.meta[(size_t)j * E + e];
            v += (m & 0xffu) + (m >> 24);
          }
        }
      }
      for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off, 64);
      if (lane == 0 && v) atomicAdd((unsigned long long*)&tc[sy * 7 + i], (unsigned long long)v);
    }
    for (int i = 0; i < 2; ++i) {
      double v = on ? s.sums[(size_t)i * E + e] : 0.0;
      for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off, 64);
      if (lane == 0) atomicAdd(&ts[sy * 2 + i], v);
    }
  }
}

// Lanes per wave of the tick kernels (one environment per lane). A wave's tick lasts as long
// as its busiest lane, and a batch of fewer than kFillWaves * 64 environments leaves SIMDs
// without a wave: such batches are spread over more waves with fewer environments each (down
// to 4), which shortens every wave's tick at no cost in issue slots.
constexpr int kFillWaves = 1024;
int lanes_per_wave(int E) {
  int lpw = 64;
  while (lpw > 4 && (E + lpw - 1) / lpw < kFillWaves) lpw >>= 1;
  return lpw;
}

template <int CM>
void launch_static_c(const SimParams& p, const EnvState& s, uint32_t k, int nt,
                     double* rew_sh, hipStream_t st) {
  const int lpw = lanes_per_wave(p.E);
  const int waves = (p.E + lpw - 1) / lpw;
  const dim3 grid((waves + 3) / 4), block(256);
  if (p.route == 3) {   // Shortest-Queue (at most 8 servers)
    if (p.K <= 2) hipLaunchKernelGGL((static_k<2, CM, true>), grid, block, 0, st, p, s, k, nt, lpw, rew_sh);
    else if (p.K <= 4) hipLaunchKernelGGL((static_k<4, CM, true>), grid, block, 0, st, p, s, k, nt, lpw, rew_sh);
    else hipLaunchKernelGGL((static_k<8, CM, true>), grid, block, 0, st, p, s, k, nt, lpw, rew_sh);
    return;
  }
  if (p.K <= 1) hipLaunchKernelGGL((static_k<1, CM, false>), grid, block, 0, st, p, s, k, nt, lpw, rew_sh);
  else if (p.K <= 4) hipLaunchKernelGGL((static_k<4, CM, false>), grid, block, 0, st, p, s, k, nt, lpw, rew_sh);
  else if (p.K <= 8) hipLaunchKernelGGL((static_k<8, CM, false>), grid, block, 0, st, p, s, k, nt, lpw, rew_sh);
  else hipLaunchKernelGGL((static_k<16, CM, false>), grid, block, 0, st, p, s, k, nt, lpw, rew_sh);
}

}  // namespace

hipError_t launch_reset(const SimParams& p, const EnvState& s, uint64_t seed, hipStream_t st) {
  hipLaunchKernelGGL(reset_k, dim3((p.E + 255) / 256), dim3(256), 0, st, p, s, seed);
  return hipGetLastError();
}

template <bool PF>
void launch_learned(const SimParams& p, const EnvState& s, uint32_t k, int lpw, dim3 grid,
                    const uint8_t* act, float* obs_out, int obs_mode, double* rew,
                    uint64_t* rchk, hipStream_t st) {
  const dim3 block(256);
  if (p.C <= 1)
    hipLaunchKernelGGL((learned_k<1, PF>), grid, block, 0, st, p, s, k, lpw, act, obs_out, obs_mode, rew, rchk);
  else if (p.C <= 2)
    hipLaunchKernelGGL((learned_k<2, PF>), grid, block, 0, st, p, s, k, lpw, act, obs_out, obs_mode, rew, rchk);
  else
    hipLaunchKernelGGL((learned_k<4, PF>), grid, block, 0, st, p, s, k, lpw, act, obs_out, obs_mode, rew, rchk);
}

hipError_t launch_step(const SimParams& p, const EnvState& s, uint32_t k,
                       const uint8_t* act, float* obs_out, int obs_mode, double* rew,
                       uint64_t* rchk, hipStream_t st) {
  if ((obs_mode & kObsBf16) && !s.obs_bf) return hipErrorInvalidValue;
  const int lpw = lanes_per_wave(p.E);
  const int waves = (p.E + lpw - 1) / lpw;
  const dim3 grid((waves + 3) / 4);
  // early end-of-tick reads when every wave has a SIMD to itself
  if (waves <= kFillWaves && p.K <= kEndChunk)
    launch_learned<true>(p, s, k, lpw, grid, act, obs_out, obs_mode, rew, rchk, st);
  else
    launch_learned<false>(p, s, k, lpw, grid, act, obs_out, obs_mode, rew, rchk, st);
  return hipGetLastError();
}

hipError_t launch_obs_pack(const SimParams& p, const EnvState& s, hipStream_t st) {
  if (!s.obs_bf) return hipErrorInvalidValue;
  const int pairs = (p.F + 1) / 2;
  hipLaunchKernelGGL(obs_pack_k, dim3((p.E + 255) / 256, pairs), dim3(256), 0, st, p, s);
  return hipGetLastError();
}

hipError_t launch_static(const SimParams& p, const EnvState& s, uint32_t k,
                         int nt, double* rew_sh, hipStream_t st) {
  if (nt < 1) return hipErrorInvalidValue;
  if (p.C <= 1) launch_static_c<1>(p, s, k, nt, rew_sh, st);
  else if (p.C <= 2) launch_static_c<2>(p, s, k, nt, rew_sh, st);
  else launch_static_c<4>(p, s, k, nt, rew_sh, st);
  return hipGetLastError();
}

hipError_t launch_counters(const SimParams& p, const EnvState& s, int64_t* cnt, double* sums,
                           hipStream_t st) {
  hipLaunchKernelGGL(counters_k, dim3((p.E + 255) / 256), dim3(256), 0, st, p, s, cnt, sums);
  return hipGetLastError();
}

hipError_t launch_totals(const SimParams& p, const EnvState& s, int64_t* d_tot_cnt,
                         double* d_tot_sum, hipStream_t st) {
  hipLaunchKernelGGL(totals_k, dim3((p.E + 255) / 256), dim3(256), 0, st, p, s, d_tot_cnt,
                     d_tot_sum);
  return hipGetLastError();
}

}  // namespace bsim
