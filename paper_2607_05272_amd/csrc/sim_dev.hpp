// sim_dev.hpp -- device code of the batched discrete-event simulator: the environments'
// state, the arrival process and its staged draws, queues, dispatch, reward and observation,
// and one tick of the learned system (learned_tick), shared by the per-tick kernel and the
// fused small-batch rollout kernel.
//
//
// One lane owns one environment for the whole tick: its structure-of-arrays state is read
// with coalesced loads into registers, the tick's events are processed in time order, and
// the state is written back. Model (paper Sec. 3.1, Sec. 4.1):
//   - arrivals from a modulated Poisson process (Poisson, MMPP or heavy-tailed ON/OFF,
//     Sec. 3.2) or an explicit trace; each arrival carries a class (model type);
//   - per-class FIFO queues holding at most N waiting requests in total, arrivals beyond
//     that are dropped (load shedding);
//   - K servers; a batch of n requests of one class occupies a server for alpha + beta*n
//     (or a lognormal / exponential time);
//   - the learned system dispatches exactly b = 2^(a%6) requests of the head-of-line class
//     to server a/6 whenever that server is idle and the class holds >= b requests;
//   - the optional shadow system applies the static rule (B requests or timeout T) to the
//     same arrivals;
//   - reward = w_thr * dispatched/dt - mean (or sum) of the class-weighted latencies of the
//     requests dispatched in the tick, attributed at dispatch.
// A batch is dispatched at the earliest event instant of the tick at which its condition
// holds; the loop visits every arrival, switch, completion of a relevant server and
// timeout instant in time order. Ties at one instant: switch, arrival, then dispatch.
//
// The learned system only touches server a/6 inside the tick, so its kernel keeps that one
// server in registers and streams over all servers once at the end of the tick
// (completions and observation). The static system needs every server inside the tick
// (lowest idle server, next completion) and runs as its own kernel with all of them in
// registers. Each system advances its own copy of the arrival process with the same
// draws, so both see the same arrivals.
#pragma once
#include "devmath.hpp"
#include "params.hpp"

namespace bsim {
namespace {

enum { C_ARR = 0, C_ACC = 1, C_DROP = 2, C_DISP = 3, C_BATCH = 4, C_DONE = 5 };
constexpr double kInf = __builtin_huge_val();

// Per-lane select from / update of a small array with compile-time bound M. Both are
// written as selects of values on every element (no conditional store), so that the
// array stays in registers: a store through a selected element address would force it
// into scratch memory.
template <int M, typename T, int L>
__device__ __forceinline__ T pick(const T (&a)[L], int i) {
  T v = a[0];
#pragma unroll
  for (int c = 1; c < M; ++c) v = i == c ? a[c] : v;
  return v;
}
template <int M, typename T, int L>
__device__ __forceinline__ void put(T (&a)[L], int i, T v) {
#pragma unroll
  for (int c = 0; c < M; ++c) a[c] = i == c ? v : a[c];
}

// ---- per-class FIFO queues of one system ---------------------------------------------------
template <int CM>
struct Queue {
  uint32_t qp, hp;  // per-class length / ring head, one byte per class
  double hts[CM];   // arrival time of each class's head request
  int qsum;
  int hh;           // head-of-line class (see hol), -1 when every queue is empty
  double hts_h;     // arrival time of its head request
  double* ring;     // this environment's rings [C][N]
  __device__ __forceinline__ int q(int c) const { return (int)((qp >> (8 * c)) & 0xffu); }
  __device__ __forceinline__ int hd(int c) const { return (int)((hp >> (8 * c)) & 0xffu); }
};

// head-of-line class: oldest head request, ties to the lower class index; -1 if empty
template <int CM>
__device__ __forceinline__ int hol(const Queue<CM>& Q, const SimParams& p, double& ts) {
  int h = -1;
  ts = 0.0;
#pragma unroll
  for (int c = 0; c < CM; ++c) {
    if (c < p.C && Q.q(c) > 0 && (h < 0 || Q.hts[c] < ts)) {
      h = c;
      ts = Q.hts[c];
    }
  }
  return h;
}

template <int CM>
__device__ __forceinline__ void load_queue(Queue<CM>& Q, const SysState& g, const SimParams& p,
                                           int e) {
  const size_t E = (size_t)p.E;
  Q.qp = g.qpack[e];
  Q.hp = g.hpack[e];
  Q.qsum = 0;
#pragma unroll
  for (int c = 0; c < CM; ++c) {
    Q.hts[c] = c < p.C ? g.hts[(size_t)c * E + e] : 0.0;
    Q.qsum += Q.q(c);
  }
  Q.ring = g.ring + (size_t)e * p.C * p.N;
  Q.hh = hol(Q, p, Q.hts_h);
}

template <int CM>
__device__ __forceinline__ void store_queue(const Queue<CM>& Q, const SysState& g,
                                            const SimParams& p, int e) {
  const size_t E = (size_t)p.E;
  g.qpack[e] = Q.qp;
  g.hpack[e] = Q.hp;
#pragma unroll
  for (int c = 0; c < CM; ++c)
    if (c < p.C) g.hts[(size_t)c * E + e] = Q.hts[c];
}


// ---- counters of one system -----------------------------------------------------------------
struct Count {
  uint32_t c[kNcnt];
  double lat, wlat;
  uint64_t chk;
  int n_k;        // requests dispatched this tick
  double Lw;      // weighted latency of this tick's dispatches (FIFO order)
  uint32_t jsvc;  // service draws this tick
};

__device__ __forceinline__ void load_count(Count& C, const SysState& g, const SimParams& p, int e) {
  const size_t E = (size_t)p.E;
#pragma unroll
  for (int i = 0; i < kNcnt; ++i) C.c[i] = g.cnt[(size_t)i * E + e];
  C.lat = g.sums[e];
  C.wlat = g.sums[E + e];
  C.chk = g.chk[e];
  C.n_k = 0;
  C.Lw = 0.0;
  C.jsvc = 0;
}

__device__ __forceinline__ void store_count(const Count& C, const SysState& g, const SimParams& p,
                                            int e) {
  const size_t E = (size_t)p.E;
#pragma unroll
  for (int i = 0; i < kNcnt; ++i) g.cnt[(size_t)i * E + e] = C.c[i];
  g.sums[e] = C.lat;
  g.sums[E + e] = C.wlat;
  g.chk[e] = C.chk;
}

// ---- arrival process (one copy per system; identical draws) ---------------------------------
struct Arrivals {
  uint32_t proc;
  double next_sw, next_arr;
  double gap;  // mean gap of the current state (a per-lane indexed read of the parameters
               // compiles to a memory load, which every arrival would otherwise wait for)
  uint32_t tr_idx;
  int tr_cnt;
  uint32_t jarr, jproc;
};

__device__ __forceinline__ void load_arrivals(Arrivals& A, const SysState& g, const SimParams& p,
                                              int e) {
  A.proc = g.proc[e];
  A.next_sw = g.next_sw[e];
  A.next_arr = g.next_arr[e];
  A.gap = pick<kMaxS>(p.mean_gap, (int)A.proc);
  A.tr_idx = 0;
  A.tr_cnt = 0;
  if (p.arrival_kind == 1) {
    A.tr_idx = g.tr_idx[e];
    const int c = p.tr_cnt[e];
    A.tr_cnt = c < 0 ? 0 : (c < p.tr_len ? c : p.tr_len);  // reset flags invalid counts
  }
  A.jarr = 0;
  A.jproc = 0;
}

__device__ __forceinline__ void store_arrivals(const Arrivals& A, const SysState& g,
                                               const SimParams& p, int e) {
  g.proc[e] = A.proc;
  g.next_sw[e] = A.next_sw;
  g.next_arr[e] = A.next_arr;
  if (p.arrival_kind == 1) g.tr_idx[e] = A.tr_idx;
}

template <bool INL = false>
__device__ __forceinline__ double dwell(const SimParams& p, int st, double u) {
  const int kind = pick<kMaxS>(p.dwell_kind, st);
  auto lg = [](double v) { return INL ? dlog_inl(v) : dlog(v); };
  auto ex = [](double v) { return INL ? dexp_inl(v) : dexp(v); };
  if (kind == 1) return -lg(u) * pick<kMaxS>(p.dwell_mean, st);
  if (kind == 2) return pick<kMaxS>(p.xm, st) * ex(-lg(u) * pick<kMaxS>(p.inv_alpha, st));
  if (kind == 3) return pick<kMaxS>(p.dwell_mean, st);  // fixed dwell: square wave
  return kInf;
}

// ---- wave-cooperative staging of ARRIVAL draws ---------------------------------------------
// Block j of purpose ARRIVAL for (env, tick) gives the exponential variate E_j = -log u(w0,w1)
// and, through the class mix, the class of uc_j = u(w2,w3); neither depends on the
// environment's state, only on j. Each lane reads them from a per-wave LDS stage of KS
// slots; when lanes run short, the whole wave refills: lane l of the wave computes work
// items l, l+64, ... of the list of (needing lane, block), so the Philox draws and
// logarithms of a few bursting environments are spread over all 64 lanes. (Service draws
// are not staged: an environment dispatches a few batches per tick at most, and the lanes
// dispatching at one instant already draw together.) The learned tick, whose LDS holds
// nothing else, stages 16 slots (fewer refills in bursts: -2.5% per C5 launch against 8); the
// static system shares the CU's LDS with its servers' busy times and stages 8.
constexpr int kStageLearned = 16, kStageStatic = 8;
template <int KS>
struct Stage {
  double E[KS][64];
  uint8_t cls[KS][64];
  uint32_t owner_j0[64];  // needing lane | first block << 6
  uint32_t tick[64];
};
// A tick takes at most kMaxEventsPerTick events and each consumes at most two ARRIVAL blocks,
// so a first block index fits the 26 bits above the lane.
static_assert(2ull * kMaxEventsPerTick + 2 * kStageLearned < (1ull << 26), "owner_j0 packing");

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Called by all 64 lanes of the wave. Lanes with `need` get blocks [jneed, jneed + n) of
// their tick k with n = KS when the arrival process can burst (`burst`: some state's rate
// exceeds KS / 4 arrivals per tick) or one of the lanes was already refilled in its tick,
// else KS / 2: at low arrival rates most lanes need one or two blocks per tick, and the work
// of a pass is n times the number of lanes served. The lanes may be at different ticks.
// fill(owner lane, tick, j) computes one block into the stage.
template <int KS, class Fill>
__device__ __forceinline__ void wave_refill(Stage<KS>& st, bool need, bool burst, uint32_t jneed,
                                            uint32_t k, uint32_t& staged_hi, int lane,
                                            Fill&& fill) {
  const uint64_t mask = __ballot(need);
  const int nneed = __popcll(mask);
  static_assert(KS >= 4 && (KS & (KS - 1)) == 0, "stage size is a power of two");
  const int lg = __ballot(need && (burst || staged_hi != 0u)) != 0ull ? __builtin_ctz(KS)
                                                                       : __builtin_ctz(KS) - 1;
  const int n = 1 << lg;
  if (need) {
    const int rank = __popcll(mask & ((1ull << lane) - 1ull));
    st.owner_j0[rank] = (uint32_t)lane | (jneed << 6);
    st.tick[rank] = k;
  }
  wave_sync_lds();
  for (int w = lane; w < n * nneed; w += 64) {
    const int r = w >> lg;
    const uint32_t oj = st.owner_j0[r];
    fill(oj & 63u, st.tick[r], (oj >> 6) + (uint32_t)(w & (n - 1)));
  }
  wave_sync_lds();
  if (need) staged_hi = jneed + (uint32_t)n;
}

// INL: the logarithm inline (kernels with registers to spare) rather than called
template <int CM, int KS, bool INL = false>
__device__ __forceinline__ void refill_arrivals(Stage<KS>& st, const SimParams& p, bool need,
                                                uint32_t jneed, uint32_t& staged_hi,
                                                uint64_t seed, int e_lane0, uint32_t k, int lane) {
  bool burst = false;
#pragma unroll
  for (int s = 0; s < kMaxS; ++s)
    if (s < p.S && p.rate[s] * p.dt * 4.0 > (double)KS) burst = true;
  wave_refill<KS>(st, need, burst, jneed, k, staged_hi, lane, [&](uint32_t own, uint32_t kk,
                                                                   uint32_t j) {
    const u32x4 d = draw(seed, (uint32_t)(e_lane0 + (int)own), kk, P_ARRIVAL, j, 0);
    st.E[j % KS][own] = -(INL ? dlog_inl(unit(d.x, d.y)) : dlog(unit(d.x, d.y)));
    const double uc = unit(d.z, d.w);
    int cls = CM - 1;
#pragma unroll
    for (int c = CM - 2; c >= 0; --c)
      if (uc < p.class_cum[c]) cls = c;
    st.cls[j % KS][own] = (uint8_t)cls;
  });
}

// Processes the switch and/or arrival due at `now` (switch first: it redraws the pending
// arrival from the switch instant). Returns the class of an arrival at `now`, or -1. ARRIVAL
// blocks are read from the stage (the caller guarantees that the two blocks an instant can
// consume, a switch redraw and an arrival, are staged).
template <int CM, int KS, bool INL = false>
__device__ __forceinline__ int advance_staged(Arrivals& A, const SimParams& p, const Stage<KS>& st,
                                              int lane, uint64_t seed, int e, uint32_t k,
                                              double now) {
  if (A.next_sw == now) {
    const u32x4 w = draw(seed, (uint32_t)e, k, P_PROCESS, A.jproc++, 0);
    int nxt;
    if (p.S == 2) {
      nxt = 1 - (int)A.proc;
    } else {
      const int idx = (int)(unit(w.z, w.w) * (double)(p.S - 1));
      nxt = idx < (int)A.proc ? idx : idx + 1;
    }
    A.proc = (uint32_t)nxt;
    A.gap = pick<kMaxS>(p.mean_gap, nxt);
    A.next_sw = now + dwell<INL>(p, nxt, unit(w.x, w.y));
    if (pick<kMaxS>(p.rate, nxt) > 0.0) {
      const uint32_t j = A.jarr++;
      A.next_arr = now + st.E[j % KS][lane] * A.gap;
    } else {
      A.next_arr = kInf;
    }
  }
  if (!(A.next_arr == now)) return -1;
  int cls;
  if (p.arrival_kind == 1) {
    const size_t base = (size_t)e * p.tr_len;
    cls = p.tr_cls[base + A.tr_idx];
    if (cls >= p.C) cls = p.C - 1;  // reset validated every class id; never index past C
    ++A.tr_idx;
    A.next_arr = (int)A.tr_idx < A.tr_cnt ? p.tr_times[base + A.tr_idx] : kInf;
  } else {
    const uint32_t j = A.jarr++;
    cls = st.cls[j % KS][lane];
    A.next_arr = now + st.E[j % KS][lane] * A.gap;
  }
  return cls;
}

// arrival at `now`: FIFO push, or drop when N requests wait (load shedding)
template <int CM>
__device__ __forceinline__ void enqueue(Queue<CM>& Q, Count& C, const SimParams& p, int cls,
                                        double now) {
  C.c[C_ARR] += 1u;
  if (Q.qsum == p.N) {
    C.c[C_DROP] += 1u;
    return;
  }
  const int qc = Q.q(cls);
  int pos = Q.hd(cls) + qc;
  if (pos >= p.N) pos -= p.N;
  Q.ring[(size_t)cls * p.N + pos] = now;
  if (qc == 0) {
    put<CM>(Q.hts, cls, now);
    // the new head is the newest request, so it is the head of line only when every queue
    // was empty, or when it ties the current head of line's time from a lower class
    if (Q.qsum == 0 || (now == Q.hts_h && cls < Q.hh)) {
      Q.hh = cls;
      Q.hts_h = now;
    }
  }
  Q.qp += 1u << (8 * cls);
  Q.qsum += 1;
  C.c[C_ACC] += 1u;
}

// The same arrival as enqueue, written as selects (the ring store aside) for the arrival runs
// of the learned tick: a loop over branchy code keeps copies of the whole queue state in
// flight, while this straight-line form updates it in place.
template <int CM>
__device__ __forceinline__ void enqueue_sel(Queue<CM>& Q, Count& C, const SimParams& p, int cls,
                                            double now) {
  const bool acc = Q.qsum != p.N;
  const int qc = Q.q(cls);
  int pos = Q.hd(cls) + qc;
  pos = pos >= p.N ? pos - p.N : pos;
  if (acc) Q.ring[(size_t)cls * p.N + pos] = now;
  const bool first = acc && qc == 0;
  const bool lead = first && (Q.qsum == 0 || (now == Q.hts_h && cls < Q.hh));
#pragma unroll
  for (int c = 0; c < CM; ++c) Q.hts[c] = first && cls == c ? now : Q.hts[c];
  Q.hh = lead ? cls : Q.hh;
  Q.hts_h = lead ? now : Q.hts_h;
  Q.qp += acc ? 1u << (8 * cls) : 0u;
  Q.qsum += acc ? 1 : 0;
  C.c[C_ARR] += 1u;
  C.c[C_DROP] += acc ? 0u : 1u;
  C.c[C_ACC] += acc ? 1u : 0u;
}

// Service time of a batch of n requests of class h. kind 0: alpha + beta n; kind 1:
// median * exp(sigma Z) + beta n with Z = sqrt(-2 log u1) cos(2 pi u2) (Box-Muller); kind 2:
// -log(u1) (alpha + beta n), with u1, u2 from SERVICE block j of (env, tick, system). Inline in
// both tick kernels: as a call it saved and restored registers through scratch memory at every
// dispatch (its fp64 elementary functions stay out of line, see devmath.hpp).
template <bool INL = false>
__device__ __forceinline__ double service_draw(int kind, double al, double be, double med,
                                            double sigma, int n, uint64_t seed, uint32_t env,
                                            uint32_t k, uint32_t j, uint32_t sys) {
  const u32x4 w = draw(seed, env, k, P_SERVICE, j, sys);
  const double u1 = unit(w.x, w.y);
  auto lg = [](double v) { return INL ? dlog_inl(v) : dlog(v); };
  if (kind == 2) return -lg(u1) * (al + be * (double)n);
  const double u2 = unit(w.z, w.w);
  const double z = sqrt(-2.0 * lg(u1)) * (INL ? dcos_inl(kTwoPi * u2) : dcos(kTwoPi * u2));
  return med * (INL ? dexp_inl(sigma * z) : dexp(sigma * z)) + be * (double)n;
}

template <int CM, bool INL = false>
__device__ __forceinline__ double service(Count& C, const SimParams& p, uint64_t seed, int e,
                                          uint32_t k, int sys, int h, int n) {
  const int kind = pick<CM>(p.svc_kind, h);
  const double al = pick<CM>(p.svc_alpha, h), be = pick<CM>(p.svc_beta, h);
  if (kind == 0) return al + be * (double)n;
  return service_draw<INL>(kind, al, be, pick<CM>(p.svc_median, h), p.svc_sigma, n, seed,
                      (uint32_t)e, k, C.jsvc++, (uint32_t)sys);
}

// Pops n requests of class h dispatched at `now` to server j, on which they complete at
// cdone = now + sv; accumulates their latencies in FIFO order. Returns cdone.
template <int CM>
__device__ __forceinline__ double pop_batch(Queue<CM>& Q, Count& C, const SimParams& p,
                                            uint32_t k, int j, int h, int n, double now,
                                            double sv) {
  const double cdone = now + sv;
  const double wh = pick<CM>(p.w_class, h);
  const int N = p.N;
  const double* rb = Q.ring + (size_t)h * N;
  const int head = Q.hd(h);
  int pos = head + n;
  pos = pos >= N ? pos - N : pos;
  const int qh = Q.q(h) - n;
  // the new head's timestamp (read even when the class empties: pos is inside the ring) and
  // the popped timestamps, eight at a time, are loaded before any of them is used
  const double next_head = rb[pos];
  double Lw = C.Lw, lat = C.lat, wlat = C.wlat;
  for (int i0 = 0; i0 < n; i0 += 8) {
    double a[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int q = head + i0 + i;
      q = q >= N ? q - N : q;
      a[i] = i0 + i < n ? rb[q] : 0.0;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (i0 + i < n) {
        const double l = cdone - a[i];
        const double wl = wh * l;
        Lw = Lw + wl;
        lat = lat + l;
        wlat = wlat + wl;
      }
    }
  }
  C.Lw = Lw; C.lat = lat; C.wlat = wlat;
  const int sh = 8 * h;
  Q.qp = (Q.qp & ~(0xffu << sh)) | ((uint32_t)qh << sh);
  Q.hp = (Q.hp & ~(0xffu << sh)) | ((uint32_t)pos << sh);
  Q.qsum -= n;
  if (qh > 0) put<CM>(Q.hts, h, next_head);
  Q.hh = hol(Q, p, Q.hts_h);
  C.c[C_DISP] += (uint32_t)n;
  C.c[C_BATCH] += 1u;
  C.chk = fnv(C.chk, ((uint64_t)(k + 1) << 32) | ((uint64_t)j << 16) | ((uint64_t)h << 8) |
                         (uint64_t)n);
  C.n_k += n;
  return cdone;
}

// end-of-tick checksum word pair and reward
template <int CM>
__device__ __forceinline__ double close_tick(const Queue<CM>& Q, Count& C, const SimParams& p,
                                             uint32_t proc, int A_k) {
  uint64_t qp = (uint64_t)Q.qp;
  if (CM < 4) qp &= (1ull << (8 * CM)) - 1;
  qp |= ((uint64_t)proc) << 32;
  qp |= ((uint64_t)(A_k & 0xffff)) << 40;
  C.chk = fnv(C.chk, qp);
  C.chk = fnv(C.chk, ((uint64_t)C.c[C_DONE] << 32) | (uint64_t)C.c[C_DROP]);
  const double thr = (double)C.n_k / p.dt;
  if (p.reward_sum) return p.w_thr * thr - C.Lw;
  return p.w_thr * thr - (C.n_k > 0 ? C.Lw / (double)C.n_k : 0.0);
}

// Writes the observation of one environment a pair of features (2m, 2m + 1) at a time, each
// feature rounded once to fp32: into the current observation [F][E] (cur, may be NULL), a
// trajectory row [F][E] (traj, may be NULL), and as the pair's two bf16 roundings packed in
// one word [F/2][E] (bf, may be NULL): what a bf16 policy reads, half the bytes of the fp32 pair.
struct ObsPairs {
  float* cur;
  float* traj;
  uint32_t* bf;
  size_t E;
  int e;
  __device__ __forceinline__ void put(int i, double v0, double v1) const {
    const float a = (float)v0, b = (float)v1;
    if (cur) {
      cur[(size_t)i * E + e] = a;
      cur[(size_t)(i + 1) * E + e] = b;
    }
    if (traj) {
      traj[(size_t)i * E + e] = a;
      traj[(size_t)(i + 1) * E + e] = b;
    }
    if (bf) bf[(size_t)(i >> 1) * E + e] = pack_bf16_pair(a, b);
  }
};

// ---- learned system: one tick ---------------------------------------------------------------
// share of the wave's lanes still in the tick that triggers a dispatch pass (1 / share)
constexpr int kLearnedDispatchShare = 4;
constexpr int kEndChunk = 8;   // server rows read per round trip at the end of the tick
// PF: the end-of-tick reads of the server rows (K <= kEndChunk) and of the arrival-rate
// averages are issued at the start of the tick instead, so that their latency passes under
// the event loop; they cost registers, which waves that have a SIMD to themselves can spare.
// Only this kernel writes those arrays, at the end of a tick, so the early reads see the same
// values. Without PF the kernel is held to four waves per SIMD (128 VGPRs): the largest grid
// fills the chip exactly at that occupancy.
// One tick k of the learned system for environments e_lane0 .. e_lane0 + lpw - 1, held by the
// first lpw lanes of the calling wave (all 64 lanes call it, and lanes past E idle); st is
// the wave's arrival stage. Reads the actions act[E], writes the observation of tick k + 1
// (obs_mode), the reward and checksum rows (if not NULL) and the environments' state.
template <int CM, bool PF>
__device__ __forceinline__ void learned_tick(const SimParams& p, const EnvState& g, uint64_t seed,
                                             uint32_t k, int e_lane0, int lpw,
                                             Stage<kStageLearned>& st,
                                             const uint8_t* __restrict__ act,
                                             float* __restrict__ obs_out, int obs_mode,
                                             double* __restrict__ rew,
                                             uint64_t* __restrict__ rchk) {
  // the fp64 logarithm, exponential and cosine of the arrival, switch and service draws
  // inline rather than called: a call waits for every outstanding memory access first and
  // saves registers, which waves that have a SIMD to themselves can spare (measured with four
  // request classes: the 8-server tick -4.9%; with fewer classes even or slower)
  constexpr bool kInl = PF && CM >= 4;
  const int lane = threadIdx.x & 63;
  const int e = e_lane0 + lane;
  // lanes without an environment stay in the loop (the wave refills together) but idle
  const bool live = lane < lpw && e < p.E;
  if (__ballot(live) == 0ull) return;
  const int ee = live ? e : 0;
  const size_t E = (size_t)p.E;
  const SysState& G = g.sys[0];
  // the state loads are issued before the action is examined: a branch on the action (and
  // the error flag's atomic, which may alias any state array) ahead of them would make every
  // environment wait out the action load first
  const int a_in = live ? act[ee] : 0;
  Queue<CM> Q;
  load_queue(Q, G, p, ee);
  Count C;
  load_count(C, G, p, ee);
  Arrivals A;
  load_arrivals(A, G, p, ee);
  const bool bad_action = a_in >= 6 * p.K;
  const int a = bad_action ? 0 : a_in;
  const int s = a / 6, b = 1 << (a % 6);
  double busy_s = G.busy[(size_t)s * E + ee];
  uint32_t meta_s = G.meta[(size_t)s * E + ee];
  if (bad_action) atomicOr(g.err, ERR_ACTION);
  bool dirty_s = false;
  double brow_pf[PF ? kEndChunk : 1], ew_pf[PF ? 4 : 1];
  uint32_t mrow_pf[PF ? kEndChunk : 1];
  if constexpr (PF) {
#pragma unroll
    for (int i = 0; i < kEndChunk; ++i) {
      brow_pf[i] = i < p.K ? G.busy[(size_t)i * E + ee] : 0.0;
      mrow_pf[i] = i < p.K ? G.meta[(size_t)i * E + ee] : 0u;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) ew_pf[i] = g.ewma[(size_t)i * E + ee];
  }

  const double t0 = (double)k * p.dt, t1 = (double)(k + 1) * p.dt;
  int A_k = 0;
  double now = t0;
  uint32_t staged_hi = 0;
  uint32_t it = 0;
  // the action's rule at `now`: exactly b requests of the head-of-line class whenever
  // server s is idle
  auto due = [&]() -> bool { return busy_s <= now && Q.qsum > 0 && Q.q(Q.hh) >= b; };
  // done: no event left in the tick; pend: a batch to dispatch at `now`. As in the static
  // system's kernel, dispatches are served in passes shared by many lanes: a lane with a batch
  // due waits (its state frozen) until a quarter of the wave's lanes still in the tick have one
  // too, or no lane can take an event. (Arrival refills are not held back here: within one
  // tick a waiting lane lengthens the tick of the whole wave.)
  bool done = !live;
  bool pend = !done && due();
  for (;;) {
    bool go = false;
    bool need = false;
    double te = now;
    if (!done && !pend) {
      te = A.next_sw < A.next_arr ? A.next_sw : A.next_arr;
      if (busy_s > now && busy_s < te) te = busy_s;
      if (!(te < t1)) {
        done = true;
      } else if (it > kMaxEventsPerTick) {
        atomicOr(g.err, ERR_EVENTS);
        done = true;
      } else {
        need = p.arrival_kind != 1 && (A.next_sw == te || A.next_arr == te) &&
               A.jarr + 2u > staged_hi;
        go = !need;
      }
    }
    if (__ballot(need) != 0ull)
      refill_arrivals<CM, kStageLearned, kInl>(st, p, need, A.jarr, staged_hi, seed, e_lane0,
                                               k, lane);
    if (go) {
      ++it;
      now = te;
      const int cls = advance_staged<CM, kStageLearned, kInl>(A, p, st, lane, seed, ee, k, now);
      if (cls >= 0) {
        ++A_k;
        enqueue(Q, C, p, cls, now);
      }
      pend = due();
      // a run of arrivals: arrivals strictly before the next switch, the tick's end and (while
      // server s is busy) its completion are the lane's only events, so they are taken here,
      // each exactly as a pass would take it (the same staged blocks, the same event bound),
      // until one makes a batch due, without the pass's wave-wide bookkeeping
      if (!pend && p.arrival_kind != 1) {
        const double wend = fmin(fmin(A.next_sw, busy_s > now ? busy_s : kInf), t1);
        bool more = A.next_arr < wend && A.jarr + 2u <= staged_hi && it <= kMaxEventsPerTick;
        while (more) {
          ++it;
          now = A.next_arr;
          const uint32_t j = A.jarr++;
          const int c = st.cls[j % kStageLearned][lane];
          A.next_arr = now + st.E[j % kStageLearned][lane] * A.gap;
          ++A_k;
          enqueue_sel(Q, C, p, c, now);
          pend = due();
          more = !pend && A.next_arr < wend && A.jarr + 2u <= staged_hi &&
                 it <= kMaxEventsPerTick;
        }
      }
    }
    const int n_act = __popcll(__ballot(!done)), n_pend = __popcll(__ballot(pend));
    const bool working = !done && !pend;
    if (n_pend > 0 && (kLearnedDispatchShare * n_pend >= n_act || __ballot(working) == 0ull) &&
        pend) {
      const int h = Q.hh;
      C.c[C_DONE] += meta_s & 0xffu;  // the previous batch on s finished at busy_s <= now
      const double sv = service<CM, kInl>(C, p, seed, ee, k, 0, h, b);
      busy_s = pop_batch(Q, C, p, k, s, h, b, now, sv);
      meta_s = (uint32_t)b | ((uint32_t)b << 8) | ((uint32_t)h << 16);
      dirty_s = true;
      pend = due();
    }
    if (__ballot(!done) == 0ull) break;
  }
  if (!live) return;

  // end of tick: completions before t1 and the per-server part of obs_{k+1}. The server rows
  // are read kEndChunk at a time, all loads of a chunk issued before any of its stores (the
  // compiler cannot reorder them across the stores, which it must assume may alias), so a
  // chunk costs one memory round trip instead of two per server.
  const ObsPairs ob{(obs_mode & kObsF32) ? g.obs : nullptr, obs_out,
                    (obs_mode & kObsBf16) ? g.obs_bf : nullptr, E, e};
  const int per = p.K > 1 ? 4 : 2;
  for (int j0 = 0; j0 < p.K; j0 += kEndChunk) {
    double brow[kEndChunk];
    uint32_t mrow[kEndChunk];
#pragma unroll
    for (int i = 0; i < kEndChunk; ++i) {
      if constexpr (PF) {
        brow[i] = brow_pf[i];
        mrow[i] = mrow_pf[i];
      } else {
        brow[i] = 0.0;
        mrow[i] = 0u;
        if (j0 + i < p.K) {
          brow[i] = G.busy[(size_t)(j0 + i) * E + e];
          mrow[i] = G.meta[(size_t)(j0 + i) * E + e];
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kEndChunk; ++i) {
      const int j = j0 + i;
      if (j >= p.K) break;
      const bool mine = j == s;
      const double bu = mine ? busy_s : brow[i];
      uint32_t m = mine ? meta_s : mrow[i];
      bool dirty = mine && dirty_s;
      const uint32_t infl = m & 0xffu;
      if (infl > 0 && bu < t1) {
        C.c[C_DONE] += infl;
        m &= ~0xffu;
        dirty = true;
      }
      if (dirty) {
        if (mine) G.busy[(size_t)j * E + e] = bu;
        G.meta[(size_t)j * E + e] = m;
      }
      const int base = 2 + per * j;
      const double bflag = bu > t1 ? 1.0 : 0.0;
      const double lb = (double)((m >> 8) & 0xffu) * 0.03125;
      ob.put(base, bflag, lb);
      if (p.K > 1) {
        const double rem = (bu > t1 ? bu - t1 : 0.0) * p.inv_tw;
        const uint32_t lc = (m >> 16) & 0xffu;
        const double lcv = (double)((lc == 0xffu ? -1 : (int)lc) + 1) * p.inv_c;
        ob.put(base + 2, rem, lcv);
      }
    }
  }
  const double r = close_tick(Q, C, p, A.proc, A_k);
  if (rew) rew[e] = r;
  if (rchk) rchk[e] = C.chk;

  // rates: exponentially weighted arrival counts with weights 1, 1/4, 1/16, 1/64
  // (all four read before the first store, for the same reason as the server rows)
  double ew[4];
  const double ewc[4] = {1.0, 0.25, 0.0625, 0.015625};
#pragma unroll
  for (int i = 0; i < 4; ++i) ew[i] = PF ? ew_pf[PF ? i : 0] : g.ewma[(size_t)i * E + e];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ew[i] = ew[i] + ewc[i] * ((double)A_k - ew[i]);
    g.ewma[(size_t)i * E + e] = ew[i];
  }
  // queue part of obs_{k+1}
  const int h = Q.hh;
  const double f0 = (double)Q.qsum * p.inv_n, f1 = (h >= 0 ? t1 - Q.hts_h : 0.0) * p.inv_tw;
  ob.put(0, f0, f1);
  int i = 2 + per * p.K;
  if (p.C > 1) {
#pragma unroll
    for (int c = 0; c < CM; ++c) {
      if (c < p.C) {
        const int qc = Q.q(c);
        const double fq = (double)qc * p.inv_n;
        const double fa = (qc > 0 ? t1 - Q.hts[c] : 0.0) * p.inv_tw;
        ob.put(i, fq, fa);
        i += 2;
      }
    }
  }
  ob.put(i, ew[0] * p.inv_rs, ew[1] * p.inv_rs);
  ob.put(i + 2, ew[2] * p.inv_rs, ew[3] * p.inv_rs);
  i += 4;
  // the padding rows past the observation's width: zero in the current observation (and its
  // bf16 pairs) since the reset or the pairs' packing (nothing else writes them), so only a
  // trajectory row needs them
  if (obs_out)
    for (; i < p.F; ++i) obs_out[(size_t)i * E + e] = 0.0f;

  store_queue(Q, G, p, e);
  store_count(C, G, p, e);
  store_arrivals(A, G, p, e);
}

}  // namespace
}  // namespace bsim
