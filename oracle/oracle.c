/* oracle.c -- plain sequential CPU oracle of the batched inference-serving rollout.
 *
 * TEST INFRASTRUCTURE: only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline
 * leg may load or call this library. It shares no code with the HIP path.
 *
 * Built with gcc -O2 -ffp-contract=off -mfma (explicit fma() calls only; no implicit
 * contraction, no fast-math). Every function processes one environment at a time, one
 * event at a time, in the order the model defines. See oracle.h for the scope and for
 * which parts are pinned by tests.
 */
#include "oracle.h"
#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2,  */
/* 3", SC'11). One round: two 32x32->64 multiplies of counter words 0 and 2 by the        */
/* multipliers; the new counter is (hi1^c1^k0, lo1, hi0^c3^k1, lo0). Between rounds the   */
/* key is bumped by the Weyl constants (golden ratio and sqrt(3)-1, scaled by 2^32).      */
/* ------------------------------------------------------------------------------------ */
#define PHX_M0 0xD2511F53u
#define PHX_M1 0xCD9E8D57u
#define PHX_W0 0x9E3779B9u
#define PHX_W1 0xBB67AE85u

static void philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; r++) {
    if (r > 0) { k0 += PHX_W0; k1 += PHX_W1; }
    uint64_t p0 = (uint64_t)PHX_M0 * (uint64_t)c0;
    uint64_t p1 = (uint64_t)PHX_M1 * (uint64_t)c2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The same construction on 64-bit words (Philox4x64-10); exported only so that tests can
 * pin the round structure against numpy's independent Philox4x64 implementation. */
static void philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
  uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint64_t k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; r++) {
    if (r > 0) { k0 += W0; k1 += W1; }
    unsigned __int128 p0 = (unsigned __int128)M0 * c0;
    unsigned __int128 p1 = (unsigned __int128)M1 * c2;
    uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    uint64_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Counter layout (R13): (env, step, purpose<<24 | j, system); key = (lo32, hi32) of seed. */
static void draw(uint64_t seed, uint32_t env, uint32_t step, uint32_t purpose, uint32_t j,
                 uint32_t sys, uint32_t out[4]) {
  uint32_t ctr[4] = {env, step, (purpose << 24) | j, sys};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  philox4x32_10(ctr, key, out);
}

/* Two words -> uniform double in (0,1): the top 53 bits of (hi:lo), centred in its cell. */
static double u01(uint32_t lo, uint32_t hi) {
  uint64_t v = ((((uint64_t)hi) << 32) | (uint64_t)lo) >> 11;
  return ((double)v + 0.5) * 0x1p-53;
}

/* ------------------------------------------------------------------------------------ */
/* Deterministic fp64 elementary functions (R14): fixed sequences of IEEE +,-,*,/ and fma */
/* so that any two IEEE-conforming implementations of the same sequence agree bit for     */
/* bit. Accuracy target: a few ulp of the correctly rounded result.                       */
/* ------------------------------------------------------------------------------------ */
#define LN2_HI 0x1.62e42fee00000p-1  /* ln 2 truncated to 32 significant bits */
#define LN2_LO 0x1.a39ef35793c76p-33 /* ln 2 - LN2_HI */
#define INV_LN2 0x1.71547652b82fep+0
#define SQRT2_D 0x1.6a09e667f3bcdp+0
#define PIO2_HI 0x1.921fb54400000p+0 /* pi/2 truncated to 32 significant bits */
#define PIO2_LO 0x1.0b4611a626331p-34
#define TWO_OVER_PI 0x1.45f306dc9c883p-1
#define TWO_PI_D 0x1.921fb54442d18p+2

/* log x for positive normal x: x = 2^e m with m in (sqrt(2)/2, sqrt(2)];
 * log m = 2 atanh(s), s = (m-1)/(m+1), atanh s = s (1 + z/3 + z^2/5 + ... ), z = s^2.
 * |s| <= 0.1716 so the series to z^11/23 reaches 2^-53. */
static double det_log(double x) {
  uint64_t bits;
  memcpy(&bits, &x, 8);
  int e = (int)((bits >> 52) & 0x7ff) - 1023;
  uint64_t mb = (bits & 0x000fffffffffffffull) | 0x3ff0000000000000ull;
  double m;
  memcpy(&m, &mb, 8);
  if (m > SQRT2_D) { m = m * 0.5; e += 1; }
  double f = m - 1.0;
  double s = f / (m + 1.0);
  double z = s * s;
  double p = 1.0 / 23.0;
  p = fma(p, z, 1.0 / 21.0);
  p = fma(p, z, 1.0 / 19.0);
  p = fma(p, z, 1.0 / 17.0);
  p = fma(p, z, 1.0 / 15.0);
  p = fma(p, z, 1.0 / 13.0);
  p = fma(p, z, 1.0 / 11.0);
  p = fma(p, z, 1.0 / 9.0);
  p = fma(p, z, 1.0 / 7.0);
  p = fma(p, z, 1.0 / 5.0);
  p = fma(p, z, 1.0 / 3.0);
  double r = fma(s * z, p, s);      /* atanh(s) */
  double lm = 2.0 * r;              /* log m */
  double de = (double)e;
  return fma(de, LN2_HI, fma(de, LN2_LO, lm));
}

/* exp x for |x| < 700: x = k ln2 + r (Cody-Waite with the split ln 2), |r| <= ln2/2,
 * exp r by its Taylor series to r^14/14!, then scaled by 2^k built from its bits. */
static double det_exp(double x) {
  double kd = floor(x * INV_LN2 + 0.5);
  int k = (int)kd;
  double r = (x - kd * LN2_HI) - kd * LN2_LO;
  double p = 1.0 / 87178291200.0;        /* 1/14! */
  p = fma(p, r, 1.0 / 6227020800.0);     /* 1/13! */
  p = fma(p, r, 1.0 / 479001600.0);      /* 1/12! */
  p = fma(p, r, 1.0 / 39916800.0);       /* 1/11! */
  p = fma(p, r, 1.0 / 3628800.0);        /* 1/10! */
  p = fma(p, r, 1.0 / 362880.0);         /* 1/9!  */
  p = fma(p, r, 1.0 / 40320.0);          /* 1/8!  */
  p = fma(p, r, 1.0 / 5040.0);           /* 1/7!  */
  p = fma(p, r, 1.0 / 720.0);            /* 1/6!  */
  p = fma(p, r, 1.0 / 120.0);            /* 1/5!  */
  p = fma(p, r, 1.0 / 24.0);             /* 1/4!  */
  p = fma(p, r, 1.0 / 6.0);              /* 1/3!  */
  p = fma(p, r, 0.5);                    /* 1/2!  */
  p = fma(p, r, 1.0);                    /* 1/1!  */
  p = fma(p, r, 1.0);                    /* 1/0!  */
  uint64_t sb = ((uint64_t)(k + 1023)) << 52;
  double sc;
  memcpy(&sc, &sb, 8);
  return p * sc;
}

/* cos x for 0 <= x <= 8: x = q pi/2 + r with |r| <= pi/4 (split pi/2), then
 * cos(x) = cos r, -sin r, -cos r, sin r for q mod 4 = 0, 1, 2, 3; Taylor series of cos to
 * z^9/18! and of sin to r^19/19!, z = r^2. */
static double det_cos(double x) {
  double qd = floor(x * TWO_OVER_PI + 0.5);
  int q = (int)qd;
  double r = (x - qd * PIO2_HI) - qd * PIO2_LO;
  double z = r * r;
  double c = 1.0 / 6402373705728000.0;   /* 1/18! */
  c = fma(c, z, -1.0 / 20922789888000.0);  /* -1/16! */
  c = fma(c, z, 1.0 / 87178291200.0);      /* 1/14! */
  c = fma(c, z, -1.0 / 479001600.0);       /* -1/12! */
  c = fma(c, z, 1.0 / 3628800.0);          /* 1/10! */
  c = fma(c, z, -1.0 / 40320.0);           /* -1/8! */
  c = fma(c, z, 1.0 / 720.0);              /* 1/6! */
  c = fma(c, z, -1.0 / 24.0);              /* -1/4! */
  c = fma(c, z, 0.5);                      /* 1/2! */
  c = fma(-c, z, 1.0);                     /* 1 - z/2 + z^2/24 - ... */
  double s = -1.0 / 121645100408832000.0;  /* -1/19! */
  s = fma(s, z, 1.0 / 355687428096000.0);  /* 1/17! */
  s = fma(s, z, -1.0 / 1307674368000.0);   /* -1/15! */
  s = fma(s, z, 1.0 / 6227020800.0);       /* 1/13! */
  s = fma(s, z, -1.0 / 39916800.0);        /* -1/11! */
  s = fma(s, z, 1.0 / 362880.0);           /* 1/9! */
  s = fma(s, z, -1.0 / 5040.0);            /* -1/7! */
  s = fma(s, z, 1.0 / 120.0);              /* 1/5! */
  s = fma(s, z, -1.0 / 6.0);               /* -1/3! */
  s = fma(s * z, r, r);                    /* r + r^3 (-1/6 + ...) */
  switch (q & 3) {
    case 0: return c;
    case 1: return -s;
    case 2: return -c;
    default: return s;
  }
}

/* ------------------------------------------------------------------------------------ */
/* Derived per-configuration constants (computed here, independently of the GPU host).   */
/* ------------------------------------------------------------------------------------ */
typedef struct derived {
  double mean_gap[ORC_MAX_S];    /* 1/lambda_i (0 rate -> no arrivals) */
  double inv_alpha[ORC_MAX_S];   /* 1/alpha of Pareto dwell */
  double stat_cum[ORC_MAX_S];    /* cumulative stationary state distribution */
  double class_cum[ORC_MAX_C];   /* cumulative class mix, last forced to 1 (R12) */
} derived;

static void derive(const orc_cfg* c, derived* d) {
  for (int i = 0; i < c->n_states; i++) {
    d->mean_gap[i] = c->rate[i] > 0.0 ? 1.0 / c->rate[i] : 0.0;
    d->inv_alpha[i] = c->dwell_kind[i] == ORC_DWELL_PARETO ? 1.0 / c->pareto_alpha[i] : 0.0;
  }
  /* time-stationary probability of a state is proportional to its mean dwell, since the
   * embedded jump chain is uniform over the other states (R11) */
  double mdw[ORC_MAX_S], tot = 0.0;
  for (int i = 0; i < c->n_states; i++) {
    if (c->dwell_kind[i] == ORC_DWELL_EXP || c->dwell_kind[i] == ORC_DWELL_DET)
      mdw[i] = c->dwell_mean[i];
    else if (c->dwell_kind[i] == ORC_DWELL_PARETO)
      mdw[i] = c->pareto_alpha[i] * c->pareto_xm[i] / (c->pareto_alpha[i] - 1.0);
    else mdw[i] = 1.0;
    tot = tot + mdw[i];
  }
  double acc = 0.0;
  for (int i = 0; i < c->n_states; i++) {
    acc = acc + mdw[i];
    d->stat_cum[i] = acc / tot;
  }
  d->stat_cum[c->n_states - 1] = 1.0;
  acc = 0.0;
  for (int i = 0; i < c->n_classes; i++) {
    acc = acc + c->class_mix[i];
    d->class_cum[i] = acc;
  }
  d->class_cum[c->n_classes - 1] = 1.0;
}

/* ------------------------------------------------------------------------------------ */
/* One queueing system of one environment (Sec. 3.1). The learned system (sys 0) follows */
/* the agent's action; the static system (sys 1) follows the timeout rule (R18).         */
/* Each system carries its own copy of the arrival process; its draws do not depend on   */
/* the system index, so both copies see the same arrivals (R13).                          */
/* ------------------------------------------------------------------------------------ */
typedef struct sys_t {
  int sys;
  /* arrival process */
  int proc;
  double next_sw, next_arr;
  int32_t tr_idx;
  /* per-class FIFO queues of arrival timestamps */
  int q[ORC_MAX_C], head[ORC_MAX_C];
  double ring[ORC_MAX_C][ORC_MAX_N];
  /* servers */
  int rr;                        /* round-robin pointer of the static system (R23) */
  double busy[ORC_MAX_K];
  int inflight[ORC_MAX_K], last_b[ORC_MAX_K], last_cls[ORC_MAX_K];
  /* Shortest-Queue routing (R27): each server's FIFO of assigned batches, at most two (the one
   * it runs and one queued behind it), completion times and sizes in order */
  int sq_cnt[ORC_MAX_K];
  double sq_c[ORC_MAX_K][2];
  int sq_n[ORC_MAX_K][2];
  double ewma[4];
  /* counters */
  int64_t arrivals, accepted, dropped, dispatched, batches, completed;
  double lat_sum, wlat_sum, wait_sum;
  uint64_t chk;
  /* exact event-by-event integrals for Little's law and queue-length averages */
  double area_n, area_q, t_area, soj_sum, horizon;
} sys_t;

typedef struct tick_ctx {
  const orc_cfg* c;
  const derived* d;
  const orc_trace* tr;
  int32_t env_idx;
  uint32_t env;
  uint64_t seed;
  uint32_t k;
  uint32_t j_arr, j_proc, j_svc, j_route;
  int n_k, ndisp, A_k;
  double Lw;
  orc_out* out;
} tick_ctx;

#define FNV_PRIME 0x100000001b3ull
#define FNV_INIT 0xcbf29ce484222325ull
static uint64_t mix(uint64_t h, uint64_t v) { return (h ^ v) * FNV_PRIME; }

static double gap_draw(const tick_ctx* t, int state, double u) {
  return -det_log(u) * t->d->mean_gap[state];
}

static double dwell_draw(const tick_ctx* t, int state, double u) {
  const orc_cfg* c = t->c;
  if (c->dwell_kind[state] == ORC_DWELL_EXP) return -det_log(u) * c->dwell_mean[state];
  if (c->dwell_kind[state] == ORC_DWELL_PARETO)
    return c->pareto_xm[state] * det_exp(-det_log(u) * t->d->inv_alpha[state]);
  if (c->dwell_kind[state] == ORC_DWELL_DET) return c->dwell_mean[state];  /* square wave (R24) */
  return INFINITY;
}

static int sumq(const sys_t* S, int C) {
  int s = 0;
  for (int c = 0; c < C; c++) s += S->q[c];
  return s;
}

/* head-of-line class: the class whose oldest request arrived first; ties to the lower
 * index (R5). Returns -1 when every queue is empty. */
static int hol(const sys_t* S, int C) {
  int h = -1;
  double best = 0.0;
  for (int c = 0; c < C; c++) {
    if (S->q[c] == 0) continue;
    double ts = S->ring[c][S->head[c]];
    if (h < 0 || ts < best) { h = c; best = ts; }
  }
  return h;
}

/* Service time of a batch of n requests of class h (R7). */
static double service(tick_ctx* t, sys_t* S, int h, int n) {
  const orc_cfg* c = t->c;
  int kind = c->service_kind[h];
  if (kind == ORC_SVC_DET) return c->svc_alpha[h] + c->svc_beta[h] * (double)n;
  uint32_t w[4];
  draw(t->seed, t->env, t->k, ORC_P_SERVICE, t->j_svc++, (uint32_t)S->sys, w);
  double u1 = u01(w[0], w[1]);
  if (kind == ORC_SVC_EXP) return -det_log(u1) * (c->svc_alpha[h] + c->svc_beta[h] * (double)n);
  double u2 = u01(w[2], w[3]);
  double z = sqrt(-2.0 * det_log(u1)) * det_cos(TWO_PI_D * u2);   /* Box-Muller */
  return c->svc_median[h] * det_exp(c->svc_sigma * z) + c->svc_beta[h] * (double)n;
}

static void take_batch(tick_ctx* t, sys_t* S, int j, int h, int n, double now, double start,
                       double cdone);

/* Dispatch n requests of class h to server j at time now (Sec. 3.1 execution model). The
 * batch's latency L_r = c - a_r of each request is known at dispatch (R8). */
static void batch(tick_ctx* t, sys_t* S, int j, int h, int n, double now) {
  if (S->inflight[j] > 0) S->completed += S->inflight[j];  /* finished at busy[j] <= now */
  double sv = service(t, S, h, n);
  double cdone = now + sv;
  take_batch(t, S, j, h, n, now, now, cdone);
  S->busy[j] = cdone;
  S->last_b[j] = n;
  S->last_cls[j] = h;
  S->inflight[j] = n;
}

/* The n oldest requests of class h leave the queue at `now` as one batch on server j that
 * starts at `start` and completes at cdone: their latencies c - a_r (Sec. 4.1 reward), waits
 * start - a_r, the counters, the dispatch record. */
static void take_batch(tick_ctx* t, sys_t* S, int j, int h, int n, double now, double start,
                       double cdone) {
  const orc_cfg* c = t->c;
  int N = c->queue_cap;
  for (int i = 0; i < n; i++) {
    double a = S->ring[h][S->head[h]];
    S->head[h] = S->head[h] + 1 == N ? 0 : S->head[h] + 1;
    double lat = cdone - a;
    double wl = c->w_class[h] * lat;
    t->Lw = t->Lw + wl;
    S->lat_sum = S->lat_sum + lat;
    S->wlat_sum = S->wlat_sum + wl;
    S->wait_sum = S->wait_sum + (start - a);
    S->soj_sum = S->soj_sum + ((cdone < S->horizon ? cdone : S->horizon) - a);
  }
  S->q[h] -= n;
  S->dispatched += n;
  S->batches += 1;
  S->chk = mix(S->chk, ((uint64_t)(t->k + 1) << 32) | ((uint64_t)j << 16) | ((uint64_t)h << 8) |
                           (uint64_t)n);
  t->n_k += n;
  t->ndisp += 1;
  orc_out* o = t->out;
  if (o && o->disp && o->disp_count < o->disp_cap) {
    orc_disp* d = &o->disp[o->disp_count];
    d->env_idx = t->env_idx; d->sys = S->sys; d->k = (int32_t)t->k; d->server = j;
    d->cls = h; d->n = n; d->t = now; d->c = cdone;
  }
  if (o && o->disp) o->disp_count++;
}

/* Learned system (R2-R4): action a = 6 s + log2 b. Whenever server s is idle and the
 * head-of-line class holds at least b requests, exactly b of them are dispatched to s. */
static int any_idle(const sys_t* S, int K, double now) {
  for (int j = 0; j < K; j++)
    if (S->busy[j] <= now) return 1;
  return 0;
}

static void dispatch_learned(tick_ctx* t, sys_t* S, int action, double now) {
  int s = action / 6, b = 1 << (action % 6);
  int C = t->c->n_classes;
  while (S->busy[s] <= now && sumq(S, C) > 0) {
    int h = hol(S, C);
    if (S->q[h] < b) break;
    batch(t, S, s, h, b, now);
  }
}

/* Server for the static system's next batch among the idle ones (R23): the lowest index;
 * uniformly at random (the idx-th idle server in index order, idx = floor(u * n_idle) with
 * u from ROUTE block j_route of (env, tick, system 1)); or round robin (the first idle
 * server at or after the pointer, cyclically; the pointer then moves past it). */
static int route_static(tick_ctx* t, sys_t* S, double now) {
  const orc_cfg* c = t->c;
  int idle[ORC_MAX_K], n_idle = 0;
  for (int i = 0; i < c->n_servers; i++)
    if (S->busy[i] <= now) idle[n_idle++] = i;
  if (n_idle == 0) return -1;
  if (c->static_route == ORC_ROUTE_RANDOM) {
    uint32_t w[4];
    draw(t->seed, t->env, t->k, ORC_P_ROUTE, t->j_route++, 1, w);
    int idx = (int)(u01(w[0], w[1]) * (double)n_idle);
    return idle[idx < n_idle ? idx : n_idle - 1];
  }
  if (c->static_route == ORC_ROUTE_ROUND_ROBIN) {
    for (int d = 0; d < c->n_servers; d++) {
      int i = (S->rr + d) % c->n_servers;
      if (S->busy[i] <= now) return i;
    }
  }
  return idle[0];
}

/* Static timeout rule (Sec. 1's "wait T or until B requests accumulate", R18): while some
 * server is idle and requests wait, dispatch min(B, Q_h) of the head-of-line class if
 * Q_h >= B or its head has waited at least T, to the server route_static chooses. */
static void dispatch_static(tick_ctx* t, sys_t* S, double now) {
  const orc_cfg* c = t->c;
  for (;;) {
    if (!any_idle(S, c->n_servers, now) || sumq(S, c->n_classes) == 0) return;
    int h = hol(S, c->n_classes);
    double head_ts = S->ring[h][S->head[h]];
    if (S->q[h] >= c->static_bmax || now >= head_ts + c->static_timeout) {
      int n = S->q[h] < c->static_bmax ? S->q[h] : c->static_bmax;
      int j = route_static(t, S, now);
      batch(t, S, j, h, n, now);
      S->rr = (j + 1) % c->n_servers;
    } else {
      return;
    }
  }
}

/* Shortest-Queue routing of the static rule's batches (Sec. 5.1 baselines, R27). Each server
 * holds the batch it runs and at most one more queued behind it, served in order. A batch
 * whose completion time has come (c <= now) has left the server; its requests count as
 * completed. */
static void sq_retire(sys_t* S, int K, double now) {
  for (int j = 0; j < K; j++) {
    while (S->sq_cnt[j] > 0 && S->sq_c[j][0] <= now) {
      S->completed += S->sq_n[j][0];
      S->sq_c[j][0] = S->sq_c[j][1];
      S->sq_n[j][0] = S->sq_n[j][1];
      S->sq_cnt[j]--;
    }
    S->busy[j] = S->sq_cnt[j] > 0 ? S->sq_c[j][0] : S->busy[j];
  }
}

static int sq_any_slot(const sys_t* S, int K) {
  for (int j = 0; j < K; j++)
    if (S->sq_cnt[j] < 2) return 1;
  return 0;
}

/* While requests wait and the static rule's condition holds (Q_h >= B, or the head of the
 * head-of-line class has waited T), the batch min(B, Q_h) goes to the server with the fewest
 * requests assigned and not completed among those with a free slot (ties to the lower index);
 * it starts when that server has finished what it holds. No free slot: the batch waits. */
static void dispatch_sq(tick_ctx* t, sys_t* S, double now) {
  const orc_cfg* c = t->c;
  sq_retire(S, c->n_servers, now);
  for (;;) {
    if (sumq(S, c->n_classes) == 0) return;
    int h = hol(S, c->n_classes);
    double head_ts = S->ring[h][S->head[h]];
    if (!(S->q[h] >= c->static_bmax || now >= head_ts + c->static_timeout)) return;
    int j = -1, best = 0;
    for (int i = 0; i < c->n_servers; i++) {
      if (S->sq_cnt[i] >= 2) continue;
      int load = 0;
      for (int b = 0; b < S->sq_cnt[i]; b++) load += S->sq_n[i][b];
      if (j < 0 || load < best) { j = i; best = load; }
    }
    if (j < 0) return;
    int n = S->q[h] < c->static_bmax ? S->q[h] : c->static_bmax;
    double start = S->sq_cnt[j] > 0 ? S->sq_c[j][S->sq_cnt[j] - 1] : now;
    double cdone = start + service(t, S, h, n);
    take_batch(t, S, j, h, n, now, start, cdone);
    S->sq_c[j][S->sq_cnt[j]] = cdone;
    S->sq_n[j][S->sq_cnt[j]] = n;
    S->sq_cnt[j]++;
    S->busy[j] = S->sq_c[j][0];
  }
}

static void do_dispatch(tick_ctx* t, sys_t* S, int action, double now) {
  if (S->sys == 0) dispatch_learned(t, S, action, now);
  else if (t->c->static_route == ORC_ROUTE_SHORTEST) dispatch_sq(t, S, now);
  else dispatch_static(t, S, now);
}

/* number in system on [t_area, te): waiting requests plus batches still in service */
static void integrate(tick_ctx* t, sys_t* S, double te) {
  const orc_cfg* c = t->c;
  int nq = sumq(S, c->n_classes);
  int ns = 0;
  if (S->sys == 1 && c->static_route == ORC_ROUTE_SHORTEST) {
    for (int j = 0; j < c->n_servers; j++)
      for (int b = 0; b < S->sq_cnt[j]; b++) ns += S->sq_n[j][b];
  } else {
    for (int j = 0; j < c->n_servers; j++)
      if (S->busy[j] > S->t_area) ns += S->last_b[j];
  }
  double dt = te - S->t_area;
  S->area_n = S->area_n + (double)(nq + ns) * dt;
  S->area_q = S->area_q + (double)nq * dt;
  S->t_area = te;
}

static void process_switch(tick_ctx* t, sys_t* S, double now) {
  const orc_cfg* c = t->c;
  uint32_t w[4];
  draw(t->seed, t->env, t->k, ORC_P_PROCESS, t->j_proc++, 0, w);
  int cur = S->proc, nxt;
  if (c->n_states == 2) {
    nxt = 1 - cur;
  } else {
    int idx = (int)(u01(w[2], w[3]) * (double)(c->n_states - 1));
    nxt = idx < cur ? idx : idx + 1;
  }
  S->proc = nxt;
  S->next_sw = now + dwell_draw(t, nxt, u01(w[0], w[1]));
  /* memoryless rate change: the pending arrival is redrawn from the switch instant (R11) */
  if (c->rate[nxt] > 0.0) {
    draw(t->seed, t->env, t->k, ORC_P_ARRIVAL, t->j_arr++, 0, w);
    S->next_arr = now + gap_draw(t, nxt, u01(w[0], w[1]));
  } else {
    S->next_arr = INFINITY;
  }
}

static void process_arrival(tick_ctx* t, sys_t* S, double now) {
  const orc_cfg* c = t->c;
  int cls;
  if (c->arrival_kind == ORC_ARR_TRACE) {
    int32_t i = t->env_idx;
    cls = t->tr->classes[(int64_t)i * t->tr->max_len + S->tr_idx];
    S->tr_idx++;
    S->next_arr = S->tr_idx < t->tr->counts[i]
                      ? t->tr->times[(int64_t)i * t->tr->max_len + S->tr_idx] : INFINITY;
  } else {
    uint32_t w[4];
    draw(t->seed, t->env, t->k, ORC_P_ARRIVAL, t->j_arr++, 0, w);
    double uc = u01(w[2], w[3]);
    cls = 0;
    while (!(uc < t->d->class_cum[cls])) cls++;
    S->next_arr = now + gap_draw(t, S->proc, u01(w[0], w[1]));
  }
  S->arrivals++;
  t->A_k++;
  /* FIFO with load shedding: an arrival finding N requests waiting is dropped (R6) */
  if (sumq(S, c->n_classes) == c->queue_cap) {
    S->dropped++;
  } else {
    int pos = S->head[cls] + S->q[cls];
    if (pos >= c->queue_cap) pos -= c->queue_cap;
    S->ring[cls][pos] = now;
    S->q[cls]++;
    S->accepted++;
  }
}

/* One tick [t_k, t_{k+1}) of one system (R1, R2, R9, R10). */
static double tick(tick_ctx* t, sys_t* S, int action) {
  const orc_cfg* c = t->c;
  double t0 = (double)t->k * c->tick_s, t1 = (double)(t->k + 1) * c->tick_s;
  t->j_arr = 0; t->j_proc = 0; t->j_svc = 0; t->j_route = 0;
  t->n_k = 0; t->ndisp = 0; t->A_k = 0; t->Lw = 0.0;
  double now = t0;
  do_dispatch(t, S, action, now);
  for (;;) {
    double te = S->next_sw;
    if (S->next_arr < te) te = S->next_arr;
    for (int j = 0; j < c->n_servers; j++)
      if (S->busy[j] > now && S->busy[j] < te) te = S->busy[j];
    const int sq = S->sys == 1 && c->static_route == ORC_ROUTE_SHORTEST;
    if (S->sys == 1 && sumq(S, c->n_classes) > 0 &&
        (sq ? sq_any_slot(S, c->n_servers) : any_idle(S, c->n_servers, now))) {
      int h = hol(S, c->n_classes);
      double tout = S->ring[h][S->head[h]] + c->static_timeout;
      if (tout > now && tout < te) te = tout;
    }
    if (!(te < t1)) break;
    integrate(t, S, te);
    now = te;
    if (S->next_sw == now) process_switch(t, S, now);
    if (S->next_arr == now) process_arrival(t, S, now);
    do_dispatch(t, S, action, now);
  }
  integrate(t, S, t1);
  /* completions of the tick: every batch finishing before t_{k+1} (R9) */
  if (S->sys == 1 && c->static_route == ORC_ROUTE_SHORTEST) {
    for (int j = 0; j < c->n_servers; j++) {
      while (S->sq_cnt[j] > 0 && S->sq_c[j][0] < t1) {
        S->completed += S->sq_n[j][0];
        S->sq_c[j][0] = S->sq_c[j][1];
        S->sq_n[j][0] = S->sq_n[j][1];
        S->sq_cnt[j]--;
      }
      S->busy[j] = S->sq_cnt[j] > 0 ? S->sq_c[j][0] : S->busy[j];
    }
  }
  for (int j = 0; j < c->n_servers; j++) {
    if (S->inflight[j] > 0 && S->busy[j] < t1) {
      S->completed += S->inflight[j];
      S->inflight[j] = 0;
    }
  }
  /* exponentially weighted arrival counts with weights 1, 1/4, 1/16, 1/64 (R15) */
  static const double ew[4] = {1.0, 0.25, 0.0625, 0.015625};
  for (int i = 0; i < 4; i++) S->ewma[i] = S->ewma[i] + ew[i] * ((double)t->A_k - S->ewma[i]);
  /* reward (Sec. 4.1, R8): throughput of the tick minus the (mean) weighted latency of the
   * requests dispatched in it */
  double thr = (double)t->n_k / c->tick_s;
  double r;
  if (c->reward_sum) r = c->w_thr * thr - t->Lw;
  else r = c->w_thr * thr - (t->n_k > 0 ? t->Lw / (double)t->n_k : 0.0);
  /* checksum of the tick's end state */
  uint64_t qp = 0;
  for (int cc = 0; cc < c->n_classes; cc++) qp |= ((uint64_t)S->q[cc]) << (8 * cc);
  qp |= ((uint64_t)S->proc) << 32;
  qp |= ((uint64_t)(t->A_k & 0xffff)) << 40;
  S->chk = mix(S->chk, qp);
  S->chk = mix(S->chk, ((uint64_t)(uint32_t)S->completed << 32) | (uint64_t)(uint32_t)S->dropped);
  return r;
}

/* Observation (Sec. 4.1, R15): every feature is a raw quantity times the reciprocal of
 * its normaliser (1/N, 1/T_w, 1/32, 1/C, 1/(lambda_ref*dt), each computed once in fp64),
 * evaluated in fp64 and rounded once to fp32. */
static void observe(const orc_cfg* c, const sys_t* S, double t, float* obs) {
  int F = c->obs_dim, K = c->n_servers, C = c->n_classes, N = c->queue_cap;
  double inv_n = 1.0 / (double)N, inv_tw = 1.0 / c->obs_tw, inv_c = 1.0 / (double)C;
  double inv_rs = 1.0 / (c->lambda_ref * c->tick_s);
  int i = 0;
  int nq = sumq(S, C);
  int h = hol(S, C);
  obs[i++] = (float)((double)nq * inv_n);
  obs[i++] = (float)((h >= 0 ? t - S->ring[h][S->head[h]] : 0.0) * inv_tw);
  for (int j = 0; j < K; j++) {
    obs[i++] = S->busy[j] > t ? 1.0f : 0.0f;
    obs[i++] = (float)((double)S->last_b[j] * 0.03125);
    if (K > 1) {
      double rem = S->busy[j] > t ? S->busy[j] - t : 0.0;
      obs[i++] = (float)(rem * inv_tw);
      obs[i++] = (float)((double)(S->last_cls[j] + 1) * inv_c);
    }
  }
  if (C > 1) {
    for (int cc = 0; cc < C; cc++) {
      obs[i++] = (float)((double)S->q[cc] * inv_n);
      double age = S->q[cc] > 0 ? t - S->ring[cc][S->head[cc]] : 0.0;
      obs[i++] = (float)(age * inv_tw);
    }
  }
  for (int r = 0; r < 4; r++) obs[i++] = (float)(S->ewma[r] * inv_rs);
  while (i < F) obs[i++] = 0.0f;
}

/* Reset (R21): empty queues, idle servers, zero counters; the modulating state is drawn
 * from its stationary law, then its dwell, then the first arrival (R11, R13). */
static void reset_sys(const orc_cfg* c, const derived* d, const orc_trace* tr, int32_t env_idx,
                      uint32_t env, uint64_t seed, int sys, double horizon, sys_t* S) {
  memset(S, 0, sizeof(*S));
  S->sys = sys;
  S->chk = FNV_INIT;
  S->horizon = horizon;
  for (int j = 0; j < c->n_servers; j++) { S->busy[j] = 0.0; S->last_cls[j] = -1; }
  S->proc = 0;
  S->next_sw = INFINITY;
  if (c->arrival_kind == ORC_ARR_TRACE) {
    S->tr_idx = 0;
    S->next_arr = tr->counts[env_idx] > 0 ? tr->times[(int64_t)env_idx * tr->max_len] : INFINITY;
    return;
  }
  uint32_t w[4];
  tick_ctx t;
  memset(&t, 0, sizeof(t));
  t.c = c; t.d = d;
  if (c->n_states > 1 && c->dwell_kind[0] == ORC_DWELL_DET) {
    /* a square wave starts in state 0 with its full dwell: same phase everywhere (R24) */
    S->proc = 0;
    S->next_sw = c->dwell_mean[0];
  } else if (c->n_states > 1) {
    draw(seed, env, ORC_STEP_RESET, ORC_P_PROCESS, 0, 0, w);
    double us = u01(w[2], w[3]);
    int s = 0;
    while (!(us < d->stat_cum[s])) s++;
    S->proc = s;
    S->next_sw = dwell_draw(&t, s, u01(w[0], w[1]));
  }
  if (c->rate[S->proc] > 0.0) {
    draw(seed, env, ORC_STEP_RESET, ORC_P_ARRIVAL, 0, 0, w);
    S->next_arr = gap_draw(&t, S->proc, u01(w[0], w[1]));
  } else {
    S->next_arr = INFINITY;
  }
}

/* ------------------------------------------------------------------------------------ */
/* Policy (Sec. 4.2, R16, R17).                                                           */
/* ------------------------------------------------------------------------------------ */
static double bf16r(double x) {
  float f = (float)x;
  uint32_t u;
  memcpy(&u, &f, 4);
  u = u + 0x7fffu + ((u >> 16) & 1u);   /* round to nearest even on the top 16 bits */
  u &= 0xffff0000u;
  memcpy(&f, &u, 4);
  return (double)f;
}

static double gelu(double x) { return 0.5 * x * (1.0 + erf(x * 0x1.6a09e667f3bcdp-1)); }

static int n_out(const orc_cfg* c) { return 6 * c->n_servers + (c->value_head ? 1 : 0); }

/* logits (and value) of one observation: F -> H1 -> H2 -> A' with GELU after each hidden
 * layer; in bf16 mode every layer input is rounded to bf16 first. */
static void mlp_forward(const orc_cfg* c, const orc_weights* w, const float* obs, double* out,
                        double* h1, double* h2) {
  int F = c->obs_dim, H1 = c->mlp_h1, H2 = c->mlp_h2, A = n_out(c);
  int bf = c->mlp_bf16;
  for (int j = 0; j < H1; j++) {
    double s = 0.0;
    for (int i = 0; i < F; i++) {
      double x = bf ? bf16r((double)obs[i]) : (double)obs[i];
      s = s + x * w->w1[(int64_t)i * H1 + j];
    }
    double v = gelu(s + w->b1[j]);
    h1[j] = bf ? bf16r(v) : v;
  }
  for (int j = 0; j < H2; j++) {
    double s = 0.0;
    for (int i = 0; i < H1; i++) s = s + h1[i] * w->w2[(int64_t)i * H2 + j];
    double v = gelu(s + w->b2[j]);
    h2[j] = bf ? bf16r(v) : v;
  }
  for (int a = 0; a < A; a++) {
    double s = 0.0;
    for (int i = 0; i < H2; i++) s = s + h2[i] * w->w3[(int64_t)i * A + a];
    out[a] = s + w->b3[a];
  }
}

/* The attention policy of Sec. 4.2 (R26), one observation, fp64, in the order the
 * definitions are stated:
 *   tokens    e_g = b_in + sum over the features i of group g of x_i W_in[i,:]
 *             (F features in attn_tokens = L contiguous groups of F/L),
 *   attention q_g, k_g, v_g = e_g W_qkv + b_qkv (query, key, value column blocks); head h
 *             takes columns [h dh, (h+1) dh) with dh = D / attn_heads and gives
 *             o_{g,h} = sum_g' softmax_g'(q_{g,h} . k_{g',h} / sqrt(dh)) v_{g',h}
 *             (scaled dot-product attention, Vaswani et al. 2017); y_g = concat_h o_{g,h}
 *             W_o + b_o,
 *   pooling   p = mean over g of y_g,
 *   heads     logits = GELU(p W_p1 + b_p1) W_p2 + b_p2 and
 *             V = GELU(p W_v1 + b_v1) W_v2 + b_v2 (a separate value MLP).
 * out[0..A) are the logits, out[A] = V when value_head = 1. */
static void attn_forward(const orc_cfg* c, const orc_weights* w, const float* obs, double* out) {
  const int F = c->obs_dim, L = c->attn_tokens, D = c->attn_embed, NH = c->attn_heads;
  const int G = F / L, dh = D / NH, A = 6 * c->n_servers;
  const int Hp = c->mlp_h1, Hv = c->mlp_h2;
  double e[ORC_ATTN_MAX_L][ORC_ATTN_MAX_D];
  double q[ORC_ATTN_MAX_L][ORC_ATTN_MAX_D], k[ORC_ATTN_MAX_L][ORC_ATTN_MAX_D];
  double v[ORC_ATTN_MAX_L][ORC_ATTN_MAX_D], o[ORC_ATTN_MAX_L][ORC_ATTN_MAX_D];
  double pool[ORC_ATTN_MAX_D];
  for (int g = 0; g < L; g++)
    for (int d = 0; d < D; d++) {
      double acc = w->b_in[d];
      for (int i = g * G; i < (g + 1) * G; i++) acc = acc + (double)obs[i] * w->w_in[i * D + d];
      e[g][d] = acc;
    }
  for (int g = 0; g < L; g++)
    for (int d = 0; d < D; d++) {
      double aq = w->b_qkv[d], ak = w->b_qkv[D + d], av = w->b_qkv[2 * D + d];
      for (int i = 0; i < D; i++) {
        aq = aq + e[g][i] * w->w_qkv[i * 3 * D + d];
        ak = ak + e[g][i] * w->w_qkv[i * 3 * D + D + d];
        av = av + e[g][i] * w->w_qkv[i * 3 * D + 2 * D + d];
      }
      q[g][d] = aq; k[g][d] = ak; v[g][d] = av;
    }
  const double scale = 1.0 / sqrt((double)dh);
  for (int h = 0; h < NH; h++)
    for (int g = 0; g < L; g++) {
      double sc[ORC_ATTN_MAX_L];
      double mx = -INFINITY;
      for (int j = 0; j < L; j++) {
        double dot = 0.0;
        for (int t = h * dh; t < (h + 1) * dh; t++) dot = dot + q[g][t] * k[j][t];
        sc[j] = dot * scale;
        if (sc[j] > mx) mx = sc[j];
      }
      double S = 0.0;
      for (int j = 0; j < L; j++) { sc[j] = exp(sc[j] - mx); S = S + sc[j]; }
      for (int t = h * dh; t < (h + 1) * dh; t++) {
        double acc = 0.0;
        for (int j = 0; j < L; j++) acc = acc + (sc[j] / S) * v[j][t];
        o[g][t] = acc;
      }
    }
  for (int d = 0; d < D; d++) pool[d] = 0.0;
  for (int g = 0; g < L; g++)
    for (int d = 0; d < D; d++) {
      double y = w->b_o[d];
      for (int i = 0; i < D; i++) y = y + o[g][i] * w->w_o[i * D + d];
      pool[d] = pool[d] + y;
    }
  for (int d = 0; d < D; d++) pool[d] = pool[d] / (double)L;
  for (int a = 0; a < A; a++) out[a] = w->bp2[a];
  for (int j = 0; j < Hp; j++) {
    double z = w->bp1[j];
    for (int d = 0; d < D; d++) z = z + pool[d] * w->wp1[d * Hp + j];
    const double h = gelu(z);
    for (int a = 0; a < A; a++) out[a] = out[a] + h * w->wp2[j * A + a];
  }
  if (c->value_head) {
    double V = w->bv2[0];
    for (int j = 0; j < Hv; j++) {
      double z = w->bv1[j];
      for (int d = 0; d < D; d++) z = z + pool[d] * w->wv1[d * Hv + j];
      V = V + gelu(z) * w->wv2[j];
    }
    out[A] = V;
  }
}

static void policy_forward(const orc_cfg* c, const orc_weights* w, const float* obs, double* out,
                           double* h1, double* h2) {
  if (c->policy_kind == ORC_POLICY_ATTN) attn_forward(c, w, obs, out);
  else mlp_forward(c, w, obs, out, h1, h2);
}

static int attn_shape_ok(const orc_cfg* c) {
  return c->attn_tokens >= 1 && c->attn_tokens <= ORC_ATTN_MAX_L && c->attn_embed >= 1 &&
         c->attn_embed <= ORC_ATTN_MAX_D && c->attn_heads >= 1 &&
         c->attn_embed % c->attn_heads == 0 && c->obs_dim % c->attn_tokens == 0 &&
         c->mlp_h1 >= 1 && c->mlp_h2 >= 1 && !c->mlp_bf16;
}

/* Action uniform (R13, R17): 23 bits of the first word of the ACTION block, centred. */
static double action_u(uint64_t seed, uint32_t env, uint32_t k) {
  uint32_t w[4];
  draw(seed, env, k, ORC_P_ACTION, 0, 0, w);
  return ((double)(w[0] >> 9) + 0.5) * 0x1p-23;
}

/* Inverse-CDF sample of the softmax of l[0..A): the first a with u*S < cum_a, where the
 * cumulative sums run in index order; falls back to A-1. */
static int sample_action(const double* l, int A, double u, double* logp, double* margin) {
  double m = l[0];
  for (int i = 1; i < A; i++)
    if (l[i] > m) m = l[i];
  double S = 0.0;
  for (int i = 0; i < A; i++) S = S + exp(l[i] - m);
  double target = u * S;
  double cum = 0.0, lo = 0.0, hi = S;
  int a = A - 1;
  int found = 0;
  for (int i = 0; i < A; i++) {
    double prev = cum;
    cum = cum + exp(l[i] - m);
    if (target < cum) { a = i; lo = prev; hi = cum; found = 1; break; }
  }
  if (!found) { lo = cum - exp(l[A - 1] - m); hi = cum; }
  double d1 = target - lo, d2 = hi - target;
  if (d1 < 0) d1 = -d1;
  if (d2 < 0) d2 = -d2;
  *margin = (d1 < d2 ? d1 : d2) / S;
  *logp = (l[a] - m) - log(S);
  return a;
}

/* ------------------------------------------------------------------------------------ */
/* Exported entry points                                                                  */
/* ------------------------------------------------------------------------------------ */
void orc_philox4x32(const uint32_t* ctr, const uint32_t* key, uint32_t* out) {
  philox4x32_10(ctr, key, out);
}
/* n counters [n][4] under one key (two words) -> [n][4] blocks */
void orc_philox4x32_batch(int64_t n, const uint32_t* ctr, const uint32_t* key, uint32_t* out) {
  for (int64_t i = 0; i < n; i++) philox4x32_10(ctr + 4 * i, key, out + 4 * i);
}
void orc_philox4x64(const uint64_t* ctr, const uint64_t* key, uint64_t* out) {
  philox4x64_10(ctr, key, out);
}
void orc_philox_constants(uint32_t* out4) {
  out4[0] = PHX_M0; out4[1] = PHX_M1; out4[2] = PHX_W0; out4[3] = PHX_W1;
}
void orc_draw(uint64_t seed, uint32_t env, uint32_t step, uint32_t purpose, uint32_t j,
              uint32_t sys, uint32_t* out) {
  draw(seed, env, step, purpose, j, sys, out);
}
double orc_u01(uint32_t lo, uint32_t hi) { return u01(lo, hi); }

void orc_det_log(const double* x, double* y, int64_t n) {
  for (int64_t i = 0; i < n; i++) y[i] = det_log(x[i]);
}
void orc_det_exp(const double* x, double* y, int64_t n) {
  for (int64_t i = 0; i < n; i++) y[i] = det_exp(x[i]);
}
void orc_det_cos(const double* x, double* y, int64_t n) {
  for (int64_t i = 0; i < n; i++) y[i] = det_cos(x[i]);
}

/* Sampler draws for distribution tests. kind: 0 uniform u01, 1 Exp(mean p0),
 * 2 Pareto(alpha p0, x_m p1), 3 standard normal (Box-Muller), 4 lognormal service
 * median p0 * exp(p1 * Z). Block i uses counter (i, 0, purpose<<24, 0). */
void orc_sample(int32_t kind, double p0, double p1, uint64_t seed, int64_t n, double* out) {
  for (int64_t i = 0; i < n; i++) {
    uint32_t w[4];
    draw(seed, (uint32_t)i, (uint32_t)(i >> 32), ORC_P_SERVICE, 0, 0, w);
    double u = u01(w[0], w[1]);
    double v = u01(w[2], w[3]);
    double z = sqrt(-2.0 * det_log(u)) * det_cos(TWO_PI_D * v);
    switch (kind) {
      case 0: out[i] = u; break;
      case 1: out[i] = -det_log(u) * p0; break;
      case 2: out[i] = p1 * det_exp(-det_log(u) * (1.0 / p0)); break;
      case 3: out[i] = z; break;
      default: out[i] = p0 * det_exp(p1 * z); break;
    }
  }
}

int orc_n_out(const orc_cfg* c) { return n_out(c); }

/* Xavier-uniform weights from the seed (R16): element i of layer l (flattened [in][out])
 * takes u from the WEIGHTS block at counter (i, 0xFFFFFFFE, WEIGHTS<<24 | l, 0):
 * w = (2u - 1) * sqrt(6 / (fan_in + fan_out)) in fp64, rounded to fp32, then to bf16 in
 * bf16 mode. Biases are zero. Output arrays are fp64 holding the rounded values. */
void orc_init_weights(const orc_cfg* c, uint64_t seed, double* w1, double* b1, double* w2,
                      double* b2, double* w3, double* b3) {
  int dims[4] = {c->obs_dim, c->mlp_h1, c->mlp_h2, n_out(c)};
  double* ws[3] = {w1, w2, w3};
  double* bs[3] = {b1, b2, b3};
  for (int l = 0; l < 3; l++) {
    int fin = dims[l], fout = dims[l + 1];
    double lim = sqrt(6.0 / (double)(fin + fout));
    for (int64_t i = 0; i < (int64_t)fin * fout; i++) {
      uint32_t wd[4];
      draw(seed, (uint32_t)i, 0xFFFFFFFEu, ORC_P_WEIGHTS, (uint32_t)l, 0, wd);
      double u = u01(wd[0], wd[1]);
      double v = (2.0 * u - 1.0) * lim;
      double f = (double)(float)v;
      ws[l][i] = c->mlp_bf16 ? bf16r(f) : f;
    }
    for (int j = 0; j < fout; j++) bs[l][j] = 0.0;
  }
}

/* Xavier-uniform weights of the attention policy (R26): its seven matrices in the order
 * W_in [F][D], W_qkv [D][3D], W_o [D][D], W_p1 [D][H1], W_p2 [H1][A], W_v1 [D][H2],
 * W_v2 [H2][1] take layer indices 0..6 of the same counter scheme as the MLP (element i of
 * matrix l from the WEIGHTS block at (i, 0xFFFFFFFE, WEIGHTS<<24 | l, 0)), limits
 * sqrt(6 / (fan_in + fan_out)), rounded to fp32; the seven biases are zero. p[14] receives
 * w_in, b_in, w_qkv, b_qkv, w_o, b_o, wp1, bp1, wp2, bp2, wv1, bv1, wv2, bv2. Returns -1 for
 * a shape it does not support. */
int orc_init_weights_attn(const orc_cfg* c, uint64_t seed, double* const* p) {
  if (!attn_shape_ok(c)) return -1;
  const int F = c->obs_dim, D = c->attn_embed, A = 6 * c->n_servers;
  const int fin[7] = {F, D, D, D, c->mlp_h1, D, c->mlp_h2};
  const int fout[7] = {D, 3 * D, D, c->mlp_h1, A, c->mlp_h2, 1};
  for (int l = 0; l < 7; l++) {
    double lim = sqrt(6.0 / (double)(fin[l] + fout[l]));
    for (int64_t i = 0; i < (int64_t)fin[l] * fout[l]; i++) {
      uint32_t wd[4];
      draw(seed, (uint32_t)i, 0xFFFFFFFEu, ORC_P_WEIGHTS, (uint32_t)l, 0, wd);
      p[2 * l][i] = (double)(float)((2.0 * u01(wd[0], wd[1]) - 1.0) * lim);
    }
    for (int j = 0; j < fout[l]; j++) p[2 * l + 1][j] = 0.0;
  }
  return 0;
}

/* Policy forward + sampler on a batch of observations [n][F]; the uniform of row i is that
 * of env env_ids[i] at step k. Outputs: logits [n][A'], actions, logp, margin. */
int orc_policy(const orc_cfg* c, const orc_weights* w, uint64_t seed, uint32_t k, int32_t n,
                const uint32_t* env_ids, const float* obs, double* logits, uint8_t* actions,
                double* logp, double* margin) {
  int A = 6 * c->n_servers, Ap = n_out(c);
  if (c->policy_kind == ORC_POLICY_ATTN && !attn_shape_ok(c)) return -1;
  double* h1 = (double*)malloc(sizeof(double) * (size_t)c->mlp_h1);
  double* h2 = (double*)malloc(sizeof(double) * (size_t)c->mlp_h2);
  double* l = (double*)malloc(sizeof(double) * (size_t)Ap);
  for (int32_t i = 0; i < n; i++) {
    policy_forward(c, w, obs + (int64_t)i * c->obs_dim, l, h1, h2);
    if (logits) memcpy(logits + (int64_t)i * Ap, l, sizeof(double) * (size_t)Ap);
    double lp, mg;
    int a = sample_action(l, A, action_u(seed, env_ids[i], k), &lp, &mg);
    if (actions) actions[i] = (uint8_t)a;
    if (logp) logp[i] = lp;
    if (margin) margin[i] = mg;
  }
  free(h1); free(h2); free(l);
  return 0;
}

/* The rollout: T ticks of each listed env, one env at a time. With actions != NULL the
 * learned system follows actions[k][i]; otherwise it follows the policy (w != NULL).
 * Returns 0, or -1 on invalid arguments. */
int orc_rollout(const orc_cfg* c, uint64_t seed, int32_t T, int32_t n, const uint32_t* env_ids,
                const uint8_t* actions, const orc_trace* tr, const orc_weights* w,
                orc_out* out) {
  if (c->n_servers < 1 || c->n_servers > ORC_MAX_K || c->n_classes < 1 ||
      c->n_classes > ORC_MAX_C || c->queue_cap < 1 || c->queue_cap > ORC_MAX_N)
    return -1;
  if (c->arrival_kind == ORC_ARR_TRACE && !tr) return -1;
  if (!actions && !w) return -1;
  if (!actions && c->policy_kind == ORC_POLICY_ATTN && !attn_shape_ok(c)) return -1;
  if (c->n_states < 1 || c->n_states > ORC_MAX_S) return -1;
  /* observation width of R15 must fit in obs_dim */
  int need = 2 + c->n_servers * (c->n_servers > 1 ? 4 : 2) + (c->n_classes > 1 ? 2 * c->n_classes : 0) + 4;
  if (need > c->obs_dim) return -1;
  derived d;
  derive(c, &d);
  int F = c->obs_dim, Ap = n_out(c), A = 6 * c->n_servers;
  double horizon = (double)T * c->tick_s;
  sys_t* S = (sys_t*)malloc(sizeof(sys_t) * 2);
  double* h1 = (double*)malloc(sizeof(double) * (size_t)(c->mlp_h1 > 0 ? c->mlp_h1 : 1));
  double* h2 = (double*)malloc(sizeof(double) * (size_t)(c->mlp_h2 > 0 ? c->mlp_h2 : 1));
  double* l = (double*)malloc(sizeof(double) * (size_t)Ap);
  float* ob = (float*)malloc(sizeof(float) * (size_t)F);
  if (out) out->disp_count = 0;
  int nsys = c->shadow ? 2 : 1;
  for (int32_t i = 0; i < n; i++) {
    uint32_t env = env_ids[i];
    for (int s = 0; s < nsys; s++) reset_sys(c, &d, tr, i, env, seed, s, horizon, &S[s]);
    observe(c, &S[0], 0.0, ob);
    if (out && out->obs) memcpy(out->obs + (int64_t)i * F, ob, sizeof(float) * (size_t)F);
    for (int32_t k = 0; k < T; k++) {
      int a;
      if (actions) {
        a = actions[(int64_t)k * n + i];
      } else {
        policy_forward(c, w, ob, l, h1, h2);
        double lp, mg;
        a = sample_action(l, A, action_u(seed, env, (uint32_t)k), &lp, &mg);
        if (out && out->actions) out->actions[(int64_t)k * n + i] = (uint8_t)a;
        if (out && out->logp) out->logp[(int64_t)k * n + i] = (float)lp;
        if (out && out->margin) out->margin[(int64_t)k * n + i] = mg;
        if (out && out->value && c->value_head) out->value[(int64_t)k * n + i] = (float)l[A];
        if (out && out->logits)
          memcpy(out->logits + ((int64_t)k * n + i) * Ap, l, sizeof(double) * (size_t)Ap);
      }
      for (int s = 0; s < nsys; s++) {
        tick_ctx t;
        memset(&t, 0, sizeof(t));
        t.c = c; t.d = &d; t.tr = tr; t.env_idx = i; t.env = env; t.seed = seed;
        t.k = (uint32_t)k; t.out = out;
        double r = tick(&t, &S[s], a);
        if (out && out->rec) {
          int32_t* rc = out->rec + (((int64_t)k * n + i) * 2 + s) * ORC_REC_W;
          rc[0] = (int32_t)t.n_k;
          rc[1] = (int32_t)t.ndisp;
          rc[2] = sumq(&S[s], c->n_classes);
          rc[3] = t.A_k;
          rc[4] = (int32_t)S[s].dropped;
          rc[5] = (int32_t)S[s].completed;
          for (int cc = 0; cc < 4; cc++) rc[6 + cc] = cc < c->n_classes ? S[s].q[cc] : 0;
        }
        if (s == 0 && out && out->reward) out->reward[(int64_t)k * n + i] = r;
        if (s == 1 && out && out->reward_shadow) out->reward_shadow[(int64_t)k * n + i] = r;
      }
      double t1 = (double)(k + 1) * c->tick_s;
      observe(c, &S[0], t1, ob);
      if (out && out->obs) memcpy(out->obs + ((int64_t)(k + 1) * n + i) * F, ob, sizeof(float) * (size_t)F);
      if (out && out->rchk) out->rchk[(int64_t)k * n + i] = S[0].chk;
    }
    if (!actions && out && out->value && c->value_head) {
      policy_forward(c, w, ob, l, h1, h2);
      out->value[(int64_t)T * n + i] = (float)l[A];
    }
    for (int s = 0; s < nsys; s++) {
      /* requests still waiting at the horizon contribute their time up to it */
      for (int cc = 0; cc < c->n_classes; cc++)
        for (int m = 0; m < S[s].q[cc]; m++) {
          int pos = S[s].head[cc] + m;
          if (pos >= c->queue_cap) pos -= c->queue_cap;
          S[s].soj_sum = S[s].soj_sum + (horizon - S[s].ring[cc][pos]);
        }
      if (out && out->chk) out->chk[(int64_t)i * 2 + s] = S[s].chk;
      if (out && out->counters) {
        int64_t* ct = out->counters + ((int64_t)i * 2 + s) * ORC_NCNT;
        int64_t infl = 0;
        for (int j = 0; j < c->n_servers; j++) {
          infl += S[s].inflight[j];
          for (int b = 0; b < S[s].sq_cnt[j]; b++) infl += S[s].sq_n[j][b];
        }
        ct[0] = S[s].arrivals; ct[1] = S[s].accepted; ct[2] = S[s].dropped;
        ct[3] = S[s].dispatched; ct[4] = S[s].batches; ct[5] = S[s].completed; ct[6] = infl;
      }
      if (out && out->sums) {
        double* sm = out->sums + ((int64_t)i * 2 + s) * ORC_NSUM;
        sm[0] = S[s].lat_sum; sm[1] = S[s].wlat_sum; sm[2] = S[s].wait_sum;
        sm[3] = S[s].area_n; sm[4] = S[s].area_q; sm[5] = S[s].soj_sum;
      }
    }
  }
  free(S); free(h1); free(h2); free(l); free(ob);
  return 0;
}

/* Discounted returns and GAE (Sec. 4.3, R19), one env at a time, backwards in t:
 *   delta_t = (r_t + gamma V_{t+1}) - V_t,  A_t = delta_t + (gamma lambda) A_{t+1},
 *   A_T = 0,  R_t = A_t + V_t.  V == NULL means V = 0 (REINFORCE with lambda = 1). */
void orc_gae(int32_t T, int32_t n, const double* r, const float* v, double gamma, double lam,
             double* adv, double* ret) {
  double gl = gamma * lam;
  for (int32_t i = 0; i < n; i++) {
    double a = 0.0;
    for (int32_t t = T - 1; t >= 0; t--) {
      double vt = v ? (double)v[(int64_t)t * n + i] : 0.0;
      double vn = v ? (double)v[(int64_t)(t + 1) * n + i] : 0.0;
      double delta = (r[(int64_t)t * n + i] + gamma * vn) - vt;
      a = delta + gl * a;
      adv[(int64_t)t * n + i] = a;
      ret[(int64_t)t * n + i] = a + vt;
    }
  }
}

int orc_sizeof_cfg(void) { return (int)sizeof(orc_cfg); }
int orc_sizeof_out(void) { return (int)sizeof(orc_out); }
int orc_sizeof_disp(void) { return (int)sizeof(orc_disp); }

/* The sampler alone, for tests: returns the action for logits l[0..A) and uniform u. */
int32_t orc_sample_logits(const double* l, int32_t A, double u, double* logp, double* margin) {
  return sample_action(l, A, u, logp, margin);
}

/* The ACTION uniform of (env, step), for tests. */
double orc_action_u(uint64_t seed, uint32_t env, uint32_t k) { return action_u(seed, env, k); }

/* The arrival process of each listed env right after reset (R11, R21), for tests of the
 * stationary start: modulating state, next switch instant and first arrival instant.
 * Returns 0, or -1 on invalid arguments. */
int orc_reset_probe(const orc_cfg* c, uint64_t seed, int32_t n, const uint32_t* env_ids,
                    int32_t* proc, double* next_sw, double* next_arr) {
  if (c->n_states < 1 || c->n_states > ORC_MAX_S || c->arrival_kind == ORC_ARR_TRACE) return -1;
  derived d;
  derive(c, &d);
  sys_t* S = (sys_t*)malloc(sizeof(sys_t));
  if (!S) return -1;
  for (int32_t i = 0; i < n; i++) {
    reset_sys(c, &d, NULL, i, env_ids[i], seed, 0, 1.0, S);
    proc[i] = S->proc;
    next_sw[i] = S->next_sw;
    next_arr[i] = S->next_arr;
  }
  free(S);
  return 0;
}
