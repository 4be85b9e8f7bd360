// attn_kernels.hip -- the attention policy of paper Sec. 4.2, fused with action sampling.
//
// Per environment (one lane each), fp32:
//   tokens    e_g = b_in + sum over the features i of group g of x_i W_in[i,:], the F features
//             split into L contiguous groups of F/L (L = 1 is the plain input projection,
//             L = F one token per state feature);
//   attention q, k, v = e W_qkv + b_qkv; per head h (D/NH columns) softmax-weighted values
//             with scores q.k / sqrt(D/NH); y_g = concat_h o_{g,h} W_o + b_o;
//   pooling   p = mean_g y_g;
//   heads     logits = GELU(p W_p1 + b_p1) W_p2 + b_p2, V = GELU(p W_v1 + b_v1) W_v2 + b_v2.
// The action is then drawn by inverse CDF of the fp32 softmax of the logits with the ACTION
// uniform of (env, step), as for the MLP policy.
//
// The network is tiny (D = 4; about 2k multiply-adds per environment), so it runs as plain
// SIMT code: every weight is read at a wave-uniform address (scalar loads through the
// scalar cache), the per-environment state stays in registers, and the observation columns
// obs[f][E] are read coalesced.
#include "devmath.hpp"
#include "params.hpp"

namespace bsim {
namespace {

constexpr int kD = 4;          // embedding width
constexpr int kBlock = 256;

__device__ __forceinline__ float gelu_exact(float x) {
  return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}

// Scores are kept in base-2 units: the queries carry the factor log2(e) / sqrt(D/NH), so each
// softmax weight is one exp2 of (score - max).
template <int L, int NH, int A>
__global__ __launch_bounds__(kBlock) void attn_policy_k(AttnParams p, const float* __restrict__ obs,
                                                        const uint64_t* __restrict__ seedp, uint32_t step,
                                                        uint8_t* __restrict__ act,
                                                        float* __restrict__ logp,
                                                        float* __restrict__ value,
                                                        float* __restrict__ logits) {
  const uint64_t seed = *seedp;   // the episode seed
  constexpr int DH = kD / NH;
  constexpr float kLog2e = 1.4426950408889634f;
  const float qscale = (DH == 1 ? 1.0f : DH == 2 ? 0.70710678118654752f : 0.5f) * kLog2e;
  const int e = blockIdx.x * kBlock + threadIdx.x;
  if (e >= p.E) return;
  const size_t E = (size_t)p.E;
  const int G = p.F / L;

  // tokens
  float tok[L][kD];
#pragma unroll
  for (int g = 0; g < L; ++g) {
#pragma unroll
    for (int d = 0; d < kD; ++d) tok[g][d] = p.b_in[d];
    for (int i = g * G; i < (g + 1) * G; ++i) {
      const float x = obs[(size_t)i * E + e];
#pragma unroll
      for (int d = 0; d < kD; ++d) tok[g][d] = fmaf(x, p.w_in[i * kD + d], tok[g][d]);
    }
  }
  // queries, keys, values
  float q[L][kD], k[L][kD], v[L][kD];
#pragma unroll
  for (int g = 0; g < L; ++g) {
#pragma unroll
    for (int d = 0; d < kD; ++d) {
      float aq = p.b_qkv[d], ak = p.b_qkv[kD + d], av = p.b_qkv[2 * kD + d];
#pragma unroll
      for (int i = 0; i < kD; ++i) {
        aq = fmaf(tok[g][i], p.w_qkv[i * 3 * kD + d], aq);
        ak = fmaf(tok[g][i], p.w_qkv[i * 3 * kD + kD + d], ak);
        av = fmaf(tok[g][i], p.w_qkv[i * 3 * kD + 2 * kD + d], av);
      }
      q[g][d] = aq * qscale;
      k[g][d] = ak;
      v[g][d] = av;
    }
  }
  // attention, output projection and mean pooling
  float pool[kD] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int g = 0; g < L; ++g) {
    float o[kD];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      float sc[L];
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < L; ++j) {
        float dot = 0.f;
#pragma unroll
        for (int t = h * DH; t < (h + 1) * DH; ++t) dot = fmaf(q[g][t], k[j][t], dot);
        sc[j] = dot;
        mx = fmaxf(mx, sc[j]);
      }
      float S = 0.f;
#pragma unroll
      for (int j = 0; j < L; ++j) {
        sc[j] = __builtin_amdgcn_exp2f(sc[j] - mx);
        S += sc[j];
      }
      const float inv = __builtin_amdgcn_rcpf(S);
#pragma unroll
      for (int t = h * DH; t < (h + 1) * DH; ++t) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < L; ++j) acc = fmaf(sc[j], v[j][t], acc);
        o[t] = acc * inv;
      }
    }
#pragma unroll
    for (int d = 0; d < kD; ++d) {
      float y = p.b_o[d];
#pragma unroll
      for (int i = 0; i < kD; ++i) y = fmaf(o[i], p.w_o[i * kD + d], y);
      pool[d] += y;
    }
  }
#pragma unroll
  for (int d = 0; d < kD; ++d) pool[d] *= 1.0f / (float)L;   // L a power of two: exact

  // policy head
  float lg[A];
#pragma unroll
  for (int a = 0; a < A; ++a) lg[a] = p.bp2[a];
  // unrolled so that the scalar weight loads of several units are in flight together
#pragma unroll 8
  for (int j = 0; j < p.Hp; ++j) {
    float z = p.bp1[j];
#pragma unroll
    for (int d = 0; d < kD; ++d) z = fmaf(pool[d], p.wp1[d * p.Hp + j], z);
    const float hj = gelu_exact(z);
    const float* w2 = p.wp2 + (size_t)j * A;
#pragma unroll
    for (int a = 0; a < A; ++a) lg[a] = fmaf(hj, w2[a], lg[a]);
  }
  // value head
  float V = 0.f;
  if (p.value_head) {
    V = p.bv2[0];
#pragma unroll 8
    for (int j = 0; j < p.Hv; ++j) {
      float z = p.bv1[j];
#pragma unroll
      for (int d = 0; d < kD; ++d) z = fmaf(pool[d], p.wv1[d * p.Hv + j], z);
      V = fmaf(gelu_exact(z), p.wv2[j], V);
    }
  }

  // sampling: fp32 max-subtracted softmax, first action whose running sum exceeds u S
  if (act || logp) {
    float mx = lg[0];
#pragma unroll
    for (int a = 1; a < A; ++a) mx = fmaxf(mx, lg[a]);
    float ex[A];
    float S = 0.f;
#pragma unroll
    for (int a = 0; a < A; ++a) {
      ex[a] = expf(lg[a] - mx);
      S += ex[a];
    }
    const u32x4 w = draw(seed, (uint32_t)e, step, P_ACTION, 0, 0);
    const float target = (((float)(w.x >> 9) + 0.5f) * 0x1p-23f) * S;
    float cum = 0.f, la = lg[A - 1];
    int pick = A - 1;
    bool found = false;
#pragma unroll
    for (int a = 0; a < A; ++a) {
      cum += ex[a];
      const bool take = !found && target < cum;
      pick = take ? a : pick;
      la = take ? lg[a] : la;
      found = found || take;
    }
    if (act) act[e] = (uint8_t)pick;
    if (logp) logp[e] = (la - mx) - logf(S);
  }
  if (value && p.value_head) value[e] = V;
  if (logits) {
#pragma unroll
    for (int a = 0; a < A; ++a) logits[(size_t)a * E + e] = lg[a];
    if (p.value_head) logits[(size_t)A * E + e] = V;
  }
}

template <int L, int NH, int A>
hipError_t run_attn(const AttnParams& p, const float* obs, const uint64_t* seed, uint32_t step,
                    uint8_t* act, float* logp, float* value, float* logits, hipStream_t st) {
  const dim3 grid((unsigned)((p.E + kBlock - 1) / kBlock)), block(kBlock);
  hipLaunchKernelGGL((attn_policy_k<L, NH, A>), grid, block, 0, st, p, obs, seed, step, act, logp,
                     value, logits);
  return hipGetLastError();
}

template <int L, int NH>
hipError_t run_attn_a(const AttnParams& p, const float* obs, const uint64_t* seed, uint32_t step,
                      uint8_t* act, float* logp, float* value, float* logits, hipStream_t st) {
  switch (p.A) {
    case 6: return run_attn<L, NH, 6>(p, obs, seed, step, act, logp, value, logits, st);
    case 12: return run_attn<L, NH, 12>(p, obs, seed, step, act, logp, value, logits, st);
    case 24: return run_attn<L, NH, 24>(p, obs, seed, step, act, logp, value, logits, st);
    default: return hipErrorInvalidValue;
  }
}

template <int L>
hipError_t run_attn_h(const AttnParams& p, const float* obs, const uint64_t* seed, uint32_t step,
                      uint8_t* act, float* logp, float* value, float* logits, hipStream_t st) {
  switch (p.NH) {
    case 1: return run_attn_a<L, 1>(p, obs, seed, step, act, logp, value, logits, st);
    case 2: return run_attn_a<L, 2>(p, obs, seed, step, act, logp, value, logits, st);
    case 4: return run_attn_a<L, 4>(p, obs, seed, step, act, logp, value, logits, st);
    default: return hipErrorInvalidValue;
  }
}

// ---- gradient of one minibatch (Sec. 4.3 losses through the Sec. 4.2 network) --------------
// One lane per sample m: the (t, env) index drawn like the MLP minibatch's, the forward in
// fp32, the loss gradient with respect to the logits and V, then the chain rule backwards.
// The pooled vector's gradient dp reaches every token's output equally (dy_g = dp / L), so
// dW_o = (sum_g o_g)^T dy, do_g = dy W_o^T is the same for every token and so is
// da_{gj} = do . v_j per head; the softmax weights are recomputed per query token. Every
// parameter's per-sample term goes to gs[param][m]; a second kernel sums over m in a fixed order.
struct AttnGradArgs {
  AttnParams p;
  int T, M, reinforce;
  const float* obs;          // [T(+1)][F][E]
  const uint8_t* act;        // [T][E]
  const float* logp_old;     // [T][E] (PPO)
  const double* adv;         // [T][E]
  const double* ret;         // [T][E]
  uint64_t seed;
  float clip, c_v, c_h;
  float* gs;                 // [P][M] per-sample gradient terms
  double* terms;             // [M][3] policy, value, entropy per sample
  int64_t* idx_out;          // optional [M]
  uint32_t* err;
  int off[14];               // start of each parameter array in the gradient vector
  int P;
};

__device__ __forceinline__ float gelu_grad(float z) {
  return 0.5f * (1.0f + erff(z * 0.70710678118654752f)) + z * expf(-0.5f * z * z) * 0.39894228040143268f;
}

template <int L, int NH, int A>
__global__ __launch_bounds__(64) void attn_grad_k(AttnGradArgs g) {
  constexpr int D = kD, DH = D / NH;
  const float rs = DH == 1 ? 1.0f : DH == 2 ? 0.70710678118654752f : 0.5f;  // 1 / sqrt(DH)
  const int m = blockIdx.x * 64 + threadIdx.x;
  if (m >= g.M) return;
  const AttnParams& p = g.p;
  const size_t E = (size_t)p.E, M = (size_t)g.M;
  const int G = p.F / L;
  auto put = [&](int k, int i, float v) { g.gs[(size_t)(g.off[k] + i) * M + m] = v; };

  const u32x4 w = draw(g.seed, (uint32_t)m, 0xFFFFFFFDu, P_MINIBATCH, 0, 0);
  long long ix = (long long)(unit(w.x, w.y) * ((double)g.T * (double)p.E));
  if (ix > (long long)g.T * p.E - 1) ix = (long long)g.T * p.E - 1;
  if (g.idx_out) g.idx_out[m] = ix;
  const int t = (int)(ix / p.E), e = (int)(ix % p.E);
  const size_t ti = (size_t)t * E + e;
  const float* xo = g.obs + (size_t)t * p.F * E + e;
  const int a_act = g.act[ti];
  if (a_act >= A) {  // invalid stored action: flag it, the sample contributes nothing
    atomicOr(g.err, ERR_ACTION);
    for (int i = 0; i < g.P; ++i) g.gs[(size_t)i * M + m] = 0.0f;
    g.terms[m * 3] = g.terms[m * 3 + 1] = g.terms[m * 3 + 2] = 0.0;
    return;
  }

  // forward
  float tok[L][D];
#pragma unroll
  for (int gg = 0; gg < L; ++gg) {
#pragma unroll
    for (int d = 0; d < D; ++d) tok[gg][d] = p.b_in[d];
    for (int i = gg * G; i < (gg + 1) * G; ++i) {
      const float x = xo[(size_t)i * E];
#pragma unroll
      for (int d = 0; d < D; ++d) tok[gg][d] = fmaf(x, p.w_in[i * D + d], tok[gg][d]);
    }
  }
  float q[L][D], k[L][D], v[L][D];
#pragma unroll
  for (int gg = 0; gg < L; ++gg)
#pragma unroll
    for (int d = 0; d < D; ++d) {
      float aq = p.b_qkv[d], ak = p.b_qkv[D + d], av = p.b_qkv[2 * D + d];
#pragma unroll
      for (int i = 0; i < D; ++i) {
        aq = fmaf(tok[gg][i], p.w_qkv[i * 3 * D + d], aq);
        ak = fmaf(tok[gg][i], p.w_qkv[i * 3 * D + D + d], ak);
        av = fmaf(tok[gg][i], p.w_qkv[i * 3 * D + 2 * D + d], av);
      }
      q[gg][d] = aq; k[gg][d] = ak; v[gg][d] = av;
    }
  // softmax weights of query gg, head h
  auto weights = [&](int gg, int h, float (&a)[L]) {
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < L; ++j) {
      float dot = 0.f;
#pragma unroll
      for (int tt = h * DH; tt < (h + 1) * DH; ++tt) dot = fmaf(q[gg][tt], k[j][tt], dot);
      a[j] = dot * rs;
      mx = fmaxf(mx, a[j]);
    }
    float S = 0.f;
#pragma unroll
    for (int j = 0; j < L; ++j) {
      a[j] = expf(a[j] - mx);
      S += a[j];
    }
    const float inv = 1.0f / S;
#pragma unroll
    for (int j = 0; j < L; ++j) a[j] *= inv;
  };
  float osum[D] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int gg = 0; gg < L; ++gg)
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      float a[L];
      weights(gg, h, a);
#pragma unroll
      for (int tt = h * DH; tt < (h + 1) * DH; ++tt) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < L; ++j) acc = fmaf(a[j], v[j][tt], acc);
        osum[tt] += acc;
      }
    }
  float pool[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    float y = 0.f;
#pragma unroll
    for (int i = 0; i < D; ++i) y = fmaf(osum[i], p.w_o[i * D + d], y);
    pool[d] = y * (1.0f / (float)L) + p.b_o[d];
  }
  float lg[A];
#pragma unroll
  for (int a = 0; a < A; ++a) lg[a] = p.bp2[a];
  for (int j = 0; j < p.Hp; ++j) {
    float z = p.bp1[j];
#pragma unroll
    for (int d = 0; d < D; ++d) z = fmaf(pool[d], p.wp1[d * p.Hp + j], z);
    const float hj = gelu_exact(z);
#pragma unroll
    for (int a = 0; a < A; ++a) lg[a] = fmaf(hj, p.wp2[(size_t)j * A + a], lg[a]);
  }
  float V = p.bv2[0];
  for (int j = 0; j < p.Hv; ++j) {
    float z = p.bv1[j];
#pragma unroll
    for (int d = 0; d < D; ++d) z = fmaf(pool[d], p.wv1[d * p.Hv + j], z);
    V = fmaf(gelu_exact(z), p.wv2[j], V);
  }

  // loss terms and their gradient with respect to the logits and V
  const float adv = (float)g.adv[ti], ret = (float)g.ret[ti];
  float mx = lg[0];
#pragma unroll
  for (int a = 1; a < A; ++a) mx = fmaxf(mx, lg[a]);
  float S = 0.f;
#pragma unroll
  for (int a = 0; a < A; ++a) S += expf(lg[a] - mx);
  const float lS = logf(S);
  float H = 0.f;
#pragma unroll
  for (int a = 0; a < A; ++a) {
    const float lp = (lg[a] - mx) - lS;
    H -= expf(lp) * lp;
  }
  float l_act = lg[0];
#pragma unroll
  for (int a = 1; a < A; ++a) l_act = a == a_act ? lg[a] : l_act;
  const float logp = (l_act - mx) - lS;
  const float invM = 1.0f / (float)g.M;
  float dlogp, pterm;
  if (g.reinforce) {
    dlogp = -adv * invM;
    pterm = -adv * logp;
  } else {
    const float rho = expf(logp - g.logp_old[ti]);
    const float lo = 1.0f - g.clip, hi = 1.0f + g.clip;
    const float rc = fminf(fmaxf(rho, lo), hi);
    const float s1 = rho * adv, s2 = rc * adv;
    const float g_rho = s1 <= s2 ? adv : ((rho > lo && rho < hi) ? adv : 0.0f);
    dlogp = -g_rho * rho * invM;
    pterm = -fminf(s1, s2);
  }
  float dl[A];
#pragma unroll
  for (int a = 0; a < A; ++a) {
    const float lp = (lg[a] - mx) - lS;
    const float pa = expf(lp);
    dl[a] = -dlogp * pa + g.c_h * invM * pa * (lp + H) + (a == a_act ? dlogp : 0.0f);
  }
  const float dV = p.value_head ? 2.0f * g.c_v * (V - ret) * invM : 0.0f;
  g.terms[m * 3] = (double)pterm;
  g.terms[m * 3 + 1] = (double)(V - ret) * (double)(V - ret);
  g.terms[m * 3 + 2] = (double)H;

  // heads backward
  float dp[D] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int a = 0; a < A; ++a) put(9, a, dl[a]);
  for (int j = 0; j < p.Hp; ++j) {
    float z = p.bp1[j];
#pragma unroll
    for (int d = 0; d < D; ++d) z = fmaf(pool[d], p.wp1[d * p.Hp + j], z);
    const float hj = gelu_exact(z);
    float dh = 0.f;
#pragma unroll
    for (int a = 0; a < A; ++a) {
      dh = fmaf(dl[a], p.wp2[(size_t)j * A + a], dh);
      put(8, j * A + a, hj * dl[a]);
    }
    const float dz = dh * gelu_grad(z);
    put(7, j, dz);
#pragma unroll
    for (int d = 0; d < D; ++d) {
      put(6, d * p.Hp + j, pool[d] * dz);
      dp[d] = fmaf(dz, p.wp1[d * p.Hp + j], dp[d]);
    }
  }
  put(13, 0, dV);
  for (int j = 0; j < p.Hv; ++j) {
    float z = p.bv1[j];
#pragma unroll
    for (int d = 0; d < D; ++d) z = fmaf(pool[d], p.wv1[d * p.Hv + j], z);
    put(12, j, gelu_exact(z) * dV);
    const float dz = dV * p.wv2[j] * gelu_grad(z);
    put(11, j, dz);
#pragma unroll
    for (int d = 0; d < D; ++d) {
      put(10, d * p.Hv + j, pool[d] * dz);
      dp[d] = fmaf(dz, p.wv1[d * p.Hv + j], dp[d]);
    }
  }
  // output projection: dy = dp / L for every token
  float dy[D], dO[D];
#pragma unroll
  for (int d = 0; d < D; ++d) dy[d] = dp[d] * (1.0f / (float)L);
#pragma unroll
  for (int i = 0; i < D; ++i) {
    float acc = 0.f;
#pragma unroll
    for (int d = 0; d < D; ++d) {
      put(4, i * D + d, osum[i] * dy[d]);
      acc = fmaf(dy[d], p.w_o[i * D + d], acc);
    }
    dO[i] = acc;
  }
#pragma unroll
  for (int d = 0; d < D; ++d) put(5, d, dp[d]);
  // attention backward, head by head
  float dq[L][D], dk[L][D], dv[L][D];
#pragma unroll
  for (int gg = 0; gg < L; ++gg)
#pragma unroll
    for (int d = 0; d < D; ++d) { dq[gg][d] = 0.f; dk[gg][d] = 0.f; dv[gg][d] = 0.f; }
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    float da[L], colsum[L];
#pragma unroll
    for (int j = 0; j < L; ++j) {
      float acc = 0.f;
#pragma unroll
      for (int tt = h * DH; tt < (h + 1) * DH; ++tt) acc = fmaf(dO[tt], v[j][tt], acc);
      da[j] = acc;
      colsum[j] = 0.f;
    }
#pragma unroll
    for (int gg = 0; gg < L; ++gg) {
      float a[L];
      weights(gg, h, a);
      float sd = 0.f;
#pragma unroll
      for (int j = 0; j < L; ++j) {
        sd = fmaf(a[j], da[j], sd);
        colsum[j] += a[j];
      }
#pragma unroll
      for (int j = 0; j < L; ++j) {
        const float ds = a[j] * (da[j] - sd) * rs;
#pragma unroll
        for (int tt = h * DH; tt < (h + 1) * DH; ++tt) {
          dq[gg][tt] = fmaf(ds, k[j][tt], dq[gg][tt]);
          dk[j][tt] = fmaf(ds, q[gg][tt], dk[j][tt]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < L; ++j)
#pragma unroll
      for (int tt = h * DH; tt < (h + 1) * DH; ++tt) dv[j][tt] = colsum[j] * dO[tt];
  }
  // q/k/v projection and the tokens
  float de[L][D];
#pragma unroll
  for (int gg = 0; gg < L; ++gg)
#pragma unroll
    for (int i = 0; i < D; ++i) de[gg][i] = 0.f;
#pragma unroll
  for (int c = 0; c < 3 * D; ++c) {
    float bsum = 0.f;
    float col[L];
#pragma unroll
    for (int gg = 0; gg < L; ++gg) {
      col[gg] = c < D ? dq[gg][c] : (c < 2 * D ? dk[gg][c - D] : dv[gg][c - 2 * D]);
      bsum += col[gg];
    }
    put(3, c, bsum);
#pragma unroll
    for (int i = 0; i < D; ++i) {
      float wsum = 0.f;
#pragma unroll
      for (int gg = 0; gg < L; ++gg) {
        wsum = fmaf(tok[gg][i], col[gg], wsum);
        de[gg][i] = fmaf(col[gg], p.w_qkv[i * 3 * D + c], de[gg][i]);
      }
      put(2, i * 3 * D + c, wsum);
    }
  }
#pragma unroll
  for (int d = 0; d < D; ++d) {
    float bsum = 0.f;
#pragma unroll
    for (int gg = 0; gg < L; ++gg) bsum += de[gg][d];
    put(1, d, bsum);
  }
#pragma unroll
  for (int gg = 0; gg < L; ++gg)
    for (int i = gg * G; i < (gg + 1) * G; ++i) {
      const float x = xo[(size_t)i * E];
#pragma unroll
      for (int d = 0; d < D; ++d) put(0, i * D + d, x * de[gg][d]);
    }
}

// grads[i] = sum over m of gs[i][m]: each of 256 threads sums a strided slice in order, then
// a fixed tree
__global__ __launch_bounds__(256) void attn_gsum_k(const float* __restrict__ gs, int M,
                                                   float* __restrict__ grads) {
  __shared__ float part[256];
  const float* row = gs + (size_t)blockIdx.x * M;
  float s = 0.f;
  for (int m = threadIdx.x; m < M; m += 256) s += row[m];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) grads[blockIdx.x] = part[0];
}

template <int L, int NH, int A>
hipError_t run_grad(const AttnGradArgs& g, hipStream_t st) {
  hipLaunchKernelGGL((attn_grad_k<L, NH, A>), dim3((unsigned)((g.M + 63) / 64)), dim3(64), 0, st, g);
  return hipGetLastError();
}
template <int L, int NH>
hipError_t run_grad_a(const AttnGradArgs& g, hipStream_t st) {
  switch (g.p.A) {
    case 6: return run_grad<L, NH, 6>(g, st);
    case 12: return run_grad<L, NH, 12>(g, st);
    case 24: return run_grad<L, NH, 24>(g, st);
    default: return hipErrorInvalidValue;
  }
}
template <int L>
hipError_t run_grad_h(const AttnGradArgs& g, hipStream_t st) {
  switch (g.p.NH) {
    case 1: return run_grad_a<L, 1>(g, st);
    case 2: return run_grad_a<L, 2>(g, st);
    case 4: return run_grad_a<L, 4>(g, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int attn_param_count(const AttnParams& p, int off[14]) {
  const int D = p.D, n[14] = {p.F * D, D, D * 3 * D, 3 * D, D * D, D, D * p.Hp, p.Hp,
                              p.Hp * p.A, p.A, D * p.Hv, p.Hv, p.Hv, 1};
  int acc = 0;
  for (int i = 0; i < 14; ++i) {
    if (off) off[i] = acc;
    acc += n[i];
  }
  return acc;
}

size_t attn_grad_scratch_bytes(const AttnParams& p, int M) {
  return (size_t)attn_param_count(p, nullptr) * M * sizeof(float) + (size_t)M * 3 * sizeof(double);
}

hipError_t launch_attn_grad(const AttnParams& p, int T, const float* obs, const uint8_t* act,
                            const float* logp_old, const double* adv, const double* ret, int M,
                            uint64_t seed, float clip, float c_v, float c_h, int reinforce,
                            void* scratch, double* loss_out, float* grads, int64_t* idx_out,
                            uint32_t* err, hipStream_t st) {
  if (!attn_shape_supported(p) || M < 1) return hipErrorInvalidValue;
  AttnGradArgs g;
  g.p = p; g.T = T; g.M = M; g.reinforce = reinforce;
  g.obs = obs; g.act = act; g.logp_old = logp_old; g.adv = adv; g.ret = ret;
  g.seed = seed; g.clip = clip; g.c_v = c_v; g.c_h = c_h;
  g.P = attn_param_count(p, g.off);
  g.gs = static_cast<float*>(scratch);
  g.terms = reinterpret_cast<double*>(g.gs + (size_t)g.P * M);
  g.idx_out = idx_out; g.err = err;
  hipError_t e;
  switch (p.L) {
    case 1: e = run_grad_h<1>(g, st); break;
    case 2: e = run_grad_h<2>(g, st); break;
    case 4: e = run_grad_h<4>(g, st); break;
    case 8: e = run_grad_h<8>(g, st); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_gsum_k, dim3((unsigned)g.P), dim3(256), 0, st, g.gs, M, grads);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_pg_loss(g.terms, M, c_v, c_h, loss_out, st);
}

bool attn_shape_supported(const AttnParams& p) {
  const bool L_ok = p.L == 1 || p.L == 2 || p.L == 4 || p.L == 8;
  const bool H_ok = p.NH == 1 || p.NH == 2 || p.NH == 4;
  const bool A_ok = p.A == 6 || p.A == 12 || p.A == 24;
  return L_ok && H_ok && A_ok && p.D == kD && p.F % p.L == 0 && p.Hp >= 1 && p.Hv >= 1;
}

hipError_t launch_attn_policy(const AttnParams& p, const float* obs, const uint64_t* seed, uint32_t step,
                              uint8_t* act, float* logp, float* value, float* logits,
                              hipStream_t st) {
  if (!attn_shape_supported(p)) return hipErrorInvalidValue;
  switch (p.L) {
    case 1: return run_attn_h<1>(p, obs, seed, step, act, logp, value, logits, st);
    case 2: return run_attn_h<2>(p, obs, seed, step, act, logp, value, logits, st);
    case 4: return run_attn_h<4>(p, obs, seed, step, act, logp, value, logits, st);
    case 8: return run_attn_h<8>(p, obs, seed, step, act, logp, value, logits, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace bsim
