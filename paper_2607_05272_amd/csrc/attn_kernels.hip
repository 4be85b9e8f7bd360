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
                                                        uint64_t seed, uint32_t step,
                                                        uint8_t* __restrict__ act,
                                                        float* __restrict__ logp,
                                                        float* __restrict__ value,
                                                        float* __restrict__ logits) {
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
hipError_t run_attn(const AttnParams& p, const float* obs, uint64_t seed, uint32_t step,
                    uint8_t* act, float* logp, float* value, float* logits, hipStream_t st) {
  const dim3 grid((unsigned)((p.E + kBlock - 1) / kBlock)), block(kBlock);
  hipLaunchKernelGGL((attn_policy_k<L, NH, A>), grid, block, 0, st, p, obs, seed, step, act, logp,
                     value, logits);
  return hipGetLastError();
}

template <int L, int NH>
hipError_t run_attn_a(const AttnParams& p, const float* obs, uint64_t seed, uint32_t step,
                      uint8_t* act, float* logp, float* value, float* logits, hipStream_t st) {
  switch (p.A) {
    case 6: return run_attn<L, NH, 6>(p, obs, seed, step, act, logp, value, logits, st);
    case 12: return run_attn<L, NH, 12>(p, obs, seed, step, act, logp, value, logits, st);
    case 24: return run_attn<L, NH, 24>(p, obs, seed, step, act, logp, value, logits, st);
    default: return hipErrorInvalidValue;
  }
}

template <int L>
hipError_t run_attn_h(const AttnParams& p, const float* obs, uint64_t seed, uint32_t step,
                      uint8_t* act, float* logp, float* value, float* logits, hipStream_t st) {
  switch (p.NH) {
    case 1: return run_attn_a<L, 1>(p, obs, seed, step, act, logp, value, logits, st);
    case 2: return run_attn_a<L, 2>(p, obs, seed, step, act, logp, value, logits, st);
    case 4: return run_attn_a<L, 4>(p, obs, seed, step, act, logp, value, logits, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool attn_shape_supported(const AttnParams& p) {
  const bool L_ok = p.L == 1 || p.L == 2 || p.L == 4 || p.L == 8;
  const bool H_ok = p.NH == 1 || p.NH == 2 || p.NH == 4;
  const bool A_ok = p.A == 6 || p.A == 12 || p.A == 24;
  return L_ok && H_ok && A_ok && p.D == kD && p.F % p.L == 0 && p.Hp >= 1 && p.Hv >= 1;
}

hipError_t launch_attn_policy(const AttnParams& p, const float* obs, uint64_t seed, uint32_t step,
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
