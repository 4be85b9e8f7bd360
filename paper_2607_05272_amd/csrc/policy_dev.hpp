// policy_dev.hpp -- device code of the policy MLP (paper Sec. 4.2) and its action sampler,
// shared by the policy kernels and the fused small-batch rollout kernel.
//
// obs [F][E] -> h1 = GELU(x W1 + b1) -> h2 = GELU(h1 W2 + b2) -> out = h2 W3 + b3, where
// out[0..A) are the logits of the categorical action distribution and out[A] (when the
// value head is on) is V(s). The epilogue of the last layer samples the action by inverse CDF
// of the fp32 softmax with the ACTION uniform of (env, step) and writes action,
// log-probability and value.
//
// Two forms. fp32 policies (v_mfma_f32_16x16x4_f32): one workgroup of 4 waves owns 16 RT
// environments whose activations live in LDS (RT = 1 for small batches, whose launch lasts as
// long as one workgroup's chain of layers; 4 otherwise); each wave produces a quarter of the
// output columns of every layer, loading all of its weight fragments of a layer from the
// repacked weights in L2 before the layer's first MFMA.
// bf16 policies: every layer's input rounded to bf16 (RNE), bf16 weights, fp32 accumulation
// (v_mfma_f32_16x16x32_bf16), bias and GELU in fp32; its layout and scheduling are described
// above policy_tile_bf16.
#pragma once
#include "devmath.hpp"
#include "params.hpp"

namespace bsim {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kThreads = 256;  // 4 waves

struct F32Mode {
  typedef float elem;
  typedef float frag;
  static constexpr int KS = 4;
  static constexpr int KL = 1;
  static constexpr int PAD = 4;
  __device__ static frag load(const elem* p) { return *p; }
  __device__ static f32x4 mfma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  __device__ static elem from_f32(float f) { return f; }
};

__device__ __forceinline__ float gelu(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }

// Where a diagnostic instantiation (DBG = true) of the policy kernels also writes every hidden
// activation it passes to the next layer: h [N][E] fp32 (bf16 values widened), for the
// workgroup's environments e0 .. The production instantiations (DBG = false) compile without
// these stores and are otherwise the same code.
struct HidOut {
  float* h;
  int E, e0;
};

// out[16 RT][N] = act_in[16 RT][K] * W^T  (W packed out-major [N][K]); epilogue: +bias, then
// GELU + rounding into act_out (hidden layers) or fp32 into lg (last layer).
template <class M, int K, int N, int RT, bool LAST, bool DBG = false>
__device__ __forceinline__ void layer(const typename M::elem* __restrict__ in,
                                      const typename M::elem* __restrict__ W,
                                      const float* __restrict__ bias,
                                      typename M::elem* __restrict__ out, float* __restrict__ lg,
                                      int lg_stride, HidOut ho = {}) {
  constexpr int NT = N / 16;             // column tiles
  // wave w owns tiles w, w + 4, ...: all NT / 4 of them, or (NT < 4) one tile or none, so
  // that no MFMA or load below sits behind a per-tile branch (which would make every MFMA wait
  // for its own operand loads)
  static_assert(NT % 4 == 0 || NT < 4, "a wave owns all of its column tiles or none");
  constexpr int NTW = NT < 4 ? 1 : NT / 4;
  constexpr int SIN = K + M::PAD;        // LDS row stride of the input
  constexpr int SOUT = N + M::PAD;
  constexpr int KSTEPS = K / M::KS;
  static_assert(K % M::KS == 0, "whole k-steps");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  if (wave >= NT) return;  // only when NT < 4; uniform over the wave
  // every weight fragment of the wave's tiles is loaded before the first MFMA: the loads are
  // independent, so the layer waits out one L2 round trip instead of one per k-step (at most
  // 64 x 64 weights per layer here: NTW * K / KS registers per lane)
  typename M::frag wfr[KSTEPS][NTW];
#pragma unroll
  for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
    for (int c = 0; c < NTW; ++c)
      wfr[ks][c] = M::load(W + (size_t)((wave + 4 * c) * 16 + r16) * K + ks * M::KS + kq * M::KL);
  f32x4 acc[RT][NTW];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int c = 0; c < NTW; ++c) acc[rt][c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < KSTEPS; ++ks) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const typename M::frag a = M::load(in + (rt * 16 + r16) * SIN + ks * M::KS + kq * M::KL);
#pragma unroll
      for (int c = 0; c < NTW; ++c) acc[rt][c] = M::mfma(a, wfr[ks][c], acc[rt][c]);
    }
  }
#pragma unroll
  for (int c = 0; c < NTW; ++c) {
    const int col = (wave + 4 * c) * 16 + r16;
    const float bv = bias[col];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = rt * 16 + kq * 4 + i;
        const float v = acc[rt][c][i] + bv;
        if (LAST) {
          lg[row * lg_stride + col] = v;
        } else {
          const typename M::elem g = M::from_f32(gelu(v));
          out[row * SOUT + col] = g;
          if constexpr (DBG)
            if (ho.e0 + row < ho.E) ho.h[(size_t)col * ho.E + ho.e0 + row] = (float)g;
        }
      }
    }
  }
}

template <class M, int FP, int H1, int H2, int AP, int RT>
struct Shape {
  typedef typename M::elem E;
  static constexpr int ROWS = 16 * RT;
  static constexpr int SX = FP + M::PAD, S1 = H1 + M::PAD, S2 = H2 + M::PAD, SL = AP + 1;
  static constexpr size_t X_BYTES = (size_t)ROWS * SX * sizeof(E);
  static constexpr size_t H1_BYTES = (size_t)ROWS * S1 * sizeof(E);
  static constexpr size_t H2_BYTES = (size_t)ROWS * S2 * sizeof(E);
  static constexpr size_t L_BYTES = (size_t)ROWS * SL * sizeof(float);
  // x shares the h2 region (dead before h2 is written), logits share the h1 region
  static constexpr size_t REGION_A = H2_BYTES > X_BYTES ? H2_BYTES : X_BYTES;
  static constexpr size_t REGION_B = H1_BYTES > L_BYTES ? H1_BYTES : L_BYTES;
  static constexpr size_t LDS = REGION_A + REGION_B;
};

// Sampling epilogue of both policy kernels: for each of the workgroup's ROWS environment rows
// of logits lg [row][sl], the action by inverse CDF of the fp32 softmax with the ACTION
// uniform of (env, step), its log-probability and the value output. G lanes per row (an
// aligned group of G lanes), each over a contiguous slice of the actions whose exponentials
// it keeps in registers; max, prefix sums and the first slice holding the target u*S by
// DPP moves within the group (below), the same operands in the same order as a chain of
// shuffles would combine, without a round trip through LDS for each of the ten steps.
//
// Cross-lane moves within aligned groups of 8 lanes (half a DPP row of 16): lane ^ 1 and
// lane ^ 2 as quad permutations, 7 - lane as the half-row mirror, lane - d (d = 1, 2, 4) as
// a row shift (lanes without a source keep 0; the callers mask them), and lane 3 of each quad.
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppQuad3 = 0xFF, kDppHalfMirror = 0x141;
constexpr int kDppShr = 0x110;   // + d: row shift right by d
template <int CTRL>
__device__ __forceinline__ int dpp8(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp8(float v) {
  return __int_as_float(dpp8<CTRL>(__float_as_int(v)));
}
// max / min over the lane's group of 8: within each quad, then across the two quads
__device__ __forceinline__ float group8_max(float v) {
  v = fmaxf(v, dpp8<kDppXor1>(v));
  v = fmaxf(v, dpp8<kDppXor2>(v));
  return fmaxf(v, dpp8<kDppHalfMirror>(v));
}
__device__ __forceinline__ int group8_min(int v) {
  v = min(v, dpp8<kDppXor1>(v));
  v = min(v, dpp8<kDppXor2>(v));
  return min(v, dpp8<kDppHalfMirror>(v));
}
// inclusive prefix sum over the group (part = lane % 8), in the order of a shift-by-1, 2, 4
// scan, and the group's total (lane 7's prefix) in every lane
__device__ __forceinline__ float group8_scan(float v, int part, float& total) {
  float t = dpp8<kDppShr + 1>(v);
  if (part >= 1) v += t;
  t = dpp8<kDppShr + 2>(v);
  if (part >= 2) v += t;
  t = dpp8<kDppShr + 4>(v);
  if (part >= 4) v += t;
  const float q3 = dpp8<kDppQuad3>(v);         // lanes 0-3: lane 3's prefix; 4-7: lane 7's
  const float m3 = dpp8<kDppHalfMirror>(q3);   // lanes 0-3: lane 7's (from lanes 7..4)
  total = part >= 4 ? q3 : m3;
  return v;
}

// The ACTION uniform of a row's environment: ((w.x >> 9) + 1/2) 2^-23 from its block.
__device__ __forceinline__ float action_uniform(uint64_t seed, uint32_t env, uint32_t step) {
  const u32x4 w = draw(seed, env, step, P_ACTION, 0, 0);
  return ((float)(w.x >> 9) + 0.5f) * 0x1p-23f;
}

// us: the rows' uniforms, drawn beforehand (one lane per row), or NULL to draw them here (every
// lane of a row's group then computes the same block).
// AC: the action count when the padded width fixes it (0: m.A at run time); with it the
// slices' bounds are compile-time and the per-logit guards vanish.
template <int AP, int ROWS, int NTHR, int AC = 0>
__device__ __forceinline__ void sample_rows(const float* lg, int sl, const MlpParams& m, int e0,
                                            uint64_t seed, uint32_t step, uint8_t* act,
                                            float* logp, float* value, float* logits,
                                            const float* us = nullptr) {
  constexpr int G = 8, KMAX = AC > 0 ? (AC + G - 1) / G : (AP + G - 1) / G;
  static_assert(NTHR % G == 0 && G == 8, "sampler groups of 8 lanes (group8_*)");
  const int tid = threadIdx.x;
  for (int row0 = 0; row0 < ROWS; row0 += NTHR / G) {
    const int row = row0 + tid / G, part = tid % G;
    const int e = e0 + row;
    const bool live = row < ROWS && e < m.E;
    const float* l = lg + (row < ROWS ? row : 0) * sl;
    const int A = AC > 0 ? AC : m.A;
    const int chunk = (A + G - 1) / G;
    const int lo = part * chunk;
    float mx = -3.0e38f;
#pragma unroll
    for (int i = 0; i < KMAX; ++i)
      if (i < chunk && lo + i < A) mx = fmaxf(mx, l[lo + i]);
    mx = group8_max(mx);
    float pe[KMAX];
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      pe[i] = (i < chunk && lo + i < A) ? __expf(l[lo + i] - mx) : 0.f;
      ps += pe[i];
    }
    float S;
    const float incl = group8_scan(ps, part, S);
    const float u = us ? us[row < ROWS ? row : 0]
                       : action_uniform(seed, (uint32_t)(live ? e : 0), step);
    const float target = u * S;
    int found = 0x7fffffff;
    float cum = incl - ps;
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      cum += pe[i];
      if (found == 0x7fffffff && i < chunk && lo + i < A && target < cum) found = lo + i;
    }
    found = group8_min(found);
    if (live && part == 0) {
      const int a = found < A ? found : A - 1;
      if (act) act[e] = (uint8_t)a;
      if (logp) logp[e] = (l[a] - mx) - __logf(S);
      if (value && m.value_head) value[e] = l[A];
    }
    if (live && logits)
      for (int i = part; i < m.Ap; i += G) logits[(size_t)i * m.E + e] = l[i];
  }
}

// One workgroup's share of the fp32 policy: environments e0 .. e0 + 16 RT - 1 (rows past E
// take zeros and write nothing), activations in smem (Shape::LDS bytes of LDS). Called by
// all kThreads threads of the workgroup, which it synchronises.
template <class M, int FP, int H1, int H2, int AP, int RT, bool DBG>
__device__ __forceinline__ void policy_tile_f32(const MlpParams& m, const float* __restrict__ obs,
                                                uint64_t seed, uint32_t step,
                                                uint8_t* __restrict__ act, float* __restrict__ logp,
                                                float* __restrict__ value,
                                                float* __restrict__ logits,
                                                float* __restrict__ hid, unsigned char* smem,
                                                int e0) {
  typedef Shape<M, FP, H1, H2, AP, RT> Sh;
  typedef typename M::elem E;
  constexpr int ROWS = Sh::ROWS;
  E* xs = reinterpret_cast<E*>(smem);
  E* h2s = reinterpret_cast<E*>(smem);
  E* h1s = reinterpret_cast<E*>(smem + Sh::REGION_A);
  float* lg = reinterpret_cast<float*>(smem + Sh::REGION_A);
  const int tid = threadIdx.x;
  // stage x: obs [F][E] fp32 -> rows of the tile, rounded to the layer's input type
  for (int idx = tid; idx < ROWS * FP; idx += kThreads) {
    const int r = idx % ROWS, f = idx / ROWS;
    const int e = e0 + r;
    float v = 0.f;
    if (f < m.F && e < m.E) v = obs[(size_t)f * m.E + e];
    xs[r * Sh::SX + f] = M::from_f32(v);
  }
  __syncthreads();
  layer<M, FP, H1, RT, false, DBG>(xs, static_cast<const E*>(m.w1), m.b1, h1s, nullptr, 0,
                               HidOut{hid, m.E, e0});
  __syncthreads();
  layer<M, H1, H2, RT, false, DBG>(h1s, static_cast<const E*>(m.w2), m.b2, h2s, nullptr, 0,
                               HidOut{DBG ? hid + (size_t)H1 * m.E : nullptr, m.E, e0});
  __syncthreads();
  layer<M, H2, AP, RT, true>(h2s, static_cast<const E*>(m.w3), m.b3, nullptr, lg, Sh::SL);
  __syncthreads();
  sample_rows<AP, ROWS, kThreads>(lg, Sh::SL, m, e0, seed, step, act, logp, value, logits);
}

// ---- bf16 policy kernel: 16*RT environments per workgroup, NW waves ------------------------
// Every layer is computed transposed, out^T = W^T act^T: the weight tile is the MFMA A
// operand (16 output units x 32 inputs, 16 contiguous bytes per lane from the weights
// repacked in fragment order) and the activation tile the B operand (32 inputs x 16 environments, 16
// contiguous bytes per lane from the row-major [env][unit] LDS buffer). A lane's four
// accumulator values are then four consecutive output units of one environment, so the
// epilogue writes them to the next layer's buffer as one 8-byte store after two packed
// fp32->bf16 conversions. Each wave owns a disjoint set of output-unit tiles, so a workgroup
// reads every weight once (from L2); weight fragments of the next k-steps are loaded while
// the current step's MFMAs run.
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) { return pack_bf16_pair(lo, hi); }

// GELU(x) = x Phi(x) = max(x, 0) - |x| Phi(-|x|) (Phi(-t) = 1 - Phi(t) folds the positive half
// onto the negative one), with Phi(-t) = 2^q(t) and q a degree-5 polynomial fitted to
// log2 Phi(-t): a least-maximum fit of the GELU error t |2^q(t) - Phi(-t)| over 0 <= t <= 8
// (largest absolute GELU error 4.8e-7; evaluated in fp32, 6.6e-7). q's leading coefficient is
// negative, so 2^q falls to 0 for large t and the result saturates to max(x, 0). One
// transcendental per activation (exp2) and no reciprocal; |x| enters every step as a source
// modifier, and max(x, 0) is an integer max of x's bits with 0 (a negative float's bits are a
// negative integer), which needs no NaN canonicalisation.
__device__ __forceinline__ float gelu_fast(float x) {
  const float t = fabsf(x);
  float q = fmaf(-0.00047566284774802625f, t, 0.007099142298102379f);
  q = fmaf(q, t, -0.051859911531209946f);
  q = fmaf(q, t, -0.45996034145355225f);
  q = fmaf(q, t, -1.150801420211792f);
  q = fmaf(q, t, -1.0000358819961548f);
  const float relu = __int_as_float(max(__float_as_int(x), 0));
  return fmaf(-t, __builtin_amdgcn_exp2f(q), relu);
}

__device__ __forceinline__ u32x2 gelu_pack4(const f32x4 v) {
  u32x2 pk;
  pk.x = pack_bf16(gelu_fast(v[0]), gelu_fast(v[1]));
  pk.y = pack_bf16(gelu_fast(v[2]), gelu_fast(v[3]));
  return pk;
}

// diagnostic store of four packed bf16 activations (units unit0 .. unit0 + 3 of tile row `row`)
template <bool DBG>
__device__ __forceinline__ void hid_store4(const HidOut& ho, int unit0, int row, u32x2 v) {
  if constexpr (DBG) {
    const int e = ho.e0 + row;
    if (e < ho.E) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t w = (i < 2 ? v.x : v.y) >> (16 * (i & 1));
        ho.h[(size_t)(unit0 + i) * ho.E + e] = __uint_as_float(w << 16);
      }
    }
  }
}

// One output tile (16 units) of a layer for RTN consecutive environment tiles starting at rt0:
// acc[rt] = act[rows] W[:, tile] + bias, with a ring of D k-steps of weight fragments in flight.
// hook(ks) runs after each k-step's MFMAs: the caller puts independent VALU work there, which
// the SIMD issues while the matrix core is busy.
template <int K, int RTN, class Hook>
__device__ __forceinline__ void mma_tile(const uint16_t* __restrict__ act, int sa,
                                         const uint16_t* __restrict__ W,
                                         const float* __restrict__ bias, int tile, int rt0,
                                         f32x4 (&acc)[RTN], Hook&& hook) {
  constexpr int KS = K / 32, D = KS < 4 ? KS : 4, S = D + 1;
  const int lane = threadIdx.x & 63, r16 = lane & 15, kq = lane >> 4;
  const f32x4 bv = *reinterpret_cast<const f32x4*>(bias + tile * 16 + kq * 4);
  const uint16_t* wp = W + (size_t)tile * KS * 512 + lane * 8;  // fragment order
  const uint16_t* brow = act + (rt0 * 16 + r16) * sa + kq * 8;
  bf16x8 w[S];
#pragma unroll
  for (int s = 0; s < D; ++s) w[s] = *reinterpret_cast<const bf16x8*>(wp + s * 512);
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (ks + D < KS) w[(ks + D) % S] = *reinterpret_cast<const bf16x8*>(wp + (ks + D) * 512);
#pragma unroll
    for (int rt = 0; rt < RTN; ++rt) {
      const bf16x8 b = *reinterpret_cast<const bf16x8*>(brow + rt * 16 * sa + ks * 32);
      acc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[ks % S], b, ks == 0 ? bv : acc[rt],
                                                        0, 0, 0);
    }
    hook(ks);
  }
}

// One hidden layer, out = bf16(GELU(act W + b)), for the wave's output tiles wave, wave + NW,
// ...: the GELU of each tile is placed inside the next tile's k-loop (the last one after it);
// the compiler is free to schedule it (pinning it there was measured slower at the 128-VGPR
// budget). A lane's four accumulator values are four consecutive units of one environment,
// written as one 8-byte store. In place (out aliases act) the packed results wait in
// registers until every wave has finished reading act.
template <int K, int N, int RT, int NW, bool kInPlace, bool DBG>
__device__ __forceinline__ void hidden_layer(const uint16_t* __restrict__ act, int sa,
                                             const uint16_t* __restrict__ W,
                                             const float* __restrict__ bias, uint16_t* out,
                                             int so, HidOut ho) {
  constexpr int NT = N / 16, CTW = NT / NW, KS = K / 32;
  static_assert(NT % NW == 0, "hidden tiles divide evenly over the waves");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  f32x4 acc[2][RT];
  u32x2 pk[kInPlace ? CTW : 1][RT];
  auto finish = [&](int c, int rt) {
    const u32x2 v = gelu_pack4(acc[c & 1][rt]);
    hid_store4<DBG>(ho, (wave + NW * c) * 16 + kq * 4, rt * 16 + r16, v);
    if (kInPlace) pk[kInPlace ? c : 0][rt] = v;
    else *reinterpret_cast<u32x2*>(out + (rt * 16 + r16) * so + (wave + NW * c) * 16 + kq * 4) = v;
  };
#pragma unroll
  for (int c = 0; c < CTW; ++c) {
    mma_tile<K, RT>(act, sa, W, bias, wave + NW * c, 0, acc[c & 1], [&](int ks) {
      if (c > 0) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          if (rt * KS / RT == ks) finish(c - 1, rt);
      }
    });
  }
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) finish(CTW - 1, rt);
  if (kInPlace) {
    __syncthreads();  // every wave has finished reading act
#pragma unroll
    for (int c = 0; c < CTW; ++c)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        *reinterpret_cast<u32x2*>(out + (rt * 16 + r16) * so + (wave + NW * c) * 16 + kq * 4) =
            pk[kInPlace ? c : 0][rt];
  }
}

// TPW output tiles (16 units each, tiles tile0 + i * tstride) of a layer for RTN consecutive
// environment tiles from rt0 in one pass over k: every activation fragment read from LDS feeds
// TPW MFMAs (the LDS traffic of a layer falls by that factor against one tile per pass), and
// a ring of D k-steps of weight fragments of all TPW tiles is kept in flight. The bias is the
// accumulators' initial value.
template <int K, int TPW, int RTN>
__device__ __forceinline__ void mma_group(const uint16_t* __restrict__ act, int sa,
                                          const uint16_t* __restrict__ W,
                                          const float* __restrict__ bias, int tile0, int tstride,
                                          int rt0, f32x4 (&acc)[TPW][RTN]) {
  constexpr int KS = K / 32, D = KS < 2 ? KS : 2, S = D + 1;
  const int lane = threadIdx.x & 63, r16 = lane & 15, kq = lane >> 4;
  const uint16_t* brow = act + (rt0 * 16 + r16) * sa + kq * 8;
  const uint16_t* wp[TPW];
#pragma unroll
  for (int i = 0; i < TPW; ++i) {
    const int tile = tile0 + i * tstride;
    wp[i] = W + (size_t)tile * KS * 512 + lane * 8;  // fragment order
    const f32x4 bv = *reinterpret_cast<const f32x4*>(bias + tile * 16 + kq * 4);
#pragma unroll
    for (int rt = 0; rt < RTN; ++rt) acc[i][rt] = bv;
  }
  bf16x8 w[S][TPW];
#pragma unroll
  for (int s = 0; s < D; ++s)
#pragma unroll
    for (int i = 0; i < TPW; ++i) w[s][i] = *reinterpret_cast<const bf16x8*>(wp[i] + s * 512);
  // software pipeline: the activation fragments of k-step ks + 1 and the weight fragments of
  // ks + D are issued before the MFMAs of ks; scheduling barriers keep the compiler from
  // sinking those loads next to their first use, where every step would wait out the L2 and
  // LDS latency
  bf16x8 b[2][RTN];
#pragma unroll
  for (int rt = 0; rt < RTN; ++rt) b[0][rt] = *reinterpret_cast<const bf16x8*>(brow + rt * 16 * sa);
  // the wave's matrix phase at a raised issue priority, so that a SIMD shared with the other
  // workgroup's waves in their GELU epilogues keeps feeding its matrix core (C5 policy -0.9%)
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (ks + 1 < KS) {
#pragma unroll
      for (int rt = 0; rt < RTN; ++rt)
        b[(ks + 1) & 1][rt] = *reinterpret_cast<const bf16x8*>(brow + rt * 16 * sa + (ks + 1) * 32);
    }
    if (ks + D < KS) {
#pragma unroll
      for (int i = 0; i < TPW; ++i)
        w[(ks + D) % S][i] = *reinterpret_cast<const bf16x8*>(wp[i] + (ks + D) * 512);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int rt = 0; rt < RTN; ++rt)
#pragma unroll
      for (int i = 0; i < TPW; ++i)
        acc[i][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[ks % S][i], b[ks & 1][rt], acc[i][rt], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  __builtin_amdgcn_s_setprio(0);
}

// Hidden layer with TPW tiles per pass (see mma_group): the wave's CTW tiles wave, wave + NW,
// ... in CTW / TPW passes, each followed by its GELU epilogue; in place, the packed results
// wait in registers until every wave has finished reading act.
template <int K, int N, int RT, int NW, int TPW, bool kInPlace, bool DBG>
__device__ __forceinline__ void hidden_layer_g(const uint16_t* __restrict__ act, int sa,
                                               const uint16_t* __restrict__ W,
                                               const float* __restrict__ bias, uint16_t* out,
                                               int so, HidOut ho) {
  constexpr int NT = N / 16, CTW = NT / NW, NG = CTW / TPW;
  static_assert(NT % NW == 0 && CTW % TPW == 0, "tiles divide evenly over waves and passes");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  u32x2 pk[kInPlace ? CTW : 1][RT];
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    f32x4 acc[TPW][RT];
    mma_group<K, TPW, RT>(act, sa, W, bias, wave + NW * TPW * g, NW, 0, acc);
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      const int c = g * TPW + i;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const u32x2 v = gelu_pack4(acc[i][rt]);
        hid_store4<DBG>(ho, (wave + NW * c) * 16 + kq * 4, rt * 16 + r16, v);
        if (kInPlace) pk[kInPlace ? c : 0][rt] = v;
        else *reinterpret_cast<u32x2*>(out + (rt * 16 + r16) * so + (wave + NW * c) * 16 + kq * 4) = v;
      }
    }
  }
  if (kInPlace) {
    __syncthreads();  // every wave has finished reading act
#pragma unroll
    for (int c = 0; c < CTW; ++c)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        *reinterpret_cast<u32x2*>(out + (rt * 16 + r16) * so + (wave + NW * c) * 16 + kq * 4) =
            pk[kInPlace ? c : 0][rt];
  }
}

__host__ __device__ constexpr int pow2_floor(int v) { return v >= 8 ? 8 : v >= 4 ? 4 : v >= 2 ? 2 : 1; }

// Output layer (logits and value, fp32 into lg, which aliases act): NT tiles x G groups of
// environment tiles are spread over the waves so that narrow heads still keep most waves busy.
template <int K, int NO, int RT, int NW>
__device__ __forceinline__ void output_layer(const uint16_t* __restrict__ act, int sa,
                                             const uint16_t* __restrict__ W,
                                             const float* __restrict__ bias, float* lg, int sl) {
  constexpr int NT = NO / 16;
  constexpr int G = pow2_floor(RT < NW / NT ? RT : (NW / NT > 0 ? NW / NT : 1));
  constexpr int RTI = RT / G, ITEMS = NT * G, IPW = (ITEMS + NW - 1) / NW;
  static_assert(RT % G == 0, "environment-tile groups");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  f32x4 acc[IPW][RTI];
#pragma unroll
  for (int i = 0; i < IPW; ++i) {
    const int item = wave + NW * i;
    if (item < ITEMS) mma_tile<K, RTI>(act, sa, W, bias, item % NT, (item / NT) * RTI, acc[i],
                                      [](int) {});
  }
  __syncthreads();  // every wave has finished reading act
#pragma unroll
  for (int i = 0; i < IPW; ++i) {
    const int item = wave + NW * i;
    if (item < ITEMS) {
      const int t = item % NT, rt0 = (item / NT) * RTI;
#pragma unroll
      for (int rt = 0; rt < RTI; ++rt)
        *reinterpret_cast<f32x4*>(lg + ((rt0 + rt) * 16 + r16) * sl + t * 16 + kq * 4) = acc[i][rt];
    }
  }
}

template <int FP, int H1, int H2, int AP, int RT, int NW>
struct BigShape {
  static constexpr int ROWS = 16 * RT;
  static constexpr int SX = FP + 8, SH = (H1 > H2 ? H1 : H2) + 8, SL = AP + 4;
  static constexpr size_t X_BYTES = (size_t)ROWS * SX * 2;
  static constexpr size_t H_BYTES = (size_t)ROWS * SH * 2;
  static constexpr size_t L_BYTES = (size_t)ROWS * SL * 4;
  static constexpr size_t HREG = H_BYTES > L_BYTES ? H_BYTES : L_BYTES;
  static constexpr size_t U_BYTES = (size_t)ROWS * 4;   // the rows' ACTION uniforms
  static constexpr size_t LDS = X_BYTES + HREG + U_BYTES;
};

// One workgroup's share of the bf16 policy: environments e0 .. e0 + 16 RT - 1 (rows past E
// take zeros and write nothing), activations in smem (BigShape::LDS bytes of LDS). Called by
// all NW * 64 threads of the workgroup, which it synchronises. obs_bf: the observation's bf16
// pairs, read instead of obs when not NULL. AC: the action count compiled into the sampler
// (0: m.A at run time).
template <int FP, int H1, int H2, int AP, int RT, int NW, int TPW, bool DBG, int AC>
__device__ __forceinline__ void policy_tile_bf16(const MlpParams& m, const float* __restrict__ obs,
                                                 const uint32_t* __restrict__ obs_bf,
                                                 uint64_t seed, uint32_t step,
                                                 uint8_t* __restrict__ act,
                                                 float* __restrict__ logp,
                                                 float* __restrict__ value,
                                                 float* __restrict__ logits,
                                                 float* __restrict__ hid, unsigned char* smem,
                                                 int e0) {
  typedef BigShape<FP, H1, H2, AP, RT, NW> Sh;
  constexpr int ROWS = Sh::ROWS, NTHR = NW * 64;
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem);
  uint16_t* hs = reinterpret_cast<uint16_t*>(smem + Sh::X_BYTES);
  float* lg = reinterpret_cast<float*>(smem + Sh::X_BYTES);
  float* us = reinterpret_cast<float*>(smem + Sh::X_BYTES + Sh::HREG);
  const int tid = threadIdx.x;
  // the sampler's uniforms, one lane per row (the first ROWS lanes), read after the layers;
  // drawn while the observation loads are in flight
  auto draw_uniforms = [&]() {
    if (tid < ROWS) us[tid] = action_uniform(seed, (uint32_t)(e0 + tid < m.E ? e0 + tid : 0), step);
  };
  // stage x: obs [F][E] fp32 -> [env][feature] bf16, two features per 4-byte store. Every
  // load of a thread's share is issued before its first store (one round trip instead of
  // one per share), except in the two-tile variant, which is at its register limit there
  // (issuing them together cost it 1%, and saved 2-5% in the others).
  constexpr int NIT = (ROWS * (FP / 2) + NTHR - 1) / NTHR;
  constexpr int NPRE = TPW == 1 ? NIT : 1;
  if (obs_bf) {
    // the observation's bf16 pairs [F/2][E] (written by the simulator's tick): one 4-byte load
    // per feature pair and environment, stored as is
    uint32_t v[NIT];
#pragma unroll
    for (int i = 0; i < NIT; ++i) {
      const int idx = tid + i * NTHR;
      const int r = idx % ROWS, f = 2 * (idx / ROWS);
      const int e = e0 + r;
      v[i] = 0u;
      if (idx < ROWS * (FP / 2) && e < m.E && f < m.F) v[i] = obs_bf[(size_t)(f / 2) * m.E + e];
    }
    draw_uniforms();
#pragma unroll
    for (int i = 0; i < NIT; ++i) {
      const int idx = tid + i * NTHR;
      const int r = idx % ROWS, f = 2 * (idx / ROWS);
      if (idx < ROWS * (FP / 2)) *reinterpret_cast<uint32_t*>(xs + r * Sh::SX + f) = v[i];
    }
  } else
  for (int it0 = 0; it0 < NIT; it0 += NPRE) {
    float v0[NPRE], v1[NPRE];
#pragma unroll
    for (int i = 0; i < NPRE; ++i) {
      const int idx = tid + (it0 + i) * NTHR;
      const int r = idx % ROWS, f = 2 * (idx / ROWS);
      const int e = e0 + r;
      v0[i] = 0.f;
      v1[i] = 0.f;
      if (it0 + i < NIT && idx < ROWS * (FP / 2) && e < m.E) {
        if (f < m.F) v0[i] = obs[(size_t)f * m.E + e];
        if (f + 1 < m.F) v1[i] = obs[(size_t)(f + 1) * m.E + e];
      }
    }
#pragma unroll
    for (int i = 0; i < NPRE; ++i) {
      const int idx = tid + (it0 + i) * NTHR;
      const int r = idx % ROWS, f = 2 * (idx / ROWS);
      if (it0 + i < NIT && idx < ROWS * (FP / 2))
        *reinterpret_cast<uint32_t*>(xs + r * Sh::SX + f) = pack_bf16(v0[i], v1[i]);
    }
  }
  if (!obs_bf) draw_uniforms();
  __syncthreads();
  const HidOut h1o{hid, m.E, e0}, h2o{DBG ? hid + (size_t)H1 * m.E : nullptr, m.E, e0};
  if constexpr (TPW == 1) {
    hidden_layer<FP, H1, RT, NW, false, DBG>(xs, Sh::SX, static_cast<const uint16_t*>(m.w1), m.b1,
                                             hs, Sh::SH, h1o);
    __syncthreads();
    hidden_layer<H1, H2, RT, NW, true, DBG>(hs, Sh::SH, static_cast<const uint16_t*>(m.w2), m.b2,
                                            hs, Sh::SH, h2o);
  } else {
    hidden_layer_g<FP, H1, RT, NW, TPW, false, DBG>(xs, Sh::SX, static_cast<const uint16_t*>(m.w1),
                                                    m.b1, hs, Sh::SH, h1o);
    __syncthreads();
    hidden_layer_g<H1, H2, RT, NW, TPW, true, DBG>(hs, Sh::SH, static_cast<const uint16_t*>(m.w2),
                                                   m.b2, hs, Sh::SH, h2o);
  }
  __syncthreads();
  output_layer<H2, AP, RT, NW>(hs, Sh::SH, static_cast<const uint16_t*>(m.w3), m.b3, lg, Sh::SL);
  __syncthreads();
  sample_rows<AP, ROWS, NTHR, AC>(lg, Sh::SL, m, e0, seed, step, act, logp, value, logits, us);
}

}  // namespace
}  // namespace bsim
