// mlp_kernels.hip -- policy MLP (paper Sec. 4.2) on MFMA, fused with action sampling.
//
// obs [F][E] -> h1 = GELU(x W1 + b1) -> h2 = GELU(h1 W2 + b2) -> out = h2 W3 + b3, where
// out[0..A) are the logits of the categorical action distribution and out[A] (when the
// value head is on) is V(s). The epilogue of the last layer samples the action by inverse CDF
// of the fp32 softmax with the ACTION uniform of (env, step) and writes action,
// log-probability and value.
//
// Two kernels. policy_k (fp32 policies, v_mfma_f32_16x16x4_f32): one workgroup of 4 waves owns
// 16 RT environments whose activations live in LDS (RT = 1 for small batches, whose launch
// lasts as long as one workgroup's chain of layers; 4 otherwise); each wave produces a quarter
// of the output columns of every layer, loading all of its weight fragments of a layer from
// the repacked weights in L2 before the layer's first MFMA.
// policy_bf16_k (bf16 policies): every layer's input rounded to bf16 (RNE), bf16 weights,
// fp32 accumulation (v_mfma_f32_16x16x32_bf16), bias and GELU in fp32; its layout and
// scheduling are described above the kernel.
#include <type_traits>

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
// shuffles within the group.
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
  static_assert(NTHR % G == 0, "sampler groups");
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
#pragma unroll
    for (int off = 1; off < G; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, G));
    float pe[KMAX];
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      pe[i] = (i < chunk && lo + i < A) ? __expf(l[lo + i] - mx) : 0.f;
      ps += pe[i];
    }
    float incl = ps;
#pragma unroll
    for (int off = 1; off < G; off <<= 1) {
      const float t = __shfl_up(incl, off, G);
      if (part >= off) incl += t;
    }
    const float S = __shfl(incl, G - 1, G);
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
#pragma unroll
    for (int off = 1; off < G; off <<= 1) found = min(found, __shfl_xor(found, off, G));
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

template <class M, int FP, int H1, int H2, int AP, int RT, bool DBG>
__global__ __launch_bounds__(kThreads) void policy_k(MlpParams m, const float* __restrict__ obs,
                                                     const uint64_t* __restrict__ seedp, uint32_t step,
                                                     uint8_t* __restrict__ act,
                                                     float* __restrict__ logp,
                                                     float* __restrict__ value,
                                                     float* __restrict__ logits,
                                                     float* __restrict__ hid) {
  const uint64_t seed = *seedp;   // the episode seed
  typedef Shape<M, FP, H1, H2, AP, RT> Sh;
  typedef typename M::elem E;
  constexpr int ROWS = Sh::ROWS;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  E* xs = reinterpret_cast<E*>(smem);
  E* h2s = reinterpret_cast<E*>(smem);
  E* h1s = reinterpret_cast<E*>(smem + Sh::REGION_A);
  float* lg = reinterpret_cast<float*>(smem + Sh::REGION_A);
  const int e0 = blockIdx.x * ROWS;
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

// packed bf16 weights in MFMA fragment order: for output tile t (16 units) and k-step ks (32
// inputs), the 64 lanes' 16-byte A fragments lie back to back, lane = kq*16 + r16 holding
// W[ks*32 + kq*8 + j][t*16 + r16], j = 0..7 (zero padded). A wave's load of one fragment is
// one contiguous kilobyte, and consecutive k-steps of a tile are consecutive kilobytes.
__global__ void repack_frag_k(const unsigned char* __restrict__ src, size_t woff, size_t boff,
                              int K, int N, int KS, int NTp, uint16_t* __restrict__ w,
                              float* __restrict__ b) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t total = (size_t)NTp * KS * 512;
  if (idx < total) {
    const int t = (int)(idx / ((size_t)KS * 512));
    const int rem = (int)(idx % ((size_t)KS * 512));
    const int ks = rem / 512, l = (rem % 512) / 8, j = rem % 8;
    const int n = t * 16 + (l & 15), k = ks * 32 + (l >> 4) * 8 + j;
    uint16_t v = 0;
    if (n < N && k < K) v = reinterpret_cast<const uint16_t*>(src + woff)[(size_t)k * N + n];
    w[idx] = v;
  }
  if (idx < (size_t)NTp * 16) {
    const int n = (int)idx;
    b[n] = n < N ? reinterpret_cast<const float*>(src + boff)[n] : 0.f;
  }
}

// packed fp32 weights: W^T [Npad][Kpad], zero padded; bias fp32 [Npad]
template <typename T>
__global__ void repack_k(const unsigned char* __restrict__ src, size_t woff, size_t boff, int K,
                         int N, int Kp, int Np, T* __restrict__ w, float* __restrict__ b) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t total = (size_t)Np * Kp;
  if (idx < total) {
    const int n = (int)(idx / Kp), k = (int)(idx % Kp);
    T v = T(0);
    if (n < N && k < K) v = reinterpret_cast<const T*>(src + woff)[(size_t)k * N + n];
    w[idx] = v;
  }
  if (idx < (size_t)Np) {
    const int n = (int)idx;
    b[n] = n < N ? reinterpret_cast<const float*>(src + boff)[n] : 0.f;
  }
}

// Xavier-uniform: element i of layer l takes u from the WEIGHTS block at counter
// (i, 0xFFFFFFFE, WEIGHTS<<24 | l, 0); w = (2u - 1) * lim in fp64, then fp32 (then bf16).
__global__ void init_w_k(uint64_t seed, int layer, size_t n, double lim, int bf16,
                         unsigned char* __restrict__ dst) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const u32x4 w = draw(seed, (uint32_t)i, 0xFFFFFFFEu, P_WEIGHTS, (uint32_t)layer, 0);
  const double u = unit(w.x, w.y);
  const float f = (float)((2.0 * u - 1.0) * lim);
  if (bf16) reinterpret_cast<uint16_t*>(dst)[i] = bf16_bits(f);
  else reinterpret_cast<float*>(dst)[i] = f;
}

__global__ void zero_f32_k(float* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.f;
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

// AC: the action count compiled into the sampler (0: m.A at run time)
template <int FP, int H1, int H2, int AP, int RT, int NW, int MINB, int TPW, bool DBG, int AC>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(NW * MINB / 4 > 0 ? NW * MINB / 4 : 1))) void policy_bf16_k(MlpParams m, const float* __restrict__ obs,
                                                               const uint32_t* __restrict__ obs_bf,
                                                               const uint64_t* __restrict__ seedp, uint32_t step,
                                                               uint8_t* __restrict__ act,
                                                               float* __restrict__ logp,
                                                               float* __restrict__ value,
                                                               float* __restrict__ logits,
                                                               float* __restrict__ hid) {
  const uint64_t seed = *seedp;   // the episode seed
  typedef BigShape<FP, H1, H2, AP, RT, NW> Sh;
  constexpr int ROWS = Sh::ROWS, NTHR = NW * 64;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem);
  uint16_t* hs = reinterpret_cast<uint16_t*>(smem + Sh::X_BYTES);
  float* lg = reinterpret_cast<float*>(smem + Sh::X_BYTES);
  float* us = reinterpret_cast<float*>(smem + Sh::X_BYTES + Sh::HREG);
  const int e0 = blockIdx.x * ROWS;
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

template <bool DBG, int FP, int H1, int H2, int AP, int RT, int NW, int MINB, int TPW, int AC>
hipError_t run_policy_bf16(const MlpParams& m, const float* obs, const uint32_t* obs_bf,
                           const uint64_t* seed, uint32_t step,
                           uint8_t* act, float* logp, float* value, float* logits, float* hid,
                           hipStream_t st) {
  typedef BigShape<FP, H1, H2, AP, RT, NW> Sh;
  static_assert(Sh::LDS <= 160 * 1024, "LDS budget");
  if (AC > 0 && m.A != AC) return hipErrorInvalidValue;
  auto kern = policy_bf16_k<FP, H1, H2, AP, RT, NW, MINB, TPW, DBG, AC>;
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)Sh::LDS);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const dim3 grid((m.E + Sh::ROWS - 1) / Sh::ROWS), block(NW * 64);
  hipLaunchKernelGGL(kern, grid, block, Sh::LDS, st, m, obs, obs_bf, seed, step, act, logp, value,
                     logits, hid);
  return hipGetLastError();
}

template <bool DBG, class M, int FP, int H1, int H2, int AP, int RT>
hipError_t run_policy(const MlpParams& m, const float* obs, const uint64_t* seed, uint32_t step,
                      uint8_t* act, float* logp, float* value, float* logits, float* hid,
                      hipStream_t st) {
  typedef Shape<M, FP, H1, H2, AP, RT> Sh;
  auto kern = policy_k<M, FP, H1, H2, AP, RT, DBG>;
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)Sh::LDS);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const dim3 grid((m.E + Sh::ROWS - 1) / Sh::ROWS), block(kThreads);
  hipLaunchKernelGGL(kern, grid, block, Sh::LDS, st, m, obs, seed, step, act, logp, value, logits,
                     hid);
  return hipGetLastError();
}

// fp32 policy row tiles per workgroup (16 environments each): small batches take small tiles,
// so that a workgroup's serial chain of layers is short
constexpr int kF32SmallE = 4096, kF32SmallRT = 1, kF32RT = 4;

struct ShapeKey { int bf16, FP, H1, H2, AP; };
constexpr ShapeKey kShapes[] = {
    {0, 8, 64, 64, 16},      // 8-64-64-6 fp32
    {1, 32, 128, 128, 16},   // 12-128-128-6 bf16
    {1, 32, 256, 256, 32},   // 32-256-256-24(+1) bf16
    {1, 64, 256, 256, 64},   // 64-256-256-48(+1) bf16
    {1, 96, 512, 512, 112},  // 96-512-512-96(+1) bf16
};

}  // namespace

static int pad_up(int x, int m) { return (x + m - 1) / m * m; }

bool policy_shape_supported(const MlpParams& m) {
  for (const ShapeKey& s : kShapes)
    if (s.bf16 == m.bf16 && s.FP == m.FP && s.H1 == m.H1 && s.H2 == m.H2 && s.AP == m.AP)
      return true;
  return false;
}

// One bf16 shape: the configurations' own action count AC0 for that width (6K of their K)
// compiled into the sampler, any other with run-time bounds (the diagnostic instantiation
// always takes the run-time bounds; AC0 = 0 compiles none). run(big, ac) launches the variant.
template <bool DBG, int AC0, class Run>
static hipError_t run_shape_bf16(const MlpParams& m, bool big, Run&& run) {
  typedef std::integral_constant<bool, true> T;
  typedef std::integral_constant<bool, false> F;
  typedef std::integral_constant<int, 0> A0;
  typedef std::integral_constant<int, DBG ? 0 : AC0> AC;
  if (!DBG && AC0 > 0 && m.A == AC0) return big ? run(T{}, AC{}) : run(F{}, AC{});
  return big ? run(T{}, A0{}) : run(F{}, A0{});
}

template <bool DBG>
static hipError_t launch_policy_t(const MlpParams& m, const float* obs, const uint32_t* obs_bf,
                                  const uint64_t* seed,
                                  uint32_t step, uint8_t* act, float* logp, float* value,
                                  float* logits, float* hid, hipStream_t st) {
  if (!m.bf16 && m.FP == 8 && m.H1 == 64 && m.H2 == 64 && m.AP == 16)
    return m.E <= kF32SmallE
               ? run_policy<DBG, F32Mode, 8, 64, 64, 16, kF32SmallRT>(m, obs, seed, step, act, logp, value, logits, hid, st)
               : run_policy<DBG, F32Mode, 8, 64, 64, 16, kF32RT>(m, obs, seed, step, act, logp, value, logits, hid, st);
  // bf16 shapes: 64-row tiles with 4 waves, two workgroups per CU, when there are enough
  // rows to fill the chip; 32-row tiles otherwise
  const bool big = m.E >= 64 * 512;
#define BSIM_BF16_ARGS (m, obs, obs_bf, seed, step, act, logp, value, logits, hid, st)
  if (m.bf16 && m.FP == 32 && m.H1 == 128 && m.H2 == 128 && m.AP == 16)
    return run_shape_bf16<DBG, 0>(m, big, [&](auto big_v, auto ac_v) {   // 6 measured slower
      constexpr bool B = decltype(big_v)::value;
      constexpr int C = decltype(ac_v)::value;
      return B ? run_policy_bf16<DBG, 32, 128, 128, 16, 4, 8, 2, 1, C> BSIM_BF16_ARGS
               : run_policy_bf16<DBG, 32, 128, 128, 16, 2, 4, 2, 1, C> BSIM_BF16_ARGS;
    });
  if (m.bf16 && m.FP == 32 && m.H1 == 256 && m.H2 == 256 && m.AP == 32)
    return run_shape_bf16<DBG, 24>(m, big, [&](auto big_v, auto ac_v) {
      constexpr bool B = decltype(big_v)::value;
      constexpr int C = decltype(ac_v)::value;
      return B ? run_policy_bf16<DBG, 32, 256, 256, 32, 4, 8, 2, 1, C> BSIM_BF16_ARGS
               : run_policy_bf16<DBG, 32, 256, 256, 32, 2, 4, 2, 1, C> BSIM_BF16_ARGS;
    });
  if (m.bf16 && m.FP == 64 && m.H1 == 256 && m.H2 == 256 && m.AP == 64)
    return run_shape_bf16<DBG, 48>(m, big, [&](auto big_v, auto ac_v) {
      constexpr bool B = decltype(big_v)::value;
      constexpr int C = decltype(ac_v)::value;
      return B ? run_policy_bf16<DBG, 64, 256, 256, 64, 4, 8, 2, 1, C> BSIM_BF16_ARGS
               : run_policy_bf16<DBG, 64, 256, 256, 64, 2, 4, 2, 1, C> BSIM_BF16_ARGS;
    });
  if (m.bf16 && m.FP == 96 && m.H1 == 512 && m.H2 == 512 && m.AP == 112)
    return run_shape_bf16<DBG, 96>(m, big, [&](auto big_v, auto ac_v) {
      constexpr bool B = decltype(big_v)::value;
      constexpr int C = decltype(ac_v)::value;
      return B ? run_policy_bf16<DBG, 96, 512, 512, 112, 4, 8, 2, 2, C> BSIM_BF16_ARGS
               : run_policy_bf16<DBG, 96, 512, 512, 112, 2, 4, 2, 1, C> BSIM_BF16_ARGS;
    });
#undef BSIM_BF16_ARGS
  return hipErrorInvalidValue;
}

hipError_t launch_policy(const MlpParams& m, const float* obs, const uint32_t* obs_bf,
                         const uint64_t* seed, uint32_t step, uint8_t* act, float* logp,
                         float* value, float* logits, float* hidden, hipStream_t st) {
  if (obs_bf && !m.bf16) return hipErrorInvalidValue;
  if (hidden)
    return launch_policy_t<true>(m, obs, obs_bf, seed, step, act, logp, value, logits, hidden, st);
  return launch_policy_t<false>(m, obs, obs_bf, seed, step, act, logp, value, logits, nullptr, st);
}

hipError_t launch_repack(const MlpParams& m, const void* d_weights, const size_t off[6],
                         void* w1, float* b1, void* w2, float* b2, void* w3, float* b3,
                         hipStream_t st) {
  const unsigned char* src = static_cast<const unsigned char*>(d_weights);
  const int Ks[3] = {m.F, m.H1, m.H2}, Ns[3] = {m.H1, m.H2, m.Ap};
  const int Kp[3] = {m.FP, m.H1, m.H2}, Np[3] = {m.H1, m.H2, m.AP};
  void* ws[3] = {w1, w2, w3};
  float* bs[3] = {b1, b2, b3};
  for (int l = 0; l < 3; ++l) {
    const size_t total = (size_t)Np[l] * Kp[l];
    const dim3 grid((unsigned)((total + 255) / 256));
    if (m.bf16)
      hipLaunchKernelGGL(repack_frag_k, grid, dim3(256), 0, st, src, off[2 * l], off[2 * l + 1],
                         Ks[l], Ns[l], Kp[l] / 32, Np[l] / 16, static_cast<uint16_t*>(ws[l]), bs[l]);
    else
      hipLaunchKernelGGL(repack_k<float>, grid, dim3(256), 0, st, src, off[2 * l], off[2 * l + 1],
                         Ks[l], Ns[l], Kp[l], Np[l], static_cast<float*>(ws[l]), bs[l]);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_init_weights(int F, int H1, int H2, int Ap, int bf16, uint64_t seed,
                               void* d_weights, const size_t off[6], hipStream_t st) {
  unsigned char* dst = static_cast<unsigned char*>(d_weights);
  const int dims[4] = {F, H1, H2, Ap};
  for (int l = 0; l < 3; ++l) {
    const size_t n = (size_t)dims[l] * dims[l + 1];
    const double lim = sqrt(6.0 / (double)(dims[l] + dims[l + 1]));
    hipLaunchKernelGGL(init_w_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, seed, l, n,
                       lim, bf16, dst + off[2 * l]);
    hipLaunchKernelGGL(zero_f32_k, dim3((dims[l + 1] + 255) / 256), dim3(256), 0, st,
                       reinterpret_cast<float*>(dst + off[2 * l + 1]), dims[l + 1]);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_init_attn(uint64_t seed, void* d_weights, const size_t off[14], const int fin[7],
                            const int fout[7], hipStream_t st) {
  unsigned char* dst = static_cast<unsigned char*>(d_weights);
  for (int l = 0; l < 7; ++l) {
    const size_t n = (size_t)fin[l] * fout[l];
    const double lim = sqrt(6.0 / (double)(fin[l] + fout[l]));
    hipLaunchKernelGGL(init_w_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, seed, l, n,
                       lim, 0, dst + off[2 * l]);
    hipLaunchKernelGGL(zero_f32_k, dim3((fout[l] + 255) / 256), dim3(256), 0, st,
                       reinterpret_cast<float*>(dst + off[2 * l + 1]), fout[l]);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace bsim
