// ppo_kernels.hip -- one policy-gradient minibatch of the MLP policy (paper Sec. 4.3): gather,
// forward, loss (PPO clipped surrogate, or REINFORCE with a learned baseline) + value +
// entropy, and its gradient with respect to every policy weight.
//
// M samples (t, env) are drawn with replacement: sample m takes u from the MINIBATCH block at
// counter (m, 0xFFFFFFFD, MINIBATCH<<24, 0) and index floor(u * T * E). The forward repeats
// the rollout policy's rounding points (every layer input rounded to bf16 in bf16 mode) with
// fp32 sums and exact GELU; gradients pass through the bf16 roundings as the identity. Loss
//   L = -mean(min(rho A, clip(rho, 1-eps, 1+eps) A)) + c_v mean((V - R)^2) - c_h mean(H),
//   rho = exp(logp_new(a) - logp_old), H the entropy of the action distribution; REINFORCE
//   replaces the first term by -mean(A log pi(a|s)) with A held constant.
//
// The eight dense products run in one MFMA GEMM template (mb_gemm_k) with the elementwise
// steps fused into its epilogues:
//   forward    Z^T = W^T X^T per layer; epilogue: + bias, GELU, bf16 rounding, GELU'(z) kept,
//              the activations stored sample-major (next layer's operand) and unit-major
//              (weight-gradient operand)
//   loss       one wavefront per sample on the outputs: dL/dout
//   backward   dZ_l^T = W_{l+1} dZ_{l+1}^T, epilogue: times GELU'(z_l)
//   weights    G_l = A_{l-1}^T dZ_l, a reduction over the samples split into chunks whose
//              partial products are summed in a fixed order, so repeated calls give identical
//              gradients; bias gradients are the samples' column sums, also in a fixed order
// bf16 mode: activations and weights are bf16 values, so their products are exact in fp32;
// the fp32 gradient operand dZ is carried as two bf16 terms hi + lo (hi = bf16(dZ),
// lo = bf16(dZ - hi), 2^-17 relative) and every backward product takes two MFMAs,
// v_mfma_f32_16x16x32_bf16. fp32 mode (fp32 policies): fp32 operands, v_mfma_f32_16x16x4_f32.
#include <mutex>

#include "devmath.hpp"
#include "params.hpp"

// Fixed device scratch of the minibatch gradient for callers that cannot allocate
// (ppo_minibatch_grad_noalloc): one copy per GPU, held until the process ends. Host code must
// use the per-device address from hipGetSymbolAddress (static_scratch below), never this
// name, which in host code is only a stand-in for the device symbol.
static __device__ __align__(256) unsigned char scratch[bsim::kStaticScratchBytes];

namespace bsim {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kThr = 256;   // 4 waves
constexpr int kTile = 64;   // output tile edge of a workgroup; every dimension is padded to it

__device__ __forceinline__ float bf16_round(float f) { return bf16_to_f32(bf16_bits(f)); }
__device__ __forceinline__ float gelu_exact(float z) {
  return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));
}
__device__ __forceinline__ float gelu_grad(float z) {
  return 0.5f * (1.0f + erff(z * 0.70710678118654752f)) + z * expf(-0.5f * z * z) * 0.39894228040143268f;
}

// Operand modes. Both MFMA shapes take, per lane l, the row (A) or column (B) l % 16 and a run
// of consecutive k (8 bf16 from k = 8 (l / 16), or one fp32 at k = l / 16): every operand
// array is stored k-contiguous, [row][k]. Their 16 x 16 results share one layout: lane l holds
// column l % 16, rows 4 (l / 16) .. + 3.
struct Bf16Mode {
  typedef uint16_t T;
  typedef bf16x8 frag;
  static constexpr int KS = 32, SPLIT = 2;
  __device__ static int koff(int lane) { return (lane >> 4) * 8; }
  __device__ static frag load(const T* p) { return *reinterpret_cast<const bf16x8*>(p); }
  __device__ static f32x4 mfma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static T act(float v) { return bf16_bits(v); }     // activation (already rounded)
  __device__ static float actf(float v) { return bf16_round(v); }
  __device__ static void split(float v, T& hi, T& lo) {
    hi = bf16_bits(v);
    lo = bf16_bits(v - bf16_to_f32(hi));
  }
  __device__ static float value(T v) { return bf16_to_f32(v); }
};

struct F32Mode {
  typedef float T;
  typedef float frag;
  static constexpr int KS = 4, SPLIT = 1;
  __device__ static int koff(int lane) { return lane >> 4; }
  __device__ static frag load(const T* p) { return *p; }
  __device__ static f32x4 mfma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  __device__ static T act(float v) { return v; }
  __device__ static float actf(float v) { return v; }
  __device__ static void split(float v, T& hi, T& lo) { hi = v; lo = 0.f; }
  __device__ static float value(T v) { return v; }
};

// C [R][N] = sum_k A[r][k] (B0[n][k] + B1[n][k]) for one kTile x kTile output tile per
// workgroup: wave w owns rows 32 (w & 1) .. + 31 and columns 32 (w >> 1) .. + 31 as 2 x 2 MFMA
// tiles. Operands are zero padded to whole tiles in every dimension, so loads need no bounds
// checks.
template <class Md, bool TWO>
__device__ __forceinline__ void gemm_tile(const typename Md::T* __restrict__ A, int lda,
                                          const typename Md::T* __restrict__ B0,
                                          const typename Md::T* __restrict__ B1, int ldb,
                                          int R0, int C0, int k0, int k1, f32x4 (&acc)[2][2]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = R0 + 32 * (wave & 1), c0 = C0 + 32 * (wave >> 1);
  const int lr = lane & 15, ko = Md::koff(lane);
  const typename Md::T* a0 = A + (size_t)(r0 + lr) * lda + ko;
  const typename Md::T* a1 = a0 + (size_t)16 * lda;
  const size_t bo0 = (size_t)(c0 + lr) * ldb + ko, bo1 = bo0 + (size_t)16 * ldb;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (k0 >= k1) return;
  // operands of step k + KS are loaded before the MFMAs of step k
  typedef typename Md::frag Fr;
  Fr fa0 = Md::load(a0 + k0), fa1 = Md::load(a1 + k0);
  Fr fb0 = Md::load(B0 + bo0 + k0), fb1 = Md::load(B0 + bo1 + k0);
  Fr gb0 = fb0, gb1 = fb1;
  if constexpr (TWO) {
    gb0 = Md::load(B1 + bo0 + k0);
    gb1 = Md::load(B1 + bo1 + k0);
  }
  for (int k = k0; k < k1; k += Md::KS) {
    const int kn = k + Md::KS < k1 ? k + Md::KS : k;
    const Fr na0 = Md::load(a0 + kn), na1 = Md::load(a1 + kn);
    const Fr nb0 = Md::load(B0 + bo0 + kn), nb1 = Md::load(B0 + bo1 + kn);
    Fr ng0 = nb0, ng1 = nb1;
    if constexpr (TWO) {
      ng0 = Md::load(B1 + bo0 + kn);
      ng1 = Md::load(B1 + bo1 + kn);
    }
    acc[0][0] = Md::mfma(fa0, fb0, acc[0][0]);
    acc[0][1] = Md::mfma(fa0, fb1, acc[0][1]);
    acc[1][0] = Md::mfma(fa1, fb0, acc[1][0]);
    acc[1][1] = Md::mfma(fa1, fb1, acc[1][1]);
    if constexpr (TWO) {
      acc[0][0] = Md::mfma(fa0, gb0, acc[0][0]);
      acc[0][1] = Md::mfma(fa0, gb1, acc[0][1]);
      acc[1][0] = Md::mfma(fa1, gb0, acc[1][0]);
      acc[1][1] = Md::mfma(fa1, gb1, acc[1][1]);
    }
    fa0 = na0; fa1 = na1; fb0 = nb0; fb1 = nb1; gb0 = ng0; gb1 = ng1;
  }
}

// A lane's 16 accumulator values into the workgroup's tile buffer [row][col] (row stride
// kTile + 1: conflict-free column and row walks in the epilogues).
typedef float Tile[kTile][kTile + 1];
__device__ __forceinline__ void stage(const f32x4 (&acc)[2][2], Tile& tile) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        tile[32 * (wave & 1) + 16 * i + 4 * (lane >> 4) + q][32 * (wave >> 1) + 16 * j + (lane & 15)] =
            acc[i][j][q];
}

struct GemmArgs {
  const void* A;
  const void* B0;
  const void* B1;   // second term of the B operand (bf16 mode's lo part) or NULL
  int lda, ldb;     // row strides in elements
  int K;            // padded
};

// One product C = A B^T over the whole k range, tile (blockIdx.y, blockIdx.x); the tile is
// staged in LDS and the epilogue writes it (rows = output units, columns = samples).
template <class Md, bool TWO, class Epi>
__global__ __launch_bounds__(kThr) void mb_gemm_k(GemmArgs g, Epi epi) {
  __shared__ Tile tile;
  f32x4 acc[2][2];
  gemm_tile<Md, TWO>(static_cast<const typename Md::T*>(g.A), g.lda,
                     static_cast<const typename Md::T*>(g.B0),
                     static_cast<const typename Md::T*>(g.B1), g.ldb, blockIdx.y * kTile,
                     blockIdx.x * kTile, 0, g.K, acc);
  stage(acc, tile);
  __syncthreads();
  epi.store(tile, blockIdx.y * kTile, blockIdx.x * kTile);
}

// ---- epilogues: tile rows = output units (from R0), columns = samples (from C0) ------------------
// Thread t walks the tile twice: unit t % 64 of samples t / 64 + 4 k (each wavefront writes a
// 64-unit run of one sample: sample-major rows), then sample t % 64 of units t / 64 + 4 k
// (a 64-sample run of one unit: unit-major rows).

// Hidden layer forward: z = acc + b, h = GELU(z) (rounded to bf16 in bf16 mode) stored
// sample-major H [Mp][N] and unit-major Ht [N][Mp], GELU'(z) into D [Mp][N]. Padded samples
// (m >= M) store zero activations.
template <class Md>
struct EpiHidden {
  typedef typename Md::T T;
  const float* bias;
  T* H;
  T* Ht;
  float* D;
  int N, Mp, M;
  __device__ void store(Tile& tile, int R0, int C0) const {
    const int t = threadIdx.x, u = t & 63;
    const float b = bias[R0 + u];
#pragma unroll 4
    for (int k = 0; k < kTile / 4; ++k) {
      const int ml = (t >> 6) + 4 * k, m = C0 + ml;
      const float z = tile[u][ml] + b;
      const float phi = 0.5f * (1.0f + erff(z * 0.70710678118654752f));
      const float h = m < M ? Md::actf(z * phi) : 0.f;
      const size_t o = (size_t)m * N + R0 + u;
      H[o] = Md::act(h);
      D[o] = phi + z * expf(-0.5f * z * z) * 0.39894228040143268f;
      tile[u][ml] = h;
    }
    __syncthreads();
    const int ml = t & 63;
#pragma unroll 4
    for (int k = 0; k < kTile / 4; ++k) {
      const int uu = (t >> 6) + 4 * k;
      Ht[(size_t)(R0 + uu) * Mp + C0 + ml] = Md::act(tile[uu][ml]);
    }
  }
};

// Output layer forward: out [Mp][Ap64] = acc + b3 for the A' real outputs, 0 in the padding.
struct EpiOut {
  const float* bias;
  float* out;
  int Ap, Ap64;
  __device__ void store(Tile& tile, int R0, int C0) const {
    const int t = threadIdx.x, a = R0 + (t & 63);
    const float b = a < Ap ? bias[a] : 0.f;
#pragma unroll 4
    for (int k = 0; k < kTile / 4; ++k) {
      const int ml = (t >> 6) + 4 * k;
      out[(size_t)(C0 + ml) * Ap64 + a] = a < Ap ? tile[t & 63][ml] + b : 0.f;
    }
  }
};

// Hidden layer backward: dz = acc * GELU'(z) as hi + lo terms, sample-major into G_hi/lo
// [Mp][N] when G_hi != NULL, and unit-major into Gt_hi/lo [N][Mp].
template <class Md>
struct EpiBack {
  typedef typename Md::T T;
  const float* D;
  T *G_hi, *G_lo, *Gt_hi, *Gt_lo;
  int N, Mp, M;
  __device__ void store(Tile& tile, int R0, int C0) const {
    const int t = threadIdx.x, u = t & 63;
#pragma unroll 4
    for (int k = 0; k < kTile / 4; ++k) {
      const int ml = (t >> 6) + 4 * k, m = C0 + ml;
      const size_t o = (size_t)m * N + R0 + u;
      const float v = m < M ? tile[u][ml] * D[o] : 0.f;
      if (G_hi) {
        T hi, lo;
        Md::split(v, hi, lo);
        G_hi[o] = hi;
        if (Md::SPLIT == 2) G_lo[o] = lo;
      }
      tile[u][ml] = v;
    }
    __syncthreads();
    const int ml = t & 63;
#pragma unroll 4
    for (int k = 0; k < kTile / 4; ++k) {
      const int uu = (t >> 6) + 4 * k;
      const size_t o = (size_t)(R0 + uu) * Mp + C0 + ml;
      T hi, lo;
      Md::split(tile[uu][ml], hi, lo);
      Gt_hi[o] = hi;
      if (Md::SPLIT == 2) Gt_lo[o] = lo;
    }
  }
};

// The three weight-gradient products in one launch: layer l's tiles (R64 / 64 x N64 / 64) times
// S sample chunks, each writing its partial product P_l [z][R64][N64] (row = input unit,
// column = output unit).
template <class Md>
struct WgDesc {
  const typename Md::T *A, *B0, *B1;   // unit-major [R64][Mp], [N64][Mp], [N64][Mp]
  float* P;
  int R64, N64, S, chunk, first;       // first block of this layer
};

template <class Md>
__global__ __launch_bounds__(kThr) void mb_wgrad_k(WgDesc<Md> d0, WgDesc<Md> d1, WgDesc<Md> d2,
                                                   int Mp) {
  const int b = blockIdx.x;
  const WgDesc<Md>& d = b >= d2.first ? d2 : (b >= d1.first ? d1 : d0);
  const int l = b - d.first, tn = d.N64 / kTile;
  const int z = l % d.S, tx = (l / d.S) % tn, ty = l / (d.S * tn);
  f32x4 acc[2][2];
  const int k0 = z * d.chunk, k1 = min(k0 + d.chunk, Mp);
  gemm_tile<Md, Md::SPLIT == 2>(d.A, Mp, d.B0, d.B1, Mp, ty * kTile, tx * kTile, k0, k1, acc);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float* p = d.P + (size_t)z * d.R64 * d.N64;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = ty * kTile + 32 * (wave & 1) + 16 * i + 4 * (lane >> 4) + q;
        const int c = tx * kTile + 32 * (wave >> 1) + 16 * j + (lane & 15);
        p[(size_t)r * d.N64 + c] = acc[i][j][q];
      }
}

// ---- elementwise kernels --------------------------------------------------------------------
// Index draw and gather for 64 samples per workgroup of kGatherThr threads: the first 64
// threads draw their sample's index (t, env); the workgroup then reads the samples'
// observations (bf16-rounded in bf16 mode), writes them sample-major into X [Mp][F64] and,
// through an LDS transpose, feature-major into Xt [F64][Mp]. Padding (f >= F or m >= M) is
// zero. Workgroups from Mp / 64 on repack the weights instead (mb_pack).
constexpr int kGatherF = 128;   // largest padded observation width
constexpr int kGatherThr = 1024;

template <class Md>
struct PackArgs {
  const void *w1, *w2, *w3;
  int F, F64, H1, H2, Ap, Ap64;
  typename Md::T *W1t, *W2t, *W3t, *W3n;
};

// Weights in the k-contiguous layouts the products read, zero padded: W1t [H1][F64] (W1^T),
// W2t [H2][H1] (W2^T), W3t [Ap64][H2] (W3^T), W3n [H2][Ap64] (W3), from the caller's [in][out]
// matrices (bf16 bits or fp32, as the policy stores them); element q of the three in order.
template <class Md>
__device__ __forceinline__ void mb_pack(const PackArgs<Md>& p, size_t q) {
  typedef typename Md::T T;
  const size_t n1 = (size_t)p.H1 * p.F64, n2 = (size_t)p.H2 * p.H1, n3 = (size_t)p.Ap64 * p.H2;
  if (q < n1) {
    const int j = (int)(q / p.F64), f = (int)(q % p.F64);
    p.W1t[q] = f < p.F ? static_cast<const T*>(p.w1)[(size_t)f * p.H1 + j] : T(0);
    return;
  }
  q -= n1;
  if (q < n2) {
    const int i = (int)(q / p.H1), j = (int)(q % p.H1);
    p.W2t[q] = static_cast<const T*>(p.w2)[(size_t)j * p.H2 + i];
    return;
  }
  q -= n2;
  if (q < n3) {
    const int a = (int)(q / p.H2), i = (int)(q % p.H2);
    const T v = a < p.Ap ? static_cast<const T*>(p.w3)[(size_t)i * p.Ap + a] : T(0);
    p.W3t[q] = v;
    p.W3n[(size_t)i * p.Ap64 + a] = v;
  }
}

template <class Md>
__global__ __launch_bounds__(kGatherThr) void mb_gather_k(uint64_t seed, int M, int Mp, int T,
                                                          int E, int F, int F64,
                                                          const float* __restrict__ obs,
                                                          int64_t* __restrict__ idx,
                                                          int64_t* __restrict__ idx_out,
                                                          typename Md::T* __restrict__ X,
                                                          typename Md::T* __restrict__ Xt,
                                                          PackArgs<Md> pk) {
  __shared__ int ts[64], es[64];
  __shared__ float xs[64][kGatherF + 1];
  const int t = threadIdx.x;
  if ((int)blockIdx.x >= Mp / 64) {   // uniform per workgroup
    mb_pack(pk, (size_t)(blockIdx.x - Mp / 64) * kGatherThr + t);
    return;
  }
  const int m0 = blockIdx.x * 64;
  if (t < 64) {
    const int m = m0 + t;
    int tt = -1, ee = 0;
    if (m < M) {
      const u32x4 w = draw(seed, (uint32_t)m, 0xFFFFFFFDu, P_MINIBATCH, 0, 0);
      const double n = (double)T * (double)E;
      long long i = (long long)(unit(w.x, w.y) * n);
      if (i > (long long)T * E - 1) i = (long long)T * E - 1;
      idx[m] = i;
      if (idx_out) idx_out[m] = i;
      tt = (int)i / E;   // T E < 2^31 (checked by the host)
      ee = (int)i - tt * E;
    }
    ts[t] = tt;
    es[t] = ee;
  }
  __syncthreads();
  for (int q = t; q < 64 * F64; q += kGatherThr) {
    const int sl = q / F64, f = q % F64;
    float v = 0.f;
    if (ts[sl] >= 0 && f < F) v = Md::actf(obs[((size_t)ts[sl] * F + f) * E + es[sl]]);
    X[(size_t)(m0 + sl) * F64 + f] = Md::act(v);
    xs[sl][f] = v;
  }
  __syncthreads();
  for (int q = t; q < 64 * F64; q += kGatherThr) {
    const int f = q / 64, sl = q % 64;
    Xt[(size_t)f * Mp + m0 + sl] = Md::act(xs[sl][f]);
  }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <class Md>
struct LossArgs {
  typedef typename Md::T T;
  int A, Ap, Ap64, M, Mp, reinforce;
  float clip, c_v, c_h;
  const float* out;                  // [Mp][Ap64] outputs with b3
  const int64_t* idx;                // [M] sampled t * E + env
  const uint8_t* act;
  const float* logp_old;
  const double* adv;
  const double* ret;
  T *d_hi, *d_lo;                    // [Mp][Ap64] dL/d(output), hi + lo
  T *dt_hi, *dt_lo;                  // [Ap64][Mp]
  double* terms;                     // [M][3] policy, value, entropy per sample
  uint32_t* err;
};

// Loss terms and the loss gradient with respect to the outputs for kLossRows samples per
// workgroup, one wavefront per sample at a time (padded samples get zero gradients): lane i
// holds outputs i and i + 64 (A' <= 128), max and sums are butterfly reductions. The gradients
// are staged in LDS and written as hi + lo terms, sample-major and output-major, in runs.
constexpr int kLossWaves = kThr / 64;
constexpr int kLossRows = 16;
template <class Md>
__global__ __launch_bounds__(kThr) void mb_loss_k(LossArgs<Md> a) {
  typedef typename Md::T T;
  __shared__ float gs[kLossRows][129];
  const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  const int m0 = blockIdx.x * kLossRows;
  const int i0 = lane, i1 = lane + 64;
  for (int sl = wave; sl < kLossRows; sl += kLossWaves) {
    const int m = m0 + sl;
    float g0 = 0.f, g1 = 0.f;
    if (m < a.M) {
      const float* l = a.out + (size_t)m * a.Ap64;
      const float v0 = i0 < a.Ap ? l[i0] : 0.0f;
      const float v1 = i1 < a.Ap ? l[i1] : 0.0f;
      double* tm = a.terms + (size_t)m * 3;
      const size_t ti = (size_t)a.idx[m];
      const int act = a.act[ti];
      if (act >= a.A) {  // invalid stored action: flag it, the sample contributes nothing
        if (lane == 0) {
          atomicOr(a.err, ERR_ACTION);
          tm[0] = tm[1] = tm[2] = 0.0;
        }
      } else {
        const bool in0 = i0 < a.A, in1 = i1 < a.A;
        const float adv = (float)a.adv[ti], ret = (float)a.ret[ti];
        const float mx = wave_max(fmaxf(in0 ? v0 : -INFINITY, in1 ? v1 : -INFINITY));
        const float S = wave_sum((in0 ? expf(v0 - mx) : 0.0f) + (in1 ? expf(v1 - mx) : 0.0f));
        const float lS = logf(S);
        const float lp0 = (v0 - mx) - lS, lp1 = (v1 - mx) - lS;
        const float p0 = in0 ? expf(lp0) : 0.0f, p1 = in1 ? expf(lp1) : 0.0f;
        const float H = -wave_sum(p0 * (in0 ? lp0 : 0.0f) + p1 * (in1 ? lp1 : 0.0f));
        // the taken action's logit and the value output, broadcast from the lanes holding them
        const float la0 = __shfl(v0, act & 63, 64), la1 = __shfl(v1, act & 63, 64);
        const float logp = ((act < 64 ? la0 : la1) - mx) - lS;
        const float va0 = __shfl(v0, a.A & 63, 64), va1 = __shfl(v1, a.A & 63, 64);
        const float v = a.A < 64 ? va0 : va1;
        const float invM = 1.0f / (float)a.M;
        float dlogp, pterm;
        if (a.reinforce) {
          // -A log pi(a|s), the advantage held constant
          dlogp = -adv * invM;
          pterm = -adv * logp;
        } else {
          const float rho = expf(logp - a.logp_old[ti]);
          const float lo = 1.0f - a.clip, hi = 1.0f + a.clip;
          const float rc = fminf(fmaxf(rho, lo), hi);
          const float s1 = rho * adv, s2 = rc * adv;
          const float g_rho = s1 <= s2 ? adv : ((rho > lo && rho < hi) ? adv : 0.0f);
          dlogp = -g_rho * rho * invM;
          pterm = -fminf(s1, s2);
        }
        const float dv = 2.0f * a.c_v * (v - ret) * invM;
        if (i0 < a.Ap) {
          g0 = in0 ? -dlogp * p0 + a.c_h * invM * p0 * (lp0 + H) : dv;
          if (i0 == act) g0 += dlogp;
        }
        if (i1 < a.Ap) {
          g1 = in1 ? -dlogp * p1 + a.c_h * invM * p1 * (lp1 + H) : dv;
          if (i1 == act) g1 += dlogp;
        }
        if (lane == 0) {
          tm[0] = (double)pterm;
          tm[1] = (double)(v - ret) * (double)(v - ret);
          tm[2] = (double)H;
        }
      }
    }
    gs[sl][i0] = g0;
    gs[sl][i1] = g1;
  }
  __syncthreads();
  T h, l;
  for (int q = threadIdx.x; q < kLossRows * a.Ap64; q += kThr) {
    const int sl = q / a.Ap64, o = q % a.Ap64;
    Md::split(gs[sl][o], h, l);
    a.d_hi[(size_t)(m0 + sl) * a.Ap64 + o] = h;
    if (Md::SPLIT == 2) a.d_lo[(size_t)(m0 + sl) * a.Ap64 + o] = l;
  }
  for (int q = threadIdx.x; q < kLossRows * a.Ap64; q += kThr) {
    const int o = q / kLossRows, sl = q % kLossRows;
    Md::split(gs[sl][o], h, l);
    a.dt_hi[(size_t)o * a.Mp + m0 + sl] = h;
    if (Md::SPLIT == 2) a.dt_lo[(size_t)o * a.Mp + m0 + sl] = l;
  }
}

// The gradients' final sums in one launch. Blocks [0, nred): weight gradients from the split-k
// partials, G_l[r][c] = sum over z in order of P_l[z][r][c] for the R_l x N_l real entries
// (row stride N_l in the gradient layout), one thread per entry, layers back to back. Blocks
// from nred: bias gradients, one workgroup per unit row of a unit-major gradient (hi + lo)
// [rows][Mp]: thread t adds samples t, t + 256, ... in order, then a pairwise tree over the
// threads.
template <class Md>
struct RedDesc {
  const float* P;
  float* G;
  int S, R64, N64, R, N, first;   // first entry of this layer in the flattened range
};
template <class Md>
struct ColDesc {
  const typename Md::T *hi, *lo;
  float* out;
  int rows;
};
// The last workgroup sums the per-sample loss terms in a fixed order into the four loss values
// (thread t adds samples t, t + 256, ... in order, then a pairwise tree).
struct LossSum {
  const double* terms;   // [M][3] policy, value, entropy
  int M;
  float c_v, c_h;
  double* out;           // total, policy, value, entropy
};
template <class Md>
__global__ __launch_bounds__(kThr) void mb_finish_k(RedDesc<Md> r0, RedDesc<Md> r1, RedDesc<Md> r2,
                                                    int nred, ColDesc<Md> c0, ColDesc<Md> c1,
                                                    ColDesc<Md> c2, int Mp, LossSum ls) {
  __shared__ float part[kThr];
  __shared__ double dpart[3][kThr];
  if (blockIdx.x == gridDim.x - 1) {   // uniform per workgroup
    double s0 = 0.0, s1 = 0.0, s2 = 0.0;
#pragma unroll 8
    for (int m = threadIdx.x; m < ls.M; m += kThr) {
      s0 += ls.terms[(size_t)m * 3];
      s1 += ls.terms[(size_t)m * 3 + 1];
      s2 += ls.terms[(size_t)m * 3 + 2];
    }
    dpart[0][threadIdx.x] = s0;
    dpart[1][threadIdx.x] = s1;
    dpart[2][threadIdx.x] = s2;
    __syncthreads();
    for (int w = kThr / 2; w > 0; w >>= 1) {
      if ((int)threadIdx.x < w)
        for (int c = 0; c < 3; ++c) dpart[c][threadIdx.x] += dpart[c][threadIdx.x + w];
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      const double pi = dpart[0][0] / ls.M, v = ls.c_v * dpart[1][0] / ls.M,
                   h = -ls.c_h * dpart[2][0] / ls.M;
      ls.out[0] = pi + v + h;
      ls.out[1] = pi;
      ls.out[2] = v;
      ls.out[3] = h;
    }
    return;
  }
  if ((int)blockIdx.x < nred) {
    const int q = blockIdx.x * kThr + threadIdx.x;
    const RedDesc<Md>& d = q >= r2.first ? r2 : (q >= r1.first ? r1 : r0);
    const int e = q - d.first;
    if (e >= d.R * d.N) return;
    const int r = e / d.N, c = e % d.N;
    const size_t o = (size_t)r * d.N64 + c, st = (size_t)d.R64 * d.N64;
    float s = 0.f;
#pragma unroll 8
    for (int z = 0; z < d.S; ++z) s += d.P[o + z * st];
    d.G[e] = s;
    return;
  }
  int r = blockIdx.x - nred;   // uniform per workgroup
  ColDesc<Md> c = c0;
  if (r >= c0.rows) {
    r -= c0.rows;
    c = c1;
    if (r >= c1.rows) {
      r -= c1.rows;
      c = c2;
    }
  }
  const typename Md::T* h = c.hi + (size_t)r * Mp;
  float s = 0.f;
  if constexpr (Md::SPLIT == 2) {
    const typename Md::T* l = c.lo + (size_t)r * Mp;
#pragma unroll 8
    for (int m = threadIdx.x; m < Mp; m += kThr) s += Md::value(h[m]) + Md::value(l[m]);
  } else {
#pragma unroll 8
    for (int m = threadIdx.x; m < Mp; m += kThr) s += Md::value(h[m]);
  }
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = kThr / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) c.out[r] = part[0];
}

// loss terms summed in a fixed order by one workgroup: each thread adds a contiguous run of
// samples in order, then a pairwise tree combines the threads' partial sums
constexpr int kSumThr = 1024;
__global__ __launch_bounds__(kSumThr) void ppo_loss_k(const double* terms, int M, float c_v,
                                                      float c_h, double* out) {
  __shared__ double part[3][kSumThr];
  const int per = (M + kSumThr - 1) / kSumThr;
  const int m0 = threadIdx.x * per;
  const int m1 = m0 + per < M ? m0 + per : M;
  double s0 = 0.0, s1 = 0.0, s2 = 0.0;
#pragma unroll 4
  for (int m = m0; m < m1; ++m) {
    s0 += terms[(size_t)m * 3];
    s1 += terms[(size_t)m * 3 + 1];
    s2 += terms[(size_t)m * 3 + 2];
  }
  part[0][threadIdx.x] = s0;
  part[1][threadIdx.x] = s1;
  part[2][threadIdx.x] = s2;
  __syncthreads();
  for (int w = kSumThr / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w)
      for (int c = 0; c < 3; ++c) part[c][threadIdx.x] += part[c][threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double pi = part[0][0] / M, v = c_v * part[1][0] / M, h = -c_h * part[2][0] / M;
    out[0] = pi + v + h;
    out[1] = pi;
    out[2] = v;
    out[3] = h;
  }
}

int pad64(int x) { return (x + 63) & ~63; }

// split of a sample reduction of length Mp into chunks (multiples of 32) for about `target`
// workgroups over `tiles` output tiles
void split_k(int Mp, int tiles, int target, int* chunk, int* S) {
  int s = target / (tiles > 0 ? tiles : 1);
  if (s < 1) s = 1;
  int c = (Mp + s - 1) / s;
  c = (c + 31) & ~31;
  if (c < 32) c = 32;
  *chunk = c;
  *S = (Mp + c - 1) / c;
}

constexpr int kWgradTarget = 256;   // workgroups per weight-gradient product

// the scratch carve-up (every piece 256-byte aligned); element size e = 2 (bf16) or 4 (fp32)
struct MbScratch {
  int64_t* idx;
  double* terms;
  void *X, *Xt, *H1, *H1t, *H2, *H2t;
  float *D1, *D2, *out, *P;
  void *dO_hi, *dO_lo, *dOt_hi, *dOt_lo, *dZ2_hi, *dZ2_lo, *dZ2t_hi, *dZ2t_lo, *dZ1t_hi, *dZ1t_lo;
  void *W1t, *W2t, *W3t, *W3n;
};

struct Dims {
  int M, Mp, F, F64, H1, H2, Ap, Ap64;
};

Dims dims_of(const MlpParams& m, int M) {
  Dims d;
  d.M = M; d.Mp = pad64(M); d.F = m.F; d.F64 = pad64(m.F); d.H1 = m.H1; d.H2 = m.H2;
  d.Ap = m.Ap; d.Ap64 = pad64(m.Ap);
  return d;
}

// the weight-gradient products in launch order (layer 3, 2, 1): padded shapes and sample chunks
struct WgShape {
  int R64, N64, R, N, S, chunk;
  size_t poff;   // offset of its partial sums in the partial buffer (floats)
};
void wg_shapes(const Dims& d, WgShape w[3], size_t* total) {
  const int R64[3] = {d.H2, d.H1, d.F64}, N64[3] = {d.Ap64, d.H2, d.H1};
  const int R[3] = {d.H2, d.H1, d.F}, N[3] = {d.Ap, d.H2, d.H1};
  size_t off = 0;
  for (int l = 0; l < 3; ++l) {
    w[l].R64 = R64[l]; w[l].N64 = N64[l]; w[l].R = R[l]; w[l].N = N[l];
    split_k(d.Mp, (R64[l] / kTile) * (N64[l] / kTile), kWgradTarget, &w[l].chunk, &w[l].S);
    w[l].poff = off;
    off += ((size_t)w[l].S * R64[l] * N64[l] + 63) & ~(size_t)63;
  }
  *total = off;
}

size_t partial_floats(const Dims& d) {
  WgShape w[3];
  size_t total;
  wg_shapes(d, w, &total);
  return total;
}

size_t carve(const MlpParams& m, int M, void* base, MbScratch* s) {
  const Dims d = dims_of(m, M);
  const size_t e = m.bf16 ? 2 : 4, two = m.bf16 ? 2 : 1;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    void* p = base ? static_cast<unsigned char*>(base) + off : nullptr;
    off += (bytes + 255) & ~(size_t)255;
    return p;
  };
  const size_t Mp = d.Mp;
  MbScratch t;
  t.idx = static_cast<int64_t*>(take((size_t)M * sizeof(int64_t)));
  t.terms = static_cast<double*>(take((size_t)M * 3 * sizeof(double)));
  t.X = take(Mp * d.F64 * e);
  t.Xt = take(Mp * d.F64 * e);
  t.H1 = take(Mp * d.H1 * e);
  t.H1t = take(Mp * d.H1 * e);
  t.H2 = take(Mp * d.H2 * e);
  t.H2t = take(Mp * d.H2 * e);
  t.D1 = static_cast<float*>(take(Mp * d.H1 * 4));
  t.D2 = static_cast<float*>(take(Mp * d.H2 * 4));
  t.out = static_cast<float*>(take(Mp * d.Ap64 * 4));
  t.dO_hi = take(Mp * d.Ap64 * e);
  t.dOt_hi = take(Mp * d.Ap64 * e);
  t.dZ2_hi = take(Mp * d.H2 * e);
  t.dZ2t_hi = take(Mp * d.H2 * e);
  t.dZ1t_hi = take(Mp * d.H1 * e);
  if (two == 2) {
    t.dO_lo = take(Mp * d.Ap64 * e);
    t.dOt_lo = take(Mp * d.Ap64 * e);
    t.dZ2_lo = take(Mp * d.H2 * e);
    t.dZ2t_lo = take(Mp * d.H2 * e);
    t.dZ1t_lo = take(Mp * d.H1 * e);
  } else {
    t.dO_lo = t.dOt_lo = t.dZ2_lo = t.dZ2t_lo = t.dZ1t_lo = nullptr;
  }
  t.W1t = take((size_t)d.H1 * d.F64 * e);
  t.W2t = take((size_t)d.H2 * d.H1 * e);
  t.W3t = take((size_t)d.Ap64 * d.H2 * e);
  t.W3n = take((size_t)d.H2 * d.Ap64 * e);
  t.P = static_cast<float*>(take(partial_floats(d) * 4));
  if (s) *s = t;
  return off;
}

unsigned blocks(size_t n, int per) { return (unsigned)((n + per - 1) / per); }

template <class Md, bool TWO, class Epi>
hipError_t gemm(const void* A, int lda, const void* B0, const void* B1, int ldb, int R, int N,
                int K, const Epi& epi, hipStream_t st) {
  GemmArgs g{A, B0, B1, lda, ldb, K};
  hipLaunchKernelGGL((mb_gemm_k<Md, TWO, Epi>), dim3(N / kTile, R / kTile), dim3(kThr), 0, st, g,
                     epi);
  return hipGetLastError();
}

template <class Md>
hipError_t run_minibatch(const MlpParams& m, const void* d_weights, const size_t off[6], int T,
                         const float* obs, const uint8_t* act, const float* logp_old,
                         const double* adv, const double* ret, int M, uint64_t seed, float clip,
                         float c_v, float c_h, int reinforce, void* scratch, double* loss_out,
                         float* grads, int64_t* idx_out, uint32_t* err, hipStream_t st) {
  typedef typename Md::T TT;
  constexpr bool TWO = Md::SPLIT == 2;
  const Dims d = dims_of(m, M);
  MbScratch s;
  carve(m, M, scratch, &s);
  const unsigned char* wb = static_cast<const unsigned char*>(d_weights);
  const float* b1 = reinterpret_cast<const float*>(wb + off[1]);
  const float* b2 = reinterpret_cast<const float*>(wb + off[3]);
  const float* b3 = reinterpret_cast<const float*>(wb + off[5]);
  const void* w2n = wb + off[2];   // W2 [H1][H2] is already k-contiguous for the backward
  hipError_t e;
  const size_t npack = (size_t)d.H1 * d.F64 + (size_t)d.H2 * d.H1 + (size_t)d.Ap64 * d.H2;
  PackArgs<Md> pk{wb + off[0], wb + off[2], wb + off[4], d.F, d.F64, d.H1, d.H2, d.Ap, d.Ap64,
                  static_cast<TT*>(s.W1t), static_cast<TT*>(s.W2t), static_cast<TT*>(s.W3t),
                  static_cast<TT*>(s.W3n)};
  hipLaunchKernelGGL(mb_gather_k<Md>, dim3(d.Mp / 64 + blocks(npack, kGatherThr)),
                     dim3(kGatherThr), 0, st, seed, M, d.Mp, T, m.E, d.F, d.F64, obs, s.idx,
                     idx_out, static_cast<TT*>(s.X), static_cast<TT*>(s.Xt), pk);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // forward: three products, columns = samples
  EpiHidden<Md> e1{b1, static_cast<TT*>(s.H1), static_cast<TT*>(s.H1t), s.D1, d.H1, d.Mp, M};
  if ((e = gemm<Md, false>(s.W1t, d.F64, s.X, nullptr, d.F64, d.H1, d.Mp, d.F64, e1, st))) return e;
  EpiHidden<Md> e2{b2, static_cast<TT*>(s.H2), static_cast<TT*>(s.H2t), s.D2, d.H2, d.Mp, M};
  if ((e = gemm<Md, false>(s.W2t, d.H1, s.H1, nullptr, d.H1, d.H2, d.Mp, d.H1, e2, st))) return e;
  EpiOut e3{b3, s.out, d.Ap, d.Ap64};
  if ((e = gemm<Md, false>(s.W3t, d.H2, s.H2, nullptr, d.H2, d.Ap64, d.Mp, d.H2, e3, st))) return e;
  // loss and dL/dout
  LossArgs<Md> la;
  la.A = m.A; la.Ap = d.Ap; la.Ap64 = d.Ap64; la.M = M; la.Mp = d.Mp; la.reinforce = reinforce;
  la.clip = clip; la.c_v = c_v; la.c_h = c_h;
  la.out = s.out; la.idx = s.idx; la.act = act; la.logp_old = logp_old; la.adv = adv; la.ret = ret;
  la.d_hi = static_cast<TT*>(s.dO_hi); la.d_lo = static_cast<TT*>(s.dO_lo);
  la.dt_hi = static_cast<TT*>(s.dOt_hi); la.dt_lo = static_cast<TT*>(s.dOt_lo);
  la.terms = s.terms; la.err = err;
  hipLaunchKernelGGL(mb_loss_k<Md>, dim3(d.Mp / kLossRows), dim3(kThr), 0, st, la);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // backward through the hidden layers, columns = samples
  EpiBack<Md> g2{s.D2, static_cast<TT*>(s.dZ2_hi), static_cast<TT*>(s.dZ2_lo),
                 static_cast<TT*>(s.dZ2t_hi), static_cast<TT*>(s.dZ2t_lo), d.H2, d.Mp, M};
  if ((e = gemm<Md, TWO>(s.W3n, d.Ap64, s.dO_hi, s.dO_lo, d.Ap64, d.H2, d.Mp, d.Ap64, g2, st)))
    return e;
  EpiBack<Md> g1{s.D1, nullptr, nullptr, static_cast<TT*>(s.dZ1t_hi), static_cast<TT*>(s.dZ1t_lo),
                 d.H1, d.Mp, M};
  if ((e = gemm<Md, TWO>(w2n, d.H2, s.dZ2_hi, s.dZ2_lo, d.H2, d.H1, d.Mp, d.H2, g1, st))) return e;
  // weight gradients, reductions over the samples: gradient layout W1 [F][H1], b1, W2 [H1][H2],
  // b2, W3 [H2][A'], b3 (fp32, contiguous)
  float* gw1 = grads;
  float* gb1 = gw1 + (size_t)d.F * d.H1;
  float* gw2 = gb1 + d.H1;
  float* gb2 = gw2 + (size_t)d.H1 * d.H2;
  float* gw3 = gb2 + d.H2;
  float* gb3 = gw3 + (size_t)d.H2 * d.Ap;
  WgShape ws[3];
  size_t ptotal;
  wg_shapes(d, ws, &ptotal);
  const TT* A_[3] = {static_cast<const TT*>(s.H2t), static_cast<const TT*>(s.H1t),
                     static_cast<const TT*>(s.Xt)};
  const TT* B0_[3] = {static_cast<const TT*>(s.dOt_hi), static_cast<const TT*>(s.dZ2t_hi),
                      static_cast<const TT*>(s.dZ1t_hi)};
  const TT* B1_[3] = {static_cast<const TT*>(s.dOt_lo), static_cast<const TT*>(s.dZ2t_lo),
                      static_cast<const TT*>(s.dZ1t_lo)};
  float* G_[3] = {gw3, gw2, gw1};
  WgDesc<Md> wd[3];
  RedDesc<Md> rd[3];
  int nblk = 0, nent = 0;
  for (int l = 0; l < 3; ++l) {
    const WgShape& q = ws[l];
    wd[l] = WgDesc<Md>{A_[l], B0_[l], B1_[l], s.P + q.poff, q.R64, q.N64, q.S, q.chunk, nblk};
    nblk += (q.R64 / kTile) * (q.N64 / kTile) * q.S;
    rd[l] = RedDesc<Md>{s.P + q.poff, G_[l], q.S, q.R64, q.N64, q.R, q.N, nent};
    nent += q.R * q.N;
  }
  hipLaunchKernelGGL(mb_wgrad_k<Md>, dim3(nblk), dim3(kThr), 0, st, wd[0], wd[1], wd[2], d.Mp);
  const int nred = (nent + kThr - 1) / kThr;
  ColDesc<Md> c3{static_cast<const TT*>(s.dOt_hi), static_cast<const TT*>(s.dOt_lo), gb3, d.Ap};
  ColDesc<Md> c2{static_cast<const TT*>(s.dZ2t_hi), static_cast<const TT*>(s.dZ2t_lo), gb2, d.H2};
  ColDesc<Md> c1{static_cast<const TT*>(s.dZ1t_hi), static_cast<const TT*>(s.dZ1t_lo), gb1, d.H1};
  LossSum ls{s.terms, M, c_v, c_h, loss_out};
  hipLaunchKernelGGL(mb_finish_k<Md>, dim3(nred + d.Ap + d.H2 + d.H1 + 1), dim3(kThr), 0, st,
                     rd[0], rd[1], rd[2], nred, c3, c2, c1, d.Mp, ls);
  return hipGetLastError();
}

}  // namespace

size_t ppo_scratch_bytes(const MlpParams& m, int M) { return carve(m, M, nullptr, nullptr); }

hipError_t static_scratch(void** ptr) {
  constexpr int kDevices = 64;
  static std::mutex mu;
  static void* addr[kDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

bool ppo_shape_supported(const MlpParams& m) {
  return m.Ap <= 128 && m.H1 % kTile == 0 && m.H2 % kTile == 0 && m.F >= 1 &&
         pad64(m.F) <= kGatherF;
}

hipError_t launch_ppo(const MlpParams& m, const void* d_weights, const size_t off[6], int T,
                      const float* obs, const uint8_t* act, const float* logp_old,
                      const double* adv, const double* ret, int M, uint64_t seed, float clip,
                      float c_v, float c_h, int reinforce, void* scratch, double* loss_out,
                      float* grads, int64_t* idx_out, uint32_t* err, hipStream_t st) {
  if (M < 1 || !ppo_shape_supported(m)) return hipErrorInvalidValue;
  if (m.bf16)
    return run_minibatch<Bf16Mode>(m, d_weights, off, T, obs, act, logp_old, adv, ret, M, seed,
                                   clip, c_v, c_h, reinforce, scratch, loss_out, grads, idx_out,
                                   err, st);
  return run_minibatch<F32Mode>(m, d_weights, off, T, obs, act, logp_old, adv, ret, M, seed, clip,
                                c_v, c_h, reinforce, scratch, loss_out, grads, idx_out, err, st);
}

hipError_t launch_pg_loss(const double* terms, int M, float c_v, float c_h, double* out,
                          hipStream_t st) {
  hipLaunchKernelGGL(ppo_loss_k, dim3(1), dim3(kSumThr), 0, st, terms, M, c_v, c_h, out);
  return hipGetLastError();
}

}  // namespace bsim
