// ppo_kernels.hip -- one policy-gradient minibatch (paper Sec. 4.3): gather, forward, loss
// (PPO clipped surrogate, or REINFORCE with a learned baseline) + value + entropy, and its
// gradient with respect to every policy weight.
//
// M samples (t, env) are drawn with replacement: sample m takes u from the MINIBATCH block at
// counter (m, 0xFFFFFFFD, MINIBATCH<<24, 0) and index floor(u * T * E). The forward repeats
// the rollout policy's rounding points (every layer input rounded to bf16) with fp32
// arithmetic and saves pre-activations; gradients pass through the bf16 roundings as the
// identity. Loss
//   L = -mean(min(rho A, clip(rho, 1-eps, 1+eps) A)) + c_v mean((V - R)^2) - c_h mean(H),
//   rho = exp(logp_new(a) - logp_old), H the entropy of the action distribution; REINFORCE
//   replaces the first term by -mean(A log pi(a|s)) with A held constant.
// Work is split into: forward (16 samples per workgroup, one output unit per thread),
// backward through the activations (same split), and weight gradients (LDS-tiled products
// over fixed sample chunks, fp32, summed in chunk order, so results are deterministic).
#include "devmath.hpp"
#include "params.hpp"

namespace bsim {
namespace {

constexpr int kSpb = 16;   // samples per workgroup
constexpr int kThr = 256;
constexpr size_t kMaxLds = 64 * 1024;  // dynamic LDS per workgroup used by the forward

__device__ __forceinline__ float bf16_round(float f) { return bf16_to_f32(bf16_bits(f)); }
__device__ __forceinline__ float gelu_exact(float z) {
  return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));
}
__device__ __forceinline__ float gelu_grad(float z) {
  return 0.5f * (1.0f + erff(z * 0.70710678118654752f)) + z * expf(-0.5f * z * z) * 0.39894228040143268f;
}

__device__ __forceinline__ float wval(const void* w, size_t i, int bf16) {
  return bf16 ? bf16_to_f32(static_cast<const uint16_t*>(w)[i]) : static_cast<const float*>(w)[i];
}

// out[s][j] = sum_i in[s][i] W[i][j] + b[j] for the workgroup's samples; W is [K][N] in-major
__device__ void dense_fwd(const float* in, int K, const void* W, const float* b, int N, int bf16,
                          float* out) {
  for (int j = threadIdx.x; j < N; j += kThr) {
    float acc[kSpb];
#pragma unroll
    for (int s = 0; s < kSpb; ++s) acc[s] = b[j];
    for (int i = 0; i < K; ++i) {
      const float wv = wval(W, (size_t)i * N + j, bf16);
#pragma unroll
      for (int s = 0; s < kSpb; ++s) acc[s] = fmaf(in[s * K + i], wv, acc[s]);
    }
#pragma unroll
    for (int s = 0; s < kSpb; ++s) out[s * N + j] = acc[s];
  }
}

struct PpoArgs {
  int F, H1, H2, A, Ap, E, T, M, bf16;
  const void* w1; const float* b1;   // ABI weights, in-major
  const void* w2; const float* b2;
  const void* w3; const float* b3;
  int AP;
  const float* obs;                  // [T(+1)][F][E]
  const uint8_t* act;
  const float* logp_old;
  const double* adv;
  const double* ret;
  uint64_t seed;
  int reinforce;                     // 0: PPO clipped surrogate; 1: REINFORCE with baseline
  float clip, c_v, c_h;
  float* x; float* z1; float* h1; float* z2; float* h2; float* dout;
  float* dz1; float* dz2;
  double* terms;                     // [M][3] policy, value, entropy per sample
  int64_t* idx_out;                  // optional [M] sampled t * E + env
  uint32_t* err;                     // device error flags
};

__global__ __launch_bounds__(kThr) void ppo_fwd_k(PpoArgs a) {
  extern __shared__ float sm[];
  float* xs = sm;                          // [kSpb][F]
  float* h1s = xs + kSpb * a.F;            // [kSpb][H1]
  float* h2s = h1s + kSpb * a.H1;          // [kSpb][H2]
  float* os = h2s + kSpb * a.H2;           // [kSpb][Ap]
  __shared__ int ts_[kSpb], es_[kSpb];
  const int m0 = blockIdx.x * kSpb;
  if (threadIdx.x < kSpb) {
    const int m = m0 + threadIdx.x;
    const u32x4 w = draw(a.seed, (uint32_t)m, 0xFFFFFFFDu, P_MINIBATCH, 0, 0);
    const double n = (double)a.T * (double)a.E;
    long long i = (long long)(unit(w.x, w.y) * n);
    if (i > (long long)a.T * a.E - 1) i = (long long)a.T * a.E - 1;
    ts_[threadIdx.x] = (int)(i / a.E);
    es_[threadIdx.x] = (int)(i % a.E);
    if (a.idx_out) a.idx_out[m] = i;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < kSpb * a.F; idx += kThr) {
    const int s = idx / a.F, f = idx % a.F;
    float v = a.obs[((size_t)ts_[s] * a.F + f) * a.E + es_[s]];
    if (a.bf16) v = bf16_round(v);
    xs[idx] = v;
    a.x[(size_t)(m0 + s) * a.F + f] = v;
  }
  __syncthreads();
  dense_fwd(xs, a.F, a.w1, a.b1, a.H1, a.bf16, h1s);
  __syncthreads();
  for (int idx = threadIdx.x; idx < kSpb * a.H1; idx += kThr) {
    const float z = h1s[idx];
    float h = gelu_exact(z);
    if (a.bf16) h = bf16_round(h);
    a.z1[(size_t)m0 * a.H1 + idx] = z;
    a.h1[(size_t)m0 * a.H1 + idx] = h;
    h1s[idx] = h;
  }
  __syncthreads();
  dense_fwd(h1s, a.H1, a.w2, a.b2, a.H2, a.bf16, h2s);
  __syncthreads();
  for (int idx = threadIdx.x; idx < kSpb * a.H2; idx += kThr) {
    const float z = h2s[idx];
    float h = gelu_exact(z);
    if (a.bf16) h = bf16_round(h);
    a.z2[(size_t)m0 * a.H2 + idx] = z;
    a.h2[(size_t)m0 * a.H2 + idx] = h;
    h2s[idx] = h;
  }
  __syncthreads();
  dense_fwd(h2s, a.H2, a.w3, a.b3, a.Ap, a.bf16, os);
  __syncthreads();
  // loss gradient with respect to the outputs, one thread per sample
  if (threadIdx.x < kSpb) {
    const int s = threadIdx.x, m = m0 + s;
    const float* l = os + s * a.Ap;
    float* d = a.dout + (size_t)m * a.Ap;
    const size_t ti = (size_t)ts_[s] * a.E + es_[s];
    const int act = a.act[ti];
    double* tm = a.terms + (size_t)m * 3;
    if (act >= a.A) {  // invalid stored action: flag it, the sample contributes nothing
      atomicOr(a.err, ERR_ACTION);
      for (int i = 0; i < a.Ap; ++i) d[i] = 0.0f;
      tm[0] = tm[1] = tm[2] = 0.0;
      return;
    }
    const float adv = (float)a.adv[ti], ret = (float)a.ret[ti];
    float mx = l[0];
    for (int i = 1; i < a.A; ++i) mx = fmaxf(mx, l[i]);
    float S = 0.f;
    for (int i = 0; i < a.A; ++i) S += expf(l[i] - mx);
    const float lS = logf(S);
    float H = 0.f;
    for (int i = 0; i < a.A; ++i) {
      const float lp = (l[i] - mx) - lS;
      H -= expf(lp) * lp;
    }
    const float logp = (l[act] - mx) - lS;
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
    for (int i = 0; i < a.A; ++i) {
      const float lp = (l[i] - mx) - lS;
      const float p = expf(lp);
      float g = -dlogp * p + a.c_h * invM * p * (lp + H);
      if (i == act) g += dlogp;
      d[i] = g;
    }
    const float v = l[a.A];
    d[a.A] = 2.0f * a.c_v * (v - ret) * invM;
    tm[0] = (double)pterm;
    tm[1] = (double)(v - ret) * (double)(v - ret);
    tm[2] = (double)H;
  }
}

// dz2 = (dout W3^T) * gelu'(z2); dz1 = (dz2 W2^T) * gelu'(z1); thread j walks row j of the
// in-major weights.
__global__ __launch_bounds__(kThr) void ppo_bwd_k(PpoArgs a) {
  extern __shared__ float sm[];
  float* ds = sm;                          // [kSpb][Ap]
  float* d2 = ds + kSpb * a.Ap;            // [kSpb][H2]
  const int m0 = blockIdx.x * kSpb;
  for (int idx = threadIdx.x; idx < kSpb * a.Ap; idx += kThr) ds[idx] = a.dout[(size_t)m0 * a.Ap + idx];
  __syncthreads();
  for (int j = threadIdx.x; j < a.H2; j += kThr) {
    float acc[kSpb];
#pragma unroll
    for (int s = 0; s < kSpb; ++s) acc[s] = 0.f;
    for (int o = 0; o < a.Ap; ++o) {
      const float wv = wval(a.w3, (size_t)j * a.Ap + o, a.bf16);
#pragma unroll
      for (int s = 0; s < kSpb; ++s) acc[s] = fmaf(ds[s * a.Ap + o], wv, acc[s]);
    }
#pragma unroll
    for (int s = 0; s < kSpb; ++s) {
      const float g = acc[s] * gelu_grad(a.z2[(size_t)(m0 + s) * a.H2 + j]);
      d2[s * a.H2 + j] = g;
      a.dz2[(size_t)(m0 + s) * a.H2 + j] = g;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < a.H1; i += kThr) {
    float acc[kSpb];
#pragma unroll
    for (int s = 0; s < kSpb; ++s) acc[s] = 0.f;
    for (int j = 0; j < a.H2; ++j) {
      const float wv = wval(a.w2, (size_t)i * a.H2 + j, a.bf16);
#pragma unroll
      for (int s = 0; s < kSpb; ++s) acc[s] = fmaf(d2[s * a.H2 + j], wv, acc[s]);
    }
#pragma unroll
    for (int s = 0; s < kSpb; ++s)
      a.dz1[(size_t)(m0 + s) * a.H1 + i] = acc[s] * gelu_grad(a.z1[(size_t)(m0 + s) * a.H1 + i]);
  }
}

// Weight gradients as one augmented product per layer: G = [A | 1]^T B, (K+1) x N, whose
// first K rows are dW = A^T B and whose last row is db = sum_m B[m]. The samples are split
// into chunks of kMC; workgroup (ti, tj, c) forms a 32 x 32 tile of chunk c's partial product
// from LDS-staged 32-sample slices (fp32, each thread 2 x 2 outputs); a second pass adds the
// chunks in order. The result does not depend on the launch, only on M.
constexpr int kWT = 32, kMS = 32, kMC = 512;

__global__ __launch_bounds__(256) void wgrad_part_k(const float* __restrict__ Am, int K,
                                                    const float* __restrict__ Bm, int N, int M,
                                                    float* __restrict__ part) {
  __shared__ float As[kMS][kWT + 1], Bs[kMS][kWT + 1];
  const int i0 = blockIdx.x * kWT, j0 = blockIdx.y * kWT, c = blockIdx.z;
  const int m0 = c * kMC, m1 = m0 + kMC < M ? m0 + kMC : M;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  float acc00 = 0.f, acc01 = 0.f, acc10 = 0.f, acc11 = 0.f;
  for (int ms = m0; ms < m1; ms += kMS) {
    for (int q = threadIdx.x; q < kMS * kWT; q += 256) {
      const int r = q / kWT, col = q % kWT, m = ms + r;
      const int i = i0 + col, j = j0 + col;
      As[r][col] = m < m1 ? (i < K ? Am[(size_t)m * K + i] : (i == K ? 1.0f : 0.0f)) : 0.0f;
      Bs[r][col] = (m < m1 && j < N) ? Bm[(size_t)m * N + j] : 0.0f;
    }
    __syncthreads();
#pragma unroll 8
    for (int r = 0; r < kMS; ++r) {
      const float a0 = As[r][2 * ty], a1 = As[r][2 * ty + 1];
      const float b0 = Bs[r][2 * tx], b1 = Bs[r][2 * tx + 1];
      acc00 = fmaf(a0, b0, acc00);
      acc01 = fmaf(a0, b1, acc01);
      acc10 = fmaf(a1, b0, acc10);
      acc11 = fmaf(a1, b1, acc11);
    }
    __syncthreads();
  }
  const int i = i0 + 2 * ty, j = j0 + 2 * tx;
  float* out = part + (size_t)c * (K + 1) * N;
  if (i <= K && j < N) out[(size_t)i * N + j] = acc00;
  if (i <= K && j + 1 < N) out[(size_t)i * N + j + 1] = acc01;
  if (i + 1 <= K && j < N) out[(size_t)(i + 1) * N + j] = acc10;
  if (i + 1 <= K && j + 1 < N) out[(size_t)(i + 1) * N + j + 1] = acc11;
}

__global__ __launch_bounds__(256) void wgrad_sum_k(const float* __restrict__ part, int nc,
                                                   size_t n, float* __restrict__ g) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= n) return;
  float s = 0.f;
  for (int c = 0; c < nc; ++c) s += part[(size_t)c * n + idx];
  g[idx] = s;
}

// loss terms summed in a fixed order by one workgroup
__global__ __launch_bounds__(kThr) void ppo_loss_k(const double* terms, int M, float c_v, float c_h,
                                                   double* out) {
  __shared__ double part[3][kThr];
  for (int c = 0; c < 3; ++c) {
    double s = 0.0;
    for (int m = threadIdx.x; m < M; m += kThr) s += terms[(size_t)m * 3 + c];
    part[c][threadIdx.x] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double t[3] = {0.0, 0.0, 0.0};
    for (int c = 0; c < 3; ++c)
      for (int i = 0; i < kThr; ++i) t[c] += part[c][i];
    const double pi = t[0] / M, v = c_v * t[1] / M, h = -c_h * t[2] / M;
    out[0] = pi + v + h;
    out[1] = pi;
    out[2] = v;
    out[3] = h;
  }
}

}  // namespace

size_t ppo_lds_bytes(const MlpParams& m) {
  return (size_t)kSpb * (m.F + m.H1 + m.H2 + m.Ap) * sizeof(float);
}

hipError_t launch_ppo(const MlpParams& m, const void* d_weights, const size_t off[6], int T,
                      const float* obs, const uint8_t* act, const float* logp_old,
                      const double* adv, const double* ret, int M, uint64_t seed, float clip,
                      float c_v, float c_h, int reinforce, float* scratch, double* loss_out,
                      float* grads, int64_t* idx_out, uint32_t* err, hipStream_t st) {
  const unsigned char* wb = static_cast<const unsigned char*>(d_weights);
  PpoArgs a;
  a.F = m.F; a.H1 = m.H1; a.H2 = m.H2; a.A = m.A; a.Ap = m.Ap; a.E = m.E; a.T = T; a.M = M;
  a.bf16 = m.bf16; a.AP = m.AP;
  a.w1 = wb + off[0]; a.b1 = reinterpret_cast<const float*>(wb + off[1]);
  a.w2 = wb + off[2]; a.b2 = reinterpret_cast<const float*>(wb + off[3]);
  a.w3 = wb + off[4]; a.b3 = reinterpret_cast<const float*>(wb + off[5]);
  a.obs = obs; a.act = act; a.logp_old = logp_old; a.adv = adv; a.ret = ret;
  a.seed = seed; a.clip = clip; a.c_v = c_v; a.c_h = c_h; a.reinforce = reinforce;
  a.idx_out = idx_out; a.err = err;
  float* p = scratch;
  a.x = p; p += (size_t)M * m.F;
  a.z1 = p; p += (size_t)M * m.H1;
  a.h1 = p; p += (size_t)M * m.H1;
  a.z2 = p; p += (size_t)M * m.H2;
  a.h2 = p; p += (size_t)M * m.H2;
  a.dout = p; p += (size_t)M * m.Ap;
  a.dz1 = p; p += (size_t)M * m.H1;
  a.dz2 = p; p += (size_t)M * m.H2;
  a.terms = reinterpret_cast<double*>(p);
  const int blocks = M / kSpb;
  const size_t lds_f = ppo_lds_bytes(m);
  if (lds_f > kMaxLds || M % kSpb) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ppo_fwd_k, dim3(blocks), dim3(kThr), lds_f, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds_b = (size_t)kSpb * (m.Ap + m.H2) * sizeof(float);
  hipLaunchKernelGGL(ppo_bwd_k, dim3(blocks), dim3(kThr), lds_b, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // gradient layout: W1 [F][H1], b1, W2 [H1][H2], b2, W3 [H2][Ap], b3 (fp32, contiguous)
  float* gw1 = grads;
  float* gb1 = gw1 + (size_t)m.F * m.H1;
  float* gw2 = gb1 + m.H1;
  float* gb2 = gw2 + (size_t)m.H1 * m.H2;
  float* gw3 = gb2 + m.H2;
  // the three augmented products [x|1]^T dz1, [h1|1]^T dz2, [h2|1]^T dout land on W,b pairs
  // that are contiguous in the gradient layout
  const struct { const float* A; int K; const float* B; int N; float* G; } g[3] = {
      {a.x, m.F, a.dz1, m.H1, gw1}, {a.h1, m.H1, a.dz2, m.H2, gw2}, {a.h2, m.H2, a.dout, m.Ap, gw3}};
  const int nc = (M + kMC - 1) / kMC;
  float* part = reinterpret_cast<float*>(a.terms + (size_t)M * 3);
  for (int l = 0; l < 3; ++l) {
    const dim3 grid((unsigned)((g[l].K + 1 + kWT - 1) / kWT), (unsigned)((g[l].N + kWT - 1) / kWT),
                    (unsigned)nc);
    hipLaunchKernelGGL(wgrad_part_k, grid, dim3(256), 0, st, g[l].A, g[l].K, g[l].B, g[l].N, M,
                       part);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t n = (size_t)(g[l].K + 1) * g[l].N;
    hipLaunchKernelGGL(wgrad_sum_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, part, nc,
                       n, g[l].G);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(ppo_loss_k, dim3(1), dim3(kThr), 0, st, a.terms, M, c_v, c_h, loss_out);
  return hipGetLastError();
}

hipError_t launch_pg_loss(const double* terms, int M, float c_v, float c_h, double* out,
                          hipStream_t st) {
  hipLaunchKernelGGL(ppo_loss_k, dim3(1), dim3(kThr), 0, st, terms, M, c_v, c_h, out);
  return hipGetLastError();
}

size_t ppo_scratch_floats(const MlpParams& m, int M) {
  // activations, per-sample loss terms (fp64), then the chunked weight-gradient partials
  const size_t nc = (size_t)(M + kMC - 1) / kMC;
  size_t kn = (size_t)(m.F + 1) * m.H1;
  if ((size_t)(m.H1 + 1) * m.H2 > kn) kn = (size_t)(m.H1 + 1) * m.H2;
  if ((size_t)(m.H2 + 1) * m.Ap > kn) kn = (size_t)(m.H2 + 1) * m.Ap;
  return (size_t)M * (m.F + 2 * m.H1 + 2 * m.H2 + m.Ap + m.H1 + m.H2) + (size_t)M * 3 * 2 +
         nc * kn + 64;
}

}  // namespace bsim
