// ppo_kernels.hip -- one policy-gradient minibatch of the MLP policy (paper Sec. 4.3): gather,
// forward, loss (PPO clipped surrogate, or REINFORCE with a learned baseline) + value +
// entropy, and its gradient with respect to every policy weight.
//
// M samples (t, env) are drawn with replacement: sample m takes u from the MINIBATCH block at
// counter (m, 0xFFFFFFFD, MINIBATCH<<24, 0) and index floor(u * T * E). The forward repeats
// the rollout policy's rounding points (every layer input rounded to bf16) with fp32
// sums and saves pre-activations; gradients pass through the bf16 roundings as the
// identity. Loss
//   L = -mean(min(rho A, clip(rho, 1-eps, 1+eps) A)) + c_v mean((V - R)^2) - c_h mean(H),
//   rho = exp(logp_new(a) - logp_old), H the entropy of the action distribution; REINFORCE
//   replaces the first term by -mean(A log pi(a|s)) with A held constant.
//
// The dense products are plain GEMMs and run in rocBLAS: the forward as bf16 x bf16 -> fp32
// products when the policy is bf16 (the products of bf16 values are exact, the sums fp32, as in
// the rollout kernel), as fp32 products otherwise; the backward through the activations and the
// weight gradients as fp32 products against fp32 copies of the weights. A layer's weight and
// bias gradients come out of one product [A | 1]^T dZ (the saved activations carry a ones
// column), whose K+1 rows land on the contiguous W, b pair of the gradient layout. The library
// runs with atomics disabled, so its sums are taken in an order fixed by the shapes and the
// gradients are deterministic. The elementwise steps around the products (index draw and
// gather, bias + GELU + bf16 rounding, the per-sample loss and its gradient, GELU') are the
// small kernels below.
#include <rocblas/rocblas.h>

#include <cstdio>

#include "devmath.hpp"
#include "params.hpp"

namespace bsim {
namespace {

constexpr int kThr = 256;
constexpr int kGs = 16;   // samples per workgroup of the gather

__device__ __forceinline__ float bf16_round(float f) { return bf16_to_f32(bf16_bits(f)); }
__device__ __forceinline__ float gelu_exact(float z) {
  return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));
}
__device__ __forceinline__ float gelu_grad(float z) {
  return 0.5f * (1.0f + erff(z * 0.70710678118654752f)) + z * expf(-0.5f * z * z) * 0.39894228040143268f;
}

// Index draw and gather: the first kGs threads draw their sample's index, then the workgroup
// copies the samples' observations (bf16-rounded in bf16 mode) into xa [M][F+1], whose last
// column is 1, and their bf16 bits into xb [M][F].
__global__ __launch_bounds__(kThr) void mb_gather_k(uint64_t seed, int M, int T, int E, int F,
                                                    int bf16, const float* __restrict__ obs,
                                                    int64_t* __restrict__ idx,
                                                    int64_t* __restrict__ idx_out,
                                                    float* __restrict__ xa,
                                                    uint16_t* __restrict__ xb) {
  __shared__ int ts_[kGs], es_[kGs];
  const int m0 = blockIdx.x * kGs;
  const int ns = M - m0 < kGs ? M - m0 : kGs;
  if ((int)threadIdx.x < ns) {
    const int m = m0 + threadIdx.x;
    const u32x4 w = draw(seed, (uint32_t)m, 0xFFFFFFFDu, P_MINIBATCH, 0, 0);
    const double n = (double)T * (double)E;
    long long i = (long long)(unit(w.x, w.y) * n);
    if (i > (long long)T * E - 1) i = (long long)T * E - 1;
    ts_[threadIdx.x] = (int)(i / E);
    es_[threadIdx.x] = (int)(i % E);
    idx[m] = i;
    if (idx_out) idx_out[m] = i;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < ns * (F + 1); q += kThr) {
    const int s = q / (F + 1), f = q % (F + 1);
    const size_t m = (size_t)(m0 + s);
    if (f == F) {
      xa[m * (F + 1) + F] = 1.0f;
      continue;
    }
    float v = obs[((size_t)ts_[s] * F + f) * E + es_[s]];
    if (bf16) {
      v = bf16_round(v);
      xb[m * F + f] = bf16_bits(v);
    }
    xa[m * (F + 1) + f] = v;
  }
}

// z [M][N] holds x W; adds the bias in place, then h = GELU(z) (bf16-rounded in bf16 mode)
// into ha [M][N+1] with a ones column and, in bf16 mode, its bits into hb [M][N].
__global__ __launch_bounds__(kThr) void mb_bias_gelu_k(int M, int N, int bf16,
                                                       const float* __restrict__ b,
                                                       float* __restrict__ z,
                                                       float* __restrict__ ha,
                                                       uint16_t* __restrict__ hb) {
  const uint32_t n = (uint32_t)M * (uint32_t)(N + 1);
  for (uint32_t q = blockIdx.x * kThr + threadIdx.x; q < n; q += gridDim.x * kThr) {
    const uint32_t m = q / (uint32_t)(N + 1), j = q % (uint32_t)(N + 1);
    if (j == (uint32_t)N) {
      ha[q] = 1.0f;
      continue;
    }
    const uint32_t zi = m * (uint32_t)N + j;
    const float v = z[zi] + b[j];
    z[zi] = v;
    float h = gelu_exact(v);
    if (bf16) {
      h = bf16_round(h);
      hb[zi] = bf16_bits(h);
    }
    ha[q] = h;
  }
}

struct LossArgs {
  int A, Ap, M, reinforce;
  float clip, c_v, c_h;
  float* out;                        // [M][Ap]: h2 W3 on entry, the outputs (with b3) on exit
  const float* b3;
  const int64_t* idx;                // [M] sampled t * E + env
  const uint8_t* act;
  const float* logp_old;
  const double* adv;
  const double* ret;
  float* dout;                       // [M][Ap] dL/d(output)
  double* terms;                     // [M][3] policy, value, entropy per sample
  uint32_t* err;
};

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

// Loss terms and the loss gradient with respect to the outputs, one wavefront per sample:
// lane i holds outputs i and i + 64 (A' <= 128), max and sums are butterfly reductions.
constexpr int kLossWaves = kThr / 64;
__global__ __launch_bounds__(kThr) void mb_loss_k(LossArgs a) {
  const int m = blockIdx.x * kLossWaves + threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  if (m >= a.M) return;   // uniform per wavefront
  float* l = a.out + (size_t)m * a.Ap;
  float* d = a.dout + (size_t)m * a.Ap;
  double* tm = a.terms + (size_t)m * 3;
  const int i0 = lane, i1 = lane + 64;
  const float v0 = i0 < a.Ap ? l[i0] + a.b3[i0] : 0.0f;
  const float v1 = i1 < a.Ap ? l[i1] + a.b3[i1] : 0.0f;
  if (i0 < a.Ap) l[i0] = v0;
  if (i1 < a.Ap) l[i1] = v1;
  const size_t ti = (size_t)a.idx[m];
  const int act = a.act[ti];
  if (act >= a.A) {  // invalid stored action: flag it, the sample contributes nothing
    if (lane == 0) {
      atomicOr(a.err, ERR_ACTION);
      tm[0] = tm[1] = tm[2] = 0.0;
    }
    if (i0 < a.Ap) d[i0] = 0.0f;
    if (i1 < a.Ap) d[i1] = 0.0f;
    return;
  }
  const bool in0 = i0 < a.A, in1 = i1 < a.A;
  const float adv = (float)a.adv[ti], ret = (float)a.ret[ti];
  const float mx = wave_max(fmaxf(in0 ? v0 : -INFINITY, in1 ? v1 : -INFINITY));
  const float S = wave_sum((in0 ? expf(v0 - mx) : 0.0f) + (in1 ? expf(v1 - mx) : 0.0f));
  const float lS = logf(S);
  const float lp0 = (v0 - mx) - lS, lp1 = (v1 - mx) - lS;
  const float p0 = in0 ? expf(lp0) : 0.0f, p1 = in1 ? expf(lp1) : 0.0f;
  const float H = -wave_sum(p0 * (in0 ? lp0 : 0.0f) + p1 * (in1 ? lp1 : 0.0f));
  // the taken action's logit and the value output, broadcast from the lanes that hold them
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
    float g = in0 ? -dlogp * p0 + a.c_h * invM * p0 * (lp0 + H) : dv;
    if (i0 == act) g += dlogp;
    d[i0] = g;
  }
  if (i1 < a.Ap) {
    float g = in1 ? -dlogp * p1 + a.c_h * invM * p1 * (lp1 + H) : dv;
    if (i1 == act) g += dlogp;
    d[i1] = g;
  }
  if (lane == 0) {
    tm[0] = (double)pterm;
    tm[1] = (double)(v - ret) * (double)(v - ret);
    tm[2] = (double)H;
  }
}

// d *= GELU'(z), elementwise over n entries
__global__ __launch_bounds__(kThr) void mb_gelu_bwd_k(uint32_t n, const float* __restrict__ z,
                                                      float* __restrict__ d) {
  for (uint32_t q = blockIdx.x * kThr + threadIdx.x; q < n; q += gridDim.x * kThr)
    d[q] = d[q] * gelu_grad(z[q]);
}

// fp32 copy of bf16 weights
__global__ __launch_bounds__(kThr) void mb_widen_k(uint32_t n, const uint16_t* __restrict__ w,
                                                   float* __restrict__ o) {
  for (uint32_t q = blockIdx.x * kThr + threadIdx.x; q < n; q += gridDim.x * kThr)
    o[q] = bf16_to_f32(w[q]);
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

unsigned grid_for(size_t n) {
  const size_t g = (n + kThr - 1) / kThr;
  return (unsigned)(g < 4096 ? (g ? g : 1) : 4096);
}

// the scratch carve-up; every piece starts on a 256-byte boundary
struct MbScratch {
  int64_t* idx;
  float *xa, *h1a, *h2a, *z1, *z2, *out, *dout, *d1, *d2, *w2f, *w3f;
  uint16_t *xb, *h1b, *h2b;
  double* terms;
};

size_t carve(const MlpParams& m, int M, void* base, MbScratch* s) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    void* p = base ? static_cast<unsigned char*>(base) + off : nullptr;
    off += (bytes + 255) & ~(size_t)255;
    return p;
  };
  const size_t Ms = (size_t)M;
  MbScratch t;
  t.idx = static_cast<int64_t*>(take(Ms * sizeof(int64_t)));
  t.xa = static_cast<float*>(take(Ms * (m.F + 1) * sizeof(float)));
  t.h1a = static_cast<float*>(take(Ms * (m.H1 + 1) * sizeof(float)));
  t.h2a = static_cast<float*>(take(Ms * (m.H2 + 1) * sizeof(float)));
  t.z1 = static_cast<float*>(take(Ms * m.H1 * sizeof(float)));
  t.z2 = static_cast<float*>(take(Ms * m.H2 * sizeof(float)));
  t.out = static_cast<float*>(take(Ms * m.Ap * sizeof(float)));
  t.dout = static_cast<float*>(take(Ms * m.Ap * sizeof(float)));
  t.d1 = static_cast<float*>(take(Ms * m.H1 * sizeof(float)));
  t.d2 = static_cast<float*>(take(Ms * m.H2 * sizeof(float)));
  t.terms = static_cast<double*>(take(Ms * 3 * sizeof(double)));
  if (m.bf16) {
    t.xb = static_cast<uint16_t*>(take(Ms * m.F * sizeof(uint16_t)));
    t.h1b = static_cast<uint16_t*>(take(Ms * m.H1 * sizeof(uint16_t)));
    t.h2b = static_cast<uint16_t*>(take(Ms * m.H2 * sizeof(uint16_t)));
    t.w2f = static_cast<float*>(take((size_t)m.H1 * m.H2 * sizeof(float)));
    t.w3f = static_cast<float*>(take((size_t)m.H2 * m.Ap * sizeof(float)));
  } else {
    t.xb = t.h1b = t.h2b = nullptr;
    t.w2f = t.w3f = nullptr;
  }
  if (s) *s = t;
  return off;
}

// rocBLAS is column-major: a row-major [R][C] array with leading dimension ld is its C x R
// column-major view, so each row-major product below is issued with its factors swapped.
struct Gemm {
  rocblas_handle h;
  const char* failed = nullptr;   // the product that failed
  rocblas_status status = rocblas_status_success;

  bool ok(rocblas_status s, const char* what) {
    if (s != rocblas_status_success && !failed) {
      failed = what;
      status = s;
    }
    return s == rocblas_status_success;
  }
  // Z [M][N] = In [M][K] (leading dimension ldi) W [K][N]
  bool fwd(bool bf16, int M, int K, int N, const void* in, int ldi, const void* w, float* z,
           const char* what) {
    const float one = 1.0f, zero = 0.0f;
    if (bf16)
      return ok(rocblas_gemm_ex(h, rocblas_operation_none, rocblas_operation_none, N, M, K, &one, w,
                                rocblas_datatype_bf16_r, N, in, rocblas_datatype_bf16_r, ldi, &zero,
                                z, rocblas_datatype_f32_r, N, z, rocblas_datatype_f32_r, N,
                                rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0,
                                rocblas_gemm_flags_none),
                what);
    return ok(rocblas_sgemm(h, rocblas_operation_none, rocblas_operation_none, N, M, K, &one,
                            static_cast<const float*>(w), N, static_cast<const float*>(in), ldi,
                            &zero, z, N),
              what);
  }
  // dIn [M][K] = dZ [M][N] W^T, W [K][N]
  bool bwd(int M, int K, int N, const float* dz, const float* w, float* din, const char* what) {
    const float one = 1.0f, zero = 0.0f;
    return ok(rocblas_sgemm(h, rocblas_operation_transpose, rocblas_operation_none, K, M, N, &one,
                            w, N, dz, N, &zero, din, K),
              what);
  }
  // G [K+1][N] = Aaug^T dZ, Aaug [M][K+1] (the activations and a ones column), dZ [M][N]
  bool wgrad(int M, int K, int N, const float* aaug, const float* dz, float* g, const char* what) {
    const float one = 1.0f, zero = 0.0f;
    return ok(rocblas_sgemm(h, rocblas_operation_none, rocblas_operation_transpose, N, K + 1, M,
                            &one, dz, N, aaug, K + 1, &zero, g, N),
              what);
  }
};

thread_local char g_blas_msg[192];

}  // namespace

void* mb_blas_create(const char** why) {
  rocblas_handle h = nullptr;
  rocblas_status s = rocblas_create_handle(&h);
  if (s == rocblas_status_success) s = rocblas_set_atomics_mode(h, rocblas_atomics_not_allowed);
  if (s == rocblas_status_success) s = rocblas_set_pointer_mode(h, rocblas_pointer_mode_host);
  if (s != rocblas_status_success) {
    if (h) (void)rocblas_destroy_handle(h);
    std::snprintf(g_blas_msg, sizeof g_blas_msg, "rocBLAS handle set-up failed: %s",
                  rocblas_status_to_string(s));
    if (why) *why = g_blas_msg;
    return nullptr;
  }
  return h;
}

void mb_blas_destroy(void* blas) {
  if (blas) (void)rocblas_destroy_handle(static_cast<rocblas_handle>(blas));
}

size_t ppo_scratch_bytes(const MlpParams& m, int M) { return carve(m, M, nullptr, nullptr); }

hipError_t launch_ppo(const MlpParams& m, const void* d_weights, const size_t off[6], int T,
                      const float* obs, const uint8_t* act, const float* logp_old,
                      const double* adv, const double* ret, int M, uint64_t seed, float clip,
                      float c_v, float c_h, int reinforce, void* scratch, double* loss_out,
                      float* grads, int64_t* idx_out, uint32_t* err, void* blas,
                      const char** why, hipStream_t st) {
  if (M < 1 || !blas || m.Ap > 128) return hipErrorInvalidValue;
  const unsigned char* wb = static_cast<const unsigned char*>(d_weights);
  const void* w1 = wb + off[0];
  const float* b1 = reinterpret_cast<const float*>(wb + off[1]);
  const void* w2 = wb + off[2];
  const float* b2 = reinterpret_cast<const float*>(wb + off[3]);
  const void* w3 = wb + off[4];
  const float* b3 = reinterpret_cast<const float*>(wb + off[5]);
  MbScratch s;
  carve(m, M, scratch, &s);
  const bool bf = m.bf16 != 0;
  Gemm g{static_cast<rocblas_handle>(blas)};
  if (!g.ok(rocblas_set_stream(g.h, st), "set_stream")) goto blas_fail;
  {
    hipLaunchKernelGGL(mb_gather_k, dim3((unsigned)((M + kGs - 1) / kGs)), dim3(kThr), 0, st, seed,
                       M, T, m.E, m.F, m.bf16, obs, s.idx, idx_out, s.xa, s.xb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (bf) {
      const uint32_t n2 = (uint32_t)m.H1 * m.H2, n3 = (uint32_t)m.H2 * m.Ap;
      hipLaunchKernelGGL(mb_widen_k, dim3(grid_for(n2)), dim3(kThr), 0, st, n2,
                         static_cast<const uint16_t*>(w2), s.w2f);
      hipLaunchKernelGGL(mb_widen_k, dim3(grid_for(n3)), dim3(kThr), 0, st, n3,
                         static_cast<const uint16_t*>(w3), s.w3f);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const float* w2f = bf ? s.w2f : static_cast<const float*>(w2);
    const float* w3f = bf ? s.w3f : static_cast<const float*>(w3);
    // forward: three products, each followed by its bias (and GELU)
    if (!g.fwd(bf, M, m.F, m.H1, bf ? (const void*)s.xb : s.xa, bf ? m.F : m.F + 1, w1, s.z1,
               "forward layer 1"))
      goto blas_fail;
    hipLaunchKernelGGL(mb_bias_gelu_k, dim3(grid_for((size_t)M * (m.H1 + 1))), dim3(kThr), 0, st,
                       M, m.H1, m.bf16, b1, s.z1, s.h1a, s.h1b);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (!g.fwd(bf, M, m.H1, m.H2, bf ? (const void*)s.h1b : s.h1a, bf ? m.H1 : m.H1 + 1, w2, s.z2,
               "forward layer 2"))
      goto blas_fail;
    hipLaunchKernelGGL(mb_bias_gelu_k, dim3(grid_for((size_t)M * (m.H2 + 1))), dim3(kThr), 0, st,
                       M, m.H2, m.bf16, b2, s.z2, s.h2a, s.h2b);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (!g.fwd(bf, M, m.H2, m.Ap, bf ? (const void*)s.h2b : s.h2a, bf ? m.H2 : m.H2 + 1, w3, s.out,
               "forward layer 3"))
      goto blas_fail;
    LossArgs la;
    la.A = m.A; la.Ap = m.Ap; la.M = M; la.reinforce = reinforce;
    la.clip = clip; la.c_v = c_v; la.c_h = c_h;
    la.out = s.out; la.b3 = b3; la.idx = s.idx; la.act = act; la.logp_old = logp_old;
    la.adv = adv; la.ret = ret; la.dout = s.dout; la.terms = s.terms; la.err = err;
    hipLaunchKernelGGL(mb_loss_k, dim3((unsigned)((M + kLossWaves - 1) / kLossWaves)), dim3(kThr), 0,
                       st, la);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // gradient layout: W1 [F][H1], b1, W2 [H1][H2], b2, W3 [H2][Ap], b3 (fp32, contiguous)
    float* gw1 = grads;
    float* gw2 = gw1 + (size_t)(m.F + 1) * m.H1;
    float* gw3 = gw2 + (size_t)(m.H1 + 1) * m.H2;
    if (!g.wgrad(M, m.H2, m.Ap, s.h2a, s.dout, gw3, "weight gradient layer 3")) goto blas_fail;
    if (!g.bwd(M, m.H2, m.Ap, s.dout, w3f, s.d2, "backward layer 3")) goto blas_fail;
    const uint32_t n2 = (uint32_t)M * m.H2, n1 = (uint32_t)M * m.H1;
    hipLaunchKernelGGL(mb_gelu_bwd_k, dim3(grid_for(n2)), dim3(kThr), 0, st, n2, s.z2, s.d2);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (!g.wgrad(M, m.H1, m.H2, s.h1a, s.d2, gw2, "weight gradient layer 2")) goto blas_fail;
    if (!g.bwd(M, m.H1, m.H2, s.d2, w2f, s.d1, "backward layer 2")) goto blas_fail;
    hipLaunchKernelGGL(mb_gelu_bwd_k, dim3(grid_for(n1)), dim3(kThr), 0, st, n1, s.z1, s.d1);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (!g.wgrad(M, m.F, m.H1, s.xa, s.d1, gw1, "weight gradient layer 1")) goto blas_fail;
    hipLaunchKernelGGL(ppo_loss_k, dim3(1), dim3(kSumThr), 0, st, s.terms, M, c_v, c_h, loss_out);
    return hipGetLastError();
  }
blas_fail:
  std::snprintf(g_blas_msg, sizeof g_blas_msg, "rocBLAS %s: %s", g.failed ? g.failed : "?",
                rocblas_status_to_string(g.status));
  if (why) *why = g_blas_msg;
  return hipErrorLaunchFailure;
}

hipError_t launch_pg_loss(const double* terms, int M, float c_v, float c_h, double* out,
                          hipStream_t st) {
  hipLaunchKernelGGL(ppo_loss_k, dim3(1), dim3(kSumThr), 0, st, terms, M, c_v, c_h, out);
  return hipGetLastError();
}

}  // namespace bsim
