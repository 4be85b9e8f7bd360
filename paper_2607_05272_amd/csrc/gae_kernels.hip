// gae_kernels.hip -- discounted returns / GAE (paper Sec. 4.3) over a [T][E] trajectory.
//
// One lane per environment walks t = T-1 .. 0:
//   delta_t = (r_t + gamma V_{t+1}) - V_t,  A_t = delta_t + (gamma*lambda) A_{t+1},
//   A_T = 0,  R_t = A_t + V_t,
// in fp64 with V read as fp32 and widened. At step t the lanes of a wave read 64
// consecutive environments of row t, so every load and store is coalesced; the recurrence
// is a two-operation dependency chain per step and the workload is HBM-streaming.
#include "params.hpp"

namespace bsim {
namespace {

__global__ __launch_bounds__(256) void gae_k(int T, int E, const double* __restrict__ r,
                                             const float* __restrict__ v, double gamma, double gl,
                                             double* __restrict__ adv, double* __restrict__ ret) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= E) return;
  const size_t sE = (size_t)E;
  double a = 0.0;
  double vn = v ? (double)v[(size_t)T * sE + e] : 0.0;
  for (int t = T - 1; t >= 0; --t) {
    const size_t i = (size_t)t * sE + e;
    const double vt = v ? (double)v[i] : 0.0;
    const double delta = (r[i] + gamma * vn) - vt;
    a = delta + gl * a;
    adv[i] = a;
    ret[i] = a + vt;
    vn = vt;
  }
}

}  // namespace

hipError_t launch_gae(int T, int E, const double* r, const float* v, double gamma, double lam,
                      double* adv, double* ret, hipStream_t st) {
  const double gl = gamma * lam;
  hipLaunchKernelGGL(gae_k, dim3((E + 255) / 256), dim3(256), 0, st, T, E, r, v, gamma, gl, adv,
                     ret);
  return hipGetLastError();
}

}  // namespace bsim
