// prim_kernels.hip -- the library's device primitives evaluated elementwise, so that their
// bit identity with a host implementation can be checked directly: the Philox4x32-10 block
// of a counter, the deterministic fp64 log/exp/cos the simulator uses for its draws, and
// fp64 square root and division (which the sampling code relies on being correctly rounded).
#include "devmath.hpp"
#include "params.hpp"

namespace bsim {
namespace {

__global__ __launch_bounds__(256) void prim_philox_k(int64_t n, uint64_t key,
                                                     const uint32_t* __restrict__ ctr,
                                                     uint32_t* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint32_t* c = ctr + 4 * i;
  const u32x4 r = philox(c[0], c[1], c[2], c[3], (uint32_t)key, (uint32_t)(key >> 32));
  out[4 * i] = r.x;
  out[4 * i + 1] = r.y;
  out[4 * i + 2] = r.z;
  out[4 * i + 3] = r.w;
}

__global__ __launch_bounds__(256) void prim_f64_k(int kind, int64_t n,
                                                  const double* __restrict__ in,
                                                  double* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  double r;
  switch (kind) {
    case PRIM_LOG: r = dlog(in[i]); break;
    case PRIM_EXP: r = dexp(in[i]); break;
    case PRIM_COS: r = dcos(in[i]); break;
    case PRIM_SQRT: r = sqrt(in[i]); break;
    default: r = in[2 * i] / in[2 * i + 1]; break;  // PRIM_DIV
  }
  out[i] = r;
}

}  // namespace

hipError_t launch_primitive(int kind, int64_t n, uint64_t key, const void* in, void* out,
                            hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const dim3 grid((unsigned)((n + 255) / 256)), block(256);
  if (kind == PRIM_PHILOX)
    hipLaunchKernelGGL(prim_philox_k, grid, block, 0, st, n, key,
                       static_cast<const uint32_t*>(in), static_cast<uint32_t*>(out));
  else
    hipLaunchKernelGGL(prim_f64_k, grid, block, 0, st, kind, n, static_cast<const double*>(in),
                       static_cast<double*>(out));
  return hipGetLastError();
}

}  // namespace bsim
