// train_kernels.hip -- parameter update of the policy (paper Sec. 4.3): Adam on fp32 master
// parameters (Kingma & Ba, "Adam: a method for stochastic optimization", ICLR 2015,
// Algorithm 1) and the conversions between the master parameters and the policy's weights.
//
// The master parameters use the gradient layout: W1 [F][H1], b1 [H1], W2 [H1][H2], b2 [H2],
// W3 [H2][A'], b3 [A'] back to back (fp32). The policy's weights are the ABI buffer (matrices
// in the element type, bf16 by round-to-nearest-even or fp32; biases fp32; each block at its
// layout offset).
#include "devmath.hpp"
#include "params.hpp"

namespace bsim {
namespace {

__global__ __launch_bounds__(256) void adam_k(float* __restrict__ p, const float* __restrict__ g,
                                              float* __restrict__ m, float* __restrict__ v, size_t n,
                                              float lr, float b1, float b2, float eps, float bc1,
                                              float bc2) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    const float gi = g[i];
    const float mi = b1 * m[i] + (1.0f - b1) * gi;
    const float vi = b2 * v[i] + (1.0f - b2) * (gi * gi);
    m[i] = mi;
    v[i] = vi;
    const float mhat = mi / bc1, vhat = vi / bc2;
    p[i] = p[i] - lr * mhat / (sqrtf(vhat) + eps);
  }
}

constexpr int kMaxSegs = 14;
struct Segs {
  int n;                   // segments in use (6 for the MLP, 14 for the attention policy)
  size_t poff[kMaxSegs];   // offset in the parameter vector
  size_t woff[kMaxSegs];   // byte offset in the weight buffer
  size_t len[kMaxSegs];
  int matrix[kMaxSegs];
};

// one thread per parameter; seg found by a short scan of the segment starts
__device__ __forceinline__ int seg_of(const Segs& s, size_t i) {
  int k = 0;
#pragma unroll
  for (int j = 1; j < kMaxSegs; ++j)
    if (j < s.n && i >= s.poff[j]) k = j;
  return k;
}

__global__ __launch_bounds__(256) void export_k(Segs s, size_t n, int bf16,
                                                const float* __restrict__ p,
                                                unsigned char* __restrict__ w) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int k = seg_of(s, i);
  const size_t j = i - s.poff[k];
  if (s.matrix[k] && bf16) reinterpret_cast<uint16_t*>(w + s.woff[k])[j] = bf16_bits(p[i]);
  else reinterpret_cast<float*>(w + s.woff[k])[j] = p[i];
}

__global__ __launch_bounds__(256) void import_k(Segs s, size_t n, int bf16,
                                                const unsigned char* __restrict__ w,
                                                float* __restrict__ p) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int k = seg_of(s, i);
  const size_t j = i - s.poff[k];
  if (s.matrix[k] && bf16) p[i] = bf16_to_f32(reinterpret_cast<const uint16_t*>(w + s.woff[k])[j]);
  else p[i] = reinterpret_cast<const float*>(w + s.woff[k])[j];
}

Segs segments(const MlpParams& m, const size_t off[6]) {
  Segs s;
  s.n = 6;
  const size_t len[6] = {(size_t)m.F * m.H1, (size_t)m.H1, (size_t)m.H1 * m.H2, (size_t)m.H2,
                         (size_t)m.H2 * m.Ap, (size_t)m.Ap};
  size_t acc = 0;
  for (int k = 0; k < 6; ++k) {
    s.poff[k] = acc;
    s.woff[k] = off[k];
    s.len[k] = len[k];
    s.matrix[k] = (k % 2) == 0;
    acc += len[k];
  }
  return s;
}

// the attention policy: fourteen fp32 arrays (nothing is rounded to bf16)
Segs attn_segments(const AttnParams& p, const size_t off[14]) {
  Segs s;
  s.n = 14;
  int po[14];
  const int P = attn_param_count(p, po);
  for (int k = 0; k < 14; ++k) {
    s.poff[k] = (size_t)po[k];
    s.woff[k] = off[k];
    s.len[k] = (size_t)((k < 13 ? po[k + 1] : P) - po[k]);
    s.matrix[k] = 0;
  }
  return s;
}

size_t total(const Segs& s) { return s.poff[s.n - 1] + s.len[s.n - 1]; }

}  // namespace

hipError_t launch_adam(float* params, const float* grads, float* m, float* v, size_t n, float lr,
                       float b1, float b2, float eps, float bc1, float bc2, hipStream_t st) {
  const unsigned blocks = (unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  hipLaunchKernelGGL(adam_k, dim3(blocks > 0 ? blocks : 1), dim3(256), 0, st, params, grads, m, v,
                     n, lr, b1, b2, eps, bc1, bc2);
  return hipGetLastError();
}

hipError_t launch_export_weights(const MlpParams& m, const float* params, void* d_weights,
                                 const size_t off[6], hipStream_t st) {
  const Segs s = segments(m, off);
  const size_t n = total(s);
  hipLaunchKernelGGL(export_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, s, n, m.bf16,
                     params, static_cast<unsigned char*>(d_weights));
  return hipGetLastError();
}

hipError_t launch_export_attn(const AttnParams& p, const float* params, void* d_weights,
                              const size_t off[14], hipStream_t st) {
  const Segs s = attn_segments(p, off);
  const size_t n = total(s);
  hipLaunchKernelGGL(export_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, s, n, 0,
                     params, static_cast<unsigned char*>(d_weights));
  return hipGetLastError();
}

hipError_t launch_import_attn(const AttnParams& p, const void* d_weights, const size_t off[14],
                              float* params, hipStream_t st) {
  const Segs s = attn_segments(p, off);
  const size_t n = total(s);
  hipLaunchKernelGGL(import_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, s, n, 0,
                     static_cast<const unsigned char*>(d_weights), params);
  return hipGetLastError();
}

hipError_t launch_import_weights(const MlpParams& m, const void* d_weights, const size_t off[6],
                                 float* params, hipStream_t st) {
  const Segs s = segments(m, off);
  const size_t n = total(s);
  hipLaunchKernelGGL(import_k, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, s, n, m.bf16,
                     static_cast<const unsigned char*>(d_weights), params);
  return hipGetLastError();
}

}  // namespace bsim
