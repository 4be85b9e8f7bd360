// mlp_kernels.hip -- the policy MLP kernels (paper Sec. 4.2), fused with action sampling:
// policy_k (fp32 policies) and policy_bf16_k (bf16 policies), each one workgroup's share of
// the batch as described in policy_dev.hpp, plus the weight repacking and initialisation.
#include <type_traits>

#include "policy_dev.hpp"

namespace bsim {
namespace {

template <class M, int FP, int H1, int H2, int AP, int RT, bool DBG>
__global__ __launch_bounds__(kThreads) void policy_k(MlpParams m, const float* __restrict__ obs,
                                                     const uint64_t* __restrict__ seedp, uint32_t step,
                                                     uint8_t* __restrict__ act,
                                                     float* __restrict__ logp,
                                                     float* __restrict__ value,
                                                     float* __restrict__ logits,
                                                     float* __restrict__ hid) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  policy_tile_f32<M, FP, H1, H2, AP, RT, DBG>(m, obs, *seedp, step, act, logp, value, logits, hid,
                                              smem, blockIdx.x * Shape<M, FP, H1, H2, AP, RT>::ROWS);
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
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  policy_tile_bf16<FP, H1, H2, AP, RT, NW, TPW, DBG, AC>(m, obs, obs_bf, *seedp, step, act, logp, value,
                                                       logits, hid, smem, blockIdx.x * (16 * RT));
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
