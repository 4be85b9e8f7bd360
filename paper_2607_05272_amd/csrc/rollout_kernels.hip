// rollout_kernels.hip -- the fused rollout of a small batch: one launch runs every tick of a
// rollout, the policy (paper Sec. 4.2) and the learned system's tick (Sec. 3.1, Sec. 4.1)
// alternating inside each workgroup.
//
// With a few thousand environments the per-tick kernels are bound by latency, not by work: a
// launch's start, its first loads of the state and its drain cost more than its arithmetic,
// twice per tick. Environments never interact, so a workgroup can own a tile of them for the
// whole rollout: per tick the policy over its tile (all waves), a workgroup barrier, the tick
// of the same environments (TW waves, ROWS / TW lanes each), another barrier. The tick writes
// the observation the next policy reads through global memory, which the barrier orders
// within the workgroup; nothing is ever exchanged between workgroups, so they run without any
// grid-wide synchronisation (a grid larger than the chip holds simply runs in rounds).
// Both phases are the per-tick kernels' own device code (policy_dev.hpp, sim_dev.hpp), so
// every output is bit-identical to the per-tick launches'.
#include "policy_dev.hpp"
#include "sim_dev.hpp"

namespace bsim {
namespace {

// fp32 policy on one 16-environment tile (4 waves)
template <int FP, int H1, int H2, int AP>
struct PolicyF32 {
  static constexpr int ROWS = 16;
  static constexpr bool kBf16 = false;
  static constexpr int kWavesPerEU = 1;
  typedef Shape<F32Mode, FP, H1, H2, AP, 1> Sh;
  static constexpr size_t LDS = Sh::LDS;
  __device__ static void run(const MlpParams& m, const float* obs, const uint32_t*, uint64_t seed,
                             uint32_t step, uint8_t* act, float* logp, float* value,
                             unsigned char* smem, int e0) {
    policy_tile_f32<F32Mode, FP, H1, H2, AP, 1, false>(m, obs, seed, step, act, logp, value,
                                                       nullptr, nullptr, smem, e0);
  }
};

// bf16 policy on one 16 RT-environment tile (4 waves, one output tile per pass); AC as in
// policy_tile_bf16; WPE: waves per SIMD the kernel is compiled for (2: at most 256 VGPRs, two
// workgroups per CU)
template <int FP, int H1, int H2, int AP, int RT, int AC, int WPE = 1>
struct PolicyBf16 {
  static constexpr int ROWS = 16 * RT;
  static constexpr bool kBf16 = true;
  static constexpr int kWavesPerEU = WPE;
  typedef BigShape<FP, H1, H2, AP, RT, 4> Sh;
  static constexpr size_t LDS = Sh::LDS;
  __device__ static void run(const MlpParams& m, const float* obs, const uint32_t* obs_bf,
                             uint64_t seed, uint32_t step, uint8_t* act, float* logp,
                             float* value, unsigned char* smem, int e0) {
    policy_tile_bf16<FP, H1, H2, AP, RT, 4, 1, false, AC>(m, obs, obs_bf, seed, step, act, logp,
                                                         value, nullptr, nullptr, smem, e0);
  }
};

// T ticks from k0 for the workgroup's ROWS environments; TW waves take the tick, ROWS / TW
// environments each. Trajectory rows as in the per-tick rollout: act, logp, value, rew and
// rchk [T][E], obs [T + 1][F][E] from row 1 (row 0, the observation before the first tick, is
// not written here), value row T for the observation after the last tick. With a bf16 policy
// the ticks write the observation's bf16 pairs (packed before the launch) and the last one
// also the fp32 observation.
template <int CM, int TW, class Pol>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(Pol::kWavesPerEU))) void rollout_fused_k(SimParams p, EnvState g, MlpParams m,
                                                       uint32_t k0, int T, RolloutOut o) {
  static_assert(Pol::ROWS % TW == 0 && TW <= 4, "tick lanes per wave");
  constexpr int LPW = Pol::ROWS / TW;
  __shared__ Stage<kStageLearned> stage[TW];
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const uint64_t seed = *g.seed;   // the episode seed, written by reset_k
  const int e0 = blockIdx.x * Pol::ROWS;
  const int wave = threadIdx.x >> 6;
  const size_t E = (size_t)p.E, F = (size_t)p.F;
  const uint32_t* obs_bf = Pol::kBf16 ? g.obs_bf : nullptr;
  for (int i = 0; i < T; ++i) {
    const uint32_t k = k0 + (uint32_t)i;
    const size_t row = (size_t)i * E;
    Pol::run(m, g.obs, obs_bf, seed, k, o.act + row, o.logp ? o.logp + row : nullptr,
             o.value ? o.value + row : nullptr, smem, e0);
    __syncthreads();   // the tile's actions are written
    if (wave < TW) {
      const int mode = !Pol::kBf16 ? kObsF32 : i + 1 < T ? kObsBf16 : kObsF32 | kObsBf16;
      learned_tick<CM, false>(p, g, seed, k, e0 + wave * LPW, LPW, stage[wave], o.act + row,
                              o.obs ? o.obs + (size_t)(i + 1) * F * E : nullptr, mode,
                              o.rew ? o.rew + row : nullptr, o.rchk ? o.rchk + row : nullptr);
    }
    __syncthreads();   // the tile's next observation and state are written
  }
  if (o.value)
    Pol::run(m, g.obs, obs_bf, seed, k0 + (uint32_t)T, nullptr, nullptr, o.value + (size_t)T * E,
             smem, e0);
}

template <int CM, int TW, class Pol>
hipError_t launch_fused(const SimParams& p, const EnvState& s, const MlpParams& m, uint32_t k0,
                        int T, const RolloutOut& o, hipStream_t st) {
  static_assert(Pol::LDS + sizeof(Stage<kStageLearned>) * TW <= 160 * 1024, "LDS budget");
  auto kern = rollout_fused_k<CM, TW, Pol>;
  static bool attr = false;   // dynamic LDS beyond the default limit, once per kernel
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute((const void*)kern,
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)Pol::LDS);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const dim3 grid((p.E + Pol::ROWS - 1) / Pol::ROWS), block(256);
  hipLaunchKernelGGL(kern, grid, block, Pol::LDS, st, p, s, m, k0, T, o);
  return hipGetLastError();
}

template <int CM, int TW, class P>
struct FusedTag {
  static constexpr int kCM = CM, kTW = TW;
  typedef P Pol;
};
template <class P>
struct PolTag {
  typedef P Pol;
};

// f(FusedTag<CM, TW, Pol>{}) for the configuration's fused kernel: the policy network's shape
// (and, where it is the configurations' own, its action count compiled into the sampler), the
// class count; hipErrorNotSupported for a network without one
template <class F>
hipError_t with_fused(const SimParams& p, const MlpParams& m, F&& f) {
  auto by_classes = [&](auto pol) -> hipError_t {
    typedef typename decltype(pol)::Pol Pol;
    if (p.C <= 1) return f(FusedTag<1, 4, Pol>{});
    if (p.C <= 2) return f(FusedTag<2, 4, Pol>{});
    return f(FusedTag<4, 4, Pol>{});
  };
  if (!m.bf16 && m.FP == 8 && m.H1 == 64 && m.H2 == 64 && m.AP == 16)
    return by_classes(PolTag<PolicyF32<8, 64, 64, 16>>{});
  if (m.bf16 && m.FP == 32 && m.H1 == 128 && m.H2 == 128 && m.AP == 16)
    return by_classes(PolTag<PolicyBf16<32, 128, 128, 16, 1, 0>>{});
  if (m.bf16 && m.FP == 32 && m.H1 == 256 && m.H2 == 256 && m.AP == 32)
    return m.A == 24 ? by_classes(PolTag<PolicyBf16<32, 256, 256, 32, 2, 24, 2>>{})
                     : by_classes(PolTag<PolicyBf16<32, 256, 256, 32, 2, 0, 2>>{});
  if (m.bf16 && m.FP == 64 && m.H1 == 256 && m.H2 == 256 && m.AP == 64)
    return m.A == 48 ? by_classes(PolTag<PolicyBf16<64, 256, 256, 64, 4, 48>>{})
                     : by_classes(PolTag<PolicyBf16<64, 256, 256, 64, 4, 0>>{});
  return hipErrorNotSupported;
}

}  // namespace

hipError_t fused_rollout_capacity(const SimParams& p, const MlpParams& m, int* max_envs) {
  *max_envs = 0;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  return with_fused(p, m, [&](auto t) -> hipError_t {
    typedef typename decltype(t)::Pol Pol;
    int per_cu = 0;
    const hipError_t e2 = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &per_cu, rollout_fused_k<decltype(t)::kCM, decltype(t)::kTW, Pol>, 256, Pol::LDS);
    if (e2 != hipSuccess) return e2;
    *max_envs = per_cu * cus * Pol::ROWS;
    return hipSuccess;
  });
}

hipError_t launch_rollout_fused(const SimParams& p, const EnvState& s, const MlpParams& m,
                                uint32_t k0, int T, const RolloutOut& o, hipStream_t st) {
  if (T < 1 || !o.act) return hipErrorInvalidValue;
  if (m.bf16 && !s.obs_bf) return hipErrorInvalidValue;
  return with_fused(p, m, [&](auto t) -> hipError_t {
    return launch_fused<decltype(t)::kCM, decltype(t)::kTW, typename decltype(t)::Pol>(
        p, s, m, k0, T, o, st);
  });
}

}  // namespace bsim
