// devmath.hpp -- device primitives of the rollout: counter-based Philox draws, uniform
// conversion, deterministic fp64 log/exp/cos, bf16 rounding, checksum mixing.
//
// Bit-exactness contract: every fp64 result here is a fixed sequence of IEEE-754
// operations (+, -, *, / and explicit fma, each correctly rounded on gfx950), compiled
// with -ffp-contract=off, so any other IEEE implementation of the same sequence gives the
// same bits. The sequences are defined by the mathematics cited at each function.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bsim {

// ---- Philox4x32-10 (Salmon et al., SC'11) ----------------------------------------------
// Round: multiply counter words 0 and 2 by the two multipliers (full 64-bit products); the
// next counter is (hi(M1*c2)^c1^k0, lo(M1*c2), hi(M0*c0)^c3^k1, lo(M0*c0)); the key is
// advanced by the Weyl increments between rounds.
struct u32x4 { uint32_t x, y, z, w; };

__device__ __forceinline__ u32x4 philox(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                        uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    // one 32 x 32 -> 64-bit multiply per word gives both halves of its product
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
    const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    k0 += 0x9E3779B9u; k1 += 0xBB67AE85u;
  }
  return {c0, c1, c2, c3};
}

enum : uint32_t { P_ARRIVAL = 1, P_PROCESS = 2, P_SERVICE = 3, P_ACTION = 4, P_WEIGHTS = 5,
                  P_MINIBATCH = 6, P_ROUTE = 7 };
constexpr uint32_t STEP_RESET = 0xFFFFFFFFu;

// Draw block j of `purpose` for (env, step, system) under `seed`.
__device__ __forceinline__ u32x4 draw(uint64_t seed, uint32_t env, uint32_t step,
                                      uint32_t purpose, uint32_t j, uint32_t sys) {
  return philox(env, step, (purpose << 24) | j, sys, (uint32_t)seed, (uint32_t)(seed >> 32));
}

// (hi:lo) -> the top 53 bits as an integer, centred in its cell of width 2^-53: (0, 1).
__device__ __forceinline__ double unit(uint32_t lo, uint32_t hi) {
  const uint64_t v = ((((uint64_t)hi) << 32) | (uint64_t)lo) >> 11;
  return ((double)v + 0.5) * 0x1p-53;
}

// ---- deterministic fp64 elementary functions ---------------------------------------------
// Split constants: ln 2 and pi/2 each as a 32-significant-bit head plus the remainder, so
// that k*head is exact for the |k| that occur.
constexpr double kLn2Hi = 0x1.62e42fee00000p-1;
constexpr double kLn2Lo = 0x1.a39ef35793c76p-33;
constexpr double kInvLn2 = 0x1.71547652b82fep+0;
constexpr double kSqrt2 = 0x1.6a09e667f3bcdp+0;
constexpr double kPio2Hi = 0x1.921fb54400000p+0;
constexpr double kPio2Lo = 0x1.0b4611a626331p-34;
constexpr double kTwoOverPi = 0x1.45f306dc9c883p-1;
constexpr double kTwoPi = 0x1.921fb54442d18p+2;

// Natural log of a positive normal x. With x = 2^e m, m in (sqrt2/2, sqrt2]:
// log m = 2 atanh s, s = (m-1)/(m+1); atanh s = s + s^3/3 + s^5/5 + ... to s^23/23.
__device__ __forceinline__ double dlog_inl(double x) {
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  int e = (int)((b >> 52) & 0x7ff) - 1023;
  double m = __longlong_as_double((long long)((b & 0x000fffffffffffffull) | 0x3ff0000000000000ull));
  if (m > kSqrt2) { m = m * 0.5; e += 1; }
  const double s = (m - 1.0) / (m + 1.0);
  const double z = s * s;
  double p = 1.0 / 23.0;
  p = __fma_rn(p, z, 1.0 / 21.0);
  p = __fma_rn(p, z, 1.0 / 19.0);
  p = __fma_rn(p, z, 1.0 / 17.0);
  p = __fma_rn(p, z, 1.0 / 15.0);
  p = __fma_rn(p, z, 1.0 / 13.0);
  p = __fma_rn(p, z, 1.0 / 11.0);
  p = __fma_rn(p, z, 1.0 / 9.0);
  p = __fma_rn(p, z, 1.0 / 7.0);
  p = __fma_rn(p, z, 1.0 / 5.0);
  p = __fma_rn(p, z, 1.0 / 3.0);
  const double lm = 2.0 * __fma_rn(s * z, p, s);
  const double de = (double)e;
  return __fma_rn(de, kLn2Hi, __fma_rn(de, kLn2Lo, lm));
}

// exp x for |x| < 700: x = k ln2 + r, |r| <= ln2/2; exp r = sum_{n<=14} r^n/n!; times 2^k.
__device__ __forceinline__ double dexp_inl(double x) {
  const double kd = floor(x * kInvLn2 + 0.5);
  const int k = (int)kd;
  const double r = (x - kd * kLn2Hi) - kd * kLn2Lo;
  double p = 1.0 / 87178291200.0;
  p = __fma_rn(p, r, 1.0 / 6227020800.0);
  p = __fma_rn(p, r, 1.0 / 479001600.0);
  p = __fma_rn(p, r, 1.0 / 39916800.0);
  p = __fma_rn(p, r, 1.0 / 3628800.0);
  p = __fma_rn(p, r, 1.0 / 362880.0);
  p = __fma_rn(p, r, 1.0 / 40320.0);
  p = __fma_rn(p, r, 1.0 / 5040.0);
  p = __fma_rn(p, r, 1.0 / 720.0);
  p = __fma_rn(p, r, 1.0 / 120.0);
  p = __fma_rn(p, r, 1.0 / 24.0);
  p = __fma_rn(p, r, 1.0 / 6.0);
  p = __fma_rn(p, r, 0.5);
  p = __fma_rn(p, r, 1.0);
  p = __fma_rn(p, r, 1.0);
  const double sc = __longlong_as_double((long long)(((uint64_t)(k + 1023)) << 52));
  return p * sc;
}

// cos x for 0 <= x <= 8: x = q pi/2 + r, |r| <= pi/4; by q mod 4 the value is cos r,
// -sin r, -cos r, sin r, with the Taylor series of cos to r^18/18! and sin to r^19/19!.
__device__ __forceinline__ double dcos_inl(double x) {
  const double qd = floor(x * kTwoOverPi + 0.5);
  const int q = (int)qd;
  const double r = (x - qd * kPio2Hi) - qd * kPio2Lo;
  const double z = r * r;
  double c = 1.0 / 6402373705728000.0;
  c = __fma_rn(c, z, -1.0 / 20922789888000.0);
  c = __fma_rn(c, z, 1.0 / 87178291200.0);
  c = __fma_rn(c, z, -1.0 / 479001600.0);
  c = __fma_rn(c, z, 1.0 / 3628800.0);
  c = __fma_rn(c, z, -1.0 / 40320.0);
  c = __fma_rn(c, z, 1.0 / 720.0);
  c = __fma_rn(c, z, -1.0 / 24.0);
  c = __fma_rn(c, z, 0.5);
  c = __fma_rn(-c, z, 1.0);
  double s = -1.0 / 121645100408832000.0;
  s = __fma_rn(s, z, 1.0 / 355687428096000.0);
  s = __fma_rn(s, z, -1.0 / 1307674368000.0);
  s = __fma_rn(s, z, 1.0 / 6227020800.0);
  s = __fma_rn(s, z, -1.0 / 39916800.0);
  s = __fma_rn(s, z, 1.0 / 362880.0);
  s = __fma_rn(s, z, -1.0 / 5040.0);
  s = __fma_rn(s, z, 1.0 / 120.0);
  s = __fma_rn(s, z, -1.0 / 6.0);
  s = __fma_rn(s * z, r, r);
  switch (q & 3) {
    case 0: return c;
    case 1: return -s;
    case 2: return -c;
    default: return s;
  }
}

// Out-of-line copies of the three (one call site each in the code, instead of the body at every
// use): kernels held to 128 VGPRs call these; kernels with registers to spare inline the
// bodies above. The same operations either way, so the results are the same bits.
__device__ __noinline__ double dlog(double x) { return dlog_inl(x); }
__device__ __noinline__ double dexp(double x) { return dexp_inl(x); }
__device__ __noinline__ double dcos(double x) { return dcos_inl(x); }

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// two fp32 values -> their bf16 roundings (nearest even, the hardware's packed conversion),
// lo in the low half of the word and hi in the high half
__device__ __forceinline__ uint32_t pack_bf16_pair(float lo, float hi) {
  typedef __attribute__((ext_vector_type(2))) float f32x2_t;
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// FNV-1a over 64-bit words: checksum of the integer state sequence.
constexpr uint64_t kFnvInit = 0xcbf29ce484222325ull;
__device__ __forceinline__ uint64_t fnv(uint64_t h, uint64_t v) { return (h ^ v) * 0x100000001b3ull; }

}  // namespace bsim
