// Device-side determinism contract: Philox4x32-10 draws, deterministic exponentials,
// 2^-40 fixed-point quantisation and exact integer decisions.
//
// Every discrete decision of the sampler and verifier (category, drafted token, accept coin,
// residual/bonus token) is taken from quantities computed here with separately rounded IEEE
// operations only, so that any other implementation of the same recipe (the CPU oracle)
// reaches the same integers bit for bit. Floating-point contraction is disabled in every
// function of this header; the intrinsics below are the correctly rounded single operations.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dbl {

// ---------------------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): 10 rounds of two 32x32->64 multiplies
// with the round constants, Weyl-sequence key schedule.
// ---------------------------------------------------------------------------------------
enum Purpose : uint32_t { kCategory = 0, kToken = 1, kAccept = 2, kResidual = 3 };

struct PhiloxPair {
  uint32_t w0, w1;  // output words 0 and 1 of one Philox4x32-10 block
};

__device__ __forceinline__ PhiloxPair philox_words01(uint32_t c0, uint32_t c1, uint32_t c2,
                                                     uint32_t c3, uint32_t k0, uint32_t k1) {
  constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;
  constexpr uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    const uint32_t hi0 = __umulhi(kM0, c0), lo0 = kM0 * c0;
    const uint32_t hi1 = __umulhi(kM1, c2), lo1 = kM1 * c2;
    const uint32_t n0 = hi1 ^ c1 ^ k0;
    const uint32_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += kW0;
    k1 += kW1;
  }
  return {c0, c1};
}

__device__ __forceinline__ uint32_t philox_word0(uint32_t c0, uint32_t c1, uint32_t c2,
                                                 uint32_t c3, uint32_t k0, uint32_t k1) {
  return philox_words01(c0, c1, c2, c3, k0, k1).w0;
}

// The uniform word for (purpose, position k) of sequence `seq` at `step` under `seed`.
__device__ __forceinline__ uint32_t draw(uint64_t seed, uint32_t purpose, uint32_t k,
                                         uint64_t seq, uint64_t step) {
  return philox_word0(k, purpose, static_cast<uint32_t>(seq), static_cast<uint32_t>(step),
                      static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32));
}

// Words 0 and 1 of the same block: the drafted token's tile (word 0) and its id within the
// tile (word 1).
__device__ __forceinline__ PhiloxPair draw2(uint64_t seed, uint32_t purpose, uint32_t k,
                                            uint64_t seq, uint64_t step) {
  return philox_words01(k, purpose, static_cast<uint32_t>(seq), static_cast<uint32_t>(step),
                        static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32));
}

// ---------------------------------------------------------------------------------------
// Deterministic exponentials (Cody-Waite reduction x = n ln2 + r with a two-word ln 2,
// Taylor polynomial of e^r in Horner form, exact scaling by 2^n).
// ---------------------------------------------------------------------------------------
// binary32: for token probabilities. Inputs above 0 are clamped to 0; inputs below -80,
// -inf and NaN give 0 (so no subnormal is ever produced).
__device__ __forceinline__ float detexp32(float x) {
#pragma clang fp contract(off)
  if (!(x > -80.0f)) return 0.0f;
  x = x > 0.0f ? 0.0f : x;
  constexpr float kLog2e = 0x1.715476p+0f;  // 1/ln 2
  constexpr float kLn2Hi = 0x1.62e4p-1f;    // ln 2 to 15 significant bits
  constexpr float kLn2Lo = 0x1.7f7d1cp-20f; // ln 2 - kLn2Hi
  const float n = rintf(__fmul_rn(x, kLog2e));
  const float r = __fsub_rn(__fsub_rn(x, __fmul_rn(n, kLn2Hi)), __fmul_rn(n, kLn2Lo));
  float p = static_cast<float>(1.0 / 5040.0);
  p = __fadd_rn(__fmul_rn(p, r), static_cast<float>(1.0 / 720.0));
  p = __fadd_rn(__fmul_rn(p, r), static_cast<float>(1.0 / 120.0));
  p = __fadd_rn(__fmul_rn(p, r), static_cast<float>(1.0 / 24.0));
  p = __fadd_rn(__fmul_rn(p, r), static_cast<float>(1.0 / 6.0));
  p = __fadd_rn(__fmul_rn(p, r), 0.5f);
  p = __fadd_rn(__fmul_rn(p, r), 1.0f);
  p = __fadd_rn(__fmul_rn(p, r), 1.0f);
  return ldexpf(p, static_cast<int>(n));
}

// binary64: for category weights. Inputs above 0 are clamped to 0; below -708, -inf and NaN
// give 0.
__device__ __forceinline__ double dexp64(double x) {
#pragma clang fp contract(off)
  if (!(x > -708.0)) return 0.0;
  x = x > 0.0 ? 0.0 : x;
  constexpr double kLog2e = 0x1.71547652b82fep+0;
  constexpr double kLn2Hi = 0x1.62e42ffp-1;            // ln 2 to 32 significant bits
  constexpr double kLn2Lo = -0x1.718432a1b0e26p-35;    // ln 2 - kLn2Hi
  const double n = rint(__dmul_rn(x, kLog2e));
  const double r = __dsub_rn(__dsub_rn(x, __dmul_rn(n, kLn2Hi)), __dmul_rn(n, kLn2Lo));
  double p = 1.0 / 6227020800.0;  // 1/13!
  p = __dadd_rn(__dmul_rn(p, r), 1.0 / 479001600.0);
  p = __dadd_rn(__dmul_rn(p, r), 1.0 / 39916800.0);
  p = __dadd_rn(__dmul_rn(p, r), 1.0 / 3628800.0);
  p = __dadd_rn(__dmul_rn(p, r), 1.0 / 362880.0);
  p = __dadd_rn(__dmul_rn(p, r), 1.0 / 40320.0);
  p = __dadd_rn(__dmul_rn(p, r), 1.0 / 5040.0);
  p = __dadd_rn(__dmul_rn(p, r), 1.0 / 720.0);
  p = __dadd_rn(__dmul_rn(p, r), 1.0 / 120.0);
  p = __dadd_rn(__dmul_rn(p, r), 1.0 / 24.0);
  p = __dadd_rn(__dmul_rn(p, r), 1.0 / 6.0);
  p = __dadd_rn(__dmul_rn(p, r), 0.5);
  p = __dadd_rn(__dmul_rn(p, r), 1.0);
  p = __dadd_rn(__dmul_rn(p, r), 1.0);
  return ldexp(p, static_cast<int>(n));
}

// ---------------------------------------------------------------------------------------
// Fixed point and integer decisions
// ---------------------------------------------------------------------------------------
// floor(y * 2^40) for binary32 y in [0, 1], exactly, from the bits of y: a normal y equals
// mant * 2^(e - 150), so y * 2^40 = mant * 2^(e - 110) and the floor is a shift of the 24-bit
// significand. Zero and subnormals (< 2^-126) give 0.
__device__ __forceinline__ uint64_t quant40(float y) {
  const uint32_t u = __float_as_uint(y);
  const int e = static_cast<int>((u >> 23) & 0xffu);
  if (e == 0) return 0;
  const uint64_t m = static_cast<uint64_t>((u & 0x7fffffu) | 0x800000u);
  const int sh = e - 110;
  return sh >= 0 ? (m << sh) : (sh > -24 ? (m >> -sh) : 0);
}
// quant40(detexp32(x)) for every binary32 x (the quantised probability of a log-probability),
// without forming detexp32(x): the same reduction n, r and polynomial p = e^r with p in
// [2^-1, 2^1), so detexp32(x) = p 2^n whenever it is normal and the floor of p 2^(n + 40) is the
// 24-bit significand of p shifted by e(p) + n - 110 <= 17, taken as one right shift of the
// significand placed at bit 17 (shift counts past 40 give 0, as the subnormal and zero results
// of detexp32 do). Inputs are clamped to [-100, 0] first: -inf, NaN and everything at or below
// -80 then have n <= -115 and quantise to 0, as the early return of detexp32 gives; branch-free.
__device__ __forceinline__ uint64_t quant_detexp32(float x) {
#pragma clang fp contract(off)
  x = fminf(fmaxf(x, -100.0f), 0.0f);
  constexpr float kLog2e = 0x1.715476p+0f;
  constexpr float kLn2Hi = 0x1.62e4p-1f;
  constexpr float kLn2Lo = 0x1.7f7d1cp-20f;
  const float n = rintf(__fmul_rn(x, kLog2e));
  const float r = __fsub_rn(__fsub_rn(x, __fmul_rn(n, kLn2Hi)), __fmul_rn(n, kLn2Lo));
  float p = static_cast<float>(1.0 / 5040.0);
  p = __fadd_rn(__fmul_rn(p, r), static_cast<float>(1.0 / 720.0));
  p = __fadd_rn(__fmul_rn(p, r), static_cast<float>(1.0 / 120.0));
  p = __fadd_rn(__fmul_rn(p, r), static_cast<float>(1.0 / 24.0));
  p = __fadd_rn(__fmul_rn(p, r), static_cast<float>(1.0 / 6.0));
  p = __fadd_rn(__fmul_rn(p, r), 0.5f);
  p = __fadd_rn(__fmul_rn(p, r), 1.0f);
  p = __fadd_rn(__fmul_rn(p, r), 1.0f);
  const uint32_t u = __float_as_uint(p);
  const uint64_t t = static_cast<uint64_t>((u & 0x7fffffu) | 0x800000u) << 17;
  const int amt = min(127 - static_cast<int>(u >> 23) - static_cast<int>(n), 63);
  return t >> amt;
}
__device__ __forceinline__ uint64_t quant40d(double y) {
  return static_cast<uint64_t>(y * 0x1p40);
}

// floor(r * Z / 2^32) exactly (r < 2^32, Z < 2^64, so the result fits 64 bits).
__device__ __forceinline__ uint64_t icdf_threshold(uint32_t r, uint64_t Z) {
  const uint64_t lo = static_cast<uint64_t>(r) * static_cast<uint32_t>(Z);
  const uint64_t hi = static_cast<uint64_t>(r) * static_cast<uint32_t>(Z >> 32);
  return hi + (lo >> 32);
}

// r * q < p * 2^32 exactly, i.e. floor(r * q / 2^32) < p (q, p < 2^41).
__device__ __forceinline__ bool accept_int(uint32_t r, uint64_t q, uint64_t p) {
  return icdf_threshold(r, q) < p;
}

// The binary32 branch log-probability fl32(tls + fl32(lmass - lse)).
__device__ __forceinline__ float flat_lq(float tls, float lmass, float lse) {
#pragma clang fp contract(off)
  return __fadd_rn(tls, __fsub_rn(lmass, lse));
}

}  // namespace dbl
