// rng.hpp -- the library's random numbers (HIP device code; gfx950).
//
// Every function is a fixed sequence of IEEE binary32 operations, so a
// translation unit that includes this header must be compiled with
// -ffp-contract=off: the results are then bitwise reproducible on any IEEE
// machine that performs the same sequence.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vase {
namespace {

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of the 4x32
// multiply-xor bijection with the published multipliers and key increments.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t lo0 = 0xD2511F53u * c.x, hi0 = __umulhi(0xD2511F53u, c.x);
    const uint32_t lo1 = 0xCD9E8D57u * c.z, hi1 = __umulhi(0xCD9E8D57u, c.z);
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// u in (0,1): odd multiple of 2^-24 chosen by the top 23 bits of x (exact in fp32).
__device__ __forceinline__ float uniform_from_word(uint32_t x) {
  return (float)(2u * (x >> 9) + 1u) * 0x1p-24f;
}

// E = -ln(u) for u in (0,1).  Reduction u = 2^e * m with m in [sqrt(1/2), sqrt(2)],
// then ln m = 2f + 2f*z*(1/3 + z/5 + z^2/7 + z^3/9) with f = (m-1)/(m+1), z = f^2
// (odd atanh series), and ln 2 split in a 15-bit head and a tail so e*head is
// exact.  Each statement is one correctly rounded binary32 operation.
__device__ __forceinline__ float neg_log(float u) {
  const uint32_t bits = __float_as_uint(u);
  int e = (int)((bits >> 23) & 0xffu) - 127;
  uint32_t mb = (bits & 0x007fffffu) | 0x3f800000u;
  if (mb > 0x3fb504f3u) {
    mb -= 0x00800000u;
    e += 1;
  }
  const float m = __uint_as_float(mb);
  const float num = m - 1.0f;
  const float den = m + 1.0f;
  const float f = num / den;
  const float z = f * f;
  float p = __builtin_fmaf(0x1.c71c72p-4f, z, 0x1.24924ap-3f);
  p = __builtin_fmaf(p, z, 0x1.99999ap-3f);
  p = __builtin_fmaf(p, z, 0x1.555556p-2f);
  const float f2 = f * 2.0f;
  const float t = z * p;
  const float lnm = __builtin_fmaf(f2, t, f2);
  const float fe = (float)e;
  const float lo = fe * 0x1.7f7d1cp-20f;
  const float s = lo + lnm;
  const float hi = fe * 0x1.62e400p-1f;
  const float r = hi + s;
  return -r;
}

// cos(2 pi u), u in (0,1): the quadrant comes from u itself (t = 4u and
// f = t - floor(t) are exact), then the Taylor series of cos(pi f/2) and
// sin(pi f/2) in f, truncated after the f^14 and f^15 terms (remainders below
// 2e-10), evaluated by Horner with fma.
__device__ __forceinline__ float cos_2pi(float u) {
  const float t = 4.0f * u;
  const float qf = floorf(t);
  const float f = t - qf;
  const int q = (int)qf & 3;
  const float z = f * f;
  // (-1)^k (pi/2)^(2k) / (2k)!, k = 7 .. 0
  float c = -0x1.b6e250p-28f;
  c = __builtin_fmaf(c, z, 0x1.f9d38ap-22f);
  c = __builtin_fmaf(c, z, -0x1.a6d1f2p-16f);
  c = __builtin_fmaf(c, z, 0x1.e1f506p-11f);
  c = __builtin_fmaf(c, z, -0x1.55d3c8p-6f);
  c = __builtin_fmaf(c, z, 0x1.03c1f0p-2f);
  c = __builtin_fmaf(c, z, -0x1.3bd3ccp+0f);
  c = __builtin_fmaf(c, z, 1.0f);
  // (-1)^k (pi/2)^(2k+1) / (2k+1)!, k = 7 .. 0, times f
  float sn = -0x1.6fadbap-31f;
  sn = __builtin_fmaf(sn, z, 0x1.e8f434p-25f);
  sn = __builtin_fmaf(sn, z, -0x1.e30750p-19f);
  sn = __builtin_fmaf(sn, z, 0x1.507834p-13f);
  sn = __builtin_fmaf(sn, z, -0x1.32d2ccp-8f);
  sn = __builtin_fmaf(sn, z, 0x1.466bc6p-4f);
  sn = __builtin_fmaf(sn, z, -0x1.4abbcep-1f);
  sn = __builtin_fmaf(sn, z, 0x1.921fb6p+0f);
  sn = sn * f;
  return q == 0 ? c : (q == 1 ? -sn : (q == 2 ? -c : sn));
}

// One entry of a VaSE-DKV projection G_t (entries N(0, 1/r)): entry e of an
// instance's [d][r] matrix takes words 2(e&1), 2(e&1)+1 of
// Philox(counter (e>>1, inst, round, 1), key seed) through Box-Muller,
// z = sqrt(2 E(u1)) cos(2 pi u2), scaled by 1/sqrt(r).
__device__ __forceinline__ float dkv_gaussian_entry(uint32_t e, uint32_t inst, uint32_t round,
                                                    uint32_t k0, uint32_t k1, float scale) {
  const uint4 x = philox4x32_10(make_uint4(e >> 1, inst, round, 1u), k0, k1);
  const uint32_t w1 = (e & 1u) ? x.z : x.x;
  const uint32_t w2 = (e & 1u) ? x.w : x.y;
  const float u1 = uniform_from_word(w1);
  const float u2 = uniform_from_word(w2);
  const float rad = __builtin_sqrtf(2.0f * neg_log(u1));
  const float z = rad * cos_2pi(u2);
  return z * scale;
}

}  // namespace
}  // namespace vase
