// device_math.h -- per-element arithmetic of the fill and the comparison,
// written for gfx950 with integer bit manipulation wherever possible so that
// no result depends on a hardware conversion or denormal mode.
//
// Floating-point contraction is disabled for every file that includes this
// header: each + - * / below rounds exactly once, in the order written.
#pragma once
#pragma clang fp contract(off)

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "asmevo.h"

namespace asmevo {

// Addresses arrive as integers in descriptor tables, so the compiler cannot
// infer that they point to global memory; these casts make the accesses
// global_load / global_store (not flat accesses, which are also checked
// against LDS and scratch).
#define AS_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ AS_GLOBAL T* gptr_mut(uint64_t addr) {
  return (AS_GLOBAL T*)(uintptr_t)addr;
}
template <typename T>
__device__ __forceinline__ const AS_GLOBAL T* gptr(const void* p) {
  return (const AS_GLOBAL T*)(uintptr_t)p;
}

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11).  One call turns a
// 128-bit counter and 64-bit key into four 32-bit words.
// ---------------------------------------------------------------------------
struct U4 {
  uint32_t x, y, z, w;
};

__device__ __forceinline__ U4 philox(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                     uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t m0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t m1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = (uint32_t)(m1 >> 32) ^ c1 ^ k0;
    const uint32_t n2 = (uint32_t)(m0 >> 32) ^ c3 ^ k1;
    c1 = (uint32_t)m1;
    c3 = (uint32_t)m0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return U4{c0, c1, c2, c3};
}

__device__ __forceinline__ uint32_t word_of(const U4& v, uint32_t k) {
  return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w;
}

// Counter layout of the fill: (lo32(j), hi32(j), alloc_id, purpose<<24 |
// aux<<16 | variant), key (lo32(seed), hi32(seed)).
enum : uint32_t { kValue = 0, kSelect = 1, kInject = 2, kCanary = 3, kPad = 5 };

__device__ __forceinline__ U4 stream(uint64_t seed, uint32_t alloc_id, uint32_t purpose,
                                     uint32_t aux, uint32_t variant, uint64_t j) {
  return philox((uint32_t)j, (uint32_t)(j >> 32), alloc_id,
                (purpose << 24) | ((aux & 0xFFu) << 16) | (variant & 0xFFFFu),
                (uint32_t)seed, (uint32_t)(seed >> 32));
}

__device__ __forceinline__ uint8_t byte_of(const U4& v, uint32_t q) {
  return (uint8_t)(word_of(v, (q >> 2) & 3u) >> (8u * (q & 3u)));
}

// ---------------------------------------------------------------------------
// Element decode: class (0 finite, 1 +Inf, 2 -Inf, 3 NaN) and the exact fp64
// value, assembled from the bit fields.
// ---------------------------------------------------------------------------
__device__ __forceinline__ double pow2i(int e) {   // 2^e for -1022 <= e <= 1023
  return __longlong_as_double((long long)(e + 1023) << 52);
}

template <int DT>
__device__ __forceinline__ int decode(uint64_t raw, double& v) {
  if constexpr (DT == ASMEVO_F32 || DT == ASMEVO_BF16) {
    const uint32_t bits = (DT == ASMEVO_F32) ? (uint32_t)raw : ((uint32_t)raw << 16);
    const uint32_t mag = bits & 0x7FFFFFFFu;
    if (mag >= 0x7F800000u) return mag > 0x7F800000u ? 3 : ((bits >> 31) ? 2 : 1);
    v = (double)__uint_as_float(bits);           // binary32 -> binary64 is exact
    return 0;
  } else if constexpr (DT == ASMEVO_F16) {
    const uint32_t h = (uint32_t)raw & 0xFFFFu;
    const uint32_t e = (h >> 10) & 0x1Fu, m = h & 0x3FFu;
    if (e == 31) return m ? 3 : ((h >> 15) ? 2 : 1);
    const double mag = e ? (double)(1024u + m) * pow2i((int)e - 25) : (double)m * pow2i(-24);
    v = (h >> 15) ? -mag : mag;
    return 0;
  } else {  // FP8 E4M3 (fn)
    const uint32_t b = (uint32_t)raw & 0xFFu;
    const uint32_t e = (b >> 3) & 0xFu, m = b & 7u;
    if ((b & 0x7Fu) == 0x7Fu) return 3;
    const double mag = e ? (double)(8u + m) * pow2i((int)e - 10) : (double)m * pow2i(-9);
    v = (b >> 7) ? -mag : mag;
    return 0;
  }
}

// ---------------------------------------------------------------------------
// Encode a binary32 value to the element type, round to nearest even.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t enc_bf16(uint32_t x) {
  if ((x & 0x7FFFFFFFu) > 0x7F800000u) return ((x >> 16) & 0x8000u) | 0x7FC0u;
  return (x + 0x7FFFu + ((x >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint32_t enc_f16(uint32_t x) {
  const uint32_t sign = (x >> 16) & 0x8000u;
  const uint32_t ax = x & 0x7FFFFFFFu;
  if (ax > 0x7F800000u) return sign | 0x7E00u;
  if (ax >= 0x477FF000u) return sign | 0x7C00u;          // >= 65520 rounds to Inf
  if (ax >= 0x38800000u) {                               // normal binary16 range
    const uint32_t r = ax + 0xFFFu + ((ax >> 13) & 1u);
    return sign | ((r >> 13) - (112u << 10));
  }
  if (ax <= 0x33000000u) return sign;                    // <= 2^-25 rounds to zero
  const uint32_t e = ax >> 23;
  const uint32_t m = (ax & 0x7FFFFFu) | 0x800000u;
  const uint32_t sh = 126u - e;                          // 14..24
  uint32_t h = m >> sh;
  const uint32_t rem = m & ((1u << sh) - 1u), half = 1u << (sh - 1u);
  h += (rem > half || (rem == half && (h & 1u))) ? 1u : 0u;
  return sign | h;
}

__device__ __forceinline__ uint32_t enc_fp8(uint32_t x, bool saturate) {
  const uint32_t sign = (x >> 24) & 0x80u;
  uint32_t ax = x & 0x7FFFFFFFu;
  if (ax > 0x7F800000u) return sign | 0x7Fu;
  if (saturate) {
    if (ax > 0x43E00000u) ax = 0x43E00000u;             // clamp to 448
  } else if (ax > 0x43E80000u) {
    return sign | 0x7Fu;                                 // above 464: no Inf, NaN
  }
  if (ax >= 0x3C800000u) {                               // >= 2^-6: normal E4M3
    uint32_t e = (ax >> 23) - 120u;
    const uint32_t mant = ax & 0x7FFFFFu;
    uint32_t r = mant >> 20;
    const uint32_t rem = mant & 0xFFFFFu;
    if (rem > 0x80000u || (rem == 0x80000u && (r & 1u))) ++r;
    if (r == 8u) {
      r = 0u;
      ++e;
    }
    return sign | (e << 3) | r;
  }
  const uint32_t e = ax >> 23;
  if (e < 1u) return sign;                               // binary32 subnormal: rounds to 0
  const uint32_t sh = 141u - e;                          // >= 21
  if (sh > 24u) return sign;
  const uint32_t m = (ax & 0x7FFFFFu) | 0x800000u;
  uint32_t h = m >> sh;
  const uint32_t rem = m & ((1u << sh) - 1u), half = 1u << (sh - 1u);
  h += (rem > half || (rem == half && (h & 1u))) ? 1u : 0u;
  return sign | h;
}

__device__ __forceinline__ uint64_t encode_f32(uint32_t dtype, float f, bool saturate) {
  const uint32_t x = __float_as_uint(f);
  switch (dtype) {
    case ASMEVO_F32: return x;
    case ASMEVO_BF16: return enc_bf16(x);
    case ASMEVO_F16: return enc_f16(x);
    default: return enc_fp8(x, saturate);
  }
}

// ---------------------------------------------------------------------------
// The fill's normal transform (Box-Muller) with a fixed operation sequence.
// ---------------------------------------------------------------------------
constexpr double kLn2 = 0x1.62e42fefa39efp-1;
constexpr double kSqrt2 = 0x1.6a09e667f3bcdp+0;
constexpr double kPio2 = 0x1.921fb54442d18p+0;

// ln((x + 1/2) 2^-32): N = 2x+1 = m 2^e, m in (sqrt2/2, sqrt2]; ln m = 2 atanh(s),
// s = (m-1)/(m+1), series to s^23.
__device__ __forceinline__ double log_u(uint32_t x) {
  const uint64_t N = 2ull * x + 1ull;
  int e = 63 - __clzll((long long)N);
  double m = (double)N * pow2i(-e);
  if (m > kSqrt2) {
    m = m * 0.5;
    e = e + 1;
  }
  const double f = m - 1.0;
  const double s = f / (2.0 + f);
  const double z = s * s;
  double p = 1.0 / 23.0;
  p = 1.0 / 21.0 + z * p;
  p = 1.0 / 19.0 + z * p;
  p = 1.0 / 17.0 + z * p;
  p = 1.0 / 15.0 + z * p;
  p = 1.0 / 13.0 + z * p;
  p = 1.0 / 11.0 + z * p;
  p = 1.0 / 9.0 + z * p;
  p = 1.0 / 7.0 + z * p;
  p = 1.0 / 5.0 + z * p;
  p = 1.0 / 3.0 + z * p;
  const double r = z * p;
  const double lnm = 2.0 * (s + s * r);
  return (double)(e - 33) * kLn2 + lnm;
}

// cos / sin of 2 pi x 2^-32: quadrant from the top two bits, fold to
// [0, pi/4] in integers, Taylor series to phi^15 (sin) and phi^16 (cos).
__device__ __forceinline__ void sincos_turns(uint32_t x, double& c_out, double& s_out) {
  const uint32_t q = x >> 30;
  uint32_t w = x & 0x3FFFFFFFu;
  const bool swap = w > (1u << 29);
  if (swap) w = (1u << 30) - w;
  const double phi = ((double)w * pow2i(-30)) * kPio2;
  const double x2 = phi * phi;
  double ps = -1.0 / 1307674368000.0;             // -1/15!
  ps = 1.0 / 6227020800.0 + x2 * ps;              // 1/13!
  ps = -1.0 / 39916800.0 + x2 * ps;               // -1/11!
  ps = 1.0 / 362880.0 + x2 * ps;                  // 1/9!
  ps = -1.0 / 5040.0 + x2 * ps;                   // -1/7!
  ps = 1.0 / 120.0 + x2 * ps;                     // 1/5!
  ps = -1.0 / 6.0 + x2 * ps;                      // -1/3!
  double sn = phi + (phi * x2) * ps;
  double pc = 1.0 / 20922789888000.0;             // 1/16!
  pc = -1.0 / 87178291200.0 + x2 * pc;            // -1/14!
  pc = 1.0 / 479001600.0 + x2 * pc;               // 1/12!
  pc = -1.0 / 3628800.0 + x2 * pc;                // -1/10!
  pc = 1.0 / 40320.0 + x2 * pc;                   // 1/8!
  pc = -1.0 / 720.0 + x2 * pc;                    // -1/6!
  pc = 1.0 / 24.0 + x2 * pc;                      // 1/4!
  pc = -1.0 / 2.0 + x2 * pc;                      // -1/2!
  double cs = 1.0 + x2 * pc;
  if (swap) {
    const double t = sn;
    sn = cs;
    cs = t;
  }
  switch (q) {
    case 0: c_out = cs; s_out = sn; break;
    case 1: c_out = -sn; s_out = cs; break;
    case 2: c_out = -cs; s_out = -sn; break;
    default: c_out = sn; s_out = -cs; break;
  }
}

// Both Box-Muller outputs of the uniform pair (xa, xb).
__device__ __forceinline__ void box_muller(uint32_t xa, uint32_t xb, double& z0, double& z1) {
  const double rho = __builtin_sqrt(-2.0 * log_u(xa));
  double c, s;
  sincos_turns(xb, c, s);
  z0 = rho * c;
  z1 = rho * s;
}

}  // namespace asmevo
