// Device arithmetic shared by the quantisers: the Philox4x32-10 stream of
// stochastic rounding, the shared exponent of a max magnitude (Eq. 1-2) and
// the rounding of one FP32 value to an integer at a given exponent (Eq. 3,
// with the rounding modes of Sec. 1).
#pragma once

#include "dfp_internal.h"

namespace dfp {

// Philox4x32-10 (Salmon et al., SC'11).
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    // one 32x32->64 multiply gives both halves of each product; the
    // three-way XORs are single bitop3 instructions (truth table 0x96)
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x, p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = make_uint4(__builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c.y, k0, 0x96), (uint32_t)p1,
                   __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c.w, k1, 0x96), (uint32_t)p0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// Exponent of the max magnitude from its bit pattern (floor(log2 m), m > 0 finite).
__device__ __forceinline__ int32_t floor_log2_bits(uint32_t mb) {
  const uint32_t eb = mb >> 23;
  if (eb != 0) return (int32_t)eb - 127;
  return (31 - __clz((int)(mb & 0x7fffffu))) - 149;
}

// Shared exponent of a tensor from its max magnitude bits (Eq. 2, clamped at
// -128), with the flags the exponent decides.  A non-finite max or an
// all-zero tensor gives exponent 0 and all-zero integers.
struct ScaleFromMax {
  int32_t es;
  uint32_t flags;  // NONFINITE | ZERO_TENSOR | EXP_CLAMPED
  bool all_zero;
};
__device__ __forceinline__ ScaleFromMax scale_from_max(uint32_t mb, int32_t bits) {
  const bool nonfinite = mb >= 0x7f800000u;
  const bool zero = mb == 0u;
  int32_t es = 0;
  bool clamped = false;
  if (!nonfinite && !zero) {
    es = floor_log2_bits(mb) - (bits - 2);
    if (es < -128) {
      es = -128;
      clamped = true;
    }
  }
  const uint32_t f = (nonfinite ? DFP_FLAG_NONFINITE : 0u) | (zero ? DFP_FLAG_ZERO_TENSOR : 0u) |
                     (clamped ? DFP_FLAG_EXP_CLAMPED : 0u);
  return {es, f, nonfinite || zero};
}

// x = f * 2^-es split as X = floor(x * 2^32) = fl * 2^32 + F, in integer
// arithmetic on the sign / exponent / significand fields.  f = S * 2^(e1 - 150)
// with S the signed 24-bit significand, so x * 2^32 = S * 2^(32 - sh) with
// sh = es + 150 - e1, and X = (S * 2^32) >> sh with an arithmetic shift (the
// floor, for either sign).  Every element of the tensor has |x| < 2^(bits-1)
// <= 2^15, which bounds sh below by 9 (|X| < 2^47); shifts are clamped at 63,
// which leaves 0 or -1 (a value below 2^-31 in magnitude).
struct Split {
  int32_t fl;   // floor(x)
  uint32_t F;   // floor(frac(x) * 2^32)
};
__device__ __forceinline__ Split split_scaled(uint32_t fb, int32_t es150) {
  const uint32_t eb = (fb >> 23) & 0xffu;
  const int32_t M = (int32_t)((fb & 0x7fffffu) | ((eb != 0u ? 1u : 0u) << 23));
  const int32_t S = (int32_t)fb < 0 ? -M : M;
  const uint32_t sh = min((uint32_t)(es150 - (int32_t)max(eb, 1u)), 63u);
  const int64_t X = (int64_t)((uint64_t)(uint32_t)S << 32) >> sh;
  return {(int32_t)(X >> 32), (uint32_t)X};
}

// Round f * 2^-es to an integer (Sec. 1 rounding modes).
//   NEAREST   ties to even: x is exact in FP32 whenever it is a normal number,
//             and every smaller |x| rounds to 0 however ldexp rounds it.
//   BIASED    floor(x + 1/2) as floor(x) + (frac(x) >= 1/2); frac is exact for
//             normal x and the decision is unchanged for smaller |x|.
//   STOCHASTIC floor(x) + (u < F), u the element's Philox word.
//   DOWN      floor(x).
template <int MODE>
__device__ __forceinline__ int32_t round_one(uint32_t fb, int32_t es, uint32_t u) {
  if (MODE == DFP_ROUND_NEAREST) {
    return (int32_t)rintf(ldexpf(__uint_as_float(fb), -es));
  } else if (MODE == DFP_ROUND_BIASED) {
    const float x = ldexpf(__uint_as_float(fb), -es);
    const float fl = floorf(x);
    return (int32_t)fl + ((x - fl) >= 0.5f ? 1 : 0);
  } else {
    const Split sp = split_scaled(fb, es + 150);
    if (MODE == DFP_ROUND_STOCHASTIC) return sp.fl + (u < sp.F ? 1 : 0);
    return sp.fl;
  }
}

}  // namespace dfp
