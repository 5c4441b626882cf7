// FP32 -> DFP quantisation (Sec. 3.1 Eq. 1-3) and the rounding modes of Sec. 1.
//
// Two HBM-bound passes: a max-magnitude reduction (integer max over the FP32
// bit patterns with the sign cleared, one atomic per block), then the rounding
// pass, which derives the shared exponent on the device from that max and
// rounds every element with integer arithmetic on its sign / exponent /
// mantissa fields (no floating-point rounding, so denormal modes cannot
// matter).  Each lane owns 4 consecutive elements: one 16-byte load, one
// Philox4x32-10 block (stochastic mode), one 8-byte store.
#include "dfp_internal.h"

namespace dfp {

namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, off, 64));
  return v;
}

// Block-wide max of one value per lane; result valid in every lane.
__device__ __forceinline__ uint32_t block_max(uint32_t v) {
  __shared__ uint32_t red[kBlock / 64];
  v = wave_max(v);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[wave] = v;
  __syncthreads();
  uint32_t m = red[0];
#pragma unroll
  for (int i = 1; i < kBlock / 64; ++i) m = max(m, red[i]);
  return m;
}

__global__ void k_scale_reset(dfp_scale* s) {
  if (threadIdx.x == 0) {
    s->amax_bits = 0u;
    s->flags = 0u;
  }
}

__global__ __launch_bounds__(kBlock) void k_amax(const float* __restrict__ src, int64_t n,
                                                 dfp_scale* __restrict__ s) {
  const uint4* src4 = reinterpret_cast<const uint4*>(src);
  const int64_t n4 = n >> 2;
  uint32_t m = 0;
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n4; i += stride) {
    uint4 v = src4[i];
    m = max(m, max(max(v.x & 0x7fffffffu, v.y & 0x7fffffffu), max(v.z & 0x7fffffffu, v.w & 0x7fffffffu)));
  }
  if (blockIdx.x == 0) {
    const uint32_t* s1 = reinterpret_cast<const uint32_t*>(src);
    for (int64_t i = 4 * n4 + threadIdx.x; i < n; i += kBlock) m = max(m, s1[i] & 0x7fffffffu);
  }
  m = block_max(m);
  // most blocks cannot raise the running max: skip their atomic after a plain read
  if (threadIdx.x == 0 && m > __atomic_load_n(&s->amax_bits, __ATOMIC_RELAXED)) atomicMax(&s->amax_bits, m);
}

// Philox4x32-10 (Salmon et al., SC'11).
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint32_t lo0 = 0xD2511F53u * c.x, hi0 = __umulhi(0xD2511F53u, c.x);
    const uint32_t lo1 = 0xCD9E8D57u * c.z, hi1 = __umulhi(0xCD9E8D57u, c.z);
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
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

// Round one FP32 value (bit pattern fb) scaled by 2^-es to an integer.
//   value = M * 2^e exactly (M the 24-bit significand); A = |x| * 2^32 = M * 2^sh.
//   X = floor(x * 2^32) as a signed 64-bit integer; fl = X >> 32; F = low word.
template <bool STOCH>
__device__ __forceinline__ int32_t round_one(uint32_t fb, int32_t es, int32_t rounding, uint32_t u) {
  const uint32_t eb = (fb >> 23) & 0xffu;
  const uint32_t man = fb & 0x7fffffu;
  const uint64_t M = eb ? (uint64_t)(man | 0x800000u) : (uint64_t)man;
  const int32_t e = (eb ? (int32_t)eb : 1) - 150;
  const int32_t sh = e - es + 32;
  uint64_t A;
  bool inexact;
  if (sh >= 0) {
    A = M << sh;  // |x| < 2^15 keeps A below 2^47
    inexact = false;
  } else if (sh > -40) {
    A = M >> (-sh);
    inexact = (M & ((1ull << (-sh)) - 1ull)) != 0ull;
  } else {
    A = 0;
    inexact = M != 0;
  }
  const int64_t X = (fb >> 31) ? -(int64_t)A - (inexact ? 1 : 0) : (int64_t)A;
  const int32_t fl = (int32_t)(X >> 32);
  const uint32_t F = (uint32_t)X;
  bool up;
  if (STOCH) {
    up = u < F;
  } else if (rounding == DFP_ROUND_NEAREST) {
    up = (F > 0x80000000u) || (F == 0x80000000u && (fl & 1));
  } else if (rounding == DFP_ROUND_BIASED) {
    up = F >= 0x80000000u;
  } else {
    up = false;
  }
  return fl + (up ? 1 : 0);
}

template <bool STOCH>
__global__ __launch_bounds__(kBlock) void k_quant_convert(const float* __restrict__ src,
                                                          int16_t* __restrict__ dst, int64_t n,
                                                          dfp_scale* __restrict__ s, int32_t bits,
                                                          int32_t rounding, uint32_t key0,
                                                          uint32_t key1, uint32_t role) {
  const uint32_t mb = s->amax_bits;
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
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    s->exp = es;
    const uint32_t f = (nonfinite ? DFP_FLAG_NONFINITE : 0u) | (zero ? DFP_FLAG_ZERO_TENSOR : 0u) |
                       (clamped ? DFP_FLAG_EXP_CLAMPED : 0u);
    if (f) atomicOr(&s->flags, f);
  }
  const bool all_zero = nonfinite || zero;
  const int32_t lim = (bits == 16) ? 32767 : 0x7fffffff;
  const int64_t groups = (n + 3) >> 2;
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  bool saturated = false;
  for (int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x; g < groups; g += stride) {
    const int64_t base = g << 2;
    uint32_t fb[4];
    const bool full = base + 4 <= n;
    if (full) {
      const uint4 v = reinterpret_cast<const uint4*>(src)[g];
      fb[0] = v.x; fb[1] = v.y; fb[2] = v.z; fb[3] = v.w;
    } else {
      const uint32_t* s1 = reinterpret_cast<const uint32_t*>(src);
#pragma unroll
      for (int i = 0; i < 4; ++i) fb[i] = (base + i < n) ? s1[base + i] : 0u;
    }
    uint32_t u[4] = {0u, 0u, 0u, 0u};
    if (STOCH) {
      const uint4 r = philox4x32_10(make_uint4((uint32_t)g, (uint32_t)((uint64_t)g >> 32), role, 0u), key0, key1);
      u[0] = r.x; u[1] = r.y; u[2] = r.z; u[3] = r.w;
    }
    int32_t iv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int32_t v = all_zero ? 0 : round_one<STOCH>(fb[i], es, rounding, u[i]);
      if (v > lim) { v = lim; saturated = true; }
      if (v < -lim) { v = -lim; saturated = true; }
      iv[i] = v;
    }
    if (full) {
      uint2 packed;
      packed.x = ((uint32_t)iv[0] & 0xffffu) | ((uint32_t)iv[1] << 16);
      packed.y = ((uint32_t)iv[2] & 0xffffu) | ((uint32_t)iv[3] << 16);
      reinterpret_cast<uint2*>(dst)[g] = packed;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (base + i < n) dst[base + i] = (int16_t)iv[i];
    }
  }
  if (saturated) atomicOr(&s->flags, DFP_FLAG_SATURATED);
}

int grid_for(int64_t work_items) {
  int64_t blocks = (work_items + kBlock - 1) / kBlock;
  if (blocks < 1) blocks = 1;
  if (blocks > 8192) blocks = 8192;
  return (int)blocks;
}

}  // namespace

dfp_status launch_scale_reset(dfp_scale* s, hipStream_t st) {
  DFP_LAUNCH(K_SCALE_RESET, k_scale_reset, dim3(1), dim3(64), 0, st, s);
  return DFP_OK;
}

dfp_status launch_amax(const float* src, int64_t n, dfp_scale* s, hipStream_t st) {
  // at most 1024 blocks: each ends with one (usually skipped) atomic on the same word
  int64_t blocks = (n / 4 + kBlock - 1) / kBlock;
  blocks = blocks < 1 ? 1 : (blocks > 1024 ? 1024 : blocks);
  DFP_LAUNCH(K_AMAX, k_amax, dim3((unsigned)blocks), dim3(kBlock), 0, st, src, n, s);
  return DFP_OK;
}

dfp_status launch_quant_convert(const float* src, int16_t* dst, int64_t n, dfp_scale* s, int32_t bits,
                                int32_t rounding, uint64_t seed, uint32_t role, hipStream_t st) {
  const dim3 grid(grid_for((n + 3) / 4));
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  if (rounding == DFP_ROUND_STOCHASTIC)
    DFP_LAUNCH(K_QUANT, k_quant_convert<true>, grid, dim3(kBlock), 0, st, src, dst, n, s, bits, rounding, k0, k1, role);
  else
    DFP_LAUNCH(K_QUANT, k_quant_convert<false>, grid, dim3(kBlock), 0, st, src, dst, n, s, bits, rounding, k0, k1, role);
  return DFP_OK;
}

}  // namespace dfp
