// FP32 -> DFP quantisation (Sec. 3.1 Eq. 1-3) and the rounding modes of Sec. 1.
//
// Two HBM-bound passes: a max-magnitude reduction (integer max over the FP32
// bit patterns with the sign cleared, one atomic per block), then the rounding
// pass, which derives the shared exponent on the device from that max.
// Stochastic rounding and round-down split every element into floor and
// 32-bit fraction with integer arithmetic on its sign / exponent / significand
// fields; nearest-even and biased rounding scale by 2^-Es with ldexp, which is
// exact for every normal result (FP32 denormals are preserved in these
// kernels, so denormal inputs scale exactly too), and the smaller results
// round the same whatever ldexp does with them.  Each lane owns 4 consecutive
// elements: one 16-byte load, one Philox4x32-10 block (stochastic mode), one
// 8-byte store.
#include <algorithm>

#include "dfp_internal.h"
#include "dfp_round.h"

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

// Max of |src| bit patterns in two stages with no atomics.  Stage 1: up to
// kAmaxMaxParts workgroups (about eight per CU) read the 16-byte vectors in
// grid-stride steps of 1024 vectors per workgroup, four loads per lane in
// flight; workgroup b stores its max in part[b].  part is the destination INT16 buffer, which the rounding pass
// overwrites only after stage 2 has read it.  Stage 2: one workgroup reduces
// the partial maxima into the scale and clears its flags.  A tensor small
// enough for one workgroup goes straight to the scale in stage 1.
constexpr int kAmaxUnroll = 4;
constexpr int kAmaxChunk = kBlock * kAmaxUnroll;  // 16-byte vectors per workgroup and step
constexpr int kAmaxMaxParts = 2048;

__device__ __forceinline__ uint32_t abs_max4(uint4 v) {
  return max(max(v.x & 0x7fffffffu, v.y & 0x7fffffffu), max(v.z & 0x7fffffffu, v.w & 0x7fffffffu));
}

// Workgroup b reads vectors b * 1024 + i .. in steps of the whole grid (1024
// vectors per workgroup and step, four loads per lane in flight), so at any
// moment the grid streams one contiguous region.
__global__ __launch_bounds__(kBlock) void k_amax(const float* __restrict__ src, int64_t n,
                                                 uint32_t* __restrict__ part, dfp_scale* __restrict__ s) {
  const uint4* src4 = reinterpret_cast<const uint4*>(src);
  const int64_t n4 = n >> 2;
  uint32_t m[kAmaxUnroll] = {0u, 0u, 0u, 0u};
  // all four loads of a step are issued before any is reduced; a load past
  // the end re-reads the last vector (the max is unchanged)
  for (int64_t base = (int64_t)blockIdx.x * kAmaxChunk + threadIdx.x; base < n4;
       base += (int64_t)gridDim.x * kAmaxChunk) {
    uint4 v[kAmaxUnroll];
#pragma unroll
    for (int k = 0; k < kAmaxUnroll; ++k) v[k] = src4[min(base + k * kBlock, n4 - 1)];
#pragma unroll
    for (int k = 0; k < kAmaxUnroll; ++k) m[k] = max(m[k], abs_max4(v[k]));
  }
  uint32_t mm = max(max(m[0], m[1]), max(m[2], m[3]));
  if (blockIdx.x == 0) {
    const uint32_t* s1 = reinterpret_cast<const uint32_t*>(src);
    for (int64_t t = 4 * n4 + threadIdx.x; t < n; t += kBlock) mm = max(mm, s1[t] & 0x7fffffffu);
  }
  mm = block_max(mm);
  if (threadIdx.x == 0) {
    if (part) {
      part[blockIdx.x] = mm;
    } else {
      s->amax_bits = mm;
      s->flags = 0u;
    }
  }
}

__global__ __launch_bounds__(kBlock) void k_amax_final(const uint32_t* __restrict__ part, int32_t nparts,
                                                       dfp_scale* __restrict__ s) {
  // eight loads per lane in flight; an index past the end re-reads the last
  // partial (the max is unchanged)
  uint32_t m = 0u;
  for (int32_t base = threadIdx.x; base < nparts; base += 8 * kBlock) {
    uint32_t v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = part[min(base + k * kBlock, nparts - 1)];
#pragma unroll
    for (int k = 0; k < 8; ++k) m = max(m, v[k]);
  }
  m = block_max(m);
  if (threadIdx.x == 0) {
    s->amax_bits = m;
    s->flags = 0u;
  }
}

// One group of four consecutive elements: four roundings with the group's
// Philox block, packed as four INT16.
template <int MODE, bool SAT>
__device__ __forceinline__ uint2 quant_group(const uint4 v, int64_t g, int32_t es, bool all_zero, uint32_t key0,
                                             uint32_t key1, uint32_t role, bool& saturated) {
  const uint32_t fb[4] = {v.x, v.y, v.z, v.w};
  uint32_t u[4] = {0u, 0u, 0u, 0u};
  if (MODE == DFP_ROUND_STOCHASTIC) {
    const uint4 r = philox4x32_10(make_uint4((uint32_t)g, (uint32_t)((uint64_t)g >> 32), role, 0u), key0, key1);
    u[0] = r.x; u[1] = r.y; u[2] = r.z; u[3] = r.w;
  }
  int32_t iv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int32_t q = round_one<MODE>(fb[i], es, u[i]);
    q = all_zero ? 0 : q;
    if (SAT) {  // P = 16: |x| < 2^15 rounds to at most 2^15
      const int32_t c = min(max(q, -32767), 32767);
      saturated |= c != q;
      q = c;
    }
    iv[i] = q;
  }
  return make_uint2(((uint32_t)iv[0] & 0xffffu) | ((uint32_t)iv[1] << 16),
                    ((uint32_t)iv[2] & 0xffffu) | ((uint32_t)iv[3] << 16));
}

template <int MODE, bool SAT>
__global__ __launch_bounds__(kBlock) void k_quant_convert(const float* __restrict__ src,
                                                          int16_t* __restrict__ dst, int64_t n,
                                                          dfp_scale* __restrict__ s, int32_t bits,
                                                          uint32_t key0, uint32_t key1, uint32_t role) {
  const ScaleFromMax sc = scale_from_max(s->amax_bits, bits);
  const int32_t es = sc.es;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    s->exp = es;
    if (sc.flags) atomicOr(&s->flags, sc.flags);
  }
  const bool all_zero = sc.all_zero;
  const int64_t full = n >> 2;  // whole groups of four
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const uint4* src4 = reinterpret_cast<const uint4*>(src);
  uint2* dst4 = reinterpret_cast<uint2*>(dst);
  bool saturated = false;
  int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  // two groups per iteration: both loads in flight before either is rounded
  for (; g + stride < full; g += 2 * stride) {
    const uint4 v0 = src4[g], v1 = src4[g + stride];
    dst4[g] = quant_group<MODE, SAT>(v0, g, es, all_zero, key0, key1, role, saturated);
    dst4[g + stride] = quant_group<MODE, SAT>(v1, g + stride, es, all_zero, key0, key1, role, saturated);
  }
  if (g < full) dst4[g] = quant_group<MODE, SAT>(src4[g], g, es, all_zero, key0, key1, role, saturated);
  if ((n & 3) && blockIdx.x == 0 && threadIdx.x == 0) {  // the last, partial group
    const uint32_t* s1 = reinterpret_cast<const uint32_t*>(src);
    const int64_t base = full << 2;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    v.x = s1[base];
    if (base + 1 < n) v.y = s1[base + 1];
    if (base + 2 < n) v.z = s1[base + 2];
    const uint2 packed = quant_group<MODE, SAT>(v, full, es, all_zero, key0, key1, role, saturated);
    dst[base] = (int16_t)(packed.x & 0xffffu);
    if (base + 1 < n) dst[base + 1] = (int16_t)(packed.x >> 16);
    if (base + 2 < n) dst[base + 2] = (int16_t)(packed.y & 0xffffu);
  }
  if (SAT && saturated) atomicOr(&s->flags, DFP_FLAG_SATURATED);
}

// Whole quantisation of a small tensor in one launch (P = 15, so no workgroup
// raises a saturation flag).  Group g (elements 4g .. 4g + 3) is group
// g mod 1024 of slice g / 1024; workgroup b rounds slice b, one group per
// thread.  Every workgroup loads the whole tensor (at most kSmallQuantElems
// elements, 16 slices; read from L2 by all but the first), thread i slice k's
// group i into register k, and its own group once more, all loads in flight
// at once; it reduces the max, derives the scale and rounds its group, with
// the same per-group Philox counters as k_quant_convert.  Workgroup 0 writes
// the scale.
constexpr int64_t kSmallQuantElems = 65536;
constexpr int kSmallThreads = 1024;
constexpr int kSmallSlices = (int)(kSmallQuantElems / 4 / kSmallThreads);  // 16

template <int MODE>
__global__ __launch_bounds__(kSmallThreads) void k_quant_small(const float* __restrict__ src,
                                                               int16_t* __restrict__ dst, int64_t n,
                                                               dfp_scale* __restrict__ s, int32_t bits,
                                                               uint32_t key0, uint32_t key1, uint32_t role) {
  __shared__ uint32_t red[kSmallThreads / 64];
  const uint4* src4 = reinterpret_cast<const uint4*>(src);
  const uint32_t* s1 = reinterpret_cast<const uint32_t*>(src);
  const int32_t n4 = (int32_t)(n >> 2);
  const int32_t groups = (int32_t)((n + 3) >> 2);
  const int32_t nsl = (groups + kSmallThreads - 1) / kSmallThreads;  // slices, one per workgroup
  const int32_t tid = (int32_t)threadIdx.x;
  const int32_t g = (int32_t)blockIdx.x * kSmallThreads + tid;  // the group this thread rounds
  // its own group, requested with the others (a second request for one of
  // them, in flight at the same time); every load is issued (an index past the
  // whole groups re-reads the last one: the max is unchanged), so that none
  // waits for another
  uint4 w4 = make_uint4(0u, 0u, 0u, 0u);
  uint4 v[kSmallSlices];
#pragma unroll
  for (int k = 0; k < kSmallSlices; ++k) v[k] = make_uint4(0u, 0u, 0u, 0u);
  if (n4 > 0) {
    w4 = src4[min(g, n4 - 1)];
#pragma unroll
    for (int k = 0; k < kSmallSlices; ++k) v[k] = src4[min(k * kSmallThreads + tid, n4 - 1)];
  }
  // the partial last group (n not a multiple of 4), from single elements
  uint4 vp = make_uint4(0u, 0u, 0u, 0u);
  if (n4 < groups && (n4 & (kSmallThreads - 1)) == tid) {
    const int64_t base = (int64_t)n4 << 2;
    vp.x = s1[base];
    if (base + 1 < n) vp.y = s1[base + 1];
    if (base + 2 < n) vp.z = s1[base + 2];
  }
  uint32_t mm = abs_max4(vp);
#pragma unroll
  for (int k = 0; k < kSmallSlices; ++k) mm = max(mm, abs_max4(v[k]));
  mm = wave_max(mm);
  if ((tid & 63) == 0) red[tid >> 6] = mm;
  __syncthreads();
  mm = red[0];
#pragma unroll
  for (int i = 1; i < kSmallThreads / 64; ++i) mm = max(mm, red[i]);
  const ScaleFromMax sc = scale_from_max(mm, bits);
  if (blockIdx.x == 0 && tid == 0) {
    s->amax_bits = mm;
    s->exp = sc.es;
    s->flags = sc.flags;
  }
  if (g >= groups) return;
  const uint4 w = g < n4 ? w4 : vp;  // g == n4: the partial group
  bool saturated = false;
  const uint2 packed = quant_group<MODE, false>(w, g, sc.es, sc.all_zero, key0, key1, role, saturated);
  if (g < n4) {
    reinterpret_cast<uint2*>(dst)[g] = packed;
  } else {  // the last, partial group
    const int64_t base = (int64_t)g << 2;
    dst[base] = (int16_t)(packed.x & 0xffffu);
    if (base + 1 < n) dst[base + 1] = (int16_t)(packed.x >> 16);
    if (base + 2 < n) dst[base + 2] = (int16_t)(packed.y & 0xffffu);
  }
}

// ---------------------------------------------------------------- DFP-32 -> DFP
// Integer down-conversion (Eq. 6 with the shift count read as in Eq. 2):
// Rs = floor(log2 max|i|) - (P - 2), E_out = E_in + Rs (clamped at -128 by
// raising Rs), and every integer rounded from i * 2^-Rs with the descriptor's
// mode.  i * 2^-Rs is split exactly as X = floor(i * 2^(32-Rs)) in 64 bits.
__device__ __forceinline__ uint32_t abs_u32(int32_t v) { return v < 0 ? 0u - (uint32_t)v : (uint32_t)v; }

__global__ __launch_bounds__(kBlock) void k_amax_i32(const int32_t* __restrict__ src, int64_t n,
                                                     uint32_t* __restrict__ part, dfp_scale* __restrict__ s) {
  const int4* src4 = reinterpret_cast<const int4*>(src);
  const int64_t n4 = n >> 2;
  uint32_t m = 0u;
  for (int64_t base = (int64_t)blockIdx.x * kAmaxChunk; base < n4; base += (int64_t)gridDim.x * kAmaxChunk) {
    if (base + kAmaxChunk <= n4) {
      int4 v[kAmaxUnroll];
#pragma unroll
      for (int k = 0; k < kAmaxUnroll; ++k) v[k] = src4[base + threadIdx.x + k * kBlock];
#pragma unroll
      for (int k = 0; k < kAmaxUnroll; ++k)
        m = max(m, max(max(abs_u32(v[k].x), abs_u32(v[k].y)), max(abs_u32(v[k].z), abs_u32(v[k].w))));
    } else {
      for (int64_t i = base + threadIdx.x; i < n4; i += kBlock) {
        const int4 v = src4[i];
        m = max(m, max(max(abs_u32(v.x), abs_u32(v.y)), max(abs_u32(v.z), abs_u32(v.w))));
      }
    }
  }
  if (blockIdx.x == 0)
    for (int64_t t = 4 * n4 + threadIdx.x; t < n; t += kBlock) m = max(m, abs_u32(src[t]));
  m = block_max(m);
  if (threadIdx.x == 0) {
    if (part) {
      part[blockIdx.x] = m;
    } else {
      s->amax_bits = m;
      s->flags = 0u;
    }
  }
}

template <int MODE>
__device__ __forceinline__ int32_t round_i32(int32_t v, int32_t rs, uint32_t u) {
  int64_t X;
  // v * 2^(32 - Rs): exact for Rs <= 32 (Rs < 0 only when max|i| < 2^(P-2), so
  // no overflow); beyond, the dropped bits lie below the 2^-32 fraction bit
  if (rs <= 32) X = (int64_t)((uint64_t)(int64_t)v << (32 - rs));
  else X = (int64_t)v >> min(rs - 32, 63);
  const int32_t fl = (int32_t)(X >> 32);
  const uint32_t F = (uint32_t)X;
  bool up;
  if (MODE == DFP_ROUND_NEAREST) up = (F > 0x80000000u) || (F == 0x80000000u && (fl & 1));
  else if (MODE == DFP_ROUND_BIASED) up = F >= 0x80000000u;
  else if (MODE == DFP_ROUND_STOCHASTIC) up = u < F;
  else up = false;
  return fl + (up ? 1 : 0);
}

template <int MODE, bool SAT>
__global__ __launch_bounds__(kBlock) void k_i32_convert(const int32_t* __restrict__ src, int16_t* __restrict__ dst,
                                                        int64_t n, const dfp_scale* __restrict__ amax_from,
                                                        const dfp_scale* __restrict__ sin, dfp_scale* sout,
                                                        int32_t bits, uint32_t key0, uint32_t key1, uint32_t role) {
  const uint32_t mx = amax_from->amax_bits;
  const int32_t e_in = sin->exp;
  const bool zero = mx == 0u;
  int32_t rs = 0, e_out = 0;
  bool clamped = false;
  if (!zero) {
    rs = (31 - __clz((int)mx)) - (bits - 2);
    e_out = e_in + rs;
    if (e_out < -128) {
      rs += -128 - e_out;
      e_out = -128;
      clamped = true;
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    sout->amax_bits = mx;
    sout->exp = e_out;
    const uint32_t f = (zero ? DFP_FLAG_ZERO_TENSOR : 0u) | (clamped ? DFP_FLAG_EXP_CLAMPED : 0u);
    // without saturation no other workgroup writes the flags: store them whole;
    // with it the launcher has cleared them and workgroups OR in SATURATED
    if (!SAT) sout->flags = f;
    else if (f) atomicOr(&sout->flags, f);
  }
  const int64_t groups = (n + 3) >> 2;
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  bool saturated = false;
  for (int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x; g < groups; g += stride) {
    const int64_t base = g << 2;
    int32_t v[4];
    const bool full = base + 4 <= n;
    if (full) {
      const int4 q = reinterpret_cast<const int4*>(src)[g];
      v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (base + i < n) ? src[base + i] : 0;
    }
    uint32_t u[4] = {0u, 0u, 0u, 0u};
    if (MODE == DFP_ROUND_STOCHASTIC) {
      const uint4 r = philox4x32_10(make_uint4((uint32_t)g, (uint32_t)((uint64_t)g >> 32), role, 0u), key0, key1);
      u[0] = r.x; u[1] = r.y; u[2] = r.z; u[3] = r.w;
    }
    int32_t iv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int32_t r = zero ? 0 : round_i32<MODE>(v[i], rs, u[i]);
      if (SAT) {
        const int32_t c = min(max(r, -32767), 32767);
        saturated |= c != r;
        r = c;
      }
      iv[i] = r;
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
  if (SAT && saturated) atomicOr(&sout->flags, DFP_FLAG_SATURATED);
}

// ---------------------------------------------------------------- Blocked-DFP
// Each block of B consecutive elements of a [rows][cols] row gets its own
// shared exponent (Eq. 1-2 on the block's max) and is rounded like a tensor of
// its own (Eq. 3), the stochastic word still that of the element's flat index.
// One wave per (row, block): a max pass, then the rounding pass.  VEC4: rows
// and blocks start at multiples of 4 elements, so a lane takes aligned groups
// of 4 (one Philox block, one 16-byte load).  s->flags starts at ZERO_TENSOR
// (k_blocked_init); a wave with a non-zero or non-finite block clears it.
__global__ void k_blocked_init(dfp_scale* s) {
  if (threadIdx.x == 0) {
    s->amax_bits = 0u;
    s->exp = 0;
    s->flags = DFP_FLAG_ZERO_TENSOR;
  }
}

template <int MODE, bool SAT, bool VEC4>
__global__ __launch_bounds__(kBlock) void k_quant_blocked(const float* __restrict__ src, int16_t* __restrict__ dst,
                                                          int8_t* __restrict__ exps, int64_t rows, int64_t cols,
                                                          int64_t B, int64_t nb, dfp_scale* s, int32_t bits,
                                                          uint32_t key0, uint32_t key1, uint32_t role,
                                                          int32_t seg_log2) {
  // a wave serves 64 >> seg_log2 blocks at a time, 2^seg_log2 lanes each, in a
  // grid-stride loop; the workgroup reports its max and flags once at the end
  const int lane = threadIdx.x & 63;
  const int S = 1 << seg_log2;
  const int sl = lane & (S - 1);
  const int64_t nblk = rows * nb;
  const int64_t stride = ((int64_t)gridDim.x * (kBlock / 64)) << (6 - seg_log2);
  uint32_t wmax = 0u;
  bool f_nonfinite = false, f_clamped = false, f_sat = false, f_nonzero = false;
  for (int64_t wave_first = ((int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6)) << (6 - seg_log2);
       wave_first < nblk; wave_first += stride) {  // uniform per wave
    const int64_t blk = wave_first + (lane >> seg_log2);
    const bool valid = blk < nblk;
    const int64_t r = valid ? blk / nb : 0, b = valid ? blk % nb : 0;
    const int64_t c0 = b * B, c1 = valid ? min(c0 + B, cols) : c0;
    const int64_t base = r * cols;
    const uint32_t* s32 = reinterpret_cast<const uint32_t*>(src) + base;
    uint32_t mb = 0u;
    if (VEC4) {
      for (int64_t c = c0 + 4 * sl; c < c1; c += 4 * S) {
        const uint4 v = *reinterpret_cast<const uint4*>(s32 + c);
        mb = max(mb, max(max(v.x & 0x7fffffffu, v.y & 0x7fffffffu), max(v.z & 0x7fffffffu, v.w & 0x7fffffffu)));
      }
    } else {
      for (int64_t c = c0 + sl; c < c1; c += S) mb = max(mb, s32[c] & 0x7fffffffu);
    }
    for (int off = S >> 1; off > 0; off >>= 1) mb = max(mb, (uint32_t)__shfl_xor((int)mb, off, 64));
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
    const bool all_zero = nonfinite || zero;
    bool saturated = false;
    auto convert = [&](uint32_t fb, uint32_t u) {
      int32_t v = all_zero ? 0 : round_one<MODE>(fb, es, u);
      if (SAT) {
        const int32_t c = min(max(v, -32767), 32767);
        saturated |= c != v;
        v = c;
      }
      return v;
    };
    if (VEC4) {
      for (int64_t c = c0 + 4 * sl; c < c1; c += 4 * S) {
        const uint4 v = *reinterpret_cast<const uint4*>(s32 + c);
        const uint64_t g = (uint64_t)(base + c) >> 2;
        uint4 rw = make_uint4(0u, 0u, 0u, 0u);
        if (MODE == DFP_ROUND_STOCHASTIC)
          rw = philox4x32_10(make_uint4((uint32_t)g, (uint32_t)(g >> 32), role, 0u), key0, key1);
        const int32_t i0 = convert(v.x, rw.x), i1 = convert(v.y, rw.y), i2 = convert(v.z, rw.z),
                      i3 = convert(v.w, rw.w);
        uint2 packed;
        packed.x = ((uint32_t)i0 & 0xffffu) | ((uint32_t)i1 << 16);
        packed.y = ((uint32_t)i2 & 0xffffu) | ((uint32_t)i3 << 16);
        *reinterpret_cast<uint2*>(dst + base + c) = packed;
      }
    } else {
      for (int64_t c = c0 + sl; c < c1; c += S) {
        const uint64_t idx = (uint64_t)(base + c);
        uint32_t u = 0u;
        if (MODE == DFP_ROUND_STOCHASTIC) {
          const uint4 rw = philox4x32_10(make_uint4((uint32_t)(idx >> 2), (uint32_t)(idx >> 34), role, 0u), key0,
                                         key1);
          const uint32_t w = idx & 3u;
          u = w == 0 ? rw.x : (w == 1 ? rw.y : (w == 2 ? rw.z : rw.w));
        }
        dst[base + c] = (int16_t)convert(s32[c], u);
      }
    }
    if (valid && sl == 0) exps[b * rows + r] = (int8_t)es;
    wmax = max(wmax, mb);
    f_nonfinite |= valid && nonfinite;
    f_clamped |= valid && clamped;
    f_sat |= saturated;
    f_nonzero |= valid && !zero;
  }
  // workgroup totals, then one guarded set of atomics
  __shared__ uint32_t red_max[kBlock / 64], red_flags[kBlock / 64];
  for (int off = 32; off > 0; off >>= 1) wmax = max(wmax, (uint32_t)__shfl_xor((int)wmax, off, 64));
  const uint32_t wf = (__any(f_nonfinite) ? DFP_FLAG_NONFINITE : 0u) | (__any(f_clamped) ? DFP_FLAG_EXP_CLAMPED : 0u) |
                      (__any(f_sat) ? DFP_FLAG_SATURATED : 0u) | (__any(f_nonzero) ? 0x80000000u : 0u);
  if (lane == 0) {
    red_max[threadIdx.x >> 6] = wmax;
    red_flags[threadIdx.x >> 6] = wf;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t m = red_max[0], f = red_flags[0];
    for (int i = 1; i < kBlock / 64; ++i) {
      m = max(m, red_max[i]);
      f |= red_flags[i];
    }
    if (m > __atomic_load_n(&s->amax_bits, __ATOMIC_RELAXED)) atomicMax(&s->amax_bits, m);
    const uint32_t fl = f & 0x7fffffffu;
    if (fl && (__atomic_load_n(&s->flags, __ATOMIC_RELAXED) & fl) != fl) atomicOr(&s->flags, fl);
    if ((f & 0x80000000u) && (__atomic_load_n(&s->flags, __ATOMIC_RELAXED) & DFP_FLAG_ZERO_TENSOR))
      atomicAnd(&s->flags, ~DFP_FLAG_ZERO_TENSOR);
  }
}

int grid_for(int64_t work_items) {
  int64_t blocks = (work_items + kBlock - 1) / kBlock;
  if (blocks < 1) blocks = 1;
  if (blocks > 8192) blocks = 8192;
  return (int)blocks;
}

}  // namespace

template <int MODE, bool SAT>
static dfp_status launch_blocked_mode(const float* src, int16_t* dst, int8_t* exps, int64_t rows, int64_t cols,
                                      int64_t B, dfp_scale* s, int32_t bits, uint32_t k0, uint32_t k1,
                                      uint32_t role, bool vec4, hipStream_t st) {
  const int64_t nb = (cols + B - 1) / B;
  // lanes per block: enough for one pass over the block, a power of two up to 64
  const int64_t lanes = vec4 ? (B + 3) / 4 : B;
  int32_t seg_log2 = 0;
  while (seg_log2 < 6 && ((int64_t)1 << seg_log2) < lanes) ++seg_log2;
  const int64_t waves = (rows * nb + (64 >> seg_log2) - 1) >> (6 - seg_log2);
  // at most 1024 workgroups (4 per CU): each reports once, so the scale sees few atomics
  const dim3 grid((unsigned)std::min<int64_t>(1024, (waves + kBlock / 64 - 1) / (kBlock / 64)));
  if (vec4)
    DFP_LAUNCH(K_QUANT_BLOCKED, (k_quant_blocked<MODE, SAT, true>), grid, dim3(kBlock), 0, st, src, dst, exps, rows,
               cols, B, nb, s, bits, k0, k1, role, seg_log2);
  else
    DFP_LAUNCH(K_QUANT_BLOCKED, (k_quant_blocked<MODE, SAT, false>), grid, dim3(kBlock), 0, st, src, dst, exps,
               rows, cols, B, nb, s, bits, k0, k1, role, seg_log2);
  return DFP_OK;
}

template <int MODE>
static dfp_status launch_blocked_sat(const float* src, int16_t* dst, int8_t* exps, int64_t rows, int64_t cols,
                                     int64_t B, dfp_scale* s, int32_t bits, uint32_t k0, uint32_t k1, uint32_t role,
                                     bool vec4, hipStream_t st) {
  if (bits == 16) return launch_blocked_mode<MODE, true>(src, dst, exps, rows, cols, B, s, bits, k0, k1, role, vec4, st);
  return launch_blocked_mode<MODE, false>(src, dst, exps, rows, cols, B, s, bits, k0, k1, role, vec4, st);
}

dfp_status launch_quantize_blocked(const float* src, int16_t* dst, int8_t* exps, int64_t rows, int64_t cols,
                                   int64_t B, dfp_scale* s, int32_t bits, int32_t rounding, uint64_t seed,
                                   uint32_t role, hipStream_t st) {
  DFP_LAUNCH(K_SCALE_RESET, k_blocked_init, dim3(1), dim3(64), 0, st, s);
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  // aligned 4-groups never straddle a block or a row
  const bool vec4 = (cols % 4) == 0 && (B % 4) == 0 && (reinterpret_cast<uintptr_t>(src) & 15) == 0 &&
                    (reinterpret_cast<uintptr_t>(dst) & 7) == 0;
  switch (rounding) {
    case DFP_ROUND_NEAREST:
      return launch_blocked_sat<DFP_ROUND_NEAREST>(src, dst, exps, rows, cols, B, s, bits, k0, k1, role, vec4, st);
    case DFP_ROUND_STOCHASTIC:
      return launch_blocked_sat<DFP_ROUND_STOCHASTIC>(src, dst, exps, rows, cols, B, s, bits, k0, k1, role, vec4, st);
    case DFP_ROUND_BIASED:
      return launch_blocked_sat<DFP_ROUND_BIASED>(src, dst, exps, rows, cols, B, s, bits, k0, k1, role, vec4, st);
    default:
      return launch_blocked_sat<DFP_ROUND_DOWN>(src, dst, exps, rows, cols, B, s, bits, k0, k1, role, vec4, st);
  }
}

dfp_status launch_scale_reset(dfp_scale* s, hipStream_t st) {
  DFP_LAUNCH(K_SCALE_RESET, k_scale_reset, dim3(1), dim3(64), 0, st, s);
  return DFP_OK;
}

dfp_status launch_amax(const float* src, int64_t n, int16_t* scratch, dfp_scale* s, hipStream_t st) {
  // about 16 KiB or more per workgroup, at most kAmaxMaxParts workgroups; the
  // partial maxima need 4 bytes each of the 2n-byte destination
  int64_t parts = (n / 4 + kBlock * kAmaxUnroll - 1) / (kBlock * kAmaxUnroll);
  parts = std::min<int64_t>(std::min<int64_t>(parts, kAmaxMaxParts), n / 2);
  if (parts <= 1) {
    DFP_LAUNCH(K_AMAX, k_amax, dim3(1), dim3(kBlock), 0, st, src, n, (uint32_t*)nullptr, s);
    return DFP_OK;
  }
  uint32_t* part = reinterpret_cast<uint32_t*>(scratch);
  DFP_LAUNCH(K_AMAX, k_amax, dim3((unsigned)parts), dim3(kBlock), 0, st, src, n, part, s);
  DFP_LAUNCH(K_AMAX, k_amax_final, dim3(1), dim3(kBlock), 0, st, part, (int32_t)parts, s);
  return DFP_OK;
}

dfp_status launch_amax_final(const uint32_t* part, int32_t nparts, dfp_scale* s, hipStream_t st) {
  DFP_LAUNCH(K_AMAX, k_amax_final, dim3(1), dim3(kBlock), 0, st, part, nparts, s);
  return DFP_OK;
}

template <int MODE>
static dfp_status launch_qc_mode(const float* src, int16_t* dst, int64_t n, dfp_scale* s, int32_t bits,
                                 uint32_t k0, uint32_t k1, uint32_t role, hipStream_t st) {
  // Without the Philox stream the pass is bound by memory: at most eight
  // workgroups per CU, so a thread rounds several groups and shares its set-up
  // (scale, exponent) among them.  Stochastic rounding is bound by its VALU
  // work and runs faster with one group per thread (more waves to interleave).
  const int64_t blocks = grid_for((n + 3) / 4);
  const dim3 grid((unsigned)(MODE == DFP_ROUND_STOCHASTIC ? blocks : std::min<int64_t>(blocks, 2048)));
  if (bits == 16)
    DFP_LAUNCH(K_QUANT, (k_quant_convert<MODE, true>), grid, dim3(kBlock), 0, st, src, dst, n, s, bits, k0, k1, role);
  else
    DFP_LAUNCH(K_QUANT, (k_quant_convert<MODE, false>), grid, dim3(kBlock), 0, st, src, dst, n, s, bits, k0, k1, role);
  return DFP_OK;
}

template <int MODE>
static dfp_status launch_small_mode(const float* src, int16_t* dst, int64_t n, dfp_scale* s, int32_t bits,
                                    uint32_t k0, uint32_t k1, uint32_t role, hipStream_t st) {
  const int64_t blocks = std::max<int64_t>(1, ((n + 3) / 4 + kSmallThreads - 1) / kSmallThreads);  // slices
  DFP_LAUNCH(K_QUANT, k_quant_small<MODE>, dim3((unsigned)blocks), dim3(kSmallThreads), 0, st, src, dst, n, s, bits,
             k0, k1, role);
  return DFP_OK;
}

dfp_status launch_quantize(const float* src, int16_t* dst, int64_t n, dfp_scale* s, int32_t bits, int32_t rounding,
                           uint64_t seed, uint32_t role, hipStream_t st) {
  if (n > kSmallQuantElems || bits != 15) {
    dfp_status rc = launch_amax(src, n, dst, s, st);
    if (rc != DFP_OK) return rc;
    return launch_quant_convert(src, dst, n, s, bits, rounding, seed, role, st);
  }
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  switch (rounding) {
    case DFP_ROUND_NEAREST: return launch_small_mode<DFP_ROUND_NEAREST>(src, dst, n, s, bits, k0, k1, role, st);
    case DFP_ROUND_STOCHASTIC: return launch_small_mode<DFP_ROUND_STOCHASTIC>(src, dst, n, s, bits, k0, k1, role, st);
    case DFP_ROUND_BIASED: return launch_small_mode<DFP_ROUND_BIASED>(src, dst, n, s, bits, k0, k1, role, st);
    default: return launch_small_mode<DFP_ROUND_DOWN>(src, dst, n, s, bits, k0, k1, role, st);
  }
}

dfp_status launch_quant_convert(const float* src, int16_t* dst, int64_t n, dfp_scale* s, int32_t bits,
                                int32_t rounding, uint64_t seed, uint32_t role, hipStream_t st) {
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  switch (rounding) {
    case DFP_ROUND_NEAREST: return launch_qc_mode<DFP_ROUND_NEAREST>(src, dst, n, s, bits, k0, k1, role, st);
    case DFP_ROUND_STOCHASTIC: return launch_qc_mode<DFP_ROUND_STOCHASTIC>(src, dst, n, s, bits, k0, k1, role, st);
    case DFP_ROUND_BIASED: return launch_qc_mode<DFP_ROUND_BIASED>(src, dst, n, s, bits, k0, k1, role, st);
    default: return launch_qc_mode<DFP_ROUND_DOWN>(src, dst, n, s, bits, k0, k1, role, st);
  }
}

template <int MODE>
static dfp_status launch_i32_mode(const int32_t* src, int16_t* dst, int64_t n, const dfp_scale* amax_from,
                                  const dfp_scale* sin, dfp_scale* sout, int32_t bits, uint32_t k0, uint32_t k1,
                                  uint32_t role, hipStream_t st) {
  const dim3 grid(grid_for((n + 3) / 4));
  if (bits == 16)
    DFP_LAUNCH(K_DC_I32, (k_i32_convert<MODE, true>), grid, dim3(kBlock), 0, st, src, dst, n, amax_from, sin, sout,
               bits, k0, k1, role);
  else
    DFP_LAUNCH(K_DC_I32, (k_i32_convert<MODE, false>), grid, dim3(kBlock), 0, st, src, dst, n, amax_from, sin, sout,
               bits, k0, k1, role);
  return DFP_OK;
}

dfp_status launch_downconvert_i32(const int32_t* src, int64_t n, const dfp_scale* sin, int16_t* dst, dfp_scale* sout,
                                  bool amax_ready, int32_t bits, int32_t rounding, uint64_t seed, uint32_t role,
                                  hipStream_t st) {
  const dfp_scale* amax_from = sin;
  if (amax_ready) {
    // P = 16 saturation flags are ORed in by every workgroup: start from zero
    if (bits == 16 && launch_scale_reset(sout, st) != DFP_OK) return DFP_ERR_HIP;
  } else {
    int64_t parts = (n / 4 + kAmaxChunk - 1) / kAmaxChunk;
    parts = std::min<int64_t>(std::min<int64_t>(parts, kAmaxMaxParts), n / 2);
    if (parts <= 1) {
      DFP_LAUNCH(K_AMAX, k_amax_i32, dim3(1), dim3(kBlock), 0, st, src, n, (uint32_t*)nullptr, sout);
    } else {
      uint32_t* part = reinterpret_cast<uint32_t*>(dst);
      DFP_LAUNCH(K_AMAX, k_amax_i32, dim3((unsigned)parts), dim3(kBlock), 0, st, src, n, part, sout);
      DFP_LAUNCH(K_AMAX, k_amax_final, dim3(1), dim3(kBlock), 0, st, part, (int32_t)parts, sout);
    }
    amax_from = sout;
  }
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  switch (rounding) {
    case DFP_ROUND_NEAREST:
      return launch_i32_mode<DFP_ROUND_NEAREST>(src, dst, n, amax_from, sin, sout, bits, k0, k1, role, st);
    case DFP_ROUND_STOCHASTIC:
      return launch_i32_mode<DFP_ROUND_STOCHASTIC>(src, dst, n, amax_from, sin, sout, bits, k0, k1, role, st);
    case DFP_ROUND_BIASED:
      return launch_i32_mode<DFP_ROUND_BIASED>(src, dst, n, amax_from, sin, sout, bits, k0, k1, role, st);
    default:
      return launch_i32_mode<DFP_ROUND_DOWN>(src, dst, n, amax_from, sin, sout, bits, k0, k1, role, st);
  }
}

}  // namespace dfp
