// VALU product path: one lane per output element, INT16 x INT16 products
// summed with 32-bit wrapping integer adds, one INT32 partial per chunk of L
// reduction indices, each converted to FP32 and added in chunk order, then
// scaled once by 2^(Ea+Eb) (Algorithm 2 and Sec. 4.3 of the paper).
//
// It walks the canonical reduction order of each direction
//   forward          t = (r*S + s)*C + c
//   backward-data    t = (r*S + s)*K + k
//   backward-weights t = (n*P + p)*Q + q   (segments of G chunks)
// and handles every shape, stride and chunk length.  It is the measured
// alternative to the MFMA path, not the default.
#include "dfp_internal.h"

namespace dfp {

namespace {

constexpr int kBlock = 256;

// Running state of one output's chunked reduction.
struct ChunkAcc {
  uint32_t acc = 0;   // INT32 partial of the current chunk (wraps mod 2^32)
  int32_t fill = 0;   // products in the current chunk so far
  int64_t j = 0;      // index of the current chunk
  float sum = 0.f;    // FP32 sum over finished chunks (or segments)
  float seg = 0.f;    // FP32 sum inside the current segment (backward-weights)
};

template <bool PARTIALS, bool SEGMENTED>
__device__ __forceinline__ void flush(ChunkAcc& st, int32_t G, int32_t* partials, int64_t O, int64_t o) {
  const float f = (float)(int32_t)st.acc;
  if (PARTIALS) partials[st.j * O + o] = (int32_t)st.acc;
  if (SEGMENTED) {
    const int64_t in_seg = st.j % G;
    st.seg = (in_seg == 0) ? f : st.seg + f;
    if (in_seg == G - 1) {
      st.sum = (st.j / G == 0) ? st.seg : st.sum + st.seg;
    }
  } else {
    st.sum = (st.j == 0) ? f : st.sum + f;
  }
  ++st.j;
  st.acc = 0;
  st.fill = 0;
}

template <bool PARTIALS, bool SEGMENTED>
__device__ __forceinline__ void push(ChunkAcc& st, int32_t prod, int32_t L, int32_t G, int32_t* partials,
                                     int64_t O, int64_t o) {
  st.acc += (uint32_t)prod;
  if (++st.fill == L) flush<PARTIALS, SEGMENTED>(st, G, partials, O, o);
}

template <bool SEGMENTED>
__device__ __forceinline__ void finish_tail(ChunkAcc& st, int32_t G) {
  if (SEGMENTED && (st.j % G) != 0) {  // close a partly filled last segment
    st.sum = (st.j / G == 0) ? st.seg : st.sum + st.seg;
  }
}

// Block max of |y| bit patterns into so->amax_bits, plus the OUTPUT_INF flag.
__device__ __forceinline__ void epilogue_amax(float y, bool active, dfp_scale* so) {
  __shared__ uint32_t red[kBlock / 64];
  uint32_t m = active ? (__float_as_uint(y) & 0x7fffffffu) : 0u;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = red[0];
    for (int i = 1; i < kBlock / 64; ++i) b = max(b, red[i]);
    if (b > __atomic_load_n(&so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&so->amax_bits, b);
    if (b == 0x7f800000u) atomicOr(&so->flags, DFP_FLAG_OUTPUT_INF);
  }
}

// Single-chunk DFP-32 output: the wrapped INT32 sum, its |.| into so->amax_bits
// (one relaxed-read-guarded atomic per lane; this path is the reference one)
// and the output exponent.
__device__ __forceinline__ void store_i32(float* out, int64_t o, uint32_t acc, dfp_scale* so, int32_t e) {
  const int32_t v = (int32_t)acc;
  reinterpret_cast<int32_t*>(out)[o] = v;
  if (so) {
    const uint32_t m = v < 0 ? 0u - (uint32_t)v : (uint32_t)v;
    if (m > __atomic_load_n(&so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&so->amax_bits, m);
    if (o == 0) so->exp = e;
  }
}

template <bool PARTIALS, bool I32 = false>
__global__ __launch_bounds__(kBlock) void k_fwd_valu(Geom g, const int16_t* __restrict__ x,
                                                    const dfp_scale* __restrict__ sx,
                                                    const int16_t* __restrict__ w,
                                                    const dfp_scale* __restrict__ sw, float* __restrict__ y,
                                                    dfp_scale* so, int32_t* __restrict__ partials) {
  const int64_t O = (int64_t)g.n * g.k * g.p * g.q;
  const int64_t o = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  const bool active = o < O;
  float yv = 0.f;
  if (active) {
    const int32_t q = (int32_t)(o % g.q), p = (int32_t)((o / g.q) % g.p);
    const int32_t k = (int32_t)((o / ((int64_t)g.q * g.p)) % g.k);
    const int64_t n = o / ((int64_t)g.q * g.p * g.k);
    const int64_t hw = (int64_t)g.h * g.w, rs = (int64_t)g.r * g.s;
    ChunkAcc st;
    for (int32_t r = 0; r < g.r; ++r) {
      const int32_t ih = p * g.sh - g.ph + r;
      for (int32_t s = 0; s < g.s; ++s) {
        const int32_t iw = q * g.sw - g.pw + s;
        const bool valid = ih >= 0 && ih < g.h && iw >= 0 && iw < g.w;
        const int16_t* xp = x + (n * g.c) * hw + (valid ? (int64_t)ih * g.w + iw : 0);
        const int16_t* wp = w + ((int64_t)k * g.c) * rs + r * g.s + s;
        for (int32_t c = 0; c < g.c; ++c) {
          const int32_t prod = valid ? (int32_t)xp[c * hw] * (int32_t)wp[c * rs] : 0;
          if (I32) st.acc += (uint32_t)prod;
          else push<PARTIALS, false>(st, prod, g.L, g.G, partials, O, o);
        }
      }
    }
    if (I32) {
      store_i32(y, o, st.acc, so, sx->exp + sw->exp);
      return;
    }
    if (st.fill) flush<PARTIALS, false>(st, g.G, partials, O, o);
    yv = ldexpf(st.sum, sx->exp + sw->exp);
    y[o] = yv;
  }
  if (so && !I32) epilogue_amax(yv, active, so);
}

template <bool PARTIALS, bool I32 = false>
__global__ __launch_bounds__(kBlock) void k_bwdd_valu(Geom g, const int16_t* __restrict__ dy,
                                                     const dfp_scale* __restrict__ sdy,
                                                     const int16_t* __restrict__ w,
                                                     const dfp_scale* __restrict__ sw, float* __restrict__ dx,
                                                     dfp_scale* so, int32_t* __restrict__ partials) {
  const int64_t O = (int64_t)g.n * g.c * g.h * g.w;
  const int64_t o = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  const bool active = o < O;
  float yv = 0.f;
  if (active) {
    const int32_t iw = (int32_t)(o % g.w), ih = (int32_t)((o / g.w) % g.h);
    const int32_t c = (int32_t)((o / ((int64_t)g.w * g.h)) % g.c);
    const int64_t n = o / ((int64_t)g.w * g.h * g.c);
    const int64_t pq = (int64_t)g.p * g.q, crs = (int64_t)g.c * g.r * g.s;
    ChunkAcc st;
    for (int32_t r = 0; r < g.r; ++r) {
      const int32_t nh = ih + g.ph - r;
      const bool vh = nh >= 0 && (nh % g.sh) == 0 && nh / g.sh < g.p;
      for (int32_t s = 0; s < g.s; ++s) {
        const int32_t nw = iw + g.pw - s;
        const bool valid = vh && nw >= 0 && (nw % g.sw) == 0 && nw / g.sw < g.q;
        const int16_t* dp = dy + (n * g.k) * pq + (valid ? (int64_t)(nh / g.sh) * g.q + nw / g.sw : 0);
        const int16_t* wp = w + ((int64_t)c * g.r + r) * g.s + s;
        for (int32_t k = 0; k < g.k; ++k) {
          const int32_t prod = valid ? (int32_t)dp[k * pq] * (int32_t)wp[k * crs] : 0;
          if (I32) st.acc += (uint32_t)prod;
          else push<PARTIALS, false>(st, prod, g.L, g.G, partials, O, o);
        }
      }
    }
    if (I32) {
      store_i32(dx, o, st.acc, so, sdy->exp + sw->exp);
      return;
    }
    if (st.fill) flush<PARTIALS, false>(st, g.G, partials, O, o);
    yv = ldexpf(st.sum, sdy->exp + sw->exp);
    dx[o] = yv;
  }
  if (so && !I32) epilogue_amax(yv, active, so);
}

template <bool PARTIALS>
__global__ __launch_bounds__(kBlock) void k_bwdw_valu(Geom g, const int16_t* __restrict__ x,
                                                     const dfp_scale* __restrict__ sx,
                                                     const int16_t* __restrict__ dy,
                                                     const dfp_scale* __restrict__ sdy, float* __restrict__ dw,
                                                     int32_t* __restrict__ partials) {
  const int64_t O = (int64_t)g.k * g.c * g.r * g.s;
  const int64_t o = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (o >= O) return;
  const int32_t s = (int32_t)(o % g.s), r = (int32_t)((o / g.s) % g.r);
  const int32_t c = (int32_t)((o / ((int64_t)g.s * g.r)) % g.c);
  const int32_t k = (int32_t)(o / ((int64_t)g.s * g.r * g.c));
  const int64_t hw = (int64_t)g.h * g.w, pq = (int64_t)g.p * g.q;
  ChunkAcc st;
  for (int32_t n = 0; n < g.n; ++n) {
    const int16_t* xn = x + ((int64_t)n * g.c + c) * hw;
    const int16_t* dn = dy + ((int64_t)n * g.k + k) * pq;
    for (int32_t p = 0; p < g.p; ++p) {
      const int32_t ih = p * g.sh - g.ph + r;
      const bool vh = ih >= 0 && ih < g.h;
      for (int32_t q = 0; q < g.q; ++q) {
        const int32_t iw = q * g.sw - g.pw + s;
        const bool valid = vh && iw >= 0 && iw < g.w;
        const int32_t prod = valid ? (int32_t)xn[(int64_t)ih * g.w + iw] * (int32_t)dn[(int64_t)p * g.q + q] : 0;
        push<PARTIALS, true>(st, prod, g.L, g.G, partials, O, o);
      }
    }
  }
  if (st.fill) flush<PARTIALS, true>(st, g.G, partials, O, o);
  finish_tail<true>(st, g.G);
  dw[o] = ldexpf(st.sum, sx->exp + sdy->exp);
}

}  // namespace

dfp_status launch_conv_valu(int32_t dir, const Geom& g, const int16_t* a, const dfp_scale* sa, const int16_t* b,
                            const dfp_scale* sb, float* out, dfp_scale* so, int32_t* partials, hipStream_t st,
                            bool i32) {
  int64_t O;
  if (dir == DFP_FWD) O = (int64_t)g.n * g.k * g.p * g.q;
  else if (dir == DFP_BWD_DATA) O = (int64_t)g.n * g.c * g.h * g.w;
  else O = (int64_t)g.k * g.c * g.r * g.s;
  const dim3 grid((unsigned)((O + kBlock - 1) / kBlock)), block(kBlock);
  if (i32) {  // forward or backward-data, one chunk
    if (dir == DFP_FWD) DFP_LAUNCH(K_FWD_I32, (k_fwd_valu<false, true>), grid, block, 0, st, g, a, sa, b, sb, out, so, partials);
    else DFP_LAUNCH(K_BWDD_I32, (k_bwdd_valu<false, true>), grid, block, 0, st, g, a, sa, b, sb, out, so, partials);
    return DFP_OK;
  }
  if (dir == DFP_FWD) {
    if (partials) DFP_LAUNCH(K_FWD_VALU, k_fwd_valu<true>, grid, block, 0, st, g, a, sa, b, sb, out, so, partials);
    else DFP_LAUNCH(K_FWD_VALU, k_fwd_valu<false>, grid, block, 0, st, g, a, sa, b, sb, out, so, partials);
  } else if (dir == DFP_BWD_DATA) {
    if (partials) DFP_LAUNCH(K_BWDD_VALU, k_bwdd_valu<true>, grid, block, 0, st, g, a, sa, b, sb, out, so, partials);
    else DFP_LAUNCH(K_BWDD_VALU, k_bwdd_valu<false>, grid, block, 0, st, g, a, sa, b, sb, out, so, partials);
  } else {
    if (partials) DFP_LAUNCH(K_BWDW_VALU, k_bwdw_valu<true>, grid, block, 0, st, g, a, sa, b, sb, out, partials);
    else DFP_LAUNCH(K_BWDW_VALU, k_bwdw_valu<false>, grid, block, 0, st, g, a, sa, b, sb, out, partials);
  }
  return DFP_OK;
}

}  // namespace dfp
