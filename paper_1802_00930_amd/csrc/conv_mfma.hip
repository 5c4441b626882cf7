// MFMA product path for the forward and backward-data convolutions.
//
// Exact INT16 x INT16 products from int8 matrix cores: every INT16 operand a
// is split into two signed byte digits, lo = a mod 256 read as int8 and
// hi = (a + 128) >> 8, so a = 256*hi + lo (exact for a in [-32768, 32639];
// DFP15 integers are within [-2^14, 2^14]).  Then
//   a*b = 65536*(hi_a*hi_b) + 256*(hi_a*lo_b + lo_a*hi_b) + lo_a*lo_b,
// and one chunk's INT32 partial is
//   P_j = (HH << 16) + (X << 8) + LL   (mod 2^32)
// with HH, X, LL three int32 MFMA accumulators over the chunk's products.
// Integer MFMA accumulation wraps modulo 2^32, so P_j equals the wrapped
// INT32 chunk sum bit for bit (Sec. 4.3 overflow semantics).
//
// Implicit GEMM: D[m][g] = sum_t A[m][t] * B[t][g], m = output channel,
// g = output pixel (n, p, q), t = canonical reduction index.
//   forward        A[k][t] = w[k,c,r,s]          t = (r*S + s)*C + c
//                  B[t][g] = x[n, c, p*sh - ph + r, q*sw - pw + s]
//   backward-data  A[c][t] = w[k,c,r,s]          t = (r*S + s)*K + k
//                  B[t][g] = dy[n, k, (h+ph-r)/sh, (w+pw-s)/sw]
// Two prep kernels rewrite the operands once per call into the workspace:
//   - A as digit planes blocked by 32 reduction indices, [kb][m][half][32 B]
//     (16 hi digits then 16 lo digits), zero-padded past T and past M;
//   - B as a zero-padded (and, for strided backward-data, zero-dilated)
//     channels-last digit tensor [n][row][col][cgroup][32 B], so every
//     (pixel, tap, 16 channels) operand is one aligned 32-byte load and
//     padding needs no bounds checks.
// Main kernel: 256 threads = 4 waves; workgroup tile 64 output channels x 128
// pixels; wave tile 64 x 32 = two v_mfma_i32_32x32x32_i8 tiles.  Per block of
// 32 reduction indices each lane loads its B column (32 B) and its two A rows
// (2 x 32 B) and issues HH, LL and the two cross products per tile.  At each
// chunk end the three accumulators are recombined, converted to FP32 and added
// to the running FP32 sum in chunk order; chunk lengths that are not a
// multiple of 32 run the block once per chunk it overlaps, with the bytes of
// the other chunks masked to zero.
#include <algorithm>
#include <type_traits>

#include "dfp_internal.h"
#include "conv_mfma.h"

// Set to 1 by the build for a kernel whose assembly fails the split-read
// check of asm_check.py (an instruction names a register of an inline-asm LDS
// read before the wait that completes it); such a kernel is not launched.
#ifndef DFP_ASM_UNSAFE_PERSIST
#define DFP_ASM_UNSAFE_PERSIST 0
#endif
#ifndef DFP_ASM_UNSAFE_PERSIST_PARTIALS
#define DFP_ASM_UNSAFE_PERSIST_PARTIALS 0
#endif
#ifndef DFP_ASM_UNSAFE_PERSIST_I32
#define DFP_ASM_UNSAFE_PERSIST_I32 0
#endif
#ifndef DFP_ASM_UNSAFE_SKEW
#define DFP_ASM_UNSAFE_SKEW 0
#endif
#ifndef DFP_ASM_UNSAFE_SKEW_PARTIALS
#define DFP_ASM_UNSAFE_SKEW_PARTIALS 0
#endif

namespace dfp {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kMT = 64;   // output channels per workgroup
static_assert(kMT == kMfmaRowTile, "row tile shared with the GEMM preps");
constexpr int kNT = 128;  // output pixels per workgroup

// Byte digits of an INT16 value.
__device__ __forceinline__ uint32_t hi_digit(int32_t a) { return (uint32_t)((a + 128) >> 8) & 0xffu; }
__device__ __forceinline__ uint32_t lo_digit(int32_t a) { return (uint32_t)a & 0xffu; }

// ---------------------------------------------------------------- A prep
// A[m][t] for t = (r*S + s)*Cin + ci.  fwd: m = k, ci = c, value w[m][ci][r][s].
// bwd-data: m = c, ci = k, value w[ci][m][r][s].  One thread per 4 digits of
// one (kb, m, half) piece: the hi and lo words it packs land 16 bytes apart.
// The same launch clears the output scale and writes the per-block B offset
// table of the main kernels.
struct PrepAArgs {
  const int16_t* w;
  uint8_t* ws;
  int32_t M, Mp, Cin, R, S, T, KB, transposed, Cw;
  dfp_scale* so;
  int2* boff;
  int32_t tap_row_bytes, tap_col_bytes;
};

// Work item idx of the filter-digit preparation: ((kb, m, half), quarter), plus
// the block offset table (idx < KB) and the output-scale reset (idx 0).
__device__ __forceinline__ void prep_a_item(const PrepAArgs& a, int32_t idx) {
  if (a.so && idx == 0) {  // the output scale starts empty; the conv epilogue raises its max
    a.so->amax_bits = 0u;
    a.so->flags = 0u;
  }
  if (idx < a.KB) {
    // block idx covers t0 .. t0+31; each 16-index half is one channel group of one tap
    // (Cin is a multiple of 16 wherever the table is read); indices past T read offset 0
    int32_t o[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int32_t t = idx * 32 + 16 * h;
      const int32_t tap = t / a.Cin, ci = t % a.Cin;
      o[h] = t < a.T ? (tap / a.S) * a.tap_row_bytes + (tap % a.S) * a.tap_col_bytes + (ci >> 4) * 32 : 0;
    }
    a.boff[idx] = make_int2(o[0], o[1]);
  }
  const int32_t total = a.KB * a.Mp * 8;
  if (idx >= total) return;
  const int32_t quarter = idx & 3;
  const int32_t piece = idx >> 2;  // (kb * Mp + m) * 2 + half
  const int32_t half = piece & 1;
  const int32_t m = (piece >> 1) % a.Mp;
  const int32_t kb = (piece >> 1) / a.Mp;
  uint32_t hi = 0u, lo = 0u;
  if (m < a.M) {
    const int32_t t0 = kb * 32 + half * 16 + quarter * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int32_t t = t0 + i;
      int32_t v = 0;
      if (t < a.T) {
        const int32_t ci = t % a.Cin, tap = t / a.Cin;
        const int32_t r = tap / a.S, s = tap % a.S;
        // forward: w[m][ci][r][s]; backward-data: w[ci][m][r][s] (Cw = C)
        const int32_t off = a.transposed ? ((ci * a.Cw + m) * a.R + r) * a.S + s : ((m * a.Cw + ci) * a.R + r) * a.S + s;
        v = a.w[off];
      }
      hi |= hi_digit(v) << (8 * i);
      lo |= lo_digit(v) << (8 * i);
    }
  }
  uint32_t* dst = reinterpret_cast<uint32_t*>(a.ws + (int64_t)piece * 32) + quarter;
  dst[0] = hi;
  dst[4] = lo;
}

__global__ __launch_bounds__(256) void k_prep_a(PrepAArgs a) { prep_a_item(a, blockIdx.x * 256 + threadIdx.x); }

// ---------------------------------------------------------------- B prep
// Xs[n][u][v][cg][32 B] = digits of src[n][cg*16 + i][(u-top)/dil_h][(v-left)/dil_w]
// when (u-top), (v-left) are non-negative multiples of the dilation inside the
// source, else 0.  One workgroup per output row (n, u): the source row of up to
// kPrepBElems / Wsrc channels is transposed into LDS as [w][channel] (16-byte
// loads along w when rows are 8-element aligned), then every lane writes the
// 32 bytes of one (v, channel group) unit from one contiguous LDS run, so the
// output row is stored contiguously.
constexpr int kPrepBElems = 16384;  // int16 elements staged per pass (32 KiB)

template <bool VEC>
__global__ __launch_bounds__(256) void k_prep_b(const int16_t* __restrict__ src, uint8_t* __restrict__ xs,
                                               int32_t N, int32_t Cs, int32_t Hs, int32_t Wsrc, int32_t Hp,
                                               int32_t Wp, int32_t CG, int32_t top, int32_t left, int32_t dil_h,
                                               int32_t dil_w) {
  extern __shared__ __align__(16) int16_t tile[];  // cgc * 16 * Wsrc elements (launcher sizes it)
  const int32_t row = blockIdx.x;  // n * Hp + u
  const int32_t n = row / Hp, u = row - n * Hp;
  const int32_t zu = u - top;
  const bool row_in = zu >= 0 && (zu % dil_h) == 0 && zu / dil_h < Hs;
  const int32_t h = row_in ? zu / dil_h : 0;
  uint4* dst = reinterpret_cast<uint4*>(xs + (int64_t)row * Wp * CG * 32);
  const int32_t cgc = max(1, min(CG, kPrepBElems / (16 * Wsrc)));  // channel groups per pass
  const int64_t plane = (int64_t)Hs * Wsrc;
  const int16_t* srow = src + (int64_t)n * Cs * plane + (int64_t)h * Wsrc;
  for (int32_t cg0 = 0; cg0 < CG; cg0 += cgc) {
    const int32_t ncg = min(cgc, CG - cg0);
    const int32_t cs = ncg * 16;  // LDS row stride in elements
    if (row_in) {
      __syncthreads();  // the previous pass has been consumed
      if (VEC) {
        const int32_t W8 = Wsrc >> 3;
        for (int32_t j = threadIdx.x; j < cs * W8; j += 256) {
          const int32_t cl = j / W8, w0 = (j - cl * W8) * 8;
          const int32_t c = cg0 * 16 + cl;
          uint4 v = make_uint4(0u, 0u, 0u, 0u);
          if (c < Cs) v = *reinterpret_cast<const uint4*>(srow + (int64_t)c * plane + w0);
          const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int k = 0; k < 8; ++k) tile[(w0 + k) * cs + cl] = (int16_t)(wv[k >> 1] >> (16 * (k & 1)));
        }
      } else {
        for (int32_t e = threadIdx.x; e < cs * Wsrc; e += 256) {
          const int32_t cl = e / Wsrc, w = e - cl * Wsrc;
          const int32_t c = cg0 * 16 + cl;
          tile[w * cs + cl] = c < Cs ? srow[(int64_t)c * plane + w] : (int16_t)0;
        }
      }
      __syncthreads();
    }
    const int32_t units = Wp * ncg;
    for (int32_t j = threadIdx.x; j < units; j += 256) {
      const int32_t v = j / ncg, cgl = j - v * ncg;
      const int32_t zv = v - left;
      const bool in = row_in && zv >= 0 && (zv % dil_w) == 0 && zv / dil_w < Wsrc;
      uint32_t hi[4] = {0u, 0u, 0u, 0u}, lo[4] = {0u, 0u, 0u, 0u};
      if (in) {
        const uint4* tp = reinterpret_cast<const uint4*>(tile + (zv / dil_w) * cs + cgl * 16);
        const uint4 p0 = tp[0], p1 = tp[1];
        const uint32_t wv[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int32_t a = (int32_t)(int16_t)(wv[i >> 1] >> (16 * (i & 1)));
          hi[i >> 2] |= hi_digit(a) << (8 * (i & 3));
          lo[i >> 2] |= lo_digit(a) << (8 * (i & 3));
        }
      }
      uint4* d = dst + (v * CG + cg0 + cgl) * 2;
      d[0] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
      d[1] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
    }
  }
}

// Plane layout Xs[n][u][cb][digit][half][v][16 B] (CG even): the hi digits of
// channel group cg = 2 cb + half at column v sit at ((cb * 4 + half) * Wp + v)
// * 16 within row u, the lo digits 2 * Wp * 16 bytes further; sources and
// zero rows / columns as for k_prep_b.  Workgroup (row block, cg, n) stages
// the group's 16 channels for up to kPlaneRows output rows in LDS as channel
// pairs, [row][pair][w] of 32-bit (even | odd << 16) words: for one channel the
// source rows of a block are adjacent (unit dilation), so the global reads are
// long runs along w, the LDS writes and reads are consecutive words across
// lanes (no bank conflicts), and the digits of each output row are written as
// two contiguous runs of Wp * 16 bytes.
constexpr int kPlaneRows = 8;
// The register-only preparation (k_prep_plane_direct) measured faster than
// the LDS-staged one on ResNet-50 conv2_x (8.0 against 8.7 us).
constexpr bool kPlaneDirect = true;
constexpr int kPlaneElems = 16384;  // int16 elements staged (32 KiB)

template <bool VEC>
__global__ __launch_bounds__(256) void k_prep_plane(const int16_t* __restrict__ src, uint8_t* __restrict__ xs,
                                                   int32_t Cs, int32_t Hs, int32_t Wsrc, int32_t Hp, int32_t Wp,
                                                   int32_t CG, int32_t top, int32_t left, int32_t dil_h,
                                                   int32_t dil_w, int32_t rb, PrepAArgs pa, int32_t with_a) {
  extern __shared__ __align__(16) uint32_t tile2[];  // [rb][8][Wsrc] channel pairs
  if (with_a && blockIdx.z == gridDim.z - 1) {  // one extra slice of workgroups prepares the filter digits
    const int32_t nthr = gridDim.x * gridDim.y * 256;
    const int32_t total = max(pa.KB * pa.Mp * 8, pa.KB);
    for (int32_t idx = (blockIdx.y * gridDim.x + blockIdx.x) * 256 + threadIdx.x; idx < total; idx += nthr)
      prep_a_item(pa, idx);
    return;
  }
  const int32_t u0 = blockIdx.x * rb, cg = blockIdx.y, n = blockIdx.z;
  const int32_t nr = min(rb, Hp - u0);
  const int64_t plane = (int64_t)Hs * Wsrc;
  const int16_t* sbase = src + ((int64_t)n * Cs + cg * 16) * plane;
  // source row of output row u0 + r, or -1 for a zero row
  auto src_row = [&](int32_t r) {
    const int32_t zu = u0 + r - top;
    return (zu >= 0 && (zu % dil_h) == 0 && zu / dil_h < Hs) ? zu / dil_h : -1;
  };
  if (VEC) {  // 8 consecutive columns of one (row, channel pair) per thread
    const int32_t W8 = Wsrc >> 3;
    for (int32_t j = threadIdx.x; j < nr * 8 * W8; j += 256) {
      const int32_t w8 = j % W8, rest = j / W8, pr = rest & 7, r = rest >> 3;
      const int32_t h = src_row(r);
      const int32_t c0 = cg * 16 + 2 * pr;
      uint4 e = make_uint4(0u, 0u, 0u, 0u), o = make_uint4(0u, 0u, 0u, 0u);
      if (h >= 0 && c0 < Cs) e = *reinterpret_cast<const uint4*>(sbase + 2 * pr * plane + (int64_t)h * Wsrc + w8 * 8);
      if (h >= 0 && c0 + 1 < Cs)
        o = *reinterpret_cast<const uint4*>(sbase + (2 * pr + 1) * plane + (int64_t)h * Wsrc + w8 * 8);
      uint4* t = reinterpret_cast<uint4*>(tile2 + ((int64_t)r * 8 + pr) * Wsrc + w8 * 8);
      t[0] = make_uint4(__builtin_amdgcn_perm(o.x, e.x, 0x05040100u), __builtin_amdgcn_perm(o.x, e.x, 0x07060302u),
                        __builtin_amdgcn_perm(o.y, e.y, 0x05040100u), __builtin_amdgcn_perm(o.y, e.y, 0x07060302u));
      t[1] = make_uint4(__builtin_amdgcn_perm(o.z, e.z, 0x05040100u), __builtin_amdgcn_perm(o.z, e.z, 0x07060302u),
                        __builtin_amdgcn_perm(o.w, e.w, 0x05040100u), __builtin_amdgcn_perm(o.w, e.w, 0x07060302u));
    }
  } else {
    for (int32_t j = threadIdx.x; j < nr * 8 * Wsrc; j += 256) {
      const int32_t w = j % Wsrc, rest = j / Wsrc, pr = rest & 7, r = rest >> 3;
      const int32_t h = src_row(r);
      const int32_t c0 = cg * 16 + 2 * pr;
      const uint32_t ev = (h >= 0 && c0 < Cs) ? (uint16_t)sbase[2 * pr * plane + (int64_t)h * Wsrc + w] : 0u;
      const uint32_t ov = (h >= 0 && c0 + 1 < Cs) ? (uint16_t)sbase[(2 * pr + 1) * plane + (int64_t)h * Wsrc + w] : 0u;
      tile2[((int64_t)r * 8 + pr) * Wsrc + w] = ev | (ov << 16);
    }
  }
  __syncthreads();
  const int64_t row_bytes = (int64_t)CG * 32 * Wp;
  const int32_t off_hi = ((cg >> 1) * 4 + (cg & 1)) * Wp;  // in 16-byte units within the row
  for (int32_t j = threadIdx.x; j < nr * Wp; j += 256) {
    const int32_t v = j % Wp, r = j / Wp;
    const int32_t zv = v - left;
    const bool in = src_row(r) >= 0 && zv >= 0 && (zv % dil_w) == 0 && zv / dil_w < Wsrc;
    uint32_t hi[4] = {0u, 0u, 0u, 0u}, lo[4] = {0u, 0u, 0u, 0u};
    if (in) {
      const uint32_t* tp = tile2 + (int64_t)r * 8 * Wsrc + zv / dil_w;
#pragma unroll
      for (int pr = 0; pr < 8; ++pr) {
        const uint32_t wv = tp[pr * Wsrc];
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
          const int i = 2 * pr + h2;
          const int32_t a = (int32_t)(int16_t)(wv >> (16 * h2));
          hi[i >> 2] |= hi_digit(a) << (8 * (i & 3));
          lo[i >> 2] |= lo_digit(a) << (8 * (i & 3));
        }
      }
    }
    uint4* d = reinterpret_cast<uint4*>(xs + ((int64_t)n * Hp + u0 + r) * row_bytes) + off_hi + v;
    d[0] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
    d[2 * Wp] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
  }
}

// Plane layout written straight from registers: workgroup (u, n) covers
// output row u of image n, a thread the 16 channels of group cg at column v
// (lanes of a wave take consecutive columns, so each of the 16 channel loads
// of a wave reads one contiguous run of the source row, and each of its two
// 16-byte stores one contiguous run of the plane).  An extra row of
// workgroups (with_a) prepares the filter digits.  Workgroup ids are mapped
// to rows so that each XCD (id mod 8) takes one contiguous range of rows of
// whole images: a 128-byte line of the source holds parts of two rows, and
// with neighbouring rows on different XCDs every such line was fetched into
// two L2s.
__global__ __launch_bounds__(256) void k_prep_plane_direct(const int16_t* __restrict__ src, uint8_t* __restrict__ xs,
                                                          int32_t Cs, int32_t Hs, int32_t Wsrc, int32_t Hp, int32_t Wp,
                                                          int32_t CG, int32_t top, int32_t left, int32_t dil_h,
                                                          int32_t dil_w, PrepAArgs pa, int32_t with_a) {
  const int32_t nwg = gridDim.x * gridDim.y, id = blockIdx.y * gridDim.x + blockIdx.x;
  const int32_t xcd = id & 7, per = nwg >> 3, rem = nwg & 7;
  const int32_t l = xcd * per + min(xcd, rem) + (id >> 3);
  const int32_t n = l / (int32_t)gridDim.x, u = l - n * (int32_t)gridDim.x;
  if (with_a && n == (int32_t)gridDim.y - 1) {
    const int32_t nthr = gridDim.x * 256;
    const int32_t total = max(pa.KB * pa.Mp * 8, pa.KB);
    for (int32_t idx = u * 256 + threadIdx.x; idx < total; idx += nthr) prep_a_item(pa, idx);
    return;
  }
  const int32_t zu = u - top;
  const bool row_in = zu >= 0 && (zu % dil_h) == 0 && zu / dil_h < Hs;
  const int32_t h = row_in ? zu / dil_h : 0;
  const int64_t plane = (int64_t)Hs * Wsrc;
  uint8_t* rowp = xs + ((int64_t)n * Hp + u) * ((int64_t)CG * 32 * Wp);
  for (int32_t j = threadIdx.x; j < CG * Wp; j += 256) {
    const int32_t cg = j / Wp, v = j - cg * Wp;
    const int32_t zv = v - left;
    const bool in = row_in && zv >= 0 && (zv % dil_w) == 0 && zv / dil_w < Wsrc;
    uint32_t hi[4] = {0u, 0u, 0u, 0u}, lo[4] = {0u, 0u, 0u, 0u};
    if (in) {
      const int16_t* sp = src + ((int64_t)n * Cs + cg * 16) * plane + (int64_t)h * Wsrc + zv / dil_w;
      int32_t a[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) a[k] = (cg * 16 + k < Cs) ? (int32_t)sp[k * plane] : 0;
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        hi[k >> 2] |= hi_digit(a[k]) << (8 * (k & 3));
        lo[k >> 2] |= lo_digit(a[k]) << (8 * (k & 3));
      }
    }
    uint4* d = reinterpret_cast<uint4*>(rowp) + ((cg >> 1) * 4 + (cg & 1)) * Wp + v;
    d[0] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
    d[2 * Wp] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
  }
}

// The same plane layout from pairs of source columns (no dilation, an even
// source width, the source 4-byte aligned): a thread loads columns 2i, 2i + 1
// of its 16 channels as one dword each (a wave's load covers 256 contiguous
// bytes of a source row instead of 128) and writes output pixels 2i + left
// and 2i + 1 + left; the remaining threads of a row write its padding columns.
__global__ __launch_bounds__(256) void k_prep_plane_pair(const int16_t* __restrict__ src, uint8_t* __restrict__ xs,
                                                        int32_t Cs, int32_t Hs, int32_t Wsrc, int32_t Hp, int32_t Wp,
                                                        int32_t CG, int32_t top, int32_t left, PrepAArgs pa,
                                                        int32_t with_a) {
  const int32_t nwg = gridDim.x * gridDim.y, id = blockIdx.y * gridDim.x + blockIdx.x;
  const int32_t xcd = id & 7, per_x = nwg >> 3, rem = nwg & 7;
  const int32_t l = xcd * per_x + min(xcd, rem) + (id >> 3);
  const int32_t n = l / (int32_t)gridDim.x, u = l - n * (int32_t)gridDim.x;
  if (with_a && n == (int32_t)gridDim.y - 1) {
    const int32_t nthr = gridDim.x * 256;
    const int32_t total = max(pa.KB * pa.Mp * 8, pa.KB);
    for (int32_t idx = u * 256 + threadIdx.x; idx < total; idx += nthr) prep_a_item(pa, idx);
    return;
  }
  const int32_t h = u - top;
  const bool row_in = h >= 0 && h < Hs;
  const int64_t plane = (int64_t)Hs * Wsrc;
  uint8_t* rowp = xs + ((int64_t)n * Hp + u) * ((int64_t)CG * 32 * Wp);
  const int32_t npair = Wsrc >> 1, per = npair + (Wp - Wsrc);
  for (int32_t j = threadIdx.x; j < CG * per; j += 256) {
    const int32_t cg = j / per, i = j - cg * per;
    uint4* d = reinterpret_cast<uint4*>(rowp) + ((cg >> 1) * 4 + (cg & 1)) * Wp;
    if (i < npair) {
      uint32_t hi0[4] = {0u, 0u, 0u, 0u}, lo0[4] = {0u, 0u, 0u, 0u}, hi1[4] = {0u, 0u, 0u, 0u},
               lo1[4] = {0u, 0u, 0u, 0u};
      if (row_in) {
        const uint32_t* sp = reinterpret_cast<const uint32_t*>(src + ((int64_t)n * Cs + cg * 16) * plane +
                                                               (int64_t)h * Wsrc + 2 * i);
        uint32_t wv[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) wv[k] = (cg * 16 + k < Cs) ? sp[k * (plane >> 1)] : 0u;
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const int32_t a0 = (int32_t)(int16_t)(wv[k] & 0xffffu), a1 = (int32_t)(int16_t)(wv[k] >> 16);
          hi0[k >> 2] |= hi_digit(a0) << (8 * (k & 3));
          lo0[k >> 2] |= lo_digit(a0) << (8 * (k & 3));
          hi1[k >> 2] |= hi_digit(a1) << (8 * (k & 3));
          lo1[k >> 2] |= lo_digit(a1) << (8 * (k & 3));
        }
      }
      const int32_t v = 2 * i + left;
      d[v] = make_uint4(hi0[0], hi0[1], hi0[2], hi0[3]);
      d[v + 1] = make_uint4(hi1[0], hi1[1], hi1[2], hi1[3]);
      d[2 * Wp + v] = make_uint4(lo0[0], lo0[1], lo0[2], lo0[3]);
      d[2 * Wp + v + 1] = make_uint4(lo1[0], lo1[1], lo1[2], lo1[3]);
    } else {  // padding columns: [0, left) and [left + Wsrc, Wp)
      const int32_t z = i - npair;
      const int32_t v = z < left ? z : Wsrc + z;
      d[v] = make_uint4(0u, 0u, 0u, 0u);
      d[2 * Wp + v] = make_uint4(0u, 0u, 0u, 0u);
    }
  }
}

// Byte mask keeping bytes [lo, hi) of a 16-byte operand (0 <= lo <= hi <= 16).
__device__ __forceinline__ v4i byte_mask16(int32_t lo, int32_t hi) {
  const uint32_t bits = ((hi >= 16 ? 0xffffu : ((1u << hi) - 1u)) & ~((1u << lo) - 1u)) & 0xffffu;
  v4i m;
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t b = (bits >> (4 * d)) & 0xfu;
    m[d] = (int)((((b * 0x00204081u) & 0x01010101u)) * 0xffu);
  }
  return m;
}

struct Acc3 {
  v16i hh, xx, ll;
};

// HH, LL and the two cross products of one 32x32 tile.  fresh: the block opens
// a chunk, so the accumulators start from zero.
__device__ __forceinline__ void mfma_tile(Acc3& acc, const v4i& ahi, const v4i& alo, const v4i& bhi,
                                          const v4i& blo, bool fresh) {
  if (fresh) {
    const v16i z = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
    acc.hh = __builtin_amdgcn_mfma_i32_32x32x32_i8(ahi, bhi, z, 0, 0, 0);
    acc.ll = __builtin_amdgcn_mfma_i32_32x32x32_i8(alo, blo, z, 0, 0, 0);
    acc.xx = __builtin_amdgcn_mfma_i32_32x32x32_i8(ahi, blo, z, 0, 0, 0);
  } else {
    acc.hh = __builtin_amdgcn_mfma_i32_32x32x32_i8(ahi, bhi, acc.hh, 0, 0, 0);
    acc.ll = __builtin_amdgcn_mfma_i32_32x32x32_i8(alo, blo, acc.ll, 0, 0, 0);
    acc.xx = __builtin_amdgcn_mfma_i32_32x32x32_i8(ahi, blo, acc.xx, 0, 0, 0);
  }
  acc.xx = __builtin_amdgcn_mfma_i32_32x32x32_i8(alo, bhi, acc.xx, 0, 0, 0);
}

// mfma_tile with the issue order HH, X(hi, lo), LL, X(lo, hi) pinned, so the
// two dependent cross products of a block are two MFMAs apart and the next
// block's first cross product follows its HH.
__device__ __forceinline__ void mfma_tile_ordered(Acc3& acc, const v4i& ahi, const v4i& alo, const v4i& bhi,
                                                  const v4i& blo, bool fresh) {
  const v16i z = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
  acc.hh = __builtin_amdgcn_mfma_i32_32x32x32_i8(ahi, bhi, fresh ? z : acc.hh, 0, 0, 0);
  __builtin_amdgcn_sched_barrier(0);
  acc.xx = __builtin_amdgcn_mfma_i32_32x32x32_i8(ahi, blo, fresh ? z : acc.xx, 0, 0, 0);
  __builtin_amdgcn_sched_barrier(0);
  acc.ll = __builtin_amdgcn_mfma_i32_32x32x32_i8(alo, blo, fresh ? z : acc.ll, 0, 0, 0);
  __builtin_amdgcn_sched_barrier(0);
  acc.xx = __builtin_amdgcn_mfma_i32_32x32x32_i8(alo, bhi, acc.xx, 0, 0, 0);
}

// ((a << 8) + b) << 8) + c as two v_lshl_add_u32.  The shift-adds are plain
// C so the compiler's hazard checks see every read of an MFMA result; the
// empty asm only stops the re-association into shift, shift, add3.
__device__ __forceinline__ uint32_t recombine(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t t = (a << 8) + b;
  asm("" : "+v"(t));
  return (t << 8) + c;
}

// Chunk end: P_j = ((HH << 8) + X) << 8) + LL modulo 2^32, converted to FP32
// (round to nearest even) and added to the running sum in chunk order.
template <bool PARTIALS>
__device__ __forceinline__ void flush_tile(const Acc3& acc, float (&sum)[16], int64_t j, int32_t* partials,
                                           int64_t O, int64_t obase, int64_t PQ, int32_t mrow0, int32_t M,
                                           bool gvalid) {
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const uint32_t p = recombine((uint32_t)acc.hh[v], (uint32_t)acc.xx[v], (uint32_t)acc.ll[v]);
    sum[v] += (float)(int32_t)p;
    if (PARTIALS) {
      const int32_t m = mrow0 + 8 * (v >> 2) + (v & 3);
      if (gvalid && m < M) partials[j * O + obase + (int64_t)m * PQ] = (int32_t)p;
    }
  }
}

// Blocked-DFP chunk end: the partial is scaled by 2^(Ea(block) + Eb(block))
// (per row and column) before it joins the running sum; no final scale.
template <bool PARTIALS>
__device__ __forceinline__ void flush_tile_blocked(const Acc3& acc, float (&sum)[16], const int32_t (&ev)[16],
                                                   int64_t j, int32_t* partials, int64_t O, int64_t obase,
                                                   int64_t PQ, int32_t mrow0, int32_t M, bool gvalid) {
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const uint32_t p = recombine((uint32_t)acc.hh[v], (uint32_t)acc.xx[v], (uint32_t)acc.ll[v]);
    sum[v] += ldexpf((float)(int32_t)p, ev[v]);
    if (PARTIALS) {
      const int32_t m = mrow0 + 8 * (v >> 2) + (v & 3);
      if (gvalid && m < M) partials[j * O + obase + (int64_t)m * PQ] = (int32_t)p;
    }
  }
}

// Single-chunk DFP-32 output: the chunk's wrapped INT32 sum itself, kept as
// raw bits in the FP32 sum registers until the epilogue stores it.
__device__ __forceinline__ void keep_tile_i32(const Acc3& acc, float (&sum)[16]) {
#pragma unroll
  for (int v = 0; v < 16; ++v)
    sum[v] = __int_as_float((int32_t)recombine((uint32_t)acc.hh[v], (uint32_t)acc.xx[v], (uint32_t)acc.ll[v]));
}

// Epilogue of one output element: FP32 path stores 2^e * sum and its |.|
// bits; the DFP-32 path stores the INT32 and |.| as an unsigned integer.
template <bool I32>
__device__ __forceinline__ uint32_t store_out(float* out, int64_t o, float sum, int32_t e) {
  if (I32) {
    const int32_t v = __float_as_int(sum);
    reinterpret_cast<int32_t*>(out)[o] = v;
    return v < 0 ? (uint32_t)0 - (uint32_t)v : (uint32_t)v;
  } else {
    const float y = ldexpf(sum, e);
    out[o] = y;
    return __float_as_uint(y) & 0x7fffffffu;
  }
}

// Operands of one block of 32 reduction indices for one lane.
struct Operands {
  v4i bhi, blo;
  v4i ahi[2], alo[2];
};

// Forward / backward-data main kernel.  Output pixels g in [0, NP) map to
// (img, po, qo) of an [Nimg][M][Po][Qo] FP32 output.
template <bool MASKED, bool PARTIALS, bool CHAN16, bool I32 = false>
__global__ __launch_bounds__(kThreads, 2) void k_conv_mfma(ConvMfmaArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int half = lane >> 5;
  const int col = lane & 31;
  const int32_t m0 = blockIdx.y * kMT;
  const int64_t g = (int64_t)blockIdx.x * kNT + wave * 32 + col;
  const bool gvalid = g < a.NP;
  const int64_t gg = gvalid ? g : 0;
  const int32_t qo = (int32_t)(gg % a.Qo);
  const int32_t po = (int32_t)((gg / a.Qo) % a.Po);
  const int64_t img = gg / ((int64_t)a.Qo * a.Po);
  // B byte address of this pixel at tap (0, 0), channel group 0
  const uint8_t* __restrict__ bpix =
      a.xs +
      (((img * a.Hp + (int64_t)po * a.ustride_h + a.roff_h) * a.Wp + (int64_t)qo * a.ustride_w + a.roff_w) * a.CG) *
          32;
  const int32_t tap_row_bytes = a.rsign * a.Wp * a.CG * 32;  // one filter row
  const int32_t tap_col_bytes = a.rsign * a.CG * 32;         // one filter column
  // A address of this lane's row in tile 0 at block 0; tile 1 is 32 rows (2048 B) further
  const uint8_t* __restrict__ apix = a.wsa + ((int64_t)(m0 + col) * 2 + half) * 32;
  const int64_t a_block_bytes = (int64_t)a.Mp * 64;
  const int64_t PQ = (int64_t)a.Po * a.Qo;
  const int64_t obase = img * a.M * PQ + (int64_t)po * a.Qo + qo;
  const int32_t T = a.T, L = a.L, Cin = a.Cin;

  Acc3 acc[2];
  float sum[2][16];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      acc[i].hh[v] = 0; acc[i].xx[v] = 0; acc[i].ll[v] = 0;
      sum[i][v] = 0.f;
    }
  }

  // Reduction position (uniform) of the first 16 indices of the next block to load.
  int32_t ld_c = 0, ld_r = 0, ld_s = 0;
  auto load = [&](int32_t kb, Operands& op) {
    const int32_t t0 = kb * 32 + half * 16;
    op.bhi = (v4i){0, 0, 0, 0};
    op.blo = (v4i){0, 0, 0, 0};
    if (CHAN16) {
      // half 0 reads channels [ld_c, ld_c+16) of tap (ld_r, ld_s); half 1 the next 16 indices
      const int32_t off0 = ld_r * tap_row_bytes + ld_s * tap_col_bytes + (ld_c >> 4) * 32;
      int32_t off1;
      if (ld_c + 16 < Cin) {
        off1 = off0 + 32;
      } else {
        const int32_t s1 = (ld_s + 1 == a.S) ? 0 : ld_s + 1;
        const int32_t r1 = (ld_s + 1 == a.S) ? ld_r + 1 : ld_r;
        off1 = r1 * tap_row_bytes + s1 * tap_col_bytes;
      }
      if (t0 < T) {
        const uint4* src = reinterpret_cast<const uint4*>(bpix + (half ? off1 : off0));
        const uint4 h4 = src[0], l4 = src[1];
        op.bhi = (v4i){(int)h4.x, (int)h4.y, (int)h4.z, (int)h4.w};
        op.blo = (v4i){(int)l4.x, (int)l4.y, (int)l4.z, (int)l4.w};
      }
      ld_c += 32;
      while (ld_c >= Cin) {
        ld_c -= Cin;
        if (++ld_s == a.S) { ld_s = 0; ++ld_r; }
      }
    } else {
      uint32_t hw[4] = {0u, 0u, 0u, 0u}, lw[4] = {0u, 0u, 0u, 0u};
      for (int i = 0; i < 16; ++i) {
        const int32_t t = t0 + i;
        if (t < T) {
          const int32_t ci = t % Cin, tap = t / Cin;
          const int32_t r = tap / a.S, s = tap % a.S;
          const uint8_t* p = bpix + r * tap_row_bytes + s * tap_col_bytes + (ci >> 4) * 32 + (ci & 15);
          hw[i >> 2] |= (uint32_t)p[0] << (8 * (i & 3));
          lw[i >> 2] |= (uint32_t)p[16] << (8 * (i & 3));
        }
      }
      op.bhi = (v4i){(int)hw[0], (int)hw[1], (int)hw[2], (int)hw[3]};
      op.blo = (v4i){(int)lw[0], (int)lw[1], (int)lw[2], (int)lw[3]};
    }
    const uint8_t* ap = apix + kb * a_block_bytes;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint4* src = reinterpret_cast<const uint4*>(ap + i * 2048);
      const uint4 h4 = src[0], l4 = src[1];
      op.ahi[i] = (v4i){(int)h4.x, (int)h4.y, (int)h4.z, (int)h4.w};
      op.alo[i] = (v4i){(int)l4.x, (int)l4.y, (int)l4.z, (int)l4.w};
    }
  };

  int64_t j = 0;           // current chunk
  int32_t blk_in_chunk = 0;  // unmasked path: blocks of the current chunk seen so far
  const int32_t chunk_blocks = L / 32;
  auto compute = [&](int32_t kb, const Operands& op) {
    if (!MASKED) {
      const bool fresh = blk_in_chunk == 0;
#pragma unroll
      for (int i = 0; i < 2; ++i) mfma_tile(acc[i], op.ahi[i], op.alo[i], op.bhi, op.blo, fresh);
      ++blk_in_chunk;
      if (blk_in_chunk == chunk_blocks || kb == a.KB - 1) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          if (I32) keep_tile_i32(acc[i], sum[i]);
          else flush_tile<PARTIALS>(acc[i], sum[i], j, a.partials, a.O, obase, PQ, m0 + 32 * i + 4 * half, a.M, gvalid);
        }
        ++j;
        blk_in_chunk = 0;
      }
    } else {
      const int32_t t0 = kb * 32 + half * 16;
      const int32_t t_lo = kb * 32, t_hi = min(kb * 32 + 32, T);
      while (true) {
        const int64_t cs = j * (int64_t)L;
        const int64_t ce = min(cs + L, (int64_t)T);
        const int32_t seg_lo = (int32_t)max((int64_t)t_lo, cs), seg_hi = (int32_t)min((int64_t)t_hi, ce);
        const v4i mk = byte_mask16(min(max(seg_lo - t0, 0), 16), min(max(seg_hi - t0, 0), 16));
        const v4i mhi = op.bhi & mk, mlo = op.blo & mk;
        const bool fresh = seg_lo == cs;
#pragma unroll
        for (int i = 0; i < 2; ++i) mfma_tile(acc[i], op.ahi[i], op.alo[i], mhi, mlo, fresh);
        if (ce <= t_hi) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
            flush_tile<PARTIALS>(acc[i], sum[i], j, a.partials, a.O, obase, PQ, m0 + 32 * i + 4 * half, a.M,
                                 gvalid);
          ++j;
        }
        if (ce >= t_hi) break;
      }
    }
  };

  // software pipeline: the next block's loads are in flight while this one computes
  Operands op0, op1;
  load(0, op0);
  int32_t kb = 0;
  for (; kb + 2 <= a.KB; kb += 2) {
    load(kb + 1, op1);
    compute(kb, op0);
    if (kb + 2 < a.KB) load(kb + 2, op0);
    compute(kb + 1, op1);
  }
  if (kb < a.KB) compute(kb, op0);

  // ---- epilogue: scale once, store, max |y|
  const int32_t e = a.ea->exp + a.eb->exp;
  uint32_t amax = 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int32_t m = m0 + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
      if (gvalid && m < a.M) amax = max(amax, store_out<I32>(a.out, obase + (int64_t)m * PQ, sum[i][v], e));
    }
  }
  if (a.so) {
    __shared__ uint32_t red[kThreads / 64];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, off, 64));
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t b = red[0];
      for (int i = 1; i < kThreads / 64; ++i) b = max(b, red[i]);
      if (b > __atomic_load_n(&a.so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&a.so->amax_bits, b);
      if (I32) {
        if (blockIdx.x == 0 && blockIdx.y == 0) a.so->exp = e;
      } else if (b == 0x7f800000u) {
        atomicOr(&a.so->flags, DFP_FLAG_OUTPUT_INF);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Pipelined variant for reduction channel counts that are multiples of 16:
// every operand block (A: 64 rows x 32 indices, B: 128 pixels x 32 indices,
// both as hi/lo digit bytes) is fetched with direct-to-LDS 16-byte loads
// (global_load_lds_dwordx4) into a ring of kStages stages, kStages-1 blocks
// ahead of the MFMAs, with one workgroup barrier per block.  Each 16-byte
// piece (row or pixel, half, digit) sits at slot row*4 + ((2*half + digit) ^
// ((row >> 2) & 3)) of its region, which keeps the ds_read_b128 operand reads
// of 16 consecutive rows (or pixels) on distinct banks.
constexpr int kStages = 4;
constexpr int kStageA = 4096;   // 64 rows x 2 halves x 32 B
constexpr int kStageB = 8192;   // 128 pixels x 2 halves x 32 B
constexpr int kStageBytes = kStageA + kStageB;

typedef __attribute__((address_space(3))) void* lds_ptr_t;

__device__ __forceinline__ int swz(int row, int piece) { return row * 4 + (piece ^ ((row >> 2) & 3)); }

// s_waitcnt vmcnt(N): this lane's direct-to-LDS loads older than the newest N
// have landed.  Issued as inline assembly together with the raw barrier below,
// because the compiler's own wait insertion treats every LDS read as aliasing
// every in-flight LDS load and would drain the whole pipeline.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// The six operand reads of one stage (B hi/lo, A hi/lo of two tiles), then a
// wait for all of them.  Stage offset STAGE_OFF is an immediate.
template <int STAGE_OFF>
__device__ __forceinline__ void read_stage(uint32_t b0, uint32_t b1, uint32_t a00, uint32_t a01, uint32_t a10,
                                           uint32_t a11, v4i& bhi, v4i& blo, v4i (&ahi)[2], v4i (&alo)[2]) {
  asm volatile(
      "ds_read_b128 %0, %6 offset:%12\n\t"
      "ds_read_b128 %1, %7 offset:%12\n\t"
      "ds_read_b128 %2, %8 offset:%12\n\t"
      "ds_read_b128 %3, %9 offset:%12\n\t"
      "ds_read_b128 %4, %10 offset:%12\n\t"
      "ds_read_b128 %5, %11 offset:%12\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(bhi), "=&v"(blo), "=&v"(ahi[0]), "=&v"(alo[0]), "=&v"(ahi[1]), "=&v"(alo[1])
      : "v"(b0), "v"(b1), "v"(a00), "v"(a01), "v"(a10), "v"(a11), "n"(STAGE_OFF)
      : "memory");
}

template <bool MASKED, bool PARTIALS>
__global__ __launch_bounds__(kThreads, 2) void k_conv_mfma_lds(ConvMfmaArgs a) {
  __shared__ __align__(16) uint8_t smem[kStages * kStageBytes];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int half = lane >> 5;
  const int col = lane & 31;
  const int32_t m0 = blockIdx.y * kMT;
  const int64_t NP = a.NP;
  const int64_t PQ = (int64_t)a.Po * a.Qo;

  // ---- output pixel of this lane (MFMA column)
  const int64_t g = (int64_t)blockIdx.x * kNT + wave * 32 + col;
  const bool gvalid = g < NP;
  int64_t img, obase;
  {
    const int64_t gg = gvalid ? g : 0;
    const int32_t qo = (int32_t)(gg % a.Qo), po = (int32_t)((gg / a.Qo) % a.Po);
    img = gg / PQ;
    obase = img * a.M * PQ + (int64_t)po * a.Qo + qo;
  }

  // ---- load assignments: A slot wave*64 + lane; B slots wave*128 + i*64 + lane
  const int a_slot = wave * 64 + lane;
  const int a_row = a_slot >> 2, a_piece = (a_slot & 3) ^ ((a_row >> 2) & 3);
  const uint8_t* a_src = a.wsa + ((int64_t)(m0 + a_row) * 2 + (a_piece >> 1)) * 32 + (a_piece & 1) * 16;
  const int64_t a_block_bytes = (int64_t)a.Mp * 64;
  const uint8_t* b_src[2];
  int b_half[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int slot = wave * 128 + i * 64 + lane;
    const int px = slot >> 2, piece = (slot & 3) ^ ((px >> 2) & 3);
    b_half[i] = piece >> 1;
    int64_t gp = (int64_t)blockIdx.x * kNT + px;
    if (gp >= NP) gp = 0;
    const int32_t qo = (int32_t)(gp % a.Qo), po = (int32_t)((gp / a.Qo) % a.Po);
    const int64_t im = gp / PQ;
    b_src[i] = a.xs +
               (((im * a.Hp + (int64_t)po * a.ustride_h + a.roff_h) * a.Wp + (int64_t)qo * a.ustride_w + a.roff_w) *
                a.CG) * 32 +
               (piece & 1) * 16;
  }
  const int32_t tap_row_bytes = a.rsign * a.Wp * a.CG * 32;
  const int32_t tap_col_bytes = a.rsign * a.CG * 32;
  const int32_t T = a.T, L = a.L, Cin = a.Cin, KB = a.KB;

  // uniform reduction position of the next block to load
  int32_t ld_c = 0, ld_r = 0, ld_s = 0;
  auto issue = [&](int32_t kb) {
    uint8_t* st = smem + (kb % kStages) * kStageBytes;
    __builtin_amdgcn_global_load_lds((const void*)(a_src + kb * a_block_bytes), (lds_ptr_t)(st + wave * 1024), 16, 0,
                                     0);
    const int32_t off0 = ld_r * tap_row_bytes + ld_s * tap_col_bytes + (ld_c >> 4) * 32;
    int32_t off1;
    if (ld_c + 16 < Cin) {
      off1 = off0 + 32;
    } else {
      const int32_t s1 = (ld_s + 1 == a.S) ? 0 : ld_s + 1;
      const int32_t r1 = (ld_s + 1 == a.S) ? ld_r + 1 : ld_r;
      off1 = r1 * tap_row_bytes + s1 * tap_col_bytes;
    }
    // indices at or past T read a valid dummy location (their A digits are zero)
    const int32_t o0 = (kb * 32 < T) ? off0 : 0;
    const int32_t o1 = (kb * 32 + 16 < T) ? off1 : 0;
#pragma unroll
    for (int i = 0; i < 2; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(b_src[i] + (b_half[i] ? o1 : o0)),
                                       (lds_ptr_t)(st + kStageA + wave * 2048 + i * 1024), 16, 0, 0);
    ld_c += 32;
    while (ld_c >= Cin) {
      ld_c -= Cin;
      if (++ld_s == a.S) { ld_s = 0; ++ld_r; }
    }
  };

  Acc3 acc[2];
  float sum[2][16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      acc[i].hh[v] = 0; acc[i].xx[v] = 0; acc[i].ll[v] = 0;
      sum[i][v] = 0.f;
    }

  // LDS read offsets of this lane's operands inside a stage
  const int b_rd0 = kStageA + swz(wave * 32 + col, 2 * half) * 16;
  const int b_rd1 = kStageA + swz(wave * 32 + col, 2 * half + 1) * 16;
  int a_rd[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int d = 0; d < 2; ++d) a_rd[i][d] = swz(32 * i + col, 2 * half + d) * 16;

  int64_t j = 0;
  int32_t blk_in_chunk = 0;
  const int32_t chunk_blocks = L / 32;

  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)smem;
  const uint32_t rb0 = lds_base + b_rd0, rb1 = lds_base + b_rd1;
  const uint32_t ra00 = lds_base + a_rd[0][0], ra01 = lds_base + a_rd[0][1];
  const uint32_t ra10 = lds_base + a_rd[1][0], ra11 = lds_base + a_rd[1][1];

  auto consume = [&](int32_t kb, const v4i& bhi, const v4i& blo, const v4i (&ahi)[2], const v4i (&alo)[2]) {
    if (!MASKED) {
      const bool fresh = blk_in_chunk == 0;
#pragma unroll
      for (int i = 0; i < 2; ++i) mfma_tile(acc[i], ahi[i], alo[i], bhi, blo, fresh);
      ++blk_in_chunk;
      if (blk_in_chunk == chunk_blocks || kb == KB - 1) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
          flush_tile<PARTIALS>(acc[i], sum[i], j, a.partials, a.O, obase, PQ, m0 + 32 * i + 4 * half, a.M, gvalid);
        ++j;
        blk_in_chunk = 0;
      }
    } else {
      const int32_t t0 = kb * 32 + half * 16;
      const int32_t t_lo = kb * 32, t_hi = min(kb * 32 + 32, T);
      while (true) {
        const int64_t cs = j * (int64_t)L;
        const int64_t ce = min(cs + L, (int64_t)T);
        const int32_t seg_lo = (int32_t)max((int64_t)t_lo, cs), seg_hi = (int32_t)min((int64_t)t_hi, ce);
        const v4i mk = byte_mask16(min(max(seg_lo - t0, 0), 16), min(max(seg_hi - t0, 0), 16));
        const v4i mhi = bhi & mk, mlo = blo & mk;
        const bool fresh = seg_lo == cs;
#pragma unroll
        for (int i = 0; i < 2; ++i) mfma_tile(acc[i], ahi[i], alo[i], mhi, mlo, fresh);
        if (ce <= t_hi) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
            flush_tile<PARTIALS>(acc[i], sum[i], j, a.partials, a.O, obase, PQ, m0 + 32 * i + 4 * half, a.M,
                                 gvalid);
          ++j;
        }
        if (ce >= t_hi) break;
      }
    }
  };

  // One block: wait for its loads (the kStages-2 newer blocks may stay in
  // flight, 3 loads each), barrier, refill the slot freed by the previous
  // block, read and consume.
  auto step = [&](int32_t kb, auto stage_tag) {
    constexpr int STAGE = decltype(stage_tag)::value;
    const int32_t ahead = min(kStages - 2, KB - 1 - kb);
    if (ahead >= 2) wait_vmcnt<6>();
    else if (ahead == 1) wait_vmcnt<3>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (kb + kStages - 1 < KB) issue(kb + kStages - 1);
    v4i bhi, blo, ahi[2], alo[2];
    read_stage<STAGE * kStageBytes>(rb0, rb1, ra00, ra01, ra10, ra11, bhi, blo, ahi, alo);
    consume(kb, bhi, blo, ahi, alo);
  };

  for (int32_t s = 0; s < kStages - 1 && s < KB; ++s) issue(s);
  int32_t kb = 0;
  for (; kb + kStages <= KB; kb += kStages) {
    step(kb + 0, std::integral_constant<int, 0>{});
    step(kb + 1, std::integral_constant<int, 1>{});
    step(kb + 2, std::integral_constant<int, 2>{});
    step(kb + 3, std::integral_constant<int, 3>{});
  }
  if (kb < KB) step(kb++, std::integral_constant<int, 0>{});
  if (kb < KB) step(kb++, std::integral_constant<int, 1>{});
  if (kb < KB) step(kb++, std::integral_constant<int, 2>{});

  // ---- epilogue: scale once, store, max |y|
  const int32_t e = a.ea->exp + a.eb->exp;
  uint32_t amax = 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int32_t m = m0 + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
      const float y = ldexpf(sum[i][v], e);
      if (gvalid && m < a.M) {
        a.out[obase + (int64_t)m * PQ] = y;
        amax = max(amax, __float_as_uint(y) & 0x7fffffffu);
      }
    }
  }
  if (a.so) {
    __shared__ uint32_t red[kThreads / 64];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, off, 64));
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t b = red[0];
      for (int i = 1; i < kThreads / 64; ++i) b = max(b, red[i]);
      if (b > __atomic_load_n(&a.so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&a.so->amax_bits, b);
      if (b == 0x7f800000u) atomicOr(&a.so->flags, DFP_FLAG_OUTPUT_INF);
    }
  }
}

// ---------------------------------------------------------------------------
// Four-waves-per-SIMD variant for chunk lengths that are multiples of 32 (no
// masking).  Workgroup = 8 waves, tile 64 output channels x 128 pixels, two
// workgroups per CU.  Each wave owns one 32 x 32 output tile: three
// accumulators, 16 running sums and one block of operands stay under 128
// VGPRs, so every SIMD holds four waves and one wave's chunk conversion
// (VALU) runs while the other waves issue MFMAs and LDS reads.  Operands pass
// through the same 4-stage LDS ring as above (waves 0-3 load the filter
// digits, every lane one B piece), one barrier per block.
constexpr int kWavesQ = 8;
constexpr int kThreadsQ = kWavesQ * 64;

// The four operand reads of one block for a single 32 x 32 tile, then a wait.
template <int STAGE_OFF>
__device__ __forceinline__ void read_stage_q(uint32_t b0, uint32_t b1, uint32_t a0, uint32_t a1, v4i& bhi,
                                             v4i& blo, v4i& ahi, v4i& alo) {
  asm volatile(
      "ds_read_b128 %0, %4 offset:%8\n\t"
      "ds_read_b128 %1, %5 offset:%8\n\t"
      "ds_read_b128 %2, %6 offset:%8\n\t"
      "ds_read_b128 %3, %7 offset:%8\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(bhi), "=&v"(blo), "=&v"(ahi), "=&v"(alo)
      : "v"(b0), "v"(b1), "v"(a0), "v"(a1), "n"(STAGE_OFF)
      : "memory");
}

// Workgroup ids are dispatched to the 8 XCDs in turn (id mod 8), each XCD
// with its own L2.  Map the ids of one XCD to a contiguous range of tiles,
// with the row tiles (blockIdx.y) of one pixel tile adjacent, so each L2 holds
// its own share of the input rows and the filter digits.
__device__ __forceinline__ void xcd_tile(int32_t& tx, int32_t& ty) {
  const int32_t nbx = gridDim.x, nby = gridDim.y, total = nbx * nby;
  const int32_t lin = blockIdx.y * nbx + blockIdx.x;
  const int32_t x = lin & 7, q = total >> 3, r = total & 7;
  const int32_t t = x * q + min(x, r) + (lin >> 3);
  ty = t % nby;
  tx = t / nby;
}

template <bool PARTIALS, bool I32 = false, bool BLOCKED = false>
__global__ __launch_bounds__(kThreadsQ, 4) void k_conv_mfma_q(ConvMfmaArgs a) {
  __shared__ __align__(16) uint8_t smem[kStages * kStageBytes];
  extern __shared__ __align__(16) int8_t qexp[];  // BLOCKED: exponents [nb][64 rows], then [nb][128 columns]
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int half = lane >> 5;
  const int col = lane & 31;
  const int wm = wave & 1, wp = wave >> 1;  // 32-row and 32-pixel sub-tile of this wave
  int32_t tx, ty;
  xcd_tile(tx, ty);
  const int32_t m0 = ty * kMT;
  // the launcher guarantees outputs and the B workspace index below 2^31
  const int32_t NP = (int32_t)a.NP;
  const int32_t PQ = a.Po * a.Qo;

  // ---- output pixel of this lane (MFMA column)
  const int32_t g = tx * kNT + wp * 32 + col;
  const bool gvalid = g < NP;
  int32_t obase;
  {
    const int32_t gg = gvalid ? g : 0;
    obase = (gg / PQ) * a.M * PQ + (gg % PQ);
  }

  // ---- load assignments: A slot tid (waves 0-3 only), B slot tid
  const bool loads_a = wave_u < 4;
  const int a_slot = threadIdx.x & 255;
  const int a_row = a_slot >> 2, a_piece = (a_slot & 3) ^ ((a_row >> 2) & 3);
  const uint32_t a_voff = (uint32_t)(((m0 + a_row) * 2 + (a_piece >> 1)) * 32 + (a_piece & 1) * 16);
  const int64_t a_block_bytes = (int64_t)a.Mp * 64;
  int32_t b_voff;
  bool b_upper;
  {
    const int slot = threadIdx.x;
    const int px = slot >> 2, piece = (slot & 3) ^ ((px >> 2) & 3);
    b_upper = (piece >> 1) != 0;
    int32_t gp = tx * kNT + px;
    if (gp >= NP) gp = 0;
    const int32_t qo = gp % a.Qo, po = (gp / a.Qo) % a.Po, im = gp / PQ;
    b_voff = ((im * a.Hp + po * a.ustride_h + a.roff_h) * a.Wp + qo * a.ustride_w + a.roff_w) * a.CG * 32 +
             (piece & 1) * 16;
  }
  const int32_t KB = a.KB;

  auto issue = [&](int32_t kb) {
    uint8_t* st = smem + (kb % kStages) * kStageBytes;
    if (loads_a)
      __builtin_amdgcn_global_load_lds((const void*)(a.wsa + kb * a_block_bytes + a_voff),
                                       (lds_ptr_t)(st + wave_u * 1024), 16, 0, 0);
    const int2 o = a.boff[kb];
    __builtin_amdgcn_global_load_lds((const void*)(a.xs + (uint32_t)(b_voff + (b_upper ? o.y : o.x))),
                                     (lds_ptr_t)(st + kStageA + wave_u * 1024), 16, 0, 0);
  };

  Acc3 acc;
  float sum[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    acc.hh[v] = 0; acc.xx[v] = 0; acc.ll[v] = 0;
    sum[v] = 0.f;
  }

  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)smem;
  const uint32_t rb0 = lds_base + kStageA + swz(wp * 32 + col, 2 * half) * 16;
  const uint32_t rb1 = lds_base + kStageA + swz(wp * 32 + col, 2 * half + 1) * 16;
  const uint32_t ra0 = lds_base + swz(wm * 32 + col, 2 * half) * 16;
  const uint32_t ra1 = lds_base + swz(wm * 32 + col, 2 * half + 1) * 16;
  const int32_t mrow0 = m0 + wm * 32 + 4 * half;

  int64_t j = 0;
  int32_t blk_in_chunk = 0;
  const int32_t chunk_blocks = a.L / 32;

  // Blocked-DFP: this workgroup's exponents staged in LDS before any DMA; a
  // lane keeps the exponent sums of its 16 outputs for the current block
  int32_t ev[16];
  uint32_t xa = 0, xb = 0;
  int32_t xblk = 0, chunk_in_xblk = 0;
  const int32_t chunks_per_xblk = BLOCKED ? a.bk / a.L : 1;
  if (BLOCKED) {
    const int32_t nb = a.nb;
    for (int32_t i = threadIdx.x; i < nb * kMT; i += kThreadsQ) {
      const int32_t b = i / kMT, row = m0 + i % kMT;
      qexp[i] = row < a.M ? a.exa[(int64_t)b * a.M + row] : (int8_t)0;
    }
    for (int32_t i = threadIdx.x; i < nb * kNT; i += kThreadsQ) {
      const int32_t b = i / kNT, cc = tx * kNT + i % kNT;
      qexp[nb * kMT + i] = cc < NP ? a.exb[(int64_t)b * NP + cc] : (int8_t)0;
    }
    __syncthreads();
    const uint32_t qb = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int8_t*)qexp;
    xa = qb + wm * 32 + 4 * half;
    xb = qb + nb * kMT + wp * 32 + col;
  }
  auto load_ev = [&]() {
    // rows mrow0 + 8*g + (0..3) are 4 consecutive bytes of the row table
    uint32_t w0, w1, w2, w3;
    int32_t eb;
    const uint32_t ra = xa + (uint32_t)xblk * kMT, rb = xb + (uint32_t)xblk * kNT;
    asm volatile(
        "ds_read_b32 %0, %5\n\t"
        "ds_read_b32 %1, %5 offset:8\n\t"
        "ds_read_b32 %2, %5 offset:16\n\t"
        "ds_read_b32 %3, %5 offset:24\n\t"
        "ds_read_i8 %4, %6\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(w0), "=&v"(w1), "=&v"(w2), "=&v"(w3), "=&v"(eb)
        : "v"(ra), "v"(rb)
        : "memory");
    const uint32_t w[4] = {w0, w1, w2, w3};
#pragma unroll
    for (int v = 0; v < 16; ++v) ev[v] = (int32_t)(int8_t)(w[v >> 2] >> (8 * (v & 3))) + eb;
  };

  // One block: wait for its loads (the two newer blocks may stay in flight:
  // two loads each in waves 0-3, one in waves 4-7), barrier, refill the slot
  // freed by the previous block, read and consume.
  auto step = [&](int32_t kb, auto stage_tag) {
    constexpr int STAGE = decltype(stage_tag)::value;
    const int32_t ahead = min(kStages - 2, KB - 1 - kb);
    if (loads_a) {
      if (ahead >= 2) wait_vmcnt<4>();
      else if (ahead == 1) wait_vmcnt<2>();
      else wait_vmcnt<0>();
    } else {
      if (ahead >= 2) wait_vmcnt<2>();
      else if (ahead == 1) wait_vmcnt<1>();
      else wait_vmcnt<0>();
    }
    __builtin_amdgcn_s_barrier();
    if (kb + kStages - 1 < KB) issue(kb + kStages - 1);
    v4i bhi, blo, ahi, alo;
    read_stage_q<STAGE * kStageBytes>(rb0, rb1, ra0, ra1, bhi, blo, ahi, alo);
    mfma_tile(acc, ahi, alo, bhi, blo, blk_in_chunk == 0);
    if (++blk_in_chunk == chunk_blocks || kb == KB - 1) {
      if (I32) {
        keep_tile_i32(acc, sum);
      } else if (BLOCKED) {
        if (chunk_in_xblk == 0) load_ev();
        flush_tile_blocked<PARTIALS>(acc, sum, ev, j, a.partials, a.O, obase, PQ, mrow0, a.M, gvalid);
        if (++chunk_in_xblk == chunks_per_xblk) {
          chunk_in_xblk = 0;
          ++xblk;
        }
      } else {
        flush_tile<PARTIALS>(acc, sum, j, a.partials, a.O, obase, PQ, mrow0, a.M, gvalid);
      }
      ++j;
      blk_in_chunk = 0;
    }
  };

  for (int32_t s = 0; s < kStages - 1 && s < KB; ++s) issue(s);
  int32_t kb = 0;
  for (; kb + kStages <= KB; kb += kStages) {
    step(kb + 0, std::integral_constant<int, 0>{});
    step(kb + 1, std::integral_constant<int, 1>{});
    step(kb + 2, std::integral_constant<int, 2>{});
    step(kb + 3, std::integral_constant<int, 3>{});
  }
  if (kb < KB) step(kb++, std::integral_constant<int, 0>{});
  if (kb < KB) step(kb++, std::integral_constant<int, 1>{});
  if (kb < KB) step(kb++, std::integral_constant<int, 2>{});

  // ---- epilogue: scale once (blocked: already scaled per chunk), store, max |y|
  const int32_t e = BLOCKED ? 0 : a.ea->exp + a.eb->exp;
  uint32_t amax = 0;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int32_t m = mrow0 + 8 * (v >> 2) + (v & 3);
    if (gvalid && m < a.M) amax = max(amax, store_out<I32>(a.out, (uint32_t)(obase + m * PQ), sum[v], e));
  }
  if (a.so) {
    __shared__ uint32_t red[kWavesQ];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, off, 64));
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t b = red[0];
      for (int i = 1; i < kWavesQ; ++i) b = max(b, red[i]);
      if (b > __atomic_load_n(&a.so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&a.so->amax_bits, b);
      if (I32) {
        if (blockIdx.x == 0 && blockIdx.y == 0) a.so->exp = e;
      } else if (b == 0x7f800000u) {
        atomicOr(&a.so->flags, DFP_FLAG_OUTPUT_INF);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Skewed variant for chunks of exactly two blocks (L = 64) when every chunk is
// full (T a multiple of 64).  At L = 64 a chunk's conversion costs as many VALU
// cycles as its MFMAs, so the two 32-row tiles of a wave run one block out of
// phase: tile 1 consumes block kb-1 while tile 0 consumes block kb.  The chunk
// end of one tile then always falls in a block where only the other tile issues
// MFMAs, and the conversion (two shift-adds, a convert and an add per output)
// is interleaved with those MFMAs instruction by instruction.
//   even kb: flush tile 0 (chunk kb/2-1) || tile 1 block kb-1; tile 0 block kb opens a chunk
//   odd  kb: flush tile 1 (chunk (kb-1)/2-1) || tile 0 block kb; tile 1 block kb-1 opens a chunk
// Operand reads of the next stage are issued before the MFMAs of this one.

// Issue the six operand reads of a stage (no wait).
template <int STAGE_OFF>
__device__ __forceinline__ void read_stage_issue(uint32_t b0, uint32_t b1, uint32_t a00, uint32_t a01, uint32_t a10,
                                                 uint32_t a11, v4i& bhi, v4i& blo, v4i& ahi0, v4i& alo0, v4i& ahi1,
                                                 v4i& alo1) {
  asm volatile(
      "ds_read_b128 %0, %6 offset:%12\n\t"
      "ds_read_b128 %1, %7 offset:%12\n\t"
      "ds_read_b128 %2, %8 offset:%12\n\t"
      "ds_read_b128 %3, %9 offset:%12\n\t"
      "ds_read_b128 %4, %10 offset:%12\n\t"
      "ds_read_b128 %5, %11 offset:%12"
      : "=&v"(bhi), "=&v"(blo), "=&v"(ahi0), "=&v"(alo0), "=&v"(ahi1), "=&v"(alo1)
      : "v"(b0), "v"(b1), "v"(a00), "v"(a01), "v"(a10), "v"(a11), "n"(STAGE_OFF)
      : "memory");
}

// Wait for outstanding LDS reads; the operands pass through so that no use
// can be scheduled before the wait.
__device__ __forceinline__ void read_stage_wait(v4i& bhi, v4i& blo, v4i& ahi0, v4i& alo0, v4i& ahi1, v4i& alo1) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(bhi), "+v"(blo), "+v"(ahi0), "+v"(alo0), "+v"(ahi1), "+v"(alo1)
               :
               : "memory");
}

// 4 MFMAs of one tile interleaved with a 64-instruction conversion block.
__device__ __forceinline__ void interleave_4x16() {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 16, 0);
  }
}

template <bool PARTIALS>
__global__ __launch_bounds__(kThreads, 2) void k_conv_mfma_skew(ConvMfmaArgs a) {
  __shared__ __align__(16) uint8_t smem[kStages * kStageBytes];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int half = lane >> 5;
  const int col = lane & 31;
  const int32_t m0 = blockIdx.y * kMT;
  const int64_t NP = a.NP;
  const int64_t PQ = (int64_t)a.Po * a.Qo;

  const int64_t g = (int64_t)blockIdx.x * kNT + wave * 32 + col;
  const bool gvalid = g < NP;
  int64_t obase;
  {
    const int64_t gg = gvalid ? g : 0;
    const int32_t qo = (int32_t)(gg % a.Qo), po = (int32_t)((gg / a.Qo) % a.Po);
    const int64_t img = gg / PQ;
    obase = img * a.M * PQ + (int64_t)po * a.Qo + qo;
  }

  const int a_slot = wave * 64 + lane;
  const int a_row = a_slot >> 2, a_piece = (a_slot & 3) ^ ((a_row >> 2) & 3);
  const uint8_t* a_src = a.wsa + ((int64_t)(m0 + a_row) * 2 + (a_piece >> 1)) * 32 + (a_piece & 1) * 16;
  const int64_t a_block_bytes = (int64_t)a.Mp * 64;
  const uint8_t* b_src[2];
  int b_half[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int slot = wave * 128 + i * 64 + lane;
    const int px = slot >> 2, piece = (slot & 3) ^ ((px >> 2) & 3);
    b_half[i] = piece >> 1;
    int64_t gp = (int64_t)blockIdx.x * kNT + px;
    if (gp >= NP) gp = 0;
    const int32_t qo = (int32_t)(gp % a.Qo), po = (int32_t)((gp / a.Qo) % a.Po);
    const int64_t im = gp / PQ;
    b_src[i] = a.xs +
               (((im * a.Hp + (int64_t)po * a.ustride_h + a.roff_h) * a.Wp + (int64_t)qo * a.ustride_w + a.roff_w) *
                a.CG) * 32 +
               (piece & 1) * 16;
  }
  const int32_t tap_row_bytes = a.rsign * a.Wp * a.CG * 32;
  const int32_t tap_col_bytes = a.rsign * a.CG * 32;
  const int32_t Cin = a.Cin, KB = a.KB;

  int32_t ld_c = 0, ld_r = 0, ld_s = 0;
  auto issue = [&](int32_t kb) {
    uint8_t* st = smem + (kb % kStages) * kStageBytes;
    __builtin_amdgcn_global_load_lds((const void*)(a_src + kb * a_block_bytes), (lds_ptr_t)(st + wave * 1024), 16, 0,
                                     0);
    const int32_t off0 = ld_r * tap_row_bytes + ld_s * tap_col_bytes + (ld_c >> 4) * 32;
    int32_t off1;
    if (ld_c + 16 < Cin) {
      off1 = off0 + 32;
    } else {
      const int32_t s1 = (ld_s + 1 == a.S) ? 0 : ld_s + 1;
      const int32_t r1 = (ld_s + 1 == a.S) ? ld_r + 1 : ld_r;
      off1 = r1 * tap_row_bytes + s1 * tap_col_bytes;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
      __builtin_amdgcn_global_load_lds((const void*)(b_src[i] + (b_half[i] ? off1 : off0)),
                                       (lds_ptr_t)(st + kStageA + wave * 2048 + i * 1024), 16, 0, 0);
    ld_c += 32;
    while (ld_c >= Cin) {
      ld_c -= Cin;
      if (++ld_s == a.S) { ld_s = 0; ++ld_r; }
    }
  };
  // wait until block kb has landed for every lane of the workgroup, then refill
  auto sync_block = [&](int32_t kb) {
    const int32_t ahead = min(kStages - 2, KB - 1 - kb);
    if (ahead >= 2) wait_vmcnt<6>();
    else if (ahead == 1) wait_vmcnt<3>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (kb + kStages - 1 < KB) issue(kb + kStages - 1);
  };

  Acc3 acc0, acc1;
  float sum0[16], sum1[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    acc0.hh[v] = 0; acc0.xx[v] = 0; acc0.ll[v] = 0;
    acc1.hh[v] = 0; acc1.xx[v] = 0; acc1.ll[v] = 0;
    sum0[v] = 0.f; sum1[v] = 0.f;
  }

  const int b_rd0 = kStageA + swz(wave * 32 + col, 2 * half) * 16;
  const int b_rd1 = kStageA + swz(wave * 32 + col, 2 * half + 1) * 16;
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)smem;
  const uint32_t rb0 = lds_base + b_rd0, rb1 = lds_base + b_rd1;
  const uint32_t ra00 = lds_base + swz(col, 2 * half) * 16, ra01 = lds_base + swz(col, 2 * half + 1) * 16;
  const uint32_t ra10 = lds_base + swz(32 + col, 2 * half) * 16, ra11 = lds_base + swz(32 + col, 2 * half + 1) * 16;
  const int32_t mrow0 = m0 + 4 * half, mrow1 = m0 + 32 + 4 * half;

  // current block operands (c*) and tile 1's lagging block operands (p*)
  v4i cbh, cbl, ca0h, ca0l, ca1h, ca1l;
  v4i pbh, pbl, pa1h, pa1l;
  auto read_issue = [&](int32_t kb) {
    switch (kb % kStages) {
      case 0: read_stage_issue<0 * kStageBytes>(rb0, rb1, ra00, ra01, ra10, ra11, cbh, cbl, ca0h, ca0l, ca1h, ca1l); break;
      case 1: read_stage_issue<1 * kStageBytes>(rb0, rb1, ra00, ra01, ra10, ra11, cbh, cbl, ca0h, ca0l, ca1h, ca1l); break;
      case 2: read_stage_issue<2 * kStageBytes>(rb0, rb1, ra00, ra01, ra10, ra11, cbh, cbl, ca0h, ca0l, ca1h, ca1l); break;
      default: read_stage_issue<3 * kStageBytes>(rb0, rb1, ra00, ra01, ra10, ra11, cbh, cbl, ca0h, ca0l, ca1h, ca1l); break;
    }
  };

  for (int32_t s = 0; s < kStages - 1 && s < KB; ++s) issue(s);
  // block 0: tile 0 opens chunk 0
  sync_block(0);
  read_issue(0);
  read_stage_wait(cbh, cbl, ca0h, ca0l, ca1h, ca1l);
  mfma_tile(acc0, ca0h, ca0l, cbh, cbl, true);
  pbh = cbh; pbl = cbl; pa1h = ca1h; pa1l = ca1l;
  // block 1: tile 0 continues chunk 0, tile 1 opens chunk 0 on block 0
  sync_block(1);
  read_issue(1);
  read_stage_wait(cbh, cbl, ca0h, ca0l, ca1h, ca1l);
  mfma_tile(acc0, ca0h, ca0l, cbh, cbl, false);
  mfma_tile(acc1, pa1h, pa1l, pbh, pbl, true);
  pbh = cbh; pbl = cbl; pa1h = ca1h; pa1l = ca1l;

  for (int32_t kb = 2; kb < KB; kb += 2) {
    // ---- even block kb: tile 0 chunk kb/2-1 ends; tile 1 finishes its chunk on block kb-1
    sync_block(kb);
    read_issue(kb);
    flush_tile<PARTIALS>(acc0, sum0, kb / 2 - 1, a.partials, a.O, obase, PQ, mrow0, a.M, gvalid);
    mfma_tile(acc1, pa1h, pa1l, pbh, pbl, false);
    interleave_4x16();
    read_stage_wait(cbh, cbl, ca0h, ca0l, ca1h, ca1l);
    mfma_tile(acc0, ca0h, ca0l, cbh, cbl, true);
    pbh = cbh; pbl = cbl; pa1h = ca1h; pa1l = ca1l;
    // ---- odd block kb+1: tile 1 chunk kb/2-1 ends; tile 0 continues
    sync_block(kb + 1);
    read_issue(kb + 1);
    read_stage_wait(cbh, cbl, ca0h, ca0l, ca1h, ca1l);
    flush_tile<PARTIALS>(acc1, sum1, kb / 2 - 1, a.partials, a.O, obase, PQ, mrow1, a.M, gvalid);
    mfma_tile(acc0, ca0h, ca0l, cbh, cbl, false);
    interleave_4x16();
    mfma_tile(acc1, pa1h, pa1l, pbh, pbl, true);
    pbh = cbh; pbl = cbl; pa1h = ca1h; pa1l = ca1l;
  }
  // tail: tile 0's last chunk ends with block KB-1; tile 1 still owes block KB-1
  flush_tile<PARTIALS>(acc0, sum0, KB / 2 - 1, a.partials, a.O, obase, PQ, mrow0, a.M, gvalid);
  mfma_tile(acc1, pa1h, pa1l, pbh, pbl, false);
  interleave_4x16();
  flush_tile<PARTIALS>(acc1, sum1, KB / 2 - 1, a.partials, a.O, obase, PQ, mrow1, a.M, gvalid);

  // ---- epilogue: scale once, store, max |y|
  const int32_t e = a.ea->exp + a.eb->exp;
  uint32_t amax = 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int32_t m = m0 + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
      const float y = ldexpf(i == 0 ? sum0[v] : sum1[v], e);
      if (gvalid && m < a.M) {
        a.out[obase + (int64_t)m * PQ] = y;
        amax = max(amax, __float_as_uint(y) & 0x7fffffffu);
      }
    }
  }
  if (a.so) {
    __shared__ uint32_t red[kThreads / 64];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, off, 64));
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t b = red[0];
      for (int i = 1; i < kThreads / 64; ++i) b = max(b, red[i]);
      if (b > __atomic_load_n(&a.so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&a.so->amax_bits, b);
      if (b == 0x7f800000u) atomicOr(&a.so->flags, DFP_FLAG_OUTPUT_INF);
    }
  }
}

constexpr int kWaves3 = 8;
constexpr int kThreads3 = kWaves3 * 64;
constexpr int kNT3 = kWaves3 * 32;           // pixels per workgroup
constexpr int kRing3 = 4;                    // B stages per wave
constexpr int kBStage3 = 2048;               // 32 pixels x 2 halves x 32 B
constexpr int kARes3Max = 20;                // resident filter blocks (80 KiB)
constexpr int kLds3 = kARes3Max * kStageA + kWaves3 * kRing3 * kBStage3;

template <int STAGE_OFF>
__device__ __forceinline__ void read_b_issue(uint32_t b0, uint32_t b1, v4i& bhi, v4i& blo) {
  asm volatile(
      "ds_read_b128 %0, %2 offset:%4\n\t"
      "ds_read_b128 %1, %3 offset:%4"
      : "=&v"(bhi), "=&v"(blo)
      : "v"(b0), "v"(b1), "n"(STAGE_OFF)
      : "memory");
}

__device__ __forceinline__ void read_a_issue(uint32_t a00, uint32_t a01, uint32_t a10, uint32_t a11, v4i& ahi0,
                                             v4i& alo0, v4i& ahi1, v4i& alo1) {
  asm volatile(
      "ds_read_b128 %0, %4\n\t"
      "ds_read_b128 %1, %5\n\t"
      "ds_read_b128 %2, %6\n\t"
      "ds_read_b128 %3, %7"
      : "=&v"(ahi0), "=&v"(alo0), "=&v"(ahi1), "=&v"(alo1)
      : "v"(a00), "v"(a01), "v"(a10), "v"(a11)
      : "memory");
}

// ---------------------------------------------------------------------------
// Persistent barrier-free variant (L = 64, full chunks, filter digits
// resident).  One workgroup of 8 waves per CU and per 64-row tile; the filter
// digits of the tile are copied into LDS once with direct-to-LDS loads.  Each
// wave then walks its own sequence of 32-pixel tiles (wave w of workgroup b
// takes tiles b*8 + w, b*8 + w + 8*grid, ...).  Its B loads form one stream
// over (tile, block) through a private 4-slot LDS ring, two blocks ahead, so
// the next tile's first blocks are in flight while the current tile finishes
// and stores its outputs.  Within a tile the two 32-row sub-tiles run one
// block out of phase (tile 1 consumes block kb-1 while tile 0 consumes block
// kb), so each chunk conversion of one sub-tile is interleaved with the other
// sub-tile's MFMAs; the operand reads of a block are in flight during the
// other sub-tile's MFMAs on the lagging block.  I32: one chunk over the whole
// reduction (no conversion until the end), INT32 outputs.
template <bool PARTIALS, bool I32 = false>
__global__ __launch_bounds__(kThreads3, 1) void k_conv_mfma_persist(ConvMfmaArgs a) {
  __shared__ __align__(16) uint8_t smem[kLds3];
  uint8_t* const sA = smem;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int half = lane >> 5;
  const int col = lane & 31;
  const int32_t m0 = blockIdx.y * kMT;
  const int32_t Cin = a.Cin, KB = a.KB;
  // the launcher guarantees outputs and the B workspace index below 2^31
  const int32_t NP = (int32_t)a.NP, Qo = a.Qo;
  const int32_t PQ = a.Po * a.Qo;
  uint8_t* const sB = smem + kARes3Max * kStageA + wave_u * (kRing3 * kBStage3);

  // ---- filter digits of this 64-row tile: KB blocks x 256 pieces of 16 B, direct to LDS
  {
    const int64_t a_block_bytes = (int64_t)a.Mp * 64;
    const int32_t insts = (KB * 256) / 64;  // one instruction fills 64 consecutive slots
    for (int32_t j = wave_u; j < insts; j += kWaves3) {
      const int32_t slot0 = j * 64;
      const int32_t sl = slot0 + lane;
      const int32_t kb = sl >> 8, sw = sl & 255;
      const int row = sw >> 2, piece = (sw & 3) ^ ((row >> 2) & 3);
      const uint8_t* src = a.wsa + kb * a_block_bytes + ((int64_t)(m0 + row) * 2 + (piece >> 1)) * 32 + (piece & 1) * 16;
      __builtin_amdgcn_global_load_lds((const void*)src, (lds_ptr_t)(sA + slot0 * 16), 16, 0, 0);
    }
  }

  const int32_t tiles = (NP + 31) / 32;
  const int32_t tile_stride = gridDim.x * kWaves3;
  const int32_t first_tile = blockIdx.x * kWaves3 + wave_u;
  const int32_t my_tiles = first_tile < tiles ? (tiles - first_tile + tile_stride - 1) / tile_stride : 0;
  const int32_t total_blocks = my_tiles * KB;

  const int32_t tap_row_bytes = a.rsign * a.Wp * a.CG * 32;
  const int32_t tap_col_bytes = a.rsign * a.CG * 32;
  // B load stream (uniform) and this lane's two pixel offsets into xs
  int32_t ld_blk = 0, ld_kb = 0, ld_c = 0, ld_r = 0, ld_s = 0;
  int32_t b_off0 = 0, b_off1 = 0;
  auto pixel_off = [&](int32_t tile, int i) {
    const int slot = i * 64 + lane;
    const int px = slot >> 2, piece = (slot & 3) ^ ((px >> 2) & 3);
    int32_t gp = tile * 32 + px;
    if (gp >= NP) gp = 0;
    const int32_t qo = gp % Qo, po = (gp / Qo) % a.Po, im = gp / PQ;
    return ((im * a.Hp + po * a.ustride_h + a.roff_h) * a.Wp + qo * a.ustride_w + a.roff_w) * a.CG * 32 +
           (piece & 1) * 16;
  };
  // slot i*64 + lane holds channel half ((slot & 3) ^ ((px >> 2) & 3)) >> 1 of pixel slot >> 2
  const bool up0 = (((lane & 3) ^ ((lane >> 4) & 3)) >> 1) != 0;
  const bool up1 = (((lane & 3) ^ (((64 + lane) >> 4) & 3)) >> 1) != 0;
  auto issue = [&]() {  // loads block ld_blk of the stream
    if (ld_kb == 0) {
      const int32_t tile = first_tile + (ld_blk / KB) * tile_stride;
      b_off0 = pixel_off(tile, 0);
      b_off1 = pixel_off(tile, 1);
      ld_c = 0; ld_r = 0; ld_s = 0;
    }
    uint8_t* st = sB + (ld_blk % kRing3) * kBStage3;
    const int32_t off0 = ld_r * tap_row_bytes + ld_s * tap_col_bytes + (ld_c >> 4) * 32;
    int32_t off1;
    if (ld_c + 16 < Cin) {
      off1 = off0 + 32;
    } else {
      const int32_t s1 = (ld_s + 1 == a.S) ? 0 : ld_s + 1;
      const int32_t r1 = (ld_s + 1 == a.S) ? ld_r + 1 : ld_r;
      off1 = r1 * tap_row_bytes + s1 * tap_col_bytes;
    }
    __builtin_amdgcn_global_load_lds((const void*)(a.xs + (uint32_t)(b_off0 + (up0 ? off1 : off0))), (lds_ptr_t)(st),
                                     16, 0, 0);
    __builtin_amdgcn_global_load_lds((const void*)(a.xs + (uint32_t)(b_off1 + (up1 ? off1 : off0))),
                                     (lds_ptr_t)(st + 1024), 16, 0, 0);
    ld_c += 32;
    while (ld_c >= Cin) {
      ld_c -= Cin;
      if (++ld_s == a.S) { ld_s = 0; ++ld_r; }
    }
    ++ld_blk;
    if (++ld_kb == KB) ld_kb = 0;
  };
  // stream block gb has landed for this wave (the newer ones may stay in flight); refill
  auto wait_block = [&](int32_t gb) {
    const int32_t ahead = min(kRing3 - 2, total_blocks - 1 - gb);
    if (ahead >= 2) wait_vmcnt<4>();
    else if (ahead == 1) wait_vmcnt<2>();
    else wait_vmcnt<0>();
    if (ld_blk < total_blocks) issue();
  };

  const uint32_t sA_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)sA;
  const uint32_t sB_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)sB;
  const uint32_t rb0 = sB_base + swz(col, 2 * half) * 16, rb1 = sB_base + swz(col, 2 * half + 1) * 16;
  // rows 32..63 sit 2048 bytes after rows 0..31 at the same swizzle position
  const uint32_t ra00 = sA_base + swz(col, 2 * half) * 16, ra01 = sA_base + swz(col, 2 * half + 1) * 16;
  const int32_t e = a.ea->exp + a.eb->exp;
  uint32_t amax = 0;

  v4i cbh, cbl, ca0h, ca0l, ca1h, ca1l;  // block kb
  v4i pbh, pbl, pa1h, pa1l;              // tile 1's lagging block kb-1
  auto read_block = [&](int32_t gb, int32_t kb) {
    switch (gb % kRing3) {
      case 0: read_b_issue<0 * kBStage3>(rb0, rb1, cbh, cbl); break;
      case 1: read_b_issue<1 * kBStage3>(rb0, rb1, cbh, cbl); break;
      case 2: read_b_issue<2 * kBStage3>(rb0, rb1, cbh, cbl); break;
      default: read_b_issue<3 * kBStage3>(rb0, rb1, cbh, cbl); break;
    }
    const uint32_t ao = (uint32_t)kb * kStageA;
    read_a_issue(ra00 + ao, ra01 + ao, ra00 + ao + 2048, ra01 + ao + 2048, ca0h, ca0l, ca1h, ca1l);
  };

  while (ld_blk < min(kRing3 - 1, total_blocks)) issue();
  wait_vmcnt<0>();  // filter digits (and the first B blocks) landed for this lane
  __syncthreads();  // ... and for every lane

  for (int32_t it = 0; it < my_tiles; ++it) {
    const int32_t gb0 = it * KB;
    const int32_t g = (first_tile + it * tile_stride) * 32 + col;
    const bool gvalid = g < NP;
    int32_t obase;
    {
      const int32_t gg = gvalid ? g : 0;
      obase = (gg / PQ) * a.M * PQ + (gg % PQ);
    }
    const int32_t mrow0 = m0 + 4 * half, mrow1 = m0 + 32 + 4 * half;
    Acc3 acc0, acc1;
    float sum0[16], sum1[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) { sum0[v] = 0.f; sum1[v] = 0.f; }

    // block 0: tile 0 opens chunk 0
    wait_block(gb0);
    read_block(gb0, 0);
    read_stage_wait(cbh, cbl, ca0h, ca0l, ca1h, ca1l);
    mfma_tile(acc0, ca0h, ca0l, cbh, cbl, true);
    pbh = cbh; pbl = cbl; pa1h = ca1h; pa1l = ca1l;
    // block 1: tile 0 continues, tile 1 opens chunk 0 on block 0
    wait_block(gb0 + 1);
    read_block(gb0 + 1, 1);
    read_stage_wait(cbh, cbl, ca0h, ca0l, ca1h, ca1l);
    mfma_tile(acc0, ca0h, ca0l, cbh, cbl, false);
    mfma_tile(acc1, pa1h, pa1l, pbh, pbl, true);
    pbh = cbh; pbl = cbl; pa1h = ca1h; pa1l = ca1l;

    for (int32_t kb = 2; kb < KB; kb += 2) {
      // even: tile 0's chunk ended at kb-1; tile 1 finishes its chunk on block kb-1
      wait_block(gb0 + kb);
      read_block(gb0 + kb, kb);
      if (!I32) flush_tile<PARTIALS>(acc0, sum0, kb / 2 - 1, a.partials, a.O, obase, PQ, mrow0, a.M, gvalid);
      mfma_tile(acc1, pa1h, pa1l, pbh, pbl, false);
      if (!I32) interleave_4x16();
      read_stage_wait(cbh, cbl, ca0h, ca0l, ca1h, ca1l);
      mfma_tile(acc0, ca0h, ca0l, cbh, cbl, !I32);
      pbh = cbh; pbl = cbl; pa1h = ca1h; pa1l = ca1l;
      // odd: tile 1's chunk ended; tile 0 continues; tile 1 opens the next chunk on block kb
      wait_block(gb0 + kb + 1);
      read_block(gb0 + kb + 1, kb + 1);
      read_stage_wait(cbh, cbl, ca0h, ca0l, ca1h, ca1l);
      if (!I32) flush_tile<PARTIALS>(acc1, sum1, kb / 2 - 1, a.partials, a.O, obase, PQ, mrow1, a.M, gvalid);
      mfma_tile(acc0, ca0h, ca0l, cbh, cbl, false);
      if (!I32) interleave_4x16();
      mfma_tile(acc1, pa1h, pa1l, pbh, pbl, !I32);
      pbh = cbh; pbl = cbl; pa1h = ca1h; pa1l = ca1l;
    }
    if (I32) {
      keep_tile_i32(acc0, sum0);
      mfma_tile(acc1, pa1h, pa1l, pbh, pbl, false);
      keep_tile_i32(acc1, sum1);
    } else {
      flush_tile<PARTIALS>(acc0, sum0, KB / 2 - 1, a.partials, a.O, obase, PQ, mrow0, a.M, gvalid);
      mfma_tile(acc1, pa1h, pa1l, pbh, pbl, false);
      interleave_4x16();
      flush_tile<PARTIALS>(acc1, sum1, KB / 2 - 1, a.partials, a.O, obase, PQ, mrow1, a.M, gvalid);
    }

    // ---- outputs of this tile (the stores drain while the next tile computes)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int32_t m = m0 + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
        if (gvalid && m < a.M)
          amax = max(amax, store_out<I32>(a.out, (uint32_t)(obase + m * PQ), i == 0 ? sum0[v] : sum1[v], e));
      }
    }
  }

  if (a.so) {
    __shared__ uint32_t red[kWaves3];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, off, 64));
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t b = red[0];
      for (int i = 1; i < kWaves3; ++i) b = max(b, red[i]);
      if (b > __atomic_load_n(&a.so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&a.so->amax_bits, b);
      if (I32) {
        if (blockIdx.x == 0 && blockIdx.y == 0) a.so->exp = e;
      } else if (b == 0x7f800000u) {
        atomicOr(&a.so->flags, DFP_FLAG_OUTPUT_INF);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Four-waves-per-SIMD persistent variant (chunks of two blocks, L = 64, or one
// chunk over the whole reduction; reduction channel counts that are multiples
// of 32; at most kW16MaxKB blocks).  One workgroup of 16 waves per CU and per
// 64-row tile keeps the tile's filter digits resident in LDS.  The work is a
// list of units (32-pixel tile, 32-row half), u = 2 * tile + half; workgroup
// b takes a contiguous range of units (ranges of one XCD adjacent, so its L2
// holds the input rows the range touches); wave w of it starts with unit w
// of the range and then takes the next unit no wave has taken (a counter in
// LDS), so a wave that the issue arbitration favours takes more units and
// the SIMDs finish close together.  Each lane loads its
// B operand (16 channels x hi / lo digits of its pixel) straight into
// registers, one chunk ahead, from the plane layout of the digit tensor, where
// the 32 lanes of a channel half read 512 consecutive bytes; the A
// operand comes from LDS.  With four waves per SIMD one wave's chunk
// conversion (VALU) runs while the others issue MFMAs, and the reduction loop
// has no data-dependent branches.
constexpr int kWaves16 = 16;
constexpr int kThreads16 = kWaves16 * 64;
constexpr int32_t kW16MaxKB = 36;

template <bool PARTIALS, bool I32 = false, bool PHASED = false>
__global__ __launch_bounds__(kThreads16, 1) void k_conv_mfma_w16(ConvMfmaArgs a) {
  __shared__ __align__(16) uint8_t sA[kW16MaxKB * kStageA];
  __shared__ __align__(8) int32_t s_boff[kW16MaxKB];
  __shared__ uint32_t red[kWaves16];
  __shared__ int32_t s_next;  // the first unit of the range no wave has taken yet
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5;
  const int col = lane & 31;
  const int32_t m0 = blockIdx.y * kMT;
  // this launch's phase: filter blocks kb0 .. kb0 + KB - 1 (whole chunks)
  const int32_t kb0 = PHASED ? a.kb0 : 0, KB = PHASED ? a.kbn : a.KB, J = KB / 2, Cin = a.Cin;
  const bool first_phase = !PHASED || (a.phase_flags & 1) != 0, last_phase = !PHASED || (a.phase_flags & 2) != 0;
  // the launcher guarantees outputs and the B workspace index below 2^31
  const int32_t NP = (int32_t)a.NP, Qo = a.Qo, PQ = a.Po * a.Qo;
  // output scale exponent, read before any other memory operation is in flight
  const int32_t e = __builtin_amdgcn_readfirstlane(a.ea->exp + a.eb->exp);

  // ---- filter digits of this 64-row tile: KB blocks x 256 pieces of 16 B, direct to LDS
  {
    const int64_t a_block_bytes = (int64_t)a.Mp * 64;
    const int32_t insts = (KB * 256) / 64;  // one instruction fills 64 consecutive slots
    for (int32_t j = wave; j < insts; j += kWaves16) {
      const int32_t slot0 = j * 64;
      const int32_t sl = slot0 + lane;
      const int32_t kb = sl >> 8, sw = sl & 255;
      const int row = sw >> 2, piece = (sw & 3) ^ ((row >> 2) & 3);
      const uint8_t* src =
          a.wsa + (kb0 + kb) * a_block_bytes + ((int64_t)(m0 + row) * 2 + (piece >> 1)) * 32 + (piece & 1) * 16;
      __builtin_amdgcn_global_load_lds((const void*)src, (lds_ptr_t)(sA + slot0 * 16), 16, 0, 0);
    }
  }
  // plane layout: row stride Cin*2*Wp bytes, column stride 16, 32-channel block stride 4*Wp*16,
  // lo digits 2*Wp*16 bytes after the hi digits, channel half `half` at Wp*16.
  // Byte offset of block kb (tap (r, s), channel block cb) from a pixel's operand:
  const int32_t cpb = Cin >> 5;  // blocks per filter tap
  const int32_t plane_bytes = a.Wp * 16;
  auto boff_of = [&](int32_t kb) {
    const int32_t tap = kb / cpb, cb = kb - tap * cpb;
    const int32_t r = tap / a.S, sx = tap - r * a.S;
    return a.rsign * (r * cpb * 4 * plane_bytes + sx * 16) + cb * 4 * plane_bytes;
  };
  if ((int32_t)threadIdx.x < KB) s_boff[threadIdx.x] = boff_of(kb0 + (int32_t)threadIdx.x);

  // ---- this workgroup's unit range (XCD x = workgroup id mod 8 gets adjacent ranges)
  // units (32-pixel tile, 32-row half); a tile whose second half lies past
  // the output rows (M - m0 <= 32) has only its first half as a unit
  const int32_t hsh = a.M - m0 > 32 ? 1 : 0;
  const int32_t units = ((NP + 31) / 32) << hsh;
  const int32_t G = gridDim.x;
  const int32_t xcd = blockIdx.x & 7, per = G >> 3, rem = G & 7;
  const int32_t vb = xcd * per + min(xcd, rem) + (blockIdx.x >> 3);
  const int32_t u0 = (int32_t)((int64_t)units * vb / G), u1 = (int32_t)((int64_t)units * (vb + 1) / G);
  const int32_t my_units = (u1 - u0 > wave) ? (u1 - u0 - wave + kWaves16 - 1) / kWaves16 : 0;
  auto unit_of = [&](int32_t i) { return u0 + wave + kWaves16 * i; };
  if (threadIdx.x == 0) s_next = u0 + kWaves16;
  // byte offset of this lane's operand for the pixel of unit u (block offsets come from s_boff)
  auto pixel_off = [&](int32_t u) -> int32_t {
    int32_t gp = (u >> hsh) * 32 + col;
    if (gp >= NP) gp = 0;
    const int32_t im = (int32_t)fdiv((uint32_t)gp, a.div_pq), rp = gp - im * PQ;
    const int32_t po = (int32_t)fdiv((uint32_t)rp, a.div_q), qo = rp - po * Qo;
    return ((im * a.Hp + po * a.ustride_h + a.roff_h) * cpb * 4 + half) * plane_bytes +
           (qo * a.ustride_w + a.roff_w) * 16;
  };
  // the loads of a block stay in stream order (hi, lo, block after block) so
  // every wait for a block's operands leaves the two newer loads in flight
  auto load_b = [&](v4i& hi, v4i& lo, int32_t pix, int32_t boff) {
    const uint32_t off = (uint32_t)(pix + boff);
    __builtin_amdgcn_sched_barrier(0);
    hi = *reinterpret_cast<const v4i*>(a.xs + off);
    lo = *reinterpret_cast<const v4i*>(a.xs + (off + 2 * plane_bytes));
    __builtin_amdgcn_sched_barrier(0);
  };

  const bool full_rows = a.M == a.Mp;  // every row of the 64-row tiles is an output channel
  // FP32 output addressed by 32-bit byte offsets (fewer than 2^30 outputs)
  const bool out_buf = a.O < (1ll << 30);
  const __amdgpu_buffer_rsrc_t rs_out =
      __builtin_amdgcn_make_buffer_rsrc(a.out, (short)0, out_buf ? (int)(a.O * 4) : 0, 0x00020000);
  uint32_t amax = 0;
  // the stream's first chunk is requested while the filter digits are in
  // flight; afterwards each block's registers are refilled with the block two
  // ahead (the next unit's first blocks at a unit's last chunk, the last
  // unit's first blocks again at the very end) as soon as its MFMAs have been
  // issued
  int32_t cur_pix = 0;
  v4i b0h, b0l, b1h, b1l;
  if (my_units > 0) {
    cur_pix = pixel_off(unit_of(0));
    load_b(b0h, b0l, cur_pix, boff_of(kb0));
    load_b(b1h, b1l, cur_pix, boff_of(kb0 + 1));
    wait_vmcnt<4>();  // filter digits landed for this lane (its four B loads may be in flight)
  } else {
    wait_vmcnt<0>();
  }
  // ... and for every lane, and the block offsets are written: a plain barrier
  // (__syncthreads would also wait for the B loads in flight)
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");

  if (my_units > 0) {
    const uint32_t ra_hi = swz(col, 2 * half) * 16, ra_lo = swz(col, 2 * half + 1) * 16;
    // wave w starts with unit w of the range and then takes the next free
    // one (a wave that runs faster takes more units)
    for (int32_t u = unit_of(0); u < u1;) {
      int32_t nu = 0;
      if (lane == 0) nu = atomicAdd(&s_next, 1);
      nu = __builtin_amdgcn_readfirstlane(nu);
      const int32_t next_pix = nu < u1 ? pixel_off(nu) : cur_pix;
      const int32_t msub = u & hsh;
      const int32_t g = (u >> hsh) * 32 + col;
      const bool gvalid = g < NP;
      int32_t obase = 0;
      if (gvalid) {
        const int32_t im = (int32_t)fdiv((uint32_t)g, a.div_pq);
        obase = im * a.M * PQ + (g - im * PQ);
      }
      const int32_t mrow0 = m0 + 32 * msub + 4 * half;
      Acc3 acc;
      float sum[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) sum[v] = 0.f;
      if (PHASED && !first_phase && gvalid) {  // the chunk sums so far, left in the output by the previous phase
        if (full_rows && out_buf) {
          const uint32_t lane_off = (uint32_t)(obase + mrow0 * PQ) * 4u;
#pragma unroll
          for (int v = 0; v < 16; ++v)
            sum[v] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                rs_out, lane_off, (uint32_t)((8 * (v >> 2) + (v & 3)) * PQ) * 4u, 0));
        } else {
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int32_t m = mrow0 + 8 * (v >> 2) + (v & 3);
            if (m < a.M) sum[v] = a.out[(uint32_t)(obase + m * PQ)];
          }
        }
      }
      const uint8_t* ab = sA + msub * 2048;
      for (int32_t c = 0; c < J; ++c, ab += 2 * kStageA) {
        const bool last = c + 1 == J;
        const int2 bo = *reinterpret_cast<const int2*>(s_boff + (last ? 0 : 2 * c + 2));
        const int32_t pix = last ? next_pix : cur_pix;
        const v4i ah0 = *reinterpret_cast<const v4i*>(ab + ra_hi);
        const v4i al0 = *reinterpret_cast<const v4i*>(ab + ra_lo);
        if (I32 && c != 0) mfma_tile(acc, ah0, al0, b0h, b0l, false);
        else mfma_tile(acc, ah0, al0, b0h, b0l, true);
        load_b(b0h, b0l, pix, bo.x);
        const v4i ah1 = *reinterpret_cast<const v4i*>(ab + kStageA + ra_hi);
        const v4i al1 = *reinterpret_cast<const v4i*>(ab + kStageA + ra_lo);
        mfma_tile(acc, ah1, al1, b1h, b1l, false);
        load_b(b1h, b1l, pix, bo.y);
        if (!I32) flush_tile<PARTIALS>(acc, sum, kb0 / 2 + c, a.partials, a.O, obase, PQ, mrow0, a.M, gvalid);
      }
      if (I32) keep_tile_i32(acc, sum);
      if (PHASED && gvalid && !last_phase) {  // unscaled sums for the next phase
        if (full_rows && out_buf) {
          const uint32_t lane_off = (uint32_t)(obase + mrow0 * PQ) * 4u;
#pragma unroll
          for (int v = 0; v < 16; ++v)
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(sum[v]), rs_out, lane_off,
                                                  (uint32_t)((8 * (v >> 2) + (v & 3)) * PQ) * 4u, 0);
        } else {
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int32_t m = mrow0 + 8 * (v >> 2) + (v & 3);
            if (m < a.M) a.out[(uint32_t)(obase + m * PQ)] = sum[v];
          }
        }
      } else if (gvalid) {
        if (!I32 && full_rows && out_buf) {
          // buffer stores at a per-lane offset plus a uniform one per output row,
          // max |y| on floats (y is never NaN), two values per v_max3
          const uint32_t lane_off = (uint32_t)(obase + mrow0 * PQ) * 4u;
          float fmx = 0.f;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const float y = ldexpf(sum[v], e);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(y), rs_out, lane_off,
                                                  (uint32_t)((8 * (v >> 2) + (v & 3)) * PQ) * 4u, 0);
            fmx = fmaxf(fmx, fabsf(y));
          }
          amax = max(amax, __float_as_uint(fmx));
        } else if (full_rows) {
#pragma unroll
          for (int v = 0; v < 16; ++v)
            amax = max(amax, store_out<I32>(a.out, (uint32_t)(obase + (mrow0 + 8 * (v >> 2) + (v & 3)) * PQ), sum[v], e));
        } else {
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int32_t m = mrow0 + 8 * (v >> 2) + (v & 3);
            if (m < a.M) amax = max(amax, store_out<I32>(a.out, (uint32_t)(obase + m * PQ), sum[v], e));
          }
        }
      }
      cur_pix = next_pix;
      u = nu;
    }
  }

  if (a.so && last_phase) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, off, 64));
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t b = red[0];
      for (int i = 1; i < kWaves16; ++i) b = max(b, red[i]);
      if (b > __atomic_load_n(&a.so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&a.so->amax_bits, b);
      if (I32) {
        if (blockIdx.x == 0 && blockIdx.y == 0) a.so->exp = e;
      } else if (b == 0x7f800000u) {
        atomicOr(&a.so->flags, DFP_FLAG_OUTPUT_INF);
      }
    }
  }
}

// Variant of the four-waves-per-SIMD kernel with 16 x 16 output tiles
// (v_mfma_i32_16x16x64_i8: one instruction covers a whole chunk of 64
// reduction indices), for layers whose 32 x 32 tiles are too few to give
// every wave of the chip work (ResNet-50's 14 x 14 and 7 x 7 layers: 3136
// and 1568 tiles of 32 x 32 for 4096 waves; 12544 and 6272 tiles of
// 16 x 16).  Same plane-layout operands and unit ranges as the 32 x 32
// kernel, but a workgroup keeps a 32-row filter slice in LDS, so a phase
// holds up to 72 blocks (a ResNet-50 14 x 14 3 x 3 layer in one phase, a
// 7 x 7 one in two); a unit is a 16-pixel tile, whose B operand a wave loads
// once per chunk and multiplies with both 16-row subtiles of the slice (only
// the first where the second lies past the output rows).  Lane l multiplies
// pixel l % 16 of the tile (B) and row l % 16 of each subtile (A) over the
// chunk's indices 16 (l / 16) .. + 15, that is channel half (l / 16) % 2 of
// block 2 c + l / 32; it accumulates rows 4 (l / 16) .. + 3 of each subtile
// at pixel l % 16.  The B registers of chunk c + 2 are loaded as soon as
// chunk c's MFMAs have issued (two register sets, chunks taken in pairs:
// every phase has an even number of chunks).  FP32 outputs only (no
// partials, no single-chunk INT32 mode).  Against units of one subtile each
// (twice as many, each loading B): ResNet-50 res4 3 x 3 forward 47.8 ->
// 43.4 us, backward-data 50.6 -> 43.3 us; res5 65 -> 57 us with one
// workgroup per CU although some waves then get no tile.
constexpr int32_t kS16Rows = 32;                   // filter rows per workgroup
constexpr int32_t kS16Block = kS16Rows * 64;        // LDS bytes of one filter block
constexpr int32_t kS16MaxKB = kW16MaxKB * kStageA / kS16Block;  // 72

template <bool PHASED>
__global__ __launch_bounds__(kThreads16, 1) void k_conv_mfma_s16(ConvMfmaArgs a) {
  __shared__ __align__(16) uint8_t sA[kS16MaxKB * kS16Block];
  __shared__ __align__(8) int32_t s_boff[kS16MaxKB];
  __shared__ uint32_t red[kWaves16];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15;  // pixel of the tile, row of the subtile
  const int kg = lane >> 4;   // index group of the chunk
  const int32_t m0 = blockIdx.y * kS16Rows;
  const int32_t kb0 = PHASED ? a.kb0 : 0, KB = PHASED ? a.kbn : a.KB, J = KB / 2, Cin = a.Cin;
  const bool first_phase = !PHASED || (a.phase_flags & 1) != 0, last_phase = !PHASED || (a.phase_flags & 2) != 0;
  const int32_t NP = (int32_t)a.NP, Qo = a.Qo, PQ = a.Po * a.Qo;
  const int32_t e = __builtin_amdgcn_readfirstlane(a.ea->exp + a.eb->exp);

  // ---- filter digits of this 32-row slice: KB blocks x 128 pieces of 16 B, direct to LDS
  {
    const int64_t a_block_bytes = (int64_t)a.Mp * 64;
    const int32_t insts = (KB * kS16Block / 16) / 64;  // one instruction fills 64 consecutive slots
    for (int32_t j = wave; j < insts; j += kWaves16) {
      const int32_t slot0 = j * 64;
      const int32_t sl = slot0 + lane;
      const int32_t kb = sl / (kS16Block / 16), sw = sl % (kS16Block / 16);
      const int row = sw >> 2, piece = (sw & 3) ^ ((row >> 2) & 3);
      const uint8_t* src =
          a.wsa + (kb0 + kb) * a_block_bytes + ((int64_t)(m0 + row) * 2 + (piece >> 1)) * 32 + (piece & 1) * 16;
      __builtin_amdgcn_global_load_lds((const void*)src, (lds_ptr_t)(sA + slot0 * 16), 16, 0, 0);
    }
  }
  const int32_t cpb = Cin >> 5;
  const int32_t plane_bytes = a.Wp * 16;
  auto boff_of = [&](int32_t kb) {
    const int32_t tap = kb / cpb, cb = kb - tap * cpb;
    const int32_t r = tap / a.S, sx = tap - r * a.S;
    return a.rsign * (r * cpb * 4 * plane_bytes + sx * 16) + cb * 4 * plane_bytes;
  };
  if ((int32_t)threadIdx.x < KB) s_boff[threadIdx.x] = boff_of(kb0 + (int32_t)threadIdx.x);

  // ---- this workgroup's unit range (XCD x = workgroup id mod 8 gets adjacent ranges)
  // units: 16-pixel tiles; both 16-row subtiles of the slice, or only the
  // first where the second lies past the output rows (M - m0 <= 16)
  const bool two_sub = a.M - m0 > 16;
  const int32_t units = (NP + 15) / 16;
  const int32_t G = gridDim.x;
  const int32_t xcd = blockIdx.x & 7, per = G >> 3, rem = G & 7;
  const int32_t vb = xcd * per + min(xcd, rem) + (blockIdx.x >> 3);
  const int32_t u0 = (int32_t)((int64_t)units * vb / G), u1 = (int32_t)((int64_t)units * (vb + 1) / G);
  const int32_t my_units = (u1 - u0 > wave) ? (u1 - u0 - wave + kWaves16 - 1) / kWaves16 : 0;
  auto unit_of = [&](int32_t i) { return u0 + wave + kWaves16 * i; };
  // byte offset of this lane's operand (pixel of unit u, channel half kg % 2)
  auto pixel_off = [&](int32_t u) -> int32_t {
    int32_t gp = u * 16 + col;
    if (gp >= NP) gp = 0;
    const int32_t im = (int32_t)fdiv((uint32_t)gp, a.div_pq), rp = gp - im * PQ;
    const int32_t po = (int32_t)fdiv((uint32_t)rp, a.div_q), qo = rp - po * Qo;
    return ((im * a.Hp + po * a.ustride_h + a.roff_h) * cpb * 4 + (kg & 1)) * plane_bytes +
           (qo * a.ustride_w + a.roff_w) * 16;
  };
  // this lane's block offset for chunk c (block 2 c + kg / 2 of the phase)
  auto boff_chunk = [&](int32_t c) {
    const int2 bo = *reinterpret_cast<const int2*>(s_boff + 2 * c);
    return (kg & 2) ? bo.y : bo.x;
  };
  auto load_b = [&](v4i& hi, v4i& lo, int32_t pix, int32_t boff) {
    const uint32_t off = (uint32_t)(pix + boff);
    __builtin_amdgcn_sched_barrier(0);
    hi = *reinterpret_cast<const v4i*>(a.xs + off);
    lo = *reinterpret_cast<const v4i*>(a.xs + (off + 2 * plane_bytes));
    __builtin_amdgcn_sched_barrier(0);
  };

  const bool full_rows = a.M == a.Mp;
  const bool out_buf = a.O < (1ll << 30);
  const __amdgpu_buffer_rsrc_t rs_out =
      __builtin_amdgcn_make_buffer_rsrc(a.out, (short)0, out_buf ? (int)(a.O * 4) : 0, 0x00020000);
  uint32_t amax = 0;
  int32_t cur_pix = 0;
  v4i b0h, b0l, b1h, b1l;
  // B of the first unit's chunks 0 and 1 while the filter digits are in flight
  if (my_units > 0) {
    cur_pix = pixel_off(unit_of(0));
    const int32_t kq = kg >> 1;
    load_b(b0h, b0l, cur_pix, boff_of(kb0 + kq));
    load_b(b1h, b1l, cur_pix, boff_of(kb0 + 2 + kq));
    wait_vmcnt<4>();
  } else {
    wait_vmcnt<0>();
  }
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");

  // The units of NSUB subtiles (rows m0 + 16 sub + 4 (l / 16) .. + 3 at
  // pixel l % 16 of the tile): the tile's B operand is loaded once per chunk
  // and multiplied with each subtile's filter rows.
  auto run_units = [&](auto nsub_c) __attribute__((always_inline)) {
    constexpr int NSUB = decltype(nsub_c)::value;
    // A: row col of the subtile, channel half kg % 2 of block kg / 2 (hi, lo pieces)
    const uint32_t ra_hi = swz(col, 2 * (kg & 1)) * 16 + (kg >> 1) * kS16Block;
    const uint32_t ra_lo = swz(col, 2 * (kg & 1) + 1) * 16 + (kg >> 1) * kS16Block;
    for (int32_t unit = 0; unit < my_units; ++unit) {
      const int32_t u = unit_of(unit);
      const int32_t next_pix = unit + 1 < my_units ? pixel_off(unit_of(unit + 1)) : cur_pix;
      const int32_t g = u * 16 + col;
      const bool gvalid = g < NP;
      int32_t obase = 0;
      if (gvalid) {
        const int32_t im = (int32_t)fdiv((uint32_t)g, a.div_pq);
        obase = im * a.M * PQ + (g - im * PQ);
      }
      const int32_t mrow0 = m0 + 4 * kg;  // row of value v of subtile sub: mrow0 + 16 sub + v
      v4i hh[NSUB], xx[NSUB], ll[NSUB];
      float sum[NSUB][4];
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
        for (int v = 0; v < 4; ++v) sum[sb][v] = 0.f;
      if (PHASED && !first_phase && gvalid) {
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int32_t m = mrow0 + 16 * sb + v;
            if (m < a.M) sum[sb][v] = a.out[(uint32_t)(obase + m * PQ)];
          }
      }
      auto chunk = [&](int32_t c, v4i& bh, v4i& bl) __attribute__((always_inline)) {
        const uint8_t* ab = sA + c * 2 * kS16Block;
        const v4i z = {0, 0, 0, 0};
        v4i ah[NSUB], al[NSUB];
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb) {
          ah[sb] = *reinterpret_cast<const v4i*>(ab + sb * 1024 + ra_hi);
          al[sb] = *reinterpret_cast<const v4i*>(ab + sb * 1024 + ra_lo);
        }
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb) {
          hh[sb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ah[sb], bh, z, 0, 0, 0);
          ll[sb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(al[sb], bl, z, 0, 0, 0);
          xx[sb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ah[sb], bl, z, 0, 0, 0);
        }
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb) xx[sb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(al[sb], bh, xx[sb], 0, 0, 0);
        // chunk c + 2 of this unit, or chunk c + 2 - J of the next one
        const int32_t nc = c + 2 < J ? c + 2 : c + 2 - J;
        load_b(bh, bl, c + 2 < J ? cur_pix : next_pix, boff_chunk(nc));
#pragma unroll
        for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const uint32_t p = recombine((uint32_t)hh[sb][v], (uint32_t)xx[sb][v], (uint32_t)ll[sb][v]);
            sum[sb][v] += (float)(int32_t)p;
          }
      };
      for (int32_t c = 0; c < J; c += 2) {
        chunk(c, b0h, b0l);
        chunk(c + 1, b1h, b1l);
      }
#pragma unroll
      for (int sb = 0; sb < NSUB; ++sb) {
        const int32_t mr = mrow0 + 16 * sb;
        if (PHASED && gvalid && !last_phase) {  // unscaled sums for the next phase
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            if (mr + v < a.M) a.out[(uint32_t)(obase + (mr + v) * PQ)] = sum[sb][v];
          }
        } else if (gvalid) {
          if (full_rows && out_buf) {
            const uint32_t lane_off = (uint32_t)(obase + mr * PQ) * 4u;
            float fmx = 0.f;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const float y = ldexpf(sum[sb][v], e);
              __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(y), rs_out, lane_off, (uint32_t)(v * PQ) * 4u, 0);
              fmx = fmaxf(fmx, fabsf(y));
            }
            amax = max(amax, __float_as_uint(fmx));
          } else {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              if (mr + v < a.M) amax = max(amax, store_out<false>(a.out, (uint32_t)(obase + (mr + v) * PQ), sum[sb][v], e));
            }
          }
        }
      }
      cur_pix = next_pix;
    }
  };
  if (my_units > 0) {
    if (two_sub) run_units(std::integral_constant<int, 2>{});
    else run_units(std::integral_constant<int, 1>{});
  }

  if (a.so && last_phase) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, off, 64));
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t b = red[0];
      for (int i = 1; i < kWaves16; ++i) b = max(b, red[i]);
      if (b > __atomic_load_n(&a.so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&a.so->amax_bits, b);
      if (b == 0x7f800000u) atomicOr(&a.so->flags, DFP_FLAG_OUTPUT_INF);
    }
  }
}

// Forward kernel for inputs with few channels (fewer than 16, such as an
// image's three colour channels), at L = 64 with FP32 outputs.  The forward
// reduction order is t = (r S + s) C + c, and for one filter row r the S C
// values (s, c) of an output pixel are contiguous in a channel-last row of the
// input (byte (q sw + s) C + c of input row p sh + r), so the 16 consecutive
// indices a lane multiplies are at most two contiguous byte runs, one at the
// end of filter row r0 and one at the start of row r0 + 1 (S C >= 16).  The
// input digits are prepared as XC[n][hp][d][row_b] (k_prep_cl); a lane loads
// 16 bytes at each run's start (byte-aligned buffer loads) and keeps the
// first n0 bytes of the first and the rest of the second (v_bfi with byte
// masks).  The offsets and masks of each (block, lane half) are a table in
// LDS.  Indices past T meet zero filter digits.  Filter digits are resident in
// LDS (at most kW16MaxKB blocks); the units, output epilogue and max are
// those of the four-waves-per-SIMD kernel; chunks are two blocks, the last one
// of an odd block count is a single block.
struct ClArgs {
  int32_t row_b;  // bytes of one digit row (at least Wp C + 16, a multiple of 16)
  int32_t SC;     // S C
  uint32_t xc_bytes;
};

template <bool PARTIALS>
__global__ __launch_bounds__(kThreads16, 1) void k_conv_mfma_cl(ConvMfmaArgs a, ClArgs cl) {
  __shared__ __align__(16) uint8_t sA[kW16MaxKB * kStageA];
  // per (block, lane half): byte offsets of the two runs, then the four dword masks of the first
  __shared__ __align__(16) int4 s_tab[2 * kW16MaxKB][2];
  __shared__ uint32_t red[kWaves16];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int half = lane >> 5;
  const int col = lane & 31;
  const int32_t m0 = blockIdx.y * kMT;
  const int32_t KB = a.KB, Cin = a.Cin;
  const int32_t NP = (int32_t)a.NP, Qo = a.Qo, PQ = a.Po * a.Qo;
  const int32_t e = __builtin_amdgcn_readfirstlane(a.ea->exp + a.eb->exp);
  const int32_t rstride = 2 * cl.row_b;  // one input row: hi and lo digit rows

  {
    const int64_t a_block_bytes = (int64_t)a.Mp * 64;
    const int32_t insts = (KB * 256) / 64;
    for (int32_t j = wave; j < insts; j += kWaves16) {
      const int32_t slot0 = j * 64;
      const int32_t sl = slot0 + lane;
      const int32_t kb = sl >> 8, sw = sl & 255;
      const int row = sw >> 2, piece = (sw & 3) ^ ((row >> 2) & 3);
      const uint8_t* src = a.wsa + kb * a_block_bytes + ((int64_t)(m0 + row) * 2 + (piece >> 1)) * 32 + (piece & 1) * 16;
      __builtin_amdgcn_global_load_lds((const void*)src, (lds_ptr_t)(sA + slot0 * 16), 16, 0, 0);
    }
  }
  if ((int32_t)threadIdx.x < 2 * KB) {
    const int32_t t0 = 16 * (int32_t)threadIdx.x;  // (block b, half h) = (i / 2, i % 2)
    const int32_t r0 = t0 / cl.SC, j0 = t0 - r0 * cl.SC, n0 = cl.SC - j0;
    int4 m;
    int* mp = reinterpret_cast<int*>(&m);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int32_t nb = min(max(n0 - 4 * k, 0), 4);
      mp[k] = nb >= 4 ? -1 : (int)((1u << (8 * nb)) - 1u);
    }
    s_tab[threadIdx.x][0] = make_int4(r0 * rstride + j0, (r0 + 1) * rstride - n0, 0, 0);
    s_tab[threadIdx.x][1] = m;
  }

  const int32_t units = 2 * ((NP + 31) / 32);
  const int32_t G = gridDim.x;
  const int32_t xcd = blockIdx.x & 7, per = G >> 3, rem = G & 7;
  const int32_t vb = xcd * per + min(xcd, rem) + (blockIdx.x >> 3);
  const int32_t u0 = (int32_t)((int64_t)units * vb / G), u1 = (int32_t)((int64_t)units * (vb + 1) / G);
  const int32_t my_units = (u1 - u0 > wave) ? (u1 - u0 - wave + kWaves16 - 1) / kWaves16 : 0;
  auto unit_of = [&](int32_t i) { return u0 + wave + kWaves16 * i; };
  // byte offset in XC of this lane's pixel of unit u at filter row 0, channel 0
  auto pixel_off = [&](int32_t u) -> int32_t {
    int32_t gp = (u >> 1) * 32 + col;
    if (gp >= NP) gp = 0;
    const int32_t im = (int32_t)fdiv((uint32_t)gp, a.div_pq), rp = gp - im * PQ;
    const int32_t po = (int32_t)fdiv((uint32_t)rp, a.div_q), qo = rp - po * Qo;
    return (im * a.Hp + po * a.ustride_h) * rstride + qo * a.ustride_w * Cin;
  };
  const __amdgpu_buffer_rsrc_t rs_x = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(a.xs), (short)0,
                                                                        (int)cl.xc_bytes, 0x00020000);
  struct Raw {
    v4i ha, hb, la, lb;
  };
  auto load_raw = [&](Raw& r, int32_t pix, int32_t kb) {
    const int4 o = s_tab[2 * kb + half][0];
    const uint32_t oa = (uint32_t)(pix + o.x), ob = (uint32_t)(pix + o.y);
    r.ha = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rs_x, oa, 0, 0));
    r.hb = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rs_x, ob, 0, 0));
    r.la = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rs_x, oa + cl.row_b, 0, 0));
    r.lb = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rs_x, ob + cl.row_b, 0, 0));
  };
  auto merge = [&](const v4i& x, const v4i& y, const int4& m) {
    return v4i{(x[0] & m.x) | (y[0] & ~m.x), (x[1] & m.y) | (y[1] & ~m.y), (x[2] & m.z) | (y[2] & ~m.z),
               (x[3] & m.w) | (y[3] & ~m.w)};
  };

  const bool full_rows = a.M == a.Mp;
  const bool out_buf = a.O < (1ll << 30);
  const __amdgpu_buffer_rsrc_t rs_out =
      __builtin_amdgcn_make_buffer_rsrc(a.out, (short)0, out_buf ? (int)(a.O * 4) : 0, 0x00020000);
  uint32_t amax = 0;
  wait_vmcnt<0>();
  __syncthreads();

  if (my_units > 0) {
    const uint32_t ra_hi = swz(col, 2 * half) * 16, ra_lo = swz(col, 2 * half + 1) * 16;
    int32_t cur_pix = pixel_off(unit_of(0));
    Raw nx;
    load_raw(nx, cur_pix, 0);
    for (int32_t unit = 0; unit < my_units; ++unit) {
      const int32_t u = unit_of(unit);
      const int32_t msub = u & 1;
      const int32_t g = (u >> 1) * 32 + col;
      const bool gvalid = g < NP;
      int32_t obase = 0;
      if (gvalid) {
        const int32_t im = (int32_t)fdiv((uint32_t)g, a.div_pq);
        obase = im * a.M * PQ + (g - im * PQ);
      }
      const int32_t mrow0 = m0 + 32 * msub + 4 * half;
      Acc3 acc;
      float sum[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) sum[v] = 0.f;
      const uint8_t* ab = sA + msub * 2048;
      for (int32_t kb = 0; kb < KB; ++kb) {
        const int4 m = s_tab[2 * kb + half][1];
        const v4i bh = merge(nx.ha, nx.hb, m), bl = merge(nx.la, nx.lb, m);
        // the next block of this unit, or the first block of the next unit
        if (kb + 1 < KB) {
          load_raw(nx, cur_pix, kb + 1);
        } else {
          if (unit + 1 < my_units) cur_pix = pixel_off(unit_of(unit + 1));
          load_raw(nx, cur_pix, 0);
        }
        const v4i ah = *reinterpret_cast<const v4i*>(ab + kb * kStageA + ra_hi);
        const v4i al = *reinterpret_cast<const v4i*>(ab + kb * kStageA + ra_lo);
        mfma_tile(acc, ah, al, bh, bl, (kb & 1) == 0);
        if ((kb & 1) == 1 || kb + 1 == KB)
          flush_tile<PARTIALS>(acc, sum, kb >> 1, a.partials, a.O, obase, PQ, mrow0, a.M, gvalid);
      }
      if (gvalid) {
        if (full_rows && out_buf) {
          const uint32_t lane_off = (uint32_t)(obase + mrow0 * PQ) * 4u;
          float fmx = 0.f;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const float y = ldexpf(sum[v], e);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(y), rs_out, lane_off,
                                                  (uint32_t)((8 * (v >> 2) + (v & 3)) * PQ) * 4u, 0);
            fmx = fmaxf(fmx, fabsf(y));
          }
          amax = max(amax, __float_as_uint(fmx));
        } else {
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int32_t m = mrow0 + 8 * (v >> 2) + (v & 3);
            if (m < a.M) amax = max(amax, store_out<false>(a.out, (uint32_t)(obase + m * PQ), sum[v], e));
          }
        }
      }
    }
  }

  if (a.so) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, off, 64));
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t b = red[0];
      for (int i = 1; i < kWaves16; ++i) b = max(b, red[i]);
      if (b > __atomic_load_n(&a.so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&a.so->amax_bits, b);
      if (b == 0x7f800000u) atomicOr(&a.so->flags, DFP_FLAG_OUTPUT_INF);
    }
  }
}

// Unit-stride 1x1 forward / backward-data from the INT16 activations through
// LDS, no operand preparation pass: D[m][pixel] = sum_c A[m][c] B[c][pixel],
// B = x (forward) or dy (backward-data) in NCHW (P*Q a multiple of 4), A = the
// filter digits [KB][Mp][2][32].  Workgroup: 64 output rows x 64 pixels, four
// waves of 32 x 32.  Per band of 64 reduction indices (two 32-channel blocks)
// the workgroup stages A (4 KiB per block, contiguous) and its 64 pixels of
// 64 channels of B: each thread loads four pixels of four channels (8-byte
// loads, 128 contiguous bytes per channel across 16 threads), splits the
// digits, transposes the 4 x 4 bytes in registers and writes, per pixel, the
// four channels' hi and lo digits as one dword each into the MFMA operand
// layout (per block and pixel: 16-byte pieces (channel half, digit),
// swizzled across banks as the filter tiles).  The loads of band b + 1 are in
// flight while band b is multiplied (two LDS buffers, one barrier per band).
// Channels past C and pixels past N*P*Q are zeros; chunks of L / 32 blocks.
constexpr int k1x1fThreads = 256;

template <bool PARTIALS>
__global__ __launch_bounds__(k1x1fThreads, 4) void k_conv1x1_s(ConvMfmaArgs a, const int16_t* __restrict__ src,
                                                             int32_t PQ, FastDiv div_pq) {
  __shared__ __align__(16) uint8_t sbuf[2][2][2 * 4096];  // [buffer][A, B][block][64 rows x 64 B]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5, lc = lane & 31;
  const int32_t m0 = blockIdx.y * 64, px0 = blockIdx.x * 64;
  const int32_t NP = (int32_t)a.NP, Cin = a.Cin, KB = a.KB;
  const int32_t e = __builtin_amdgcn_readfirstlane(a.ea->exp + a.eb->exp);
  // B staging: pixels px0 + 4 pg .. + 3 (one image) of channels 4 cg .. + 3 of the band
  const int32_t pg = (int32_t)threadIdx.x & 15, cg = (int32_t)threadIdx.x >> 4;
  const int32_t gpix = px0 + 4 * pg;
  const bool pin = gpix < NP;
  int32_t img = 0, pq = 0;
  if (pin) {
    img = (int32_t)fdiv((uint32_t)gpix, div_pq);
    pq = gpix - img * PQ;
  }
  const int16_t* sp = src + ((int64_t)img * Cin) * PQ + pq;
  const int64_t a_block_bytes = (int64_t)a.Mp * 64;
  uint2 rb[4];
  uint4 ra[2];
  auto load_band = [&](int32_t kb) {  // blocks kb, kb + 1
#pragma unroll
    for (int ch = 0; ch < 4; ++ch) {
      const int32_t c = kb * 32 + 4 * cg + ch;
      rb[ch] = make_uint2(0u, 0u);
      if (pin && c < Cin) rb[ch] = *reinterpret_cast<const uint2*>(sp + (int64_t)c * PQ);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      ra[j] = make_uint4(0u, 0u, 0u, 0u);
      if (kb + j < KB)
        ra[j] = *reinterpret_cast<const uint4*>(a.wsa + (kb + j) * a_block_bytes + (int64_t)m0 * 64 + threadIdx.x * 16);
    }
  };
  auto write_band = [&](int buf) {
    // A: piece i = thread of 256 per block, row i / 4, piece i % 4 (channel half, digit)
#pragma unroll
    for (int j = 0; j < 2; ++j)
      *reinterpret_cast<uint4*>(&sbuf[buf][0][j * 4096 + swz((int)threadIdx.x >> 2, (int)threadIdx.x & 3) * 16]) = ra[j];
    // B: split, transpose 4 channels x 4 pixels, one dword per (pixel, digit)
    uint32_t w[4][2], h[4][2];
#pragma unroll
    for (int ch = 0; ch < 4; ++ch) {
      w[ch][0] = rb[ch].x;
      w[ch][1] = rb[ch].y;
#pragma unroll
      for (int d = 0; d < 2; ++d)
        h[ch][d] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, w[ch][d]) + (u16x2){128, 128});
    }
    const int32_t blk = cg >> 3, khalf = (cg >> 2) & 1, sub = (cg & 3) * 4;
#pragma unroll
    for (int d = 0; d < 2; ++d) {  // pixels 2d, 2d + 1
      // lo digits: byte 0 (pixel 2d) and byte 2 (pixel 2d + 1) of each channel's dword
      const uint32_t l01 = __builtin_amdgcn_perm(w[1][d], w[0][d], 0x06020400u);
      const uint32_t l23 = __builtin_amdgcn_perm(w[3][d], w[2][d], 0x06020400u);
      const uint32_t h01 = __builtin_amdgcn_perm(h[1][d], h[0][d], 0x07030501u);
      const uint32_t h23 = __builtin_amdgcn_perm(h[3][d], h[2][d], 0x07030501u);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int row = 4 * pg + 2 * d + k;
        const uint32_t lo = __builtin_amdgcn_perm(l23, l01, k ? 0x07060302u : 0x05040100u);
        const uint32_t hi = __builtin_amdgcn_perm(h23, h01, k ? 0x07060302u : 0x05040100u);
        uint8_t* bb = &sbuf[buf][1][blk * 4096];
        *reinterpret_cast<uint32_t*>(bb + swz(row, 2 * khalf) * 16 + sub) = hi;
        *reinterpret_cast<uint32_t*>(bb + swz(row, 2 * khalf + 1) * 16 + sub) = lo;
      }
    }
  };

  Acc3 acc;
  float sum[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) sum[v] = 0.f;
  const int arow = (wave >> 1) * 32 + lc, brow = (wave & 1) * 32 + lc;
  const uint32_t oa_hi = swz(arow, 2 * half) * 16, oa_lo = swz(arow, 2 * half + 1) * 16;
  const uint32_t ob_hi = swz(brow, 2 * half) * 16, ob_lo = swz(brow, 2 * half + 1) * 16;
  const int32_t g = px0 + brow;
  const bool gvalid = g < NP;
  int32_t obase = 0;
  if (gvalid) {
    const int32_t im = (int32_t)fdiv((uint32_t)g, div_pq);
    obase = im * a.M * PQ + (g - im * PQ);
  }
  const int32_t mrow0 = m0 + (wave >> 1) * 32 + 4 * half;
  const int32_t chunk_blocks = a.L / 32;
  int32_t blk_in_chunk = 0, j = 0;
  load_band(0);
  int buf = 0;
  for (int32_t kb = 0; kb < KB; kb += 2, buf ^= 1) {
    write_band(buf);
    __syncthreads();
    if (kb + 2 < KB) load_band(kb + 2);
    const int32_t nblk = min(2, KB - kb);
    for (int32_t b = 0; b < nblk; ++b) {
      const uint8_t* pa = &sbuf[buf][0][b * 4096];
      const uint8_t* pb = &sbuf[buf][1][b * 4096];
      const v4i ah = *reinterpret_cast<const v4i*>(pa + oa_hi), al = *reinterpret_cast<const v4i*>(pa + oa_lo);
      const v4i bh = *reinterpret_cast<const v4i*>(pb + ob_hi), bl = *reinterpret_cast<const v4i*>(pb + ob_lo);
      mfma_tile(acc, ah, al, bh, bl, blk_in_chunk == 0);
      if (++blk_in_chunk == chunk_blocks || kb + b == KB - 1) {
        flush_tile<PARTIALS>(acc, sum, j++, a.partials, a.O, obase, PQ, mrow0, a.M, gvalid);
        blk_in_chunk = 0;
      }
    }
  }

  uint32_t amax = 0;
  if (gvalid) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int32_t m = mrow0 + 8 * (v >> 2) + (v & 3);
      if (m < a.M) amax = max(amax, store_out<false>(a.out, (int64_t)obase + (int64_t)m * PQ, sum[v], e));
    }
  }
  if (a.so) {
    __shared__ uint32_t red[k1x1fThreads / 64];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, off, 64));
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t b = max(max(red[0], red[1]), max(red[2], red[3]));
      if (b > __atomic_load_n(&a.so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&a.so->amax_bits, b);
      if (b == 0x7f800000u) atomicOr(&a.so->flags, DFP_FLAG_OUTPUT_INF);
    }
  }
}

// XC[n][hp][d][row_b] for k_conv_mfma_cl: byte wp C + c of digit row d (0 hi,
// 1 lo) holds that digit of x[n][c][hp - ph][wp - pw] (zero outside the
// image); thread (n, hp, group of four columns).  Bytes past Wp C stay unset
// (they only ever meet zero filter digits or a mask).
__global__ __launch_bounds__(256) void k_prep_cl(const int16_t* __restrict__ x, uint8_t* __restrict__ xc, int32_t N,
                                                int32_t C, int32_t H, int32_t W, int32_t Hp, int32_t Wp, int32_t ph,
                                                int32_t pw, int32_t row_b) {
  const int32_t W4 = (Wp + 3) / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)N * Hp * W4) return;
  const int32_t w4 = (int32_t)(i % W4);
  const int64_t r = i / W4;  // n * Hp + hp
  const int32_t hp = (int32_t)(r % Hp), n = (int32_t)(r / Hp);
  const int32_t h = hp - ph;
  uint8_t* hi = xc + r * 2 * row_b + 4 * w4 * C;
  uint8_t* lo = hi + row_b;
  for (int32_t k = 0; k < 4 * C; k += 4) {  // four bytes: (column, channel) = divmod(4 w4 C + k + b, C)
    uint32_t dh = 0u, dl = 0u;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int32_t idx = k + b, wq = 4 * w4 + idx / C, c = idx - (idx / C) * C;
      const int32_t w = wq - pw;
      int32_t v = 0;
      if (wq < Wp && h >= 0 && h < H && w >= 0 && w < W) v = x[(((int64_t)n * C + c) * H + h) * W + w];
      dh |= hi_digit(v) << (8 * b);
      dl |= lo_digit(v) << (8 * b);
    }
    *reinterpret_cast<uint32_t*>(hi + k) = dh;
    *reinterpret_cast<uint32_t*>(lo + k) = dl;
  }
}

inline int64_t align256(int64_t v) { return (v + 255) & ~(int64_t)255; }

}  // namespace

// The 16 x 16-tile kernel serves FP32 outputs at L = 64 without partials
// when the 32 x 32 tiles are fewer than the chip's wave slots (16 per CU), or
// the output has at most 16 rows (a 16-row subtile then wastes half as many
// rows as a 32-row half), and every phase (whole chunks, at most kS16MaxKB
// blocks, as equal as possible) has an even number of chunks.
static bool use_s16(int64_t NP, int32_t M, int32_t Mp, int32_t KB, bool partials, int cus) {
  if (partials || (M > 16 && 2 * ((NP + 31) / 32) * (Mp / kMT) >= (int64_t)cus * kWaves16)) return false;
  const int32_t chunks = KB / 2, nph = (KB + kS16MaxKB - 1) / kS16MaxKB;
  for (int32_t ph = 0; ph < nph; ++ph) {
    const int32_t n = chunks * (ph + 1) / nph - chunks * ph / nph;
    if (n < 2 || n % 2 != 0) return false;
  }
  return true;
}

static int device_cus() {
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess) hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  return cus;
}

bool conv_w16_eligible(int32_t Cin, int32_t T, int32_t L, bool i32) {
  // FP32 outputs at L = 64 take any number of blocks in phases of at most
  // kW16MaxKB; single-chunk INT32 outputs one phase
  return (Cin % 32) == 0 && (T % 64) == 0 && (i32 ? T / 32 <= kW16MaxKB : L == 64);
}

bool conv_mfma_supported(const Geom& g, int32_t dir) {
  const int32_t wsrc = dir == DFP_FWD ? g.w : g.q;
  return 16 * wsrc <= kPrepBElems;
}

// Workspace layout of the forward / backward-data MFMA path.
ConvMfmaPlan plan_conv_mfma(const Geom& g, int32_t dir) {
  ConvMfmaPlan p{};
  const bool fwd = dir == DFP_FWD;
  p.M = fwd ? g.k : g.c;
  p.Cin = fwd ? g.c : g.k;
  p.T = p.Cin * g.r * g.s;
  p.KB = (p.T + 31) / 32;
  p.Mp = (p.M + kMT - 1) / kMT * kMT;
  p.CG = (p.Cin + 15) / 16;
  if (fwd) {
    p.Hp = g.h + 2 * g.ph;
    p.Wp = g.w + 2 * g.pw;
    p.top = g.ph; p.left = g.pw; p.dil_h = 1; p.dil_w = 1;
    p.Po = g.p; p.Qo = g.q;
  } else {
    p.Hp = g.h + g.r - 1;
    p.Wp = g.w + g.s - 1;
    p.top = g.r - 1 - g.ph;
    p.left = g.s - 1 - g.pw;
    p.dil_h = g.sh;
    p.dil_w = g.sw;
    p.Po = g.h; p.Qo = g.w;
  }
  p.ws_a_bytes = align256((int64_t)p.KB * p.Mp * 2 * 32);
  p.ws_b_bytes = align256((int64_t)g.n * p.Hp * p.Wp * p.CG * 32);
  p.ws_t_bytes = align256((int64_t)p.KB * 8);
  p.bytes = p.ws_a_bytes + p.ws_b_bytes + p.ws_t_bytes;
  return p;
}

dfp_status launch_conv_mfma(int32_t dir, const Geom& g, const int16_t* a, const dfp_scale* sa, const int16_t* b,
                            const dfp_scale* sb, float* out, dfp_scale* so, int32_t* partials, void* ws,
                            hipStream_t st, bool i32, bool prefer_w16, bool so_reset) {
  // fwd: a = x (B source), b = w.  bwd-data: a = dy (B source), b = w.
  const ConvMfmaPlan p = plan_conv_mfma(g, dir);
  const bool fwd = dir == DFP_FWD;
  uint8_t* wsa = reinterpret_cast<uint8_t*>(ws);
  uint8_t* xs = wsa + p.ws_a_bytes;
  int2* boff = reinterpret_cast<int2*>(xs + p.ws_b_bytes);
  const int32_t rsign = fwd ? 1 : -1;
  const int32_t tap_row_bytes = rsign * p.Wp * p.CG * 32, tap_col_bytes = rsign * p.CG * 32;
  bool plane = conv_w16_eligible(p.Cin, p.T, g.L, i32) && (int64_t)g.n * p.Po * p.Qo * p.M < (1ll << 31) &&
               p.ws_b_bytes < (1ll << 31);
  if (plane && p.KB > kW16MaxKB && !prefer_w16) {
    // phases pay the kernel's fixed cost once each: taken only when there are
    // at least as many 16 x 16 (32 x 32) output tiles per workgroup as it has
    // waves, in each phase
    const int cus = device_cus();
    const int64_t NP = (int64_t)g.n * p.Po * p.Qo;
    if (use_s16(NP, p.M, p.Mp, p.KB, partials != nullptr, cus)) {
      const int64_t gx = std::max<int64_t>(1, cus / ((p.M + kS16Rows - 1) / kS16Rows));
      plane = 2 * ((NP + 15) / 16) >= gx * kWaves16 || p.KB <= kS16MaxKB;
    } else {
      const int64_t gx = std::max<int64_t>(1, cus / (p.Mp / kMT));
      plane = 2 * ((NP + 31) / 32) >= gx * kWaves16;
    }
  }
  // the filter preparation clears so (unless a previous launch of the same
  // output has already raised it) before the main kernel raises it
  const PrepAArgs pa{b, wsa, p.M, p.Mp, p.Cin, g.r, g.s, p.T, p.KB, fwd ? 0 : 1, g.c, so_reset ? so : nullptr, boff,
                     tap_row_bytes, tap_col_bytes};
  // unit-stride 1x1 without padding (forward, or backward-data as the 1x1 of dy
  // with the transposed filter): the activations are read in NCHW through LDS.
  // Taken for many pixels and short reductions (at most 256 channels), where
  // the plane preparation of a large tensor costs more than the filter
  // restaging per workgroup (measured on ResNet-50: 56 x 56 layers 2-11%
  // faster steps, 28 x 28 with 128 channels about even, 14 x 14 slower)
  const int32_t PQ1 = p.Po * p.Qo;
  if (!i32 && g.r == 1 && g.s == 1 && g.sh == 1 && g.sw == 1 && g.ph == 0 && g.pw == 0 && (g.L % 32) == 0 &&
      PQ1 % 4 == 0 && (reinterpret_cast<uintptr_t>(a) & 7) == 0 && p.KB <= 8 && (int64_t)g.n * PQ1 >= 32768 &&
      (int64_t)g.n * std::max(p.Cin, p.M) * PQ1 < (1ll << 31)) {
    const int64_t a_items = (int64_t)p.KB * p.Mp * 8;
    DFP_LAUNCH(K_WPREP, k_prep_a, dim3((unsigned)((a_items + 255) / 256)), dim3(256), 0, st, pa);
    ConvMfmaArgs args{};
    args.wsa = wsa;
    args.ea = sa;
    args.eb = sb;
    args.out = out;
    args.so = so;
    args.partials = partials;
    args.M = p.M; args.Mp = p.Mp; args.Cin = p.Cin; args.T = p.T; args.KB = p.KB; args.L = g.L;
    args.NP = (int64_t)g.n * PQ1;
    args.O = args.NP * p.M;
    const dim3 grid((unsigned)((args.NP + 63) / 64), (unsigned)(p.Mp / 64));
    const FastDiv dpq = make_fastdiv((uint32_t)PQ1);
    const int kid = fwd ? K_FWD_MFMA : K_BWDD_MFMA;
    if (partials) DFP_LAUNCH(kid, (k_conv1x1_s<true>), grid, dim3(k1x1fThreads), 0, st, args, a, PQ1, dpq);
    else DFP_LAUNCH(kid, (k_conv1x1_s<false>), grid, dim3(k1x1fThreads), 0, st, args, a, PQ1, dpq);
    return DFP_OK;
  }
  const int64_t a_total = (int64_t)p.KB * p.Mp * 8;
  // the plane-layout preparation takes the filter digits in an extra slice of
  // its grid when that slice needs at most 8 items per thread
  const int32_t rb_plane = std::max(1, std::min(kPlaneRows, kPlaneElems / (16 * (fwd ? g.w : g.q))));
  const int64_t slice_threads =
      kPlaneDirect ? (int64_t)p.Hp * 256 : (int64_t)((p.Hp + rb_plane - 1) / rb_plane) * p.CG * 256;
  const bool merge_a = plane && a_total <= 8 * slice_threads;
  if (!merge_a) DFP_LAUNCH(K_WPREP, k_prep_a, dim3((unsigned)((a_total + 255) / 256)), dim3(256), 0, st, pa);
  // few input channels (forward, L = 64, FP32 outputs): channel-last digit rows
  const int32_t cl_row_b = (p.Wp * p.Cin + 31) / 16 * 16;
  const int64_t cl_bytes = ((int64_t)g.n * p.Hp + 2) * 2 * cl_row_b;
  if (fwd && !i32 && g.L == 64 && p.Cin < 16 && g.s * p.Cin >= 16 && p.KB <= kW16MaxKB &&
      cl_bytes <= p.ws_b_bytes && cl_bytes < (1ll << 31) && (int64_t)g.n * p.Po * p.Qo * p.M < (1ll << 30)) {
    const int64_t items = (int64_t)g.n * p.Hp * ((p.Wp + 3) / 4);
    DFP_LAUNCH(K_XPREP, k_prep_cl, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, st, a, xs, g.n, p.Cin, g.h,
               g.w, p.Hp, p.Wp, g.ph, g.pw, cl_row_b);
    ConvMfmaArgs args{};
    args.xs = xs;
    args.wsa = wsa;
    args.ea = sa;
    args.eb = sb;
    args.out = out;
    args.so = so;
    args.partials = partials;
    args.M = p.M; args.Mp = p.Mp; args.Cin = p.Cin; args.S = g.s; args.T = p.T; args.KB = p.KB; args.L = g.L;
    args.Hp = p.Hp; args.Wp = p.Wp; args.Po = p.Po; args.Qo = p.Qo;
    args.NP = (int64_t)g.n * p.Po * p.Qo;
    args.O = args.NP * p.M;
    args.ustride_h = g.sh;
    args.ustride_w = g.sw;
    args.div_pq = make_fastdiv((uint32_t)(p.Po * p.Qo));
    args.div_q = make_fastdiv((uint32_t)p.Qo);
    const ClArgs cla{cl_row_b, g.s * p.Cin, (uint32_t)cl_bytes};
    const int cus = device_cus();
    const int64_t units = 2 * ((args.NP + 31) / 32), mtiles = p.Mp / kMT;
    int64_t gx = std::max<int64_t>(1, cus / mtiles);
    gx = std::min<int64_t>(gx, (units + kWaves16 - 1) / kWaves16);
    const dim3 grid((unsigned)gx, (unsigned)mtiles);
    if (partials) DFP_LAUNCH(K_FWD_MFMA, (k_conv_mfma_cl<true>), grid, dim3(kThreads16), 0, st, args, cla);
    else DFP_LAUNCH(K_FWD_MFMA, (k_conv_mfma_cl<false>), grid, dim3(kThreads16), 0, st, args, cla);
    return DFP_OK;
  }
  {
    const int32_t Cs = fwd ? g.c : g.k, Hs = fwd ? g.h : g.p, Wsrc = fwd ? g.w : g.q;
    const bool vec = (Wsrc % 8) == 0 && (reinterpret_cast<uintptr_t>(a) & 15) == 0;
    const int32_t cgc = std::max(1, std::min(p.CG, kPrepBElems / (16 * Wsrc)));  // as in the kernel
    const size_t lds = (size_t)cgc * 16 * Wsrc * 2;
    if (plane) {
      const int32_t rb = rb_plane;
      const dim3 grid((unsigned)((p.Hp + rb - 1) / rb), (unsigned)p.CG, (unsigned)(g.n + (merge_a ? 1 : 0)));
      const size_t plds = (size_t)rb * Wsrc * 16 * 2;
      const int32_t wa = merge_a ? 1 : 0;
      const dim3 gridd((unsigned)p.Hp, (unsigned)(g.n + (merge_a ? 1 : 0)));
      if (kPlaneDirect && p.dil_h == 1 && p.dil_w == 1 && (Wsrc % 2) == 0 &&
          (reinterpret_cast<uintptr_t>(a) & 3) == 0 && p.left >= 0 && p.left + Wsrc <= p.Wp) {
        DFP_LAUNCH(K_XPREP, k_prep_plane_pair, gridd, dim3(256), 0, st, a, xs, Cs, Hs, Wsrc, p.Hp, p.Wp, p.CG,
                   p.top, p.left, pa, wa);
      } else if (kPlaneDirect) {
        DFP_LAUNCH(K_XPREP, k_prep_plane_direct, gridd, dim3(256), 0, st, a, xs, Cs, Hs, Wsrc, p.Hp, p.Wp, p.CG,
                   p.top, p.left, p.dil_h, p.dil_w, pa, wa);
      } else if (vec)
        DFP_LAUNCH(K_XPREP, k_prep_plane<true>, grid, dim3(256), plds, st, a, xs, Cs, Hs, Wsrc, p.Hp, p.Wp, p.CG,
                   p.top, p.left, p.dil_h, p.dil_w, rb, pa, wa);
      else
        DFP_LAUNCH(K_XPREP, k_prep_plane<false>, grid, dim3(256), plds, st, a, xs, Cs, Hs, Wsrc, p.Hp, p.Wp, p.CG,
                   p.top, p.left, p.dil_h, p.dil_w, rb, pa, wa);
    } else if (vec) {
      DFP_LAUNCH(K_XPREP, k_prep_b<true>, dim3((unsigned)(g.n * p.Hp)), dim3(256), lds, st, a, xs, g.n, Cs, Hs, Wsrc,
                 p.Hp, p.Wp, p.CG, p.top, p.left, p.dil_h, p.dil_w);
    } else {
      DFP_LAUNCH(K_XPREP, k_prep_b<false>, dim3((unsigned)(g.n * p.Hp)), dim3(256), lds, st, a, xs, g.n, Cs, Hs, Wsrc,
                 p.Hp, p.Wp, p.CG, p.top, p.left, p.dil_h, p.dil_w);
    }
  }
  ConvMfmaArgs args{};
  args.xs = xs;
  args.wsa = wsa;
  args.boff = boff;
  args.ea = sa;
  args.eb = sb;
  args.out = out;
  args.so = so;
  args.partials = partials;
  args.M = p.M; args.Mp = p.Mp; args.Cin = p.Cin; args.S = g.s; args.T = p.T; args.KB = p.KB; args.L = g.L;
  args.CG = p.CG; args.Hp = p.Hp; args.Wp = p.Wp; args.Po = p.Po; args.Qo = p.Qo;
  args.NP = (int64_t)g.n * p.Po * p.Qo;
  args.O = args.NP * p.M;
  args.plane = plane ? 1 : 0;
  if (fwd) {
    args.ustride_h = g.sh;
    args.ustride_w = g.sw;
    args.rsign = 1;
    args.roff_h = 0;
    args.roff_w = 0;
  } else {
    args.ustride_h = 1;
    args.ustride_w = 1;
    args.rsign = -1;
    args.roff_h = g.r - 1;
    args.roff_w = g.s - 1;
  }
  return launch_mfma_main(args, p.ws_b_bytes, fwd ? K_FWD_MFMA : K_BWDD_MFMA, fwd ? K_FWD_I32 : K_BWDD_I32, i32, st);
}

dfp_status launch_mfma_main(ConvMfmaArgs& args, int64_t ws_b_bytes, int kid, int kid32, bool i32, hipStream_t st) {
  const dim3 grid((unsigned)((args.NP + kNT - 1) / kNT), (unsigned)(args.Mp / kMT));
  const bool masked = (args.L % 32) != 0;
  const bool chan16 = (args.Cin % 16) == 0;
  const bool partials = args.partials != nullptr;
  // persistent grid: one workgroup per CU for each 64-row tile of the output channels
  auto persist_grid = [&]() {
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess) hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int64_t wave_tiles = (args.NP + 31) / 32;
    const int64_t mtiles = args.Mp / kMT;
    int64_t gx = std::max<int64_t>(1, cus / mtiles);
    gx = std::min<int64_t>(gx, (wave_tiles + kWaves3 - 1) / kWaves3);
    return dim3((unsigned)gx, (unsigned)mtiles);
  };
  const bool small_index = args.O < (1ll << 31) && ws_b_bytes < (1ll << 31);
  if (args.exa) {
    // Blocked-DFP: the shared-ring kernel with per-chunk block scales
    if (i32 || masked || !chan16 || !small_index || args.nb > kBlockedMaxBlocks || args.bk % args.L != 0)
      return DFP_ERR_PARAM;
    const size_t lds = (size_t)args.nb * (kMT + kNT);
    if (partials) DFP_LAUNCH(kid, (k_conv_mfma_q<true, false, true>), grid, dim3(kThreadsQ), lds, st, args);
    else DFP_LAUNCH(kid, (k_conv_mfma_q<false, false, true>), grid, dim3(kThreadsQ), lds, st, args);
    return DFP_OK;
  }
  const bool persist_ok = chan16 && (args.T % 64) == 0 && args.KB >= 4 && args.KB <= kARes3Max && small_index;
  // four waves per SIMD: 32-channel blocks (each block inside one filter tap), full chunks of two blocks
  const bool w16_ok = args.plane != 0 && small_index;
  args.div_pq = make_fastdiv((uint32_t)(args.Po * args.Qo));
  args.div_q = make_fastdiv((uint32_t)args.Qo);
  auto w16_grid = [&]() {
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess) hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int64_t units = 2 * ((args.NP + 31) / 32);
    const int64_t mtiles = args.Mp / kMT;
    int64_t gx = std::max<int64_t>(1, cus / mtiles);
    gx = std::min<int64_t>(gx, (units + kWaves16 - 1) / kWaves16);
    return dim3((unsigned)gx, (unsigned)mtiles);
  };
  args.kb0 = 0;
  args.kbn = args.KB;
  args.phase_flags = 3;
  if (i32) {
    // DFP-32 output: one chunk over the whole reduction (the caller checked L >= T)
    args.L = args.KB * 32;
    if (w16_ok)
      DFP_LAUNCH(kid32, (k_conv_mfma_w16<false, true>), w16_grid(), dim3(kThreads16), 0, st, args);
    else if (persist_ok && !DFP_ASM_UNSAFE_PERSIST_I32 &&
             no_scratch(reinterpret_cast<const void*>(&k_conv_mfma_persist<false, true>)))
      DFP_LAUNCH(kid32, (k_conv_mfma_persist<false, true>), persist_grid(), dim3(kThreads3), 0, st, args);
    else if (chan16 && small_index)
      DFP_LAUNCH(kid32, (k_conv_mfma_q<false, true>), grid, dim3(kThreadsQ), 0, st, args);
    else if (chan16)
      DFP_LAUNCH(kid32, (k_conv_mfma<false, false, true, true>), grid, dim3(kThreads), 0, st, args);
    else
      DFP_LAUNCH(kid32, (k_conv_mfma<false, false, false, true>), grid, dim3(kThreads), 0, st, args);
    return DFP_OK;
  }
#define DFP_CONV_MFMA_CASE(MK, PT, CH)                                                      \
  if (masked == MK && partials == PT && chan16 == CH) {                                    \
    DFP_LAUNCH(kid, (k_conv_mfma<MK, PT, CH>), grid, dim3(kThreads), 0, st, args);          \
    return DFP_OK;                                                                          \
  }
  if (w16_ok && args.L == 64) {
    // phases of whole chunks, at most kW16MaxKB blocks each, as equal as possible;
    // each launch continues the chunk sums the previous one left in the output
    const int32_t chunks = args.KB / 2;
    const int32_t nph = (args.KB + kW16MaxKB - 1) / kW16MaxKB;
    const int cus = device_cus();
    const int64_t mtiles = args.Mp / kMT;
    if (use_s16(args.NP, args.M, args.Mp, args.KB, partials, cus)) {
      // 32-row filter slices up to the last output row
      // (one workgroup per CU, even where some waves get no 16-pixel tile, but
      // at least 8 tiles per workgroup: every workgroup copies its filter slice)
      const int64_t stiles = (args.M + kS16Rows - 1) / kS16Rows;
      const int32_t nph16 = (args.KB + kS16MaxKB - 1) / kS16MaxKB;
      const int64_t gx = std::max<int64_t>(1, std::min<int64_t>(cus / stiles, (args.NP + 16 * 8 - 1) / (16 * 8)));
      const dim3 grid_s((unsigned)gx, (unsigned)stiles);
      for (int32_t ph = 0; ph < nph16; ++ph) {
        const int32_t c0 = chunks * ph / nph16, c1 = chunks * (ph + 1) / nph16;
        args.kb0 = 2 * c0;
        args.kbn = 2 * (c1 - c0);
        args.phase_flags = (ph == 0 ? 1 : 0) | (ph == nph16 - 1 ? 2 : 0);
        if (nph16 == 1) DFP_LAUNCH(kid, (k_conv_mfma_s16<false>), grid_s, dim3(kThreads16), 0, st, args);
        else DFP_LAUNCH(kid, (k_conv_mfma_s16<true>), grid_s, dim3(kThreads16), 0, st, args);
      }
      return DFP_OK;
    }
    const dim3 grid16 = w16_grid();
    for (int32_t ph = 0; ph < nph; ++ph) {
      const int32_t c0 = chunks * ph / nph, c1 = chunks * (ph + 1) / nph;
      args.kb0 = 2 * c0;
      args.kbn = 2 * (c1 - c0);
      args.phase_flags = (ph == 0 ? 1 : 0) | (ph == nph - 1 ? 2 : 0);
      if (nph == 1 && partials) DFP_LAUNCH(kid, (k_conv_mfma_w16<true>), grid16, dim3(kThreads16), 0, st, args);
      else if (nph == 1) DFP_LAUNCH(kid, (k_conv_mfma_w16<false>), grid16, dim3(kThreads16), 0, st, args);
      else if (partials)
        DFP_LAUNCH(kid, (k_conv_mfma_w16<true, false, true>), grid16, dim3(kThreads16), 0, st, args);
      else DFP_LAUNCH(kid, (k_conv_mfma_w16<false, false, true>), grid16, dim3(kThreads16), 0, st, args);
    }
    return DFP_OK;
  }
  // the persistent and skewed kernels wait for their inline-assembly LDS reads
  // in a later statement: a build of them with scratch is not used (see
  // no_scratch); the shared-ring and LDS kernels wait inside the same asm
  // (the build's assembly check can also take them out of use, DFP_ASM_UNSAFE_*)
  static const bool persist_safe[2] = {
      !DFP_ASM_UNSAFE_PERSIST && no_scratch(reinterpret_cast<const void*>(&k_conv_mfma_persist<false>)),
      !DFP_ASM_UNSAFE_PERSIST_PARTIALS && no_scratch(reinterpret_cast<const void*>(&k_conv_mfma_persist<true>))};
  static const bool skew_safe[2] = {
      !DFP_ASM_UNSAFE_SKEW && no_scratch(reinterpret_cast<const void*>(&k_conv_mfma_skew<false>)),
      !DFP_ASM_UNSAFE_SKEW_PARTIALS && no_scratch(reinterpret_cast<const void*>(&k_conv_mfma_skew<true>))};
  if (persist_ok && args.L == 64 && persist_safe[partials ? 1 : 0]) {
    const dim3 grid3 = persist_grid();
    if (partials) DFP_LAUNCH(kid, (k_conv_mfma_persist<true>), grid3, dim3(kThreads3), 0, st, args);
    else DFP_LAUNCH(kid, (k_conv_mfma_persist<false>), grid3, dim3(kThreads3), 0, st, args);
    return DFP_OK;
  }
  if (chan16 && !masked && small_index) {
    if (partials) DFP_LAUNCH(kid, (k_conv_mfma_q<true>), grid, dim3(kThreadsQ), 0, st, args);
    else DFP_LAUNCH(kid, (k_conv_mfma_q<false>), grid, dim3(kThreadsQ), 0, st, args);
    return DFP_OK;
  }
  if (chan16 && args.L == 64 && (args.T % 64) == 0 && args.KB >= 4 && skew_safe[partials ? 1 : 0]) {
    if (partials) DFP_LAUNCH(kid, (k_conv_mfma_skew<true>), grid, dim3(kThreads), 0, st, args);
    else DFP_LAUNCH(kid, (k_conv_mfma_skew<false>), grid, dim3(kThreads), 0, st, args);
    return DFP_OK;
  }
  if (chan16) {
    if (!masked && !partials) DFP_LAUNCH(kid, (k_conv_mfma_lds<false, false>), grid, dim3(kThreads), 0, st, args);
    else if (!masked) DFP_LAUNCH(kid, (k_conv_mfma_lds<false, true>), grid, dim3(kThreads), 0, st, args);
    else if (!partials) DFP_LAUNCH(kid, (k_conv_mfma_lds<true, false>), grid, dim3(kThreads), 0, st, args);
    else DFP_LAUNCH(kid, (k_conv_mfma_lds<true, true>), grid, dim3(kThreads), 0, st, args);
    return DFP_OK;
  }
  DFP_CONV_MFMA_CASE(false, false, false)
  DFP_CONV_MFMA_CASE(false, true, false)
  DFP_CONV_MFMA_CASE(true, false, false)
  DFP_CONV_MFMA_CASE(true, true, false)
#undef DFP_CONV_MFMA_CASE
  return DFP_ERR_PARAM;
}

// Backward-data of a 1x1 convolution without padding and with stride
// (sh, sw): dx[n][c][h][w] has the single term set k = 0 .. K-1 of
// dy[n][k][h/sh][w/sw] w[k][c] where sh divides h and sw divides w, and no term
// elsewhere (0).  The sampled pixels are the unit-stride backward-data over
// the P x Q grid, with the same reduction index k and hence the same chunks,
// so that runs into the end of the workspace and k_scatter_strided spreads it
// over dx; the zeros leave the epilogue's max unchanged.  (The general route
// runs the reduction over a zero-dilated dy, three quarters of it zeros at
// stride 2.)
namespace {
// Thread (x, y): in-plane position hw of every dx plane (n, c) = y, y +
// gridDim.y, ...; the position's row / column split is done once.
__global__ __launch_bounds__(256) void k_scatter_strided(const float* __restrict__ sub, float* __restrict__ dx,
                                                         int64_t planes, int32_t H, int32_t W, int32_t P, int32_t Q,
                                                         int32_t sh, int32_t sw) {
  const int32_t hw = blockIdx.x * 256 + threadIdx.x;
  if (hw >= H * W) return;
  const int32_t h = hw / W, w = hw - h * W, p = h / sh, q = w / sw;
  const bool hit = h == p * sh && w == q * sw && p < P && q < Q;
  const int32_t pq = hit ? p * Q + q : 0;
  for (int64_t nc = blockIdx.y; nc < planes; nc += gridDim.y)
    dx[nc * H * W + hw] = hit ? sub[nc * P * Q + pq] : 0.f;
}
Geom unit_grid(const Geom& g) {
  Geom u = g;
  u.h = g.p;
  u.w = g.q;
  u.sh = u.sw = 1;
  return u;
}
}  // namespace

int64_t conv_bwd_data_sub_bytes(const Geom& g) {
  if (g.r != 1 || g.s != 1 || g.ph != 0 || g.pw != 0 || (g.sh == 1 && g.sw == 1)) return 0;
  // k_scatter_strided indexes a plane (and sizes its grid) with 32 bits
  if ((int64_t)g.h * g.w >= (1ll << 31) - 256) return 0;
  const Geom u = unit_grid(g);
  if (!conv_mfma_supported(u, DFP_BWD_DATA)) return 0;
  return plan_conv_mfma(u, DFP_BWD_DATA).bytes + align256((int64_t)g.n * g.c * g.p * g.q * 4);
}

dfp_status launch_conv_bwd_data_sub(const Geom& g, const int16_t* dy, const dfp_scale* sdy, const int16_t* w,
                                    const dfp_scale* sw, float* dx, dfp_scale* so, void* ws, hipStream_t st,
                                    bool prefer_w16) {
  const Geom u = unit_grid(g);
  float* sub = reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(ws) + plan_conv_mfma(u, DFP_BWD_DATA).bytes);
  dfp_status rc = launch_conv_mfma(DFP_BWD_DATA, u, dy, sdy, w, sw, sub, so, nullptr, ws, st, false, prefer_w16);
  if (rc != DFP_OK) return rc;
  const int64_t planes = (int64_t)g.n * g.c;
  const int32_t gx = (g.h * g.w + 255) / 256;
  const int64_t gy = std::max<int64_t>(1, std::min<int64_t>(planes, std::max(1, 16384 / gx)));
  DFP_LAUNCH(K_XPREP, k_scatter_strided, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0, st, sub, dx, planes, g.h,
             g.w, g.p, g.q, g.sh, g.sw);
  return DFP_OK;
}


namespace {

// Strided backward-data split by output phase.  A pixel (h, w) of dx with
// h = alpha + sh*i and w = beta + sw*j receives only the filter taps
// r = r0 + sh*m, s = s0 + sw*m' with r0 = (alpha + ph) mod sh (s0 likewise),
// from dy[n][k][i + a0 - m][j + b0 - m'] with a0 = (alpha + ph - r0) / sh
// (b0 likewise): a unit-stride backward-data over the undilated dy with the
// sub-filter of those taps (in their canonical order) and padding (a0, b0),
// whose output is the phase's Ha x Wb grid of pixels.  When K is a multiple
// of L every chunk of the reduction t = (r*S + s)*K + k lies inside one tap,
// so the chunks of the other taps, whose products all vanish at these pixels,
// have partial 0, and leaving them out of the FP32 sum (+0.0 added to a sum
// that is never -0.0) changes nothing: each phase is bit-identical to the
// strided sum.  The phases run one after another into the end of the
// workspace, and each is spread over its pixels of dx.
struct Phase {
  Geom g;  // the unit-stride sub-problem (g.h, g.w: the phase grid; g.p, g.q: dy)
  int32_t alpha, beta, r0, s0;
  bool empty;  // no tap reaches these pixels (or no pixel has this phase): zeros
};
Phase phase_of(const Geom& g, int32_t idx) {
  Phase f{};
  f.alpha = idx / g.sw;
  f.beta = idx - f.alpha * g.sw;
  f.r0 = (f.alpha + g.ph) % g.sh;
  f.s0 = (f.beta + g.pw) % g.sw;
  const int32_t Mr = f.r0 < g.r ? (g.r - f.r0 + g.sh - 1) / g.sh : 0;
  const int32_t Ms = f.s0 < g.s ? (g.s - f.s0 + g.sw - 1) / g.sw : 0;
  const int32_t Ha = f.alpha < g.h ? (g.h - f.alpha + g.sh - 1) / g.sh : 0;
  const int32_t Wb = f.beta < g.w ? (g.w - f.beta + g.sw - 1) / g.sw : 0;
  f.g = g;
  f.g.h = Ha;
  f.g.w = Wb;
  f.g.r = Mr;
  f.g.s = Ms;
  f.g.sh = f.g.sw = 1;
  f.g.ph = (f.alpha + g.ph - f.r0) / g.sh;
  f.g.pw = (f.beta + g.pw - f.s0) / g.sw;
  f.empty = Mr == 0 || Ms == 0 || Ha == 0 || Wb == 0;
  return f;
}

// wsub[kc][m][m'] = w[kc][r0 + sh*m][s0 + sw*m'] (kc = k*C + c)
__global__ __launch_bounds__(256) void k_gather_taps(const int16_t* __restrict__ w, int16_t* __restrict__ wsub,
                                                    int64_t KC, int32_t R, int32_t S, int32_t r0, int32_t sh,
                                                    int32_t Mr, int32_t s0, int32_t sw, int32_t Ms) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= KC * Mr * Ms) return;
  const int64_t kc = i / (Mr * Ms);
  const int32_t t = (int32_t)(i - kc * (Mr * Ms)), m = t / Ms, mm = t - m * Ms;
  wsub[i] = w[(kc * R + r0 + sh * m) * S + s0 + sw * mm];
}

// dx[nc][alpha + sh*i][beta + sw*j] = sub[nc][i][j] (0 where sub is null)
__global__ __launch_bounds__(256) void k_scatter_phase(const float* __restrict__ sub, float* __restrict__ dx,
                                                      int64_t planes, int32_t H, int32_t W, int32_t Ha, int32_t Wb,
                                                      int32_t alpha, int32_t beta, int32_t sh, int32_t sw) {
  const int32_t ij = blockIdx.x * 256 + threadIdx.x;
  if (ij >= Ha * Wb) return;
  const int32_t i = ij / Wb, j = ij - i * Wb;
  const int64_t o = (int64_t)(alpha + sh * i) * W + beta + sw * j;
  for (int64_t nc = blockIdx.y; nc < planes; nc += gridDim.y)
    dx[nc * H * W + o] = sub ? sub[nc * Ha * Wb + ij] : 0.f;
}

}  // namespace

int64_t conv_bwd_data_phase_bytes(const Geom& g) {
  if ((g.sh == 1 && g.sw == 1) || g.L < 1 || g.k % g.L != 0 || conv_bwd_data_sub_bytes(g) > 0) return 0;
  // k_scatter_phase indexes a plane (and sizes its grid) with 32 bits
  if ((int64_t)g.h * g.w >= (1ll << 31) - 256) return 0;
  int64_t conv = 0, wsub = 0, out = 0;
  for (int32_t idx = 0; idx < g.sh * g.sw; ++idx) {
    const Phase f = phase_of(g, idx);
    if (f.empty) continue;
    // every phase on the plane-layout kernels, whose preparation takes any
    // padding; a 1x1 phase without padding must cover dy exactly (the 1x1
    // route reads its input with the output's pixel count)
    if (!conv_mfma_supported(f.g, DFP_BWD_DATA) ||
        !conv_w16_eligible(g.k, g.k * f.g.r * f.g.s, g.L, false) ||
        (f.g.r == 1 && f.g.s == 1 && f.g.ph == 0 && f.g.pw == 0 && (f.g.h != g.p || f.g.w != g.q)))
      return 0;
    conv = std::max(conv, plan_conv_mfma(f.g, DFP_BWD_DATA).bytes);
    wsub = std::max(wsub, align256((int64_t)g.k * g.c * f.g.r * f.g.s * 2));
    out = std::max(out, align256((int64_t)g.n * g.c * f.g.h * f.g.w * 4));
  }
  return conv > 0 ? conv + wsub + out : 0;
}

dfp_status launch_conv_bwd_data_phases(const Geom& g, const int16_t* dy, const dfp_scale* sdy, const int16_t* w,
                                       const dfp_scale* sw, float* dx, dfp_scale* so, void* ws, hipStream_t st,
                                       bool prefer_w16) {
  int64_t conv = 0, wsub_b = 0;
  for (int32_t idx = 0; idx < g.sh * g.sw; ++idx) {
    const Phase f = phase_of(g, idx);
    if (f.empty) continue;
    conv = std::max(conv, plan_conv_mfma(f.g, DFP_BWD_DATA).bytes);
    wsub_b = std::max(wsub_b, align256((int64_t)g.k * g.c * f.g.r * f.g.s * 2));
  }
  int16_t* wsub = reinterpret_cast<int16_t*>(reinterpret_cast<uint8_t*>(ws) + conv);
  float* sub = reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(ws) + conv + wsub_b);
  const int64_t planes = (int64_t)g.n * g.c;
  bool first = true;
  for (int32_t idx = 0; idx < g.sh * g.sw; ++idx) {
    const Phase f = phase_of(g, idx);
    const int32_t Ha = f.alpha < g.h ? (g.h - f.alpha + g.sh - 1) / g.sh : 0;
    const int32_t Wb = f.beta < g.w ? (g.w - f.beta + g.sw - 1) / g.sw : 0;
    if (Ha == 0 || Wb == 0) continue;
    if (!f.empty) {
      const int64_t n_sub = (int64_t)g.k * g.c * f.g.r * f.g.s;
      DFP_LAUNCH(K_WPREP, k_gather_taps, dim3((unsigned)((n_sub + 255) / 256)), dim3(256), 0, st, w, wsub,
                 (int64_t)g.k * g.c, g.r, g.s, f.r0, g.sh, f.g.r, f.s0, g.sw, f.g.s);
      const dfp_status rc = launch_conv_mfma(DFP_BWD_DATA, f.g, dy, sdy, wsub, sw, sub, so, nullptr, ws, st, false,
                                             prefer_w16, first);
      if (rc != DFP_OK) return rc;
      first = false;
    }
    const int32_t gx = (Ha * Wb + 255) / 256;
    const int64_t gy = std::max<int64_t>(1, std::min<int64_t>(planes, std::max(1, 16384 / gx)));
    DFP_LAUNCH(K_XPREP, k_scatter_phase, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0, st,
               f.empty ? nullptr : sub, dx, planes, g.h, g.w, Ha, Wb, f.alpha, f.beta, g.sh, g.sw);
  }
  if (first && so) return launch_scale_reset(so, st);  // no tap reached any pixel: dx is zero
  return DFP_OK;
}

}  // namespace dfp
