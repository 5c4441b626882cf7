// DFP16 GEMM (the paper's INT16 kernels serve "convolutions and GEMM",
// Sec. 4): D[i][j] = sum over t of opA[i][t] * opB[t][j], with the forward
// convolution's numeric contract (Algorithm 2, Sec. 4.3): INT32 partials over
// chunks of L consecutive t (mod 2^32), each converted to FP32 and added in
// chunk order, one scale 2^(Ea+Eb) at the end.
//
// A GEMM is the 1x1 forward convolution whose pixels are the columns of D:
// the matrix-core path prepares opA as the filter digit planes and opB as the
// channels-last activation digit planes (reduction padded with zero digits to
// a multiple of 32) and runs the convolution's main kernels on them.  The
// VALU kernel below serves P = 16 and path = VALU.
#include <algorithm>

#include "dfp_internal.h"
#include "conv_mfma.h"

namespace dfp {

namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ uint32_t hi_byte(int32_t a) { return (uint32_t)((a + 128) >> 8) & 0xffu; }
__device__ __forceinline__ uint32_t lo_byte(int32_t a) { return (uint32_t)a & 0xffu; }

// Digit planes of one operand view: element (row, t) = src[row * rs + t * ts]
// for row < rows and t < K, else 0.  Unit (row, g) covers t in [16g, 16g+16)
// and is stored as 16 hi bytes then 16 lo bytes at
//   A layout (a_layout = 1): ((g / 2) * rows_pad + row) * 64 + (g % 2) * 32
//   B layout (a_layout = 0): (row * G16 + g) * 32
// One thread per unit.  ROW_FAST: consecutive threads take consecutive rows
// (coalesced when t is the strided index), else consecutive g.  The A launch
// also clears the output scale and writes the per-block B offset table.
template <bool ROW_FAST>
__global__ __launch_bounds__(kBlock) void k_gemm_digits(const int16_t* __restrict__ src, int64_t rs, int64_t ts,
                                                        int32_t rows, int32_t rows_pad, int32_t K, int32_t G16,
                                                        uint8_t* __restrict__ dst, int32_t a_layout,
                                                        dfp_scale* so, int2* boff) {
  const int64_t idx = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (a_layout) {
    if (so && idx == 0) {
      so->amax_bits = 0u;
      so->flags = 0u;
    }
    // block kb reads its two 16-index halves at byte offsets 32*(2kb), 32*(2kb+1)
    // of a column; halves at or past K read offset 0 (their A digits are zero)
    if (idx < G16 / 2) {
      const int32_t t0 = (int32_t)idx * 32;
      boff[idx] = make_int2(t0 < K ? (t0 >> 4) * 32 : 0, t0 + 16 < K ? ((t0 + 16) >> 4) * 32 : 0);
    }
  }
  const int64_t units = (int64_t)rows_pad * G16;
  if (idx >= units) return;
  int32_t row, g;
  if (ROW_FAST) {
    row = (int32_t)(idx % rows_pad);
    g = (int32_t)(idx / rows_pad);
  } else {
    g = (int32_t)(idx % G16);
    row = (int32_t)(idx / G16);
  }
  uint32_t hi[4] = {0u, 0u, 0u, 0u}, lo[4] = {0u, 0u, 0u, 0u};
  if (row < rows) {
    const int16_t* p = src + (int64_t)row * rs;
    const int32_t t0 = g * 16;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int32_t t = t0 + i;
      const int32_t v = t < K ? (int32_t)p[(int64_t)t * ts] : 0;
      hi[i >> 2] |= hi_byte(v) << (8 * (i & 3));
      lo[i >> 2] |= lo_byte(v) << (8 * (i & 3));
    }
  }
  const int64_t off = a_layout ? (((int64_t)(g >> 1) * rows_pad + row) * 64 + (g & 1) * 32)
                               : (((int64_t)row * G16 + g) * 32);
  uint4* d = reinterpret_cast<uint4*>(dst + off);
  d[0] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
  d[1] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
}

// VALU GEMM: one lane per output, chunked INT32 partials, FP32 fold in chunk
// order, one scale; epilogue max |D| into so (cleared by the launcher).
template <bool PARTIALS>
__global__ __launch_bounds__(kBlock) void k_gemm_valu(const int16_t* __restrict__ a, int64_t ars, int64_t ats,
                                                      const int16_t* __restrict__ b, int64_t bts, int64_t bcs,
                                                      int32_t m, int32_t n, int32_t K, int32_t L,
                                                      const dfp_scale* __restrict__ sa,
                                                      const dfp_scale* __restrict__ sb, float* __restrict__ d,
                                                      dfp_scale* so, int32_t* __restrict__ partials) {
  const int64_t O = (int64_t)m * n;
  const int64_t o = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  const bool active = o < O;
  float y = 0.f;
  if (active) {
    const int64_t i = o / n, j = o % n;
    const int16_t* pa = a + i * ars;
    const int16_t* pb = b + j * bcs;
    float sum = 0.f;
    int64_t chunk = 0;
    for (int32_t t0 = 0; t0 < K; t0 += L, ++chunk) {
      const int32_t t1 = min(K, t0 + L);
      uint32_t acc = 0u;
      for (int32_t t = t0; t < t1; ++t) acc += (uint32_t)((int32_t)pa[t * ats] * (int32_t)pb[t * bts]);
      if (PARTIALS) partials[chunk * O + o] = (int32_t)acc;
      const float f = (float)(int32_t)acc;
      sum = chunk == 0 ? f : sum + f;
    }
    y = ldexpf(sum, sa->exp + sb->exp);
    d[o] = y;
  }
  if (so) {
    __shared__ uint32_t red[kBlock / 64];
    uint32_t mx = active ? (__float_as_uint(y) & 0x7fffffffu) : 0u;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off, 64));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t bm = red[0];
      for (int w = 1; w < kBlock / 64; ++w) bm = max(bm, red[w]);
      if (bm > __atomic_load_n(&so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&so->amax_bits, bm);
      if (bm == 0x7f800000u) atomicOr(&so->flags, DFP_FLAG_OUTPUT_INF);
    }
  }
}

// VALU Blocked-DFP GEMM (t contiguous in both operands): every chunk partial is
// scaled by 2^(ea[blk][i] + eb[blk][j]) before it joins the FP32 sum.
template <bool PARTIALS>
__global__ __launch_bounds__(kBlock) void k_gemm_blocked_valu(const int16_t* __restrict__ a,
                                                              const int8_t* __restrict__ ea,
                                                              const int16_t* __restrict__ b,
                                                              const int8_t* __restrict__ eb, int32_t m, int32_t n,
                                                              int32_t K, int32_t L, int32_t bk,
                                                              float* __restrict__ d, dfp_scale* so,
                                                              int32_t* __restrict__ partials) {
  const int64_t O = (int64_t)m * n;
  const int64_t o = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  const bool active = o < O;
  float y = 0.f;
  if (active) {
    const int64_t i = o / n, j = o % n;
    const int16_t* pa = a + i * K;
    const int16_t* pb = b + j * K;
    float sum = 0.f;
    int64_t chunk = 0;
    for (int32_t t0 = 0; t0 < K; t0 += L, ++chunk) {
      const int32_t t1 = min(K, t0 + L);
      uint32_t acc = 0u;
      for (int32_t t = t0; t < t1; ++t) acc += (uint32_t)((int32_t)pa[t] * (int32_t)pb[t]);
      if (PARTIALS) partials[chunk * O + o] = (int32_t)acc;
      const int32_t blk = t0 / bk;
      const float term = ldexpf((float)(int32_t)acc, (int32_t)ea[(int64_t)blk * m + i] + (int32_t)eb[(int64_t)blk * n + j]);
      sum = chunk == 0 ? term : sum + term;
    }
    y = sum;
    d[o] = y;
  }
  if (so) {
    __shared__ uint32_t red[kBlock / 64];
    uint32_t mx = active ? (__float_as_uint(y) & 0x7fffffffu) : 0u;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off, 64));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t bm = red[0];
      for (int w = 1; w < kBlock / 64; ++w) bm = max(bm, red[w]);
      if (bm > __atomic_load_n(&so->amax_bits, __ATOMIC_RELAXED)) atomicMax(&so->amax_bits, bm);
      if (bm == 0x7f800000u) atomicOr(&so->flags, DFP_FLAG_OUTPUT_INF);
    }
  }
}

inline int64_t align256(int64_t v) { return (v + 255) & ~(int64_t)255; }

}  // namespace

GemmPlan plan_gemm(int32_t m, int32_t n, int32_t k) {
  GemmPlan p{};
  p.KB = (k + 31) / 32;
  p.G16 = p.KB * 2;
  p.Mp = (m + kMfmaRowTile - 1) / kMfmaRowTile * kMfmaRowTile;
  p.a_bytes = align256((int64_t)p.KB * p.Mp * 64);
  p.b_bytes = align256((int64_t)n * p.G16 * 32);
  p.t_bytes = align256((int64_t)p.KB * 8);
  p.bytes = p.a_bytes + p.b_bytes + p.t_bytes;
  return p;
}

dfp_status launch_gemm_mfma(int32_t m, int32_t n, int32_t k, int32_t trans_a, int32_t trans_b, int32_t L,
                            const int16_t* a, const dfp_scale* sa, const int16_t* b, const dfp_scale* sb,
                            float* d, dfp_scale* so, int32_t* partials, void* ws, hipStream_t st,
                            const int8_t* exa, const int8_t* exb, int32_t bk) {
  const GemmPlan p = plan_gemm(m, n, k);
  uint8_t* wsa = reinterpret_cast<uint8_t*>(ws);
  uint8_t* xs = wsa + p.a_bytes;
  int2* boff = reinterpret_cast<int2*>(xs + p.b_bytes);
  {
    // opA[i][t] = a[i*k + t] or a[t*m + i]
    const int64_t rs = trans_a ? 1 : k, ts = trans_a ? m : 1;
    const int64_t units = std::max<int64_t>((int64_t)p.Mp * p.G16, p.KB);
    const dim3 grid((unsigned)((units + kBlock - 1) / kBlock));
    if (trans_a)
      DFP_LAUNCH(K_GEMM_PREP, k_gemm_digits<true>, grid, dim3(kBlock), 0, st, a, rs, ts, m, p.Mp, k, p.G16, wsa,
                 1, so, boff);
    else
      DFP_LAUNCH(K_GEMM_PREP, k_gemm_digits<false>, grid, dim3(kBlock), 0, st, a, rs, ts, m, p.Mp, k, p.G16, wsa,
                 1, so, boff);
  }
  {
    // column j of opB: opB[t][j] = b[t*n + j] or b[j*k + t]
    const int64_t rs = trans_b ? k : 1, ts = trans_b ? 1 : n;
    const int64_t units = (int64_t)n * p.G16;
    const dim3 grid((unsigned)((units + kBlock - 1) / kBlock));
    if (trans_b)
      DFP_LAUNCH(K_GEMM_PREP, k_gemm_digits<false>, grid, dim3(kBlock), 0, st, b, rs, ts, n, n, k, p.G16, xs, 0,
                 (dfp_scale*)nullptr, (int2*)nullptr);
    else
      DFP_LAUNCH(K_GEMM_PREP, k_gemm_digits<true>, grid, dim3(kBlock), 0, st, b, rs, ts, n, n, k, p.G16, xs, 0,
                 (dfp_scale*)nullptr, (int2*)nullptr);
  }
  ConvMfmaArgs args{};
  args.xs = xs;
  args.wsa = wsa;
  args.boff = boff;
  args.ea = sa;
  args.eb = sb;
  args.out = d;
  args.so = so;
  args.partials = partials;
  args.M = m; args.Mp = p.Mp; args.Cin = p.KB * 32; args.S = 1; args.T = k; args.KB = p.KB; args.L = L;
  args.CG = p.G16; args.Hp = 1; args.Wp = n; args.Po = 1; args.Qo = n;
  args.NP = n;
  args.O = (int64_t)m * n;
  args.ustride_h = 1; args.ustride_w = 1; args.rsign = 1; args.roff_h = 0; args.roff_w = 0;
  args.exa = exa;
  args.exb = exb;
  args.bk = bk;
  args.nb = exa ? (k + bk - 1) / bk : 0;
  return launch_mfma_main(args, p.b_bytes, exa ? K_GEMM_BLOCKED : K_GEMM, K_GEMM, false, st);
}

dfp_status launch_gemm_blocked_valu(int32_t m, int32_t n, int32_t k, int32_t L, int32_t bk, const int16_t* a,
                                    const int8_t* ea, const int16_t* b, const int8_t* eb, float* d, dfp_scale* so,
                                    int32_t* partials, hipStream_t st) {
  const int64_t O = (int64_t)m * n;
  const dim3 grid((unsigned)((O + kBlock - 1) / kBlock));
  if (partials)
    DFP_LAUNCH(K_GEMM_BLOCKED, k_gemm_blocked_valu<true>, grid, dim3(kBlock), 0, st, a, ea, b, eb, m, n, k, L, bk, d,
               so, partials);
  else
    DFP_LAUNCH(K_GEMM_BLOCKED, k_gemm_blocked_valu<false>, grid, dim3(kBlock), 0, st, a, ea, b, eb, m, n, k, L, bk,
               d, so, partials);
  return DFP_OK;
}

dfp_status launch_gemm_valu(int32_t m, int32_t n, int32_t k, int32_t trans_a, int32_t trans_b, int32_t L,
                            const int16_t* a, const dfp_scale* sa, const int16_t* b, const dfp_scale* sb,
                            float* d, dfp_scale* so, int32_t* partials, hipStream_t st) {
  const int64_t ars = trans_a ? 1 : k, ats = trans_a ? m : 1;
  const int64_t bts = trans_b ? 1 : n, bcs = trans_b ? k : 1;
  const int64_t O = (int64_t)m * n;
  const dim3 grid((unsigned)((O + kBlock - 1) / kBlock));
  if (partials)
    DFP_LAUNCH(K_GEMM, k_gemm_valu<true>, grid, dim3(kBlock), 0, st, a, ars, ats, b, bts, bcs, m, n, k, L, sa, sb, d,
               so, partials);
  else
    DFP_LAUNCH(K_GEMM, k_gemm_valu<false>, grid, dim3(kBlock), 0, st, a, ars, ats, b, bts, bcs, m, n, k, L, sa, sb,
               d, so, partials);
  return DFP_OK;
}

}  // namespace dfp
