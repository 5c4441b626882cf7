// The FP32 steps either side of a layer's convolutions in a DFP16 training
// step (Sec. 4.1, Fig. 2): batch normalisation with an optional residual add
// and ReLU on an up-converted DFP16 tensor, its backward pass, and FP32 SGD on
// master weights; each ends in the quantiser of its output (Q_a, Q_e, Q_w).
//
// Batch-norm statistics need no floating-point accumulation: a channel's
// values are i * 2^E with integer i, so sum i and sum i^2 (and in the backward
// pass the masked sums of dz and dz * y) are exact in 64-bit integers and
// independent of the reduction order.  Per-channel values are computed once
// in float64 and rounded to FP32; per-element work is FP32 with a fixed
// operation order, every step one IEEE rounding (no contraction in this
// file), so the rounding pass can recompute an element bit for bit instead of
// reading it back.
//
// Passes (all HBM-bound):
//   forward   k_bn_stats (y) -> k_bn_finalize -> [res: k_bn_amax + max reduce]
//             -> k_bn_convert (y [, res]) writing zq [and z]
//   backward  k_bn_stats (y, dz [, res]) -> k_bn_finalize -> k_bn_amax (writes
//             dy / dres if asked) -> max reduce -> k_bn_convert
//   SGD       k_sgd (update + max) -> max reduce -> the tensor quantiser
// Without a residual the forward output is a monotone function of the input
// integer within a channel (ReLU of an affine map evaluated with monotone
// roundings), so its max is the larger of the values at the channel's
// smallest and largest integer and the max pass over z is skipped.
#pragma clang fp contract(off)

#include <algorithm>
#include <climits>

#include "dfp_internal.h"
#include "dfp_round.h"

namespace dfp {

namespace {

constexpr int kBlock = 256;
constexpr int kMaxParts = 1024;

struct Chan {
  float mean, inv, gamma, beta;
};
__device__ __forceinline__ Chan load_chan(const float* mean, const float* inv, const float* gamma,
                                          const float* beta, int32_t c) {
  return {mean[c], inv[c], gamma[c], beta[c]};
}

// xhat = (i 2^E - mean) * inv_std; i 2^E is exact for |i| < 2^24.
__device__ __forceinline__ float bn_xhat(int32_t yi, int32_t ey, const Chan& p) {
  return __fmul_rn(__fsub_rn(ldexpf((float)yi, ey), p.mean), p.inv);
}
// Pre-activation gamma * xhat + beta (fused), plus the residual if any.
__device__ __forceinline__ float bn_pre(float xh, const Chan& p, const float* res, int32_t idx) {
  const float zp = __fmaf_rn(xh, p.gamma, p.beta);
  return res ? __fadd_rn(zp, res[idx]) : zp;
}
__device__ __forceinline__ float relu(float v) { return v > 0.0f ? v : 0.0f; }

// Gradient at y of one element: dy = fma(k1, g, fma(k2, xhat, k3)) with
// g = pre > 0 ? dz 2^Edz : 0; also returns g (the gradient at res).
__device__ __forceinline__ float bn_dy(int32_t yi, int32_t dzi, int32_t ey, int32_t edz, const Chan& p,
                                       const float4& k, const float* res, int32_t idx, float* g_out) {
  const float xh = bn_xhat(yi, ey, p);
  const float pre = bn_pre(xh, p, res, idx);
  const float g = pre > 0.0f ? ldexpf((float)dzi, edz) : 0.0f;
  *g_out = g;
  return __fmaf_rn(k.x, g, __fmaf_rn(k.y, xh, k.z));
}

__device__ __forceinline__ int32_t lo16(uint32_t w) { return (int32_t)(int16_t)(w & 0xffffu); }
__device__ __forceinline__ int32_t hi16(uint32_t w) { return (int32_t)w >> 16; }

// ------------------------------------------------------------ statistics
// Workgroup (s, c) reduces channel c over images [N s / S, N (s+1) / S).
// Forward: S1 = sum i, S2 = sum i^2, min i, max i.  Backward: D = sum g_i,
// Pd = sum g_i * y_i with g_i = dz_i where the recomputed pre-activation is
// positive, else 0.  Partials: part[(s*C + c)*3 + {0, 1, 2}], slot 2 holding
// (max << 32) | (uint32)min.  VEC: 8 elements per unit (hw % 8 == 0).
template <bool BWD, bool VEC>
__global__ __launch_bounds__(kBlock) void k_bn_stats(const int16_t* __restrict__ y, const int16_t* __restrict__ dz,
                                                     const float* __restrict__ res, const float* __restrict__ mean,
                                                     const float* __restrict__ inv, const float* __restrict__ gamma,
                                                     const float* __restrict__ beta, const dfp_scale* __restrict__ sy,
                                                     const dfp_scale* __restrict__ sdz, int32_t N, int32_t C,
                                                     int32_t HW, int32_t S, FastDiv upr_div,
                                                     int64_t* __restrict__ part, dfp_scale* __restrict__ sz) {
  const int32_t s = blockIdx.x, c = blockIdx.y;
  if (sz && s == 0 && c == 0 && threadIdx.x == 0) {  // the finalize kernel max-reduces into it
    sz->amax_bits = 0u;
    sz->flags = 0u;
  }
  const int32_t n0 = (int32_t)((int64_t)N * s / S), n1 = (int32_t)((int64_t)N * (s + 1) / S);
  constexpr int V = VEC ? 8 : 1;
  const int32_t upr = HW / V;
  const int32_t units = (n1 - n0) * upr;
  int64_t a = 0, b = 0;
  int32_t mn = INT_MAX, mx = INT_MIN;
  Chan p{};
  int32_t ey = 0;
  if (BWD) {
    p = load_chan(mean, inv, gamma, beta, c);
    ey = sy->exp;
  }
  (void)sdz;
  for (int32_t j = threadIdx.x; j < units; j += kBlock) {
    const int32_t r = (int32_t)fdiv((uint32_t)j, upr_div);
    const int32_t off = ((n0 + r) * C + c) * HW + (j - r * upr) * V;
    int32_t yv[V], dv[V];
    if (VEC) {
      const uint4 w = *reinterpret_cast<const uint4*>(y + off);
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) { yv[2 * q] = lo16(ws[q]); yv[2 * q + 1] = hi16(ws[q]); }
      if (BWD) {
        const uint4 d = *reinterpret_cast<const uint4*>(dz + off);
        const uint32_t ds[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) { dv[2 * q] = lo16(ds[q]); dv[2 * q + 1] = hi16(ds[q]); }
      }
    } else {
      yv[0] = y[off];
      if (BWD) dv[0] = dz[off];
    }
#pragma unroll
    for (int q = 0; q < V; ++q) {
      if (BWD) {
        const float pre = bn_pre(bn_xhat(yv[q], ey, p), p, res, off + q);
        const int32_t g = pre > 0.0f ? dv[q] : 0;
        a += g;
        b += g * yv[q];  // |g y| <= 2^30
      } else {
        a += yv[q];
        b += yv[q] * yv[q];
        mn = min(mn, yv[q]);
        mx = max(mx, yv[q]);
      }
    }
  }
  __shared__ int64_t ra[kBlock], rb[kBlock];
  __shared__ int32_t rmn[kBlock], rmx[kBlock];
  ra[threadIdx.x] = a;
  rb[threadIdx.x] = b;
  rmn[threadIdx.x] = mn;
  rmx[threadIdx.x] = mx;
  __syncthreads();
  for (int w = kBlock / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      ra[threadIdx.x] += ra[threadIdx.x + w];
      rb[threadIdx.x] += rb[threadIdx.x + w];
      rmn[threadIdx.x] = min(rmn[threadIdx.x], rmn[threadIdx.x + w]);
      rmx[threadIdx.x] = max(rmx[threadIdx.x], rmx[threadIdx.x + w]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    int64_t* o = part + ((int64_t)s * C + c) * 3;
    o[0] = ra[0];
    o[1] = rb[0];
    o[2] = (int64_t)(((uint64_t)(uint32_t)rmx[0] << 32) | (uint32_t)rmn[0]);
  }
}

// -------------------------------------------------------------- finalize
// One wave per channel: the lanes add the channel's S partials (exact
// integers), lane 0 derives the per-channel values.
// Forward: mean / inv_std from the exact sums (float64, rounded once), and
// without a residual the output max from the channel's extreme integers,
// max-reduced into the output scale (cleared by the statistics kernel).
// Backward: dbeta, dgamma and the per-element coefficients k1..k3.
template <bool BWD>
__global__ __launch_bounds__(kBlock) void k_bn_finalize(const int64_t* __restrict__ part, int32_t S, int32_t C,
                                                        int64_t cnt, const dfp_scale* __restrict__ sy,
                                                        const dfp_scale* __restrict__ sdz, float eps,
                                                        const float* __restrict__ gamma,
                                                        const float* __restrict__ beta, float* __restrict__ mean,
                                                        float* __restrict__ inv, int64_t* __restrict__ sums,
                                                        float* __restrict__ dgamma, float* __restrict__ dbeta,
                                                        float4* __restrict__ kco, dfp_scale* __restrict__ sz,
                                                        bool write_max) {
  const int lane = threadIdx.x & 63;
  const int32_t c = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  if (c >= C) return;
  int64_t a = 0, b = 0;
  int32_t mn = INT_MAX, mx = INT_MIN;
  for (int32_t s = lane; s < S; s += 64) {
    const int64_t* o = part + ((int64_t)s * C + c) * 3;
    a += o[0];
    b += o[1];
    const uint64_t e = (uint64_t)o[2];
    mn = min(mn, (int32_t)(uint32_t)e);
    mx = max(mx, (int32_t)(uint32_t)(e >> 32));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a += __shfl_xor(a, off, 64);
    b += __shfl_xor(b, off, 64);
    mn = min(mn, __shfl_xor(mn, off, 64));
    mx = max(mx, __shfl_xor(mx, off, 64));
  }
  if (lane != 0) return;
  const int32_t ey = sy->exp;
  const double dcnt = (double)cnt;
  if (sums) {
    sums[2 * c] = a;
    sums[2 * c + 1] = b;
  }
  if (!BWD) {
    const double mu = __ddiv_rn(ldexp((double)a, ey), dcnt);
    double var = __dsub_rn(__ddiv_rn(ldexp((double)b, 2 * ey), dcnt), __dmul_rn(mu, mu));
    if (var < 0.0) var = 0.0;
    const float mf = (float)mu;
    const float t = __fadd_rn((float)var, eps);
    const float sq = (float)__dsqrt_rn((double)t);  // correctly rounded FP32 square root
    const float iv = __fdiv_rn(1.0f, sq);
    mean[c] = mf;
    inv[c] = iv;
    if (write_max) {
      const Chan p{mf, iv, gamma[c], beta[c]};
      const float zlo = relu(bn_pre(bn_xhat(mn, ey, p), p, nullptr, 0));
      const float zhi = relu(bn_pre(bn_xhat(mx, ey, p), p, nullptr, 0));
      const uint32_t m = max(__float_as_uint(zlo), __float_as_uint(zhi)) & 0x7fffffffu;
      if (m) atomicMax(&sz->amax_bits, m);
    }
  } else {
    const int32_t edz = sdz->exp;
    const double mf = (double)mean[c], iv = (double)inv[c];
    const double db = ldexp((double)a, edz);
    const double dg = __dmul_rn(iv, ldexp(__dsub_rn(ldexp((double)b, ey), __dmul_rn(mf, (double)a)), edz));
    const float dbf = (float)db, dgf = (float)dg;
    dbeta[c] = dbf;
    dgamma[c] = dgf;
    const double al = __dmul_rn((double)gamma[c], iv);  // exact: two FP32 factors
    kco[c] = make_float4((float)al, (float)__ddiv_rn(__dmul_rn(-al, (double)dgf), dcnt),
                         (float)__ddiv_rn(__dmul_rn(-al, (double)dbf), dcnt), 0.0f);
  }
}

// ------------------------------------------------------ element groups
// Flat groups of four consecutive elements (the Philox block of stochastic
// rounding).  Channel of element idx: (idx / hw) mod C.
struct Elems {
  const int16_t* y;
  const int16_t* dz;
  const float* res;
  const float* mean;
  const float* inv;
  const float* gamma;
  const float* beta;
  const float4* kco;
  const dfp_scale* sy;
  const dfp_scale* sdz;
  int32_t total, C;
  FastDiv hw_div, c_div;
  bool hw4;  // hw % 4 == 0: a group lies in one channel
};

__device__ __forceinline__ int32_t chan_of(const Elems& e, int32_t idx) {
  const uint32_t row = fdiv((uint32_t)idx, e.hw_div);
  return (int32_t)(row - fdiv(row, e.c_div) * (uint32_t)e.C);
}

// Values of the group starting at base (valid lanes < cnt): the forward output
// z or the backward gradient dy (and g, the gradient at res).
template <bool BWD>
__device__ __forceinline__ void group_values(const Elems& e, int32_t base, int32_t cnt, int32_t ey, int32_t edz,
                                             float v[4], float g[4]) {
  int32_t yi[4] = {0, 0, 0, 0}, di[4] = {0, 0, 0, 0};
  if (cnt == 4) {
    const uint2 w = *reinterpret_cast<const uint2*>(e.y + base);
    yi[0] = lo16(w.x); yi[1] = hi16(w.x); yi[2] = lo16(w.y); yi[3] = hi16(w.y);
    if (BWD) {
      const uint2 d = *reinterpret_cast<const uint2*>(e.dz + base);
      di[0] = lo16(d.x); di[1] = hi16(d.x); di[2] = lo16(d.y); di[3] = hi16(d.y);
    }
  } else {
    for (int q = 0; q < cnt; ++q) {
      yi[q] = e.y[base + q];
      if (BWD) di[q] = e.dz[base + q];
    }
  }
  Chan p{};
  float4 k{};
  int32_t c0 = -1;
  if (e.hw4) {
    c0 = chan_of(e, base);
    p = load_chan(e.mean, e.inv, e.gamma, e.beta, c0);
    if (BWD) k = e.kco[c0];
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    v[q] = 0.0f;
    g[q] = 0.0f;
    if (q >= cnt) continue;
    if (!e.hw4) {
      const int32_t c = chan_of(e, base + q);
      p = load_chan(e.mean, e.inv, e.gamma, e.beta, c);
      if (BWD) k = e.kco[c];
    }
    if (BWD) v[q] = bn_dy(yi[q], di[q], ey, edz, p, k, e.res, base + q, &g[q]);
    else v[q] = relu(bn_pre(bn_xhat(yi[q], ey, p), p, e.res, base + q));
  }
}

// Max pass: part[workgroup] = max |v| bits over its groups (part == nullptr:
// a single workgroup writes the scale directly and clears its flags).
// Backward: also stores dy and dres when asked.
template <bool BWD>
__global__ __launch_bounds__(kBlock) void k_bn_amax(Elems e, float* __restrict__ dy, float* __restrict__ dres,
                                                    uint32_t* __restrict__ part, dfp_scale* __restrict__ s) {
  const int32_t ey = e.sy->exp;
  const int32_t edz = BWD ? e.sdz->exp : 0;
  const int32_t groups = (e.total + 3) >> 2;
  uint32_t m = 0u;
  for (int32_t gi = blockIdx.x * kBlock + threadIdx.x; gi < groups; gi += gridDim.x * kBlock) {
    const int32_t base = gi << 2;
    const int32_t cnt = min(4, e.total - base);
    float v[4], g[4];
    group_values<BWD>(e, base, cnt, ey, edz, v, g);
#pragma unroll
    for (int q = 0; q < 4; ++q) m = max(m, __float_as_uint(v[q]) & 0x7fffffffu);
    if (BWD) {
      if (cnt == 4) {
        if (dy) *reinterpret_cast<float4*>(dy + base) = make_float4(v[0], v[1], v[2], v[3]);
        if (dres) *reinterpret_cast<float4*>(dres + base) = make_float4(g[0], g[1], g[2], g[3]);
      } else {
        for (int q = 0; q < cnt; ++q) {
          if (dy) dy[base + q] = v[q];
          if (dres) dres[base + q] = g[q];
        }
      }
    }
  }
  __shared__ uint32_t red[kBlock / 64];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = red[0];
    for (int i = 1; i < kBlock / 64; ++i) r = max(r, red[i]);
    if (part) {
      part[blockIdx.x] = r;
    } else {
      s->amax_bits = r;
      s->flags = 0u;
    }
  }
}

// Rounding pass: recomputes each element's value, rounds it with the shared
// exponent of the tensor max (Eq. 2-3, the descriptor's mode), writes the
// INT16 result and, forward, the FP32 value when z != nullptr.
template <bool BWD, int MODE, bool SAT>
__global__ __launch_bounds__(kBlock) void k_bn_convert(Elems e, float* __restrict__ z, int16_t* __restrict__ dst,
                                                       dfp_scale* __restrict__ s, int32_t bits, uint32_t key0,
                                                       uint32_t key1, uint32_t role) {
  const ScaleFromMax sc = scale_from_max(s->amax_bits, bits);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    s->exp = sc.es;
    if (sc.flags) atomicOr(&s->flags, sc.flags);
  }
  const int32_t ey = e.sy->exp;
  const int32_t edz = BWD ? e.sdz->exp : 0;
  const int32_t groups = (e.total + 3) >> 2;
  bool saturated = false;
  for (int32_t gi = blockIdx.x * kBlock + threadIdx.x; gi < groups; gi += gridDim.x * kBlock) {
    const int32_t base = gi << 2;
    const int32_t cnt = min(4, e.total - base);
    float v[4], g[4];
    group_values<BWD>(e, base, cnt, ey, edz, v, g);
    uint32_t u[4] = {0u, 0u, 0u, 0u};
    if (MODE == DFP_ROUND_STOCHASTIC) {
      const uint4 r = philox4x32_10(make_uint4((uint32_t)gi, 0u, role, 0u), key0, key1);
      u[0] = r.x; u[1] = r.y; u[2] = r.z; u[3] = r.w;
    }
    int32_t iv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      int32_t t = round_one<MODE>(__float_as_uint(v[q]), sc.es, u[q]);
      t = sc.all_zero ? 0 : t;
      if (SAT) {
        const int32_t cl = min(max(t, -32767), 32767);
        saturated |= cl != t;
        t = cl;
      }
      iv[q] = t;
    }
    if (cnt == 4) {
      uint2 packed;
      packed.x = ((uint32_t)iv[0] & 0xffffu) | ((uint32_t)iv[1] << 16);
      packed.y = ((uint32_t)iv[2] & 0xffffu) | ((uint32_t)iv[3] << 16);
      *reinterpret_cast<uint2*>(dst + base) = packed;
      if (!BWD && z) *reinterpret_cast<float4*>(z + base) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
      for (int q = 0; q < cnt; ++q) {
        dst[base + q] = (int16_t)iv[q];
        if (!BWD && z) z[base + q] = v[q];
      }
    }
  }
  if (SAT && saturated) atomicOr(&s->flags, DFP_FLAG_SATURATED);
}

// ------------------------------------------------------------------ SGD
// g = fma(wd, w, dw); v = fma(mu, v, g); w = fma(-lr, v, w), in place, and the
// max |w| per workgroup (as k_bn_amax).
__global__ __launch_bounds__(kBlock) void k_sgd(int64_t n, float lr, float mu, float wd, float* __restrict__ w,
                                                float* __restrict__ v, const float* __restrict__ dw,
                                                uint32_t* __restrict__ part, dfp_scale* __restrict__ s) {
  const int64_t groups = (n + 3) >> 2;
  uint32_t m = 0u;
  for (int64_t gi = (int64_t)blockIdx.x * kBlock + threadIdx.x; gi < groups; gi += (int64_t)gridDim.x * kBlock) {
    const int64_t base = gi << 2;
    if (base + 4 <= n) {
      float4 w4 = reinterpret_cast<const float4*>(w)[gi];
      float4 v4 = reinterpret_cast<const float4*>(v)[gi];
      const float4 d4 = reinterpret_cast<const float4*>(dw)[gi];
      float* wp = &w4.x;
      float* vp = &v4.x;
      const float* dp = &d4.x;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float g = __fmaf_rn(wd, wp[q], dp[q]);
        vp[q] = __fmaf_rn(mu, vp[q], g);
        wp[q] = __fmaf_rn(-lr, vp[q], wp[q]);
        m = max(m, __float_as_uint(wp[q]) & 0x7fffffffu);
      }
      reinterpret_cast<float4*>(w)[gi] = w4;
      reinterpret_cast<float4*>(v)[gi] = v4;
    } else {
      for (int64_t i = base; i < n; ++i) {
        const float g = __fmaf_rn(wd, w[i], dw[i]);
        const float vn = __fmaf_rn(mu, v[i], g);
        const float wn = __fmaf_rn(-lr, vn, w[i]);
        v[i] = vn;
        w[i] = wn;
        m = max(m, __float_as_uint(wn) & 0x7fffffffu);
      }
    }
  }
  __shared__ uint32_t red[kBlock / 64];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = red[0];
    for (int i = 1; i < kBlock / 64; ++i) r = max(r, red[i]);
    if (part) {
      part[blockIdx.x] = r;
    } else {
      s->amax_bits = r;
      s->flags = 0u;
    }
  }
}

// ------------------------------------------------------------ host side
int32_t bn_splits(const dfp_bn_desc& d) {
  const int32_t want = (2048 + d.c - 1) / d.c;
  return std::max(1, std::min(want, d.n));
}

struct BnWs {
  int64_t* part;
  float4* kco;
};
BnWs bn_ws(const dfp_bn_desc& d, void* ws) {
  const int64_t part_bytes = ((int64_t)bn_splits(d) * d.c * 24 + 255) / 256 * 256;
  return {reinterpret_cast<int64_t*>(ws), reinterpret_cast<float4*>(reinterpret_cast<uint8_t*>(ws) + part_bytes)};
}

// Workgroups of a max pass over `groups` groups of four whose per-workgroup
// maxima are kept in an INT16 buffer of `n` elements (4 bytes each); <= 1
// means one workgroup writing the scale directly.
int32_t max_parts(int64_t groups, int64_t n) {
  int64_t parts = (groups + kBlock - 1) / kBlock;
  parts = std::min<int64_t>(std::min<int64_t>(parts, kMaxParts), n / 2);
  return (int32_t)std::max<int64_t>(parts, 1);
}

dfp_status launch_stats(bool bwd, const dfp_bn_desc& d, const int16_t* y, const int16_t* dz, const float* res,
                        const float* mean, const float* inv, const float* gamma, const float* beta,
                        const dfp_scale* sy, const dfp_scale* sdz, int64_t* part, dfp_scale* sz, hipStream_t st) {
  const int32_t S = bn_splits(d);
  const bool vec = (d.hw % 8) == 0 && ((uintptr_t)y & 15) == 0 && (!bwd || ((uintptr_t)dz & 15) == 0);
  const FastDiv upr = make_fastdiv((uint32_t)(vec ? d.hw / 8 : d.hw));
  const dim3 grid((unsigned)S, (unsigned)d.c);
  if (bwd) {
    if (vec)
      DFP_LAUNCH(K_BN_STATS, (k_bn_stats<true, true>), grid, dim3(kBlock), 0, st, y, dz, res, mean, inv, gamma, beta,
                 sy, sdz, d.n, d.c, d.hw, S, upr, part, sz);
    else
      DFP_LAUNCH(K_BN_STATS, (k_bn_stats<true, false>), grid, dim3(kBlock), 0, st, y, dz, res, mean, inv, gamma,
                 beta, sy, sdz, d.n, d.c, d.hw, S, upr, part, sz);
  } else {
    if (vec)
      DFP_LAUNCH(K_BN_STATS, (k_bn_stats<false, true>), grid, dim3(kBlock), 0, st, y, dz, res, mean, inv, gamma,
                 beta, sy, sdz, d.n, d.c, d.hw, S, upr, part, sz);
    else
      DFP_LAUNCH(K_BN_STATS, (k_bn_stats<false, false>), grid, dim3(kBlock), 0, st, y, dz, res, mean, inv, gamma,
                 beta, sy, sdz, d.n, d.c, d.hw, S, upr, part, sz);
  }
  return DFP_OK;
}

Elems make_elems(const dfp_bn_desc& d, const int16_t* y, const int16_t* dz, const float* res, const float* mean,
                 const float* inv, const float* gamma, const float* beta, const float4* kco, const dfp_scale* sy,
                 const dfp_scale* sdz) {
  Elems e{};
  e.y = y; e.dz = dz; e.res = res; e.mean = mean; e.inv = inv; e.gamma = gamma; e.beta = beta; e.kco = kco;
  e.sy = sy; e.sdz = sdz;
  e.total = d.n * d.c * d.hw;
  e.C = d.c;
  e.hw_div = make_fastdiv((uint32_t)d.hw);
  e.c_div = make_fastdiv((uint32_t)d.c);
  e.hw4 = (d.hw % 4) == 0;
  return e;
}

// Max pass (k_bn_amax + the max reduce) into s.
template <bool BWD>
dfp_status launch_max(const Elems& e, float* dy, float* dres, int16_t* scratch, dfp_scale* s, hipStream_t st) {
  const int32_t parts = max_parts((e.total + 3) / 4, e.total);
  if (parts <= 1) {
    DFP_LAUNCH(K_BN_AMAX, k_bn_amax<BWD>, dim3(1), dim3(kBlock), 0, st, e, dy, dres, (uint32_t*)nullptr, s);
    return DFP_OK;
  }
  uint32_t* part = reinterpret_cast<uint32_t*>(scratch);
  DFP_LAUNCH(K_BN_AMAX, k_bn_amax<BWD>, dim3((unsigned)parts), dim3(kBlock), 0, st, e, dy, dres, part, s);
  return launch_amax_final(part, parts, s, st);
}

template <bool BWD, int MODE>
dfp_status launch_convert_mode(const Elems& e, float* z, int16_t* dst, dfp_scale* s, int32_t bits, uint64_t seed,
                               uint32_t role, hipStream_t st) {
  int64_t blocks = ((int64_t)(e.total + 3) / 4 + kBlock - 1) / kBlock;
  blocks = std::max<int64_t>(1, std::min<int64_t>(blocks, 8192));
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  if (bits == 16)
    DFP_LAUNCH(K_BN_CONVERT, (k_bn_convert<BWD, MODE, true>), dim3((unsigned)blocks), dim3(kBlock), 0, st, e, z, dst,
               s, bits, k0, k1, role);
  else
    DFP_LAUNCH(K_BN_CONVERT, (k_bn_convert<BWD, MODE, false>), dim3((unsigned)blocks), dim3(kBlock), 0, st, e, z,
               dst, s, bits, k0, k1, role);
  return DFP_OK;
}

template <bool BWD>
dfp_status launch_convert(const Elems& e, float* z, int16_t* dst, dfp_scale* s, int32_t bits, int32_t rounding,
                          uint64_t seed, uint32_t role, hipStream_t st) {
  switch (rounding) {
    case DFP_ROUND_NEAREST: return launch_convert_mode<BWD, DFP_ROUND_NEAREST>(e, z, dst, s, bits, seed, role, st);
    case DFP_ROUND_STOCHASTIC:
      return launch_convert_mode<BWD, DFP_ROUND_STOCHASTIC>(e, z, dst, s, bits, seed, role, st);
    case DFP_ROUND_BIASED: return launch_convert_mode<BWD, DFP_ROUND_BIASED>(e, z, dst, s, bits, seed, role, st);
    default: return launch_convert_mode<BWD, DFP_ROUND_DOWN>(e, z, dst, s, bits, seed, role, st);
  }
}

}  // namespace

size_t bn_workspace_bytes(const dfp_bn_desc& d) {
  const int64_t part_bytes = ((int64_t)bn_splits(d) * d.c * 24 + 255) / 256 * 256;
  const int64_t k_bytes = ((int64_t)d.c * 16 + 255) / 256 * 256;
  return (size_t)(part_bytes + k_bytes);
}

dfp_status launch_bn_relu_fwd(const dfp_bn_desc& d, const int16_t* y, const dfp_scale* sy, const float* gamma,
                              const float* beta, const float* res, float* z, int16_t* zq, dfp_scale* sz, float* mean,
                              float* inv_std, int64_t* sums, void* ws, hipStream_t st) {
  const BnWs w = bn_ws(d, ws);
  dfp_status rc;
  if ((rc = launch_stats(false, d, y, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, sy, nullptr, w.part,
                         res ? nullptr : sz, st)) != DFP_OK)
    return rc;
  const int64_t cnt = (int64_t)d.n * d.hw;
  DFP_LAUNCH(K_BN_FINAL, k_bn_finalize<false>, dim3((unsigned)((d.c + 3) / 4)), dim3(kBlock), 0, st, w.part, bn_splits(d), d.c, cnt, sy,
             (const dfp_scale*)nullptr, d.eps, gamma, beta, mean, inv_std, sums, (float*)nullptr, (float*)nullptr,
             (float4*)nullptr, sz, res == nullptr);
  const Elems e = make_elems(d, y, nullptr, res, mean, inv_std, gamma, beta, nullptr, sy, nullptr);
  if (res && (rc = launch_max<false>(e, nullptr, nullptr, zq, sz, st)) != DFP_OK) return rc;
  return launch_convert<false>(e, z, zq, sz, d.bits, d.rounding, d.seed, DFP_ROLE_X, st);
}

dfp_status launch_bn_relu_bwd(const dfp_bn_desc& d, const int16_t* dz, const dfp_scale* sdz, const int16_t* y,
                              const dfp_scale* sy, const float* gamma, const float* beta, const float* res,
                              const float* mean, const float* inv_std, float* dy, int16_t* dyq, dfp_scale* sdy,
                              float* dgamma, float* dbeta, float* dres, int64_t* sums, void* ws, hipStream_t st) {
  const BnWs w = bn_ws(d, ws);
  dfp_status rc;
  if ((rc = launch_stats(true, d, y, dz, res, mean, inv_std, gamma, beta, sy, sdz, w.part, nullptr, st)) != DFP_OK)
    return rc;
  const int64_t cnt = (int64_t)d.n * d.hw;
  DFP_LAUNCH(K_BN_FINAL, k_bn_finalize<true>, dim3((unsigned)((d.c + 3) / 4)), dim3(kBlock), 0, st, w.part, bn_splits(d), d.c, cnt, sy, sdz,
             d.eps, gamma, beta, const_cast<float*>(mean), const_cast<float*>(inv_std), sums, dgamma, dbeta, w.kco,
             (dfp_scale*)nullptr, false);
  const Elems e = make_elems(d, y, dz, res, mean, inv_std, gamma, beta, w.kco, sy, sdz);
  if ((rc = launch_max<true>(e, dy, dres, dyq, sdy, st)) != DFP_OK) return rc;
  return launch_convert<true>(e, nullptr, dyq, sdy, d.bits, d.rounding, d.seed, DFP_ROLE_DY, st);
}

dfp_status launch_sgd_quantize(int64_t n, float lr, float mu, float wd, int32_t bits, int32_t rounding,
                               uint64_t seed, float* w, float* v, const float* dw, int16_t* wq, dfp_scale* sw,
                               hipStream_t st) {
  const int32_t parts = max_parts((n + 3) / 4, n);
  if (parts <= 1) {
    DFP_LAUNCH(K_SGD, k_sgd, dim3(1), dim3(kBlock), 0, st, n, lr, mu, wd, w, v, dw, (uint32_t*)nullptr, sw);
  } else {
    uint32_t* part = reinterpret_cast<uint32_t*>(wq);
    DFP_LAUNCH(K_SGD, k_sgd, dim3((unsigned)parts), dim3(kBlock), 0, st, n, lr, mu, wd, w, v, dw, part, sw);
    dfp_status rc;
    if ((rc = launch_amax_final(part, parts, sw, st)) != DFP_OK) return rc;
  }
  return launch_quant_convert(w, wq, n, sw, bits, rounding, seed, DFP_ROLE_W, st);
}

}  // namespace dfp
