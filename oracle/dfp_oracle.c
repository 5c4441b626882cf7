/*
 * dfp_oracle.c -- CPU oracle for Dynamic Fixed Point (DFP) INT16 convolution
 * (Das et al., "Mixed Precision Training of Convolutional Neural Networks using
 * Integer Operations", ICLR 2018).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline leg do.  It shares no code, header, table or helper with the HIP
 * path.
 *
 * Plain, slow and obviously correct on purpose: scalar loops, int64 products,
 * exact float64 arithmetic where the method needs rational values, and one
 * output element at a time, each chunk of its reduction visited in order.
 * OpenMP only splits the loop over independent output elements.
 *
 * What each part follows (paper sections / equations / algorithms):
 *   - Shared exponent from the tensor-wide max magnitude: Sec. 3.1, Eq. 1-2.
 *   - Meaning of a DFP value (i * 2^Es): Sec. 3.1, Eq. 3.
 *   - Product exponent is the sum of the operand exponents, and every product
 *     of a multiply-accumulate chain shares it: Sec. 3.1, Eq. 4 and the note
 *     after Eq. 5.
 *   - Down-conversion of an output using the max of the current output and
 *     nearest / stochastic / biased rounding: Sec. 1 (list of ingredients),
 *     Sec. 3.1 Eq. 6, Sec. 4.1 (quantisers after FP and BP).
 *   - INT16 x INT16 -> INT32 multiply-accumulate over short chains, each INT32
 *     partial converted to FP32 and added into the FP32 result with the scale
 *     2^(Ea+Eb): Sec. 4.2 (Algorithm 2, the FPROP loop) and Sec. 4.3.
 *   - 1-bit input shift, i.e. DFP15 tensors: Sec. 4.3.
 *
 * Readings where the paper is silent or garbled (all also listed in the
 * design notes):
 *   - E(.) in Eq. 1 is floor(log2 |.|), subnormals included.
 *   - bits P in {15, 16}; P = 15 (the paper's experimental DFP15) quantises
 *     directly with Es = Efmax - 13 (single rounding).
 *   - Es is an 8-bit signed integer (Sec. 3): clamped at -128.  An all-zero
 *     tensor gets Es = 0.  A tensor holding NaN or Inf gets all-zero integers,
 *     Es = 0 and the NONFINITE flag.
 *   - Rounding: NEAREST = ties to even, BIASED = ties toward +inf (round half
 *     up), STOCHASTIC = floor(x + u) with u = U / 2^32, U a Philox4x32-10 word,
 *     DOWN = floor (the bare shift of Eq. 6), offered as an extra mode.
 *   - P = 15 never saturates; P = 16 clamps to [-32767, 32767].
 *   - An INT32 partial that overflows wraps modulo 2^32 (two's complement).
 *   - A chunk is L consecutive indices of a canonical flat reduction order:
 *       fwd       t = (r*S + s)*C + c
 *       bwd-data  t = (r*S + s)*K + k
 *       bwd-wt    t = (n*P + p)*Q + q
 *     A tap that falls in the padding (or, for bwd-data, between strided
 *     rows/columns) contributes 0 but keeps its slot t.
 *   - FP32 accumulation is strictly sequential in chunk order; the scale
 *     2^(Ea+Eb) is applied once at the end with a single rounding.  bwd-wt
 *     sums chunks into segments of G chunks first (each sequential), then the
 *     segment sums sequentially.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_ROUND_NEAREST 0
#define ORC_ROUND_STOCHASTIC 1
#define ORC_ROUND_BIASED 2
#define ORC_ROUND_DOWN 3

#define ORC_FLAG_NONFINITE 1u
#define ORC_FLAG_EXP_CLAMPED 2u
#define ORC_FLAG_SATURATED 4u
#define ORC_FLAG_ZERO_TENSOR 8u
/* Stochastic-stream roles of the quantisers (the same numbering as the library's) */
#define ORC_ROLE_X 0u
#define ORC_ROLE_W 1u
#define ORC_ROLE_DY 2u
#define ORC_FLAG_OUTPUT_INF 16u

/* Convolution geometry, mirrored by a ctypes Structure on the Python side. */
typedef struct {
  int32_t n, c, h, w;  /* activations, NCHW */
  int32_t k, r, s;     /* filters, KCRS */
  int32_t stride_h, stride_w, pad_h, pad_w;
} orc_geom;

static int64_t out_p(const orc_geom *g) { return (g->h + 2 * g->pad_h - g->r) / g->stride_h + 1; }
static int64_t out_q(const orc_geom *g) { return (g->w + 2 * g->pad_w - g->s) / g->stride_w + 1; }

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as   */
/* easy as 1, 2, 3", SC'11).  Ten rounds; each round multiplies counter     */
/* words 0 and 2 by the two round multipliers, swaps and xors with the key; */
/* the key is bumped by the two Weyl constants between rounds.              */
/* ------------------------------------------------------------------------ */
void orc_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  const uint64_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += W0;
      k1 += W1;
    }
    uint64_t p0 = M0 * (uint64_t)c0;
    uint64_t p1 = M1 * (uint64_t)c2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    uint32_t n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The uniform word U used to round element idx of a tensor with the given role:
 * counter = (q mod 2^32, q div 2^32, role, 0) with q = idx div 4, key = seed,
 * U = word (idx mod 4) of the Philox output block. */
uint32_t orc_rng_word(uint64_t seed, uint32_t role, uint64_t idx) {
  uint64_t q = idx / 4;
  uint32_t ctr[4] = {(uint32_t)(q & 0xffffffffu), (uint32_t)(q >> 32), role, 0u};
  uint32_t key[2] = {(uint32_t)(seed & 0xffffffffu), (uint32_t)(seed >> 32)};
  uint32_t out[4];
  orc_philox4x32_10(ctr, key, out);
  return out[idx % 4];
}

/* ------------------------------------------------------------------------ */
/* Quantisation FP32 -> DFP-P (Eq. 1-3) and the rounding step.              */
/* ------------------------------------------------------------------------ */

/* Shared exponent from the max magnitude m (Eq. 1-2). Returns flags. */
static uint32_t shared_exponent(double m, int bits, int32_t *es_out) {
  if (m == 0.0) {
    *es_out = 0;
    return ORC_FLAG_ZERO_TENSOR;
  }
  int e2;
  frexp(m, &e2);          /* m = fr * 2^e2, fr in [0.5, 1)  */
  int efmax = e2 - 1;     /* Eq. 1: exponent of the max, floor(log2 m) */
  int es = efmax - (bits - 2); /* Eq. 2 */
  uint32_t flags = 0;
  if (es < -128) {
    es = -128;
    flags |= ORC_FLAG_EXP_CLAMPED;
  }
  *es_out = es;
  return flags;
}

/* Round one scaled value x = f * 2^-Es (exact in float64) to an integer.
 * X = floor(x * 2^32) is exact; its integer part fl = floor(x) and the
 * fraction word F = X - fl * 2^32 in [0, 2^32) decide the rounding. */
static int64_t round_scaled(double x, int rounding, uint32_t u) {
  double xs = ldexp(x, 32);
  double Xd = floor(xs);
  double fld = floor(x);
  int64_t X = (int64_t)Xd;
  int64_t fl = (int64_t)fld;
  int64_t F = X - fl * ((int64_t)1 << 32);
  int up = 0;
  const int64_t half = (int64_t)1 << 31;
  switch (rounding) {
    case ORC_ROUND_NEAREST:
      up = (F > half) || (F == half && (fl % 2 != 0));
      break;
    case ORC_ROUND_BIASED:
      up = (F >= half);
      break;
    case ORC_ROUND_STOCHASTIC:
      up = ((int64_t)u < F);
      break;
    case ORC_ROUND_DOWN:
    default:
      up = 0;
      break;
  }
  return fl + up;
}

/* Quantise n FP32 values to DFP-`bits` integers with one shared exponent.
 * Returns the flags word; writes the exponent and the integers. */
uint32_t orc_quantize(const float *src, int64_t n, int bits, int rounding, uint64_t seed,
                      uint32_t role, int16_t *dst, int32_t *es_out) {
  double m = 0.0;
  int nonfinite = 0;
  for (int64_t i = 0; i < n; ++i) {
    double a = fabs((double)src[i]);
    if (!isfinite(a)) nonfinite = 1;
    else if (a > m) m = a;
  }
  if (nonfinite) {
    memset(dst, 0, (size_t)n * sizeof(int16_t));
    *es_out = 0;
    return ORC_FLAG_NONFINITE;
  }
  int32_t es;
  uint32_t flags = shared_exponent(m, bits, &es);
  if (flags & ORC_FLAG_ZERO_TENSOR) {
    memset(dst, 0, (size_t)n * sizeof(int16_t));
    *es_out = 0;
    return flags;
  }
  const int64_t lim = (bits == 16) ? 32767 : ((int64_t)1 << (bits - 1));
  int saturated = 0;
#pragma omp parallel for schedule(static) reduction(| : saturated)
  for (int64_t i = 0; i < n; ++i) {
    double x = ldexp((double)src[i], -es); /* exact: 24-bit mantissa, power-of-two scale */
    uint32_t u = (rounding == ORC_ROUND_STOCHASTIC) ? orc_rng_word(seed, role, (uint64_t)i) : 0u;
    int64_t v = round_scaled(x, rounding, u);
    if (bits == 16) {
      if (v > lim) { v = lim; saturated = 1; }
      if (v < -lim) { v = -lim; saturated = 1; }
    }
    dst[i] = (int16_t)v;
  }
  if (saturated) flags |= ORC_FLAG_SATURATED;
  *es_out = es;
  return flags;
}

/* Integer down-conversion of a DFP-32 tensor <I, E> to DFP-`bits` (Eq. 6 with
 * the shift count read so that the max lands at bit P-2, the same place Eq. 2
 * puts it):  Rs = floor(log2 max|i|) - (P - 2), new exponent E + Rs, and the
 * integers rounded from i * 2^-Rs with the given mode (Rs may be negative: an
 * exact left shift).  Same exponent clamp and saturation rules as above. */
uint32_t orc_downconvert_i32(const int32_t *src, int64_t n, int32_t e_in, int bits, int rounding,
                             uint64_t seed, uint32_t role, int16_t *dst, int32_t *es_out) {
  int64_t mx = 0;
  for (int64_t i = 0; i < n; ++i) {
    int64_t a = src[i] < 0 ? -(int64_t)src[i] : (int64_t)src[i];
    if (a > mx) mx = a;
  }
  if (mx == 0) {
    memset(dst, 0, (size_t)n * sizeof(int16_t));
    *es_out = 0;
    return ORC_FLAG_ZERO_TENSOR;
  }
  int lz = 0; /* leading-zero count of max|i| in a 32-bit accumulator */
  while (lz < 32 && !((uint64_t)mx & ((uint64_t)1 << (31 - lz)))) ++lz;
  int top = 31 - lz; /* floor(log2 max|i|) */
  int rs = top - (bits - 2);
  int64_t enew = (int64_t)e_in + rs;
  uint32_t flags = 0;
  if (enew < -128) {
    rs += (int)(-128 - enew);
    enew = -128;
    flags |= ORC_FLAG_EXP_CLAMPED;
  }
  const int64_t lim = (bits == 16) ? 32767 : ((int64_t)1 << (bits - 1));
  int saturated = 0;
  for (int64_t i = 0; i < n; ++i) {
    double x = ldexp((double)src[i], -rs); /* exact: |i| < 2^31 */
    uint32_t u = (rounding == ORC_ROUND_STOCHASTIC) ? orc_rng_word(seed, role, (uint64_t)i) : 0u;
    int64_t v = round_scaled(x, rounding, u);
    if (bits == 16) {
      if (v > lim) { v = lim; saturated = 1; }
      if (v < -lim) { v = -lim; saturated = 1; }
    }
    dst[i] = (int16_t)v;
  }
  if (saturated) flags |= ORC_FLAG_SATURATED;
  *es_out = (int32_t)enew;
  return flags;
}

/* ------------------------------------------------------------------------ */
/* Convolutions: INT16 x INT16 products summed in INT32 over chunks of L     */
/* consecutive reduction indices, each chunk's partial converted to FP32 and */
/* added in chunk order, then scaled by 2^(Ea+Eb) (Alg. 2, Sec. 4.3, Eq. 4). */
/* ------------------------------------------------------------------------ */

/* Reduce an exact int64 sum modulo 2^32 into [-2^31, 2^31). */
static int64_t wrap32(int64_t v) {
  uint64_t u = (uint64_t)v & 0xffffffffull;
  return (u >= 0x80000000ull) ? (int64_t)u - ((int64_t)1 << 32) : (int64_t)u;
}

/* Scale an FP32 sum by 2^e with one rounding to FP32 (float64 holds S*2^e
 * exactly for every S and e that can occur here). */
static float scale_out(float s, int32_t e) { return (float)ldexp((double)s, e); }

/* Product term number t of output `o` for each direction; 0 for a padding tap
 * or a stride hole.  o is the flat logical output index. */
static int64_t fwd_term(const orc_geom *g, const int16_t *x, const int16_t *w, int64_t o, int64_t t) {
  int64_t P = out_p(g), Q = out_q(g);
  int64_t q = o % Q, p = (o / Q) % P, k = (o / (Q * P)) % g->k, n = o / (Q * P * g->k);
  int64_t c = t % g->c, s = (t / g->c) % g->s, r = t / ((int64_t)g->c * g->s);
  int64_t ih = p * g->stride_h - g->pad_h + r;
  int64_t iw = q * g->stride_w - g->pad_w + s;
  if (ih < 0 || ih >= g->h || iw < 0 || iw >= g->w) return 0;
  int64_t xv = x[((n * g->c + c) * g->h + ih) * g->w + iw];
  int64_t wv = w[((k * g->c + c) * g->r + r) * g->s + s];
  return xv * wv;
}

static int64_t bwd_data_term(const orc_geom *g, const int16_t *dy, const int16_t *w, int64_t o, int64_t t) {
  int64_t P = out_p(g), Q = out_q(g);
  int64_t iw = o % g->w, ih = (o / g->w) % g->h, c = (o / ((int64_t)g->w * g->h)) % g->c;
  int64_t n = o / ((int64_t)g->w * g->h * g->c);
  int64_t k = t % g->k, s = (t / g->k) % g->s, r = t / ((int64_t)g->k * g->s);
  int64_t nh = ih + g->pad_h - r, nw = iw + g->pad_w - s;
  if (nh < 0 || nw < 0 || nh % g->stride_h != 0 || nw % g->stride_w != 0) return 0;
  int64_t p = nh / g->stride_h, q = nw / g->stride_w;
  if (p >= P || q >= Q) return 0;
  int64_t dv = dy[((n * g->k + k) * P + p) * Q + q];
  int64_t wv = w[((k * g->c + c) * g->r + r) * g->s + s];
  return dv * wv;
}

static int64_t bwd_wt_term(const orc_geom *g, const int16_t *x, const int16_t *dy, int64_t o, int64_t t) {
  int64_t P = out_p(g), Q = out_q(g);
  int64_t s = o % g->s, r = (o / g->s) % g->r, c = (o / ((int64_t)g->s * g->r)) % g->c;
  int64_t k = o / ((int64_t)g->s * g->r * g->c);
  int64_t q = t % Q, p = (t / Q) % P, n = t / (Q * P);
  int64_t ih = p * g->stride_h - g->pad_h + r;
  int64_t iw = q * g->stride_w - g->pad_w + s;
  if (ih < 0 || ih >= g->h || iw < 0 || iw >= g->w) return 0;
  int64_t xv = x[((n * g->c + c) * g->h + ih) * g->w + iw];
  int64_t dv = dy[((n * g->k + k) * P + p) * Q + q];
  return xv * dv;
}

enum { DIR_FWD = 0, DIR_BWD_DATA = 1, DIR_BWD_WT = 2 };

static int64_t reduction_len(const orc_geom *g, int dir) {
  if (dir == DIR_FWD) return (int64_t)g->c * g->r * g->s;
  if (dir == DIR_BWD_DATA) return (int64_t)g->k * g->r * g->s;
  return (int64_t)g->n * out_p(g) * out_q(g);
}

static int64_t output_len(const orc_geom *g, int dir) {
  if (dir == DIR_FWD) return (int64_t)g->n * g->k * out_p(g) * out_q(g);
  if (dir == DIR_BWD_DATA) return (int64_t)g->n * g->c * g->h * g->w;
  return (int64_t)g->k * g->c * g->r * g->s;
}

int64_t orc_num_chunks(const orc_geom *g, int dir, int32_t L) {
  int64_t T = reduction_len(g, dir);
  return (T + L - 1) / L;
}

int64_t orc_output_len(const orc_geom *g, int dir) { return output_len(g, dir); }

int32_t orc_default_seg_chunks(int32_t L) { return (4096 / L) > 1 ? (4096 / L) : 1; }

/* One output element: chunk partials (optionally stored, stride `pstride`
 * between chunks), the FP32 sum in chunk order (two-level for bwd-wt) and the
 * final scaling.  Returns the number of chunks whose INT32 partial wrapped. */
static int64_t one_output(const orc_geom *g, int dir, const int16_t *a, const int16_t *b,
                          int32_t e, int32_t L, int32_t G, int64_t o, float *y_out,
                          int32_t *part, int64_t pstride) {
  int64_t T = reduction_len(g, dir);
  int64_t J = (T + L - 1) / L;
  int64_t overflow = 0;
  float total = 0.0f, seg = 0.0f;
  for (int64_t j = 0; j < J; ++j) {
    int64_t exact = 0;
    int64_t t_end = (j + 1) * (int64_t)L < T ? (j + 1) * (int64_t)L : T;
    for (int64_t t = j * (int64_t)L; t < t_end; ++t) {
      if (dir == DIR_FWD) exact += fwd_term(g, a, b, o, t);
      else if (dir == DIR_BWD_DATA) exact += bwd_data_term(g, a, b, o, t);
      else exact += bwd_wt_term(g, a, b, o, t);
    }
    int64_t pj = wrap32(exact);
    if (pj != exact) ++overflow;
    if (part) part[j * pstride] = (int32_t)pj;
    float fj = (float)pj; /* IEEE round-to-nearest-even */
    if (dir == DIR_BWD_WT) {
      /* segment g = j / G: sequential inside the segment ... */
      seg = (j % G == 0) ? fj : seg + fj;
      if (j % G == G - 1 || j == J - 1) {
        /* ... then the segment sums, sequential over g */
        total = (j / G == 0) ? seg : total + seg;
      }
    } else {
      total = (j == 0) ? fj : total + fj;
    }
  }
  *y_out = scale_out(total, e);
  return overflow;
}

/* Full convolution in one direction.  a, b are the two INT16 operands:
 *   fwd:      a = x  [N,C,H,W], b = w  [K,C,R,S] -> y  [N,K,P,Q]
 *   bwd-data: a = dy [N,K,P,Q], b = w  [K,C,R,S] -> dx [N,C,H,W]
 *   bwd-wt:   a = x  [N,C,H,W], b = dy [N,K,P,Q] -> dw [K,C,R,S]
 * e = Ea + Eb.  partials (nullable) is [J][outputs].  G is the bwd-wt segment
 * size in chunks (0 = default).  Returns the number of wrapped partials. */
int64_t orc_conv(const orc_geom *g, int dir, const int16_t *a, const int16_t *b, int32_t e,
                 int32_t L, int32_t G, float *out, int32_t *partials) {
  int64_t O = output_len(g, dir);
  if (G <= 0) G = orc_default_seg_chunks(L);
  int64_t overflow = 0;
#pragma omp parallel for schedule(dynamic, 64) reduction(+ : overflow)
  for (int64_t o = 0; o < O; ++o) {
    overflow += one_output(g, dir, a, b, e, L, G, o, &out[o], partials ? &partials[o] : NULL, O);
  }
  return overflow;
}

/* The same computation at a list of output indices only.  out[i] and
 * partials[i*J + j] (nullable) belong to output idx[i]. */
int64_t orc_conv_at(const orc_geom *g, int dir, const int16_t *a, const int16_t *b, int32_t e,
                    int32_t L, int32_t G, const int64_t *idx, int64_t count, float *out,
                    int32_t *partials) {
  if (G <= 0) G = orc_default_seg_chunks(L);
  int64_t J = orc_num_chunks(g, dir, L);
  int64_t overflow = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(+ : overflow)
  for (int64_t i = 0; i < count; ++i) {
    overflow += one_output(g, dir, a, b, e, L, G, idx[i], &out[i], partials ? &partials[i * J] : NULL, 1);
  }
  return overflow;
}

/* Flags a finished FP32 output would carry: Inf after scaling. */
uint32_t orc_output_flags(const float *y, int64_t n) {
  for (int64_t i = 0; i < n; ++i)
    if (isinf(y[i])) return ORC_FLAG_OUTPUT_INF;
  return 0;
}

/* ------------------------------------------------------------------------ */
/* GEMM (the paper applies the same INT16 kernels to "convolutions and GEMM",
 * Sec. 4): D[i][j] = sum over t of opA[i][t] * opB[t][j], t in [0, k), with
 * the forward convolution's contract (Alg. 2, Sec. 4.3): INT32 partials over
 * chunks of L consecutive t (mod 2^32), converted to FP32 and added in chunk
 * order, scaled once by 2^e.  opA[i][t] = a[i*k + t] (trans_a = 0) or
 * a[t*m + i] (trans_a = 1); opB[t][j] = b[t*n + j] (trans_b = 0) or
 * b[j*k + t] (trans_b = 1).  D is row-major [m][n]; partials (nullable) is
 * [J][m*n].  Returns the number of wrapped partials. */
/* ------------------------------------------------------------------------ */
int64_t orc_gemm(int64_t m, int64_t n, int64_t k, int trans_a, int trans_b, const int16_t *a,
                 const int16_t *b, int32_t e, int32_t L, float *out, int32_t *partials) {
  int64_t J = (k + L - 1) / L;
  int64_t overflow = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(+ : overflow)
  for (int64_t o = 0; o < m * n; ++o) {
    int64_t i = o / n, j = o % n;
    float total = 0.0f;
    for (int64_t c = 0; c < J; ++c) {
      int64_t exact = 0;
      int64_t t_end = (c + 1) * (int64_t)L < k ? (c + 1) * (int64_t)L : k;
      for (int64_t t = c * (int64_t)L; t < t_end; ++t) {
        int64_t av = trans_a ? a[t * m + i] : a[i * k + t];
        int64_t bv = trans_b ? b[j * k + t] : b[t * n + j];
        exact += av * bv;
      }
      int64_t pc = wrap32(exact);
      if (pc != exact) ++overflow;
      if (partials) partials[c * m * n + o] = (int32_t)pc;
      float fc = (float)pc;
      total = (c == 0) ? fc : total + fc;
    }
    out[o] = scale_out(total, e);
  }
  return overflow;
}

/* ------------------------------------------------------------------------ */
/* Blocked-DFP (Sec. 3: several exponents per tensor, each shared by a small  */
/* block of integers).  A [rows][cols] tensor is split along cols into blocks */
/* of B consecutive elements (the last one per row possibly shorter); every   */
/* block is quantised like a tensor of its own (Eq. 1-3, same clamp, zero and */
/* non-finite rules), the stochastic word of an element still taken from its  */
/* flat index in the whole tensor.  exps is [nb][rows] (block-major), nb =    */
/* ceil(cols / B).  Returned flags: NONFINITE, EXP_CLAMPED, SATURATED if any  */
/* block has them; ZERO_TENSOR only if every block is zero.                   */
/* ------------------------------------------------------------------------ */
uint32_t orc_quantize_blocked(const float *src, int64_t rows, int64_t cols, int64_t B, int bits, int rounding,
                              uint64_t seed, uint32_t role, int16_t *dst, int8_t *exps) {
  const int64_t nb = (cols + B - 1) / B;
  const int64_t lim = (bits == 16) ? 32767 : ((int64_t)1 << (bits - 1));
  uint32_t any = 0;
  int all_zero = 1;
#pragma omp parallel for schedule(static) reduction(| : any) reduction(& : all_zero)
  for (int64_t rb = 0; rb < rows * nb; ++rb) {
    const int64_t r = rb / nb, b = rb % nb;
    const int64_t c0 = b * B, c1 = (c0 + B < cols) ? c0 + B : cols;
    const int64_t base = r * cols;
    double m = 0.0;
    int nonfinite = 0;
    for (int64_t c = c0; c < c1; ++c) {
      double a = fabs((double)src[base + c]);
      if (!isfinite(a)) nonfinite = 1;
      else if (a > m) m = a;
    }
    int32_t es = 0;
    uint32_t f = 0;
    if (nonfinite) {
      f = ORC_FLAG_NONFINITE;
      all_zero = 0; /* a non-finite block is not a zero block */
    } else {
      f = shared_exponent(m, bits, &es);
    }
    if (nonfinite || (f & ORC_FLAG_ZERO_TENSOR)) {
      for (int64_t c = c0; c < c1; ++c) dst[base + c] = 0;
      es = 0;
    } else {
      all_zero = 0;
      for (int64_t c = c0; c < c1; ++c) {
        const int64_t idx = base + c;
        double x = ldexp((double)src[idx], -es);
        uint32_t u = (rounding == ORC_ROUND_STOCHASTIC) ? orc_rng_word(seed, role, (uint64_t)idx) : 0u;
        int64_t v = round_scaled(x, rounding, u);
        if (bits == 16) {
          if (v > lim) { v = lim; f |= ORC_FLAG_SATURATED; }
          if (v < -lim) { v = -lim; f |= ORC_FLAG_SATURATED; }
        }
        dst[idx] = (int16_t)v;
      }
    }
    exps[b * rows + r] = (int8_t)es;
    any |= f & (ORC_FLAG_NONFINITE | ORC_FLAG_EXP_CLAMPED | ORC_FLAG_SATURATED);
  }
  return any | (all_zero ? ORC_FLAG_ZERO_TENSOR : 0u);
}

/* Blocked-DFP GEMM: D[i][j] = sum over t of a[i][t] * b[j][t] (both stored
 * with t contiguous), exponents ea [nb][m] and eb [nb][n] per block of Bk
 * consecutive t.  Chunks of L (Bk a multiple of L) lie inside one block; each
 * chunk's INT32 partial (mod 2^32) is converted to FP32, scaled by
 * 2^(ea[blk][i] + eb[blk][j]) and added to the FP32 sum in chunk order (the
 * per-chunk scaling of Alg. 2).  partials (nullable): [J][m*n]. */
int64_t orc_gemm_blocked(int64_t m, int64_t n, int64_t k, const int16_t *a, const int8_t *ea, const int16_t *b,
                         const int8_t *eb, int64_t Bk, int32_t L, float *out, int32_t *partials) {
  const int64_t J = (k + L - 1) / L;
  int64_t overflow = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(+ : overflow)
  for (int64_t o = 0; o < m * n; ++o) {
    const int64_t i = o / n, j = o % n;
    float total = 0.0f;
    for (int64_t c = 0; c < J; ++c) {
      const int64_t t0 = c * (int64_t)L, t1 = (t0 + L < k) ? t0 + L : k;
      int64_t exact = 0;
      for (int64_t t = t0; t < t1; ++t) exact += (int64_t)a[i * k + t] * (int64_t)b[j * k + t];
      const int64_t pc = wrap32(exact);
      if (pc != exact) ++overflow;
      if (partials) partials[c * m * n + o] = (int32_t)pc;
      const int64_t blk = t0 / Bk;
      const float term = scale_out((float)pc, (int32_t)ea[blk * m + i] + (int32_t)eb[blk * n + j]);
      total = (c == 0) ? term : total + term;
    }
    out[o] = total;
  }
  return overflow;
}

/* ------------------------------------------------------------------------ */
/* One layer's steps either side of the convolutions (Sec. 4.1, Fig. 2).     */
/* Batch normalisation reads DFP16 tensors and up-converts them; with the    */
/* integers I and exponent E of a channel's n = N*H*W elements the sums     */
/* S1 = sum I, S2 = sum I^2 (and in the backward pass D = sum g, P = sum g*I */
/* over the ReLU-masked gradient integers g) are exact in 64-bit integers,  */
/* so the statistics need no FP32 accumulation at all.  Per-channel values  */
/* are computed in float64 and rounded once to FP32; per-element work is    */
/* FP32 with the stated operation order (fmaf = fused multiply-add).         */
/* ------------------------------------------------------------------------ */

/* Per-channel statistics of a DFP16 tensor [N][C][HW]. */
static void bn_channel_stats(const int16_t *y, int64_t N, int64_t C, int64_t HW, int64_t c, int64_t *s1,
                             int64_t *s2) {
  int64_t a = 0, b = 0;
  for (int64_t n = 0; n < N; ++n)
    for (int64_t i = 0; i < HW; ++i) {
      int64_t v = y[(n * C + c) * HW + i];
      a += v;
      b += v * v;
    }
  *s1 = a;
  *s2 = b;
}

/* mean = S1 2^E / n, var = S2 2^2E / n - mean^2 (biased, clamped at 0), both
 * in float64; mean_f = fl32(mean), inv_std = 1 / sqrt(fl32(var) + eps) in FP32. */
static void bn_mean_inv_std(int64_t s1, int64_t s2, int32_t e, int64_t cnt, float eps, float *mean_f,
                            float *inv_std_f) {
  double mean = ldexp((double)s1, e) / (double)cnt;
  double var = ldexp((double)s2, 2 * e) / (double)cnt - mean * mean;
  if (var < 0.0) var = 0.0;
  *mean_f = (float)mean;
  float vf = (float)var;
  *inv_std_f = 1.0f / sqrtf(vf + eps);
}

/* BN + (residual add) + ReLU forward of one element. */
static float bn_relu_elem(int16_t yi, int32_t e, float mean_f, float inv_std_f, float g, float b, const float *res,
                          int64_t idx, float *pre) {
  float yv = ldexpf((float)yi, e);          /* exact: |yi| < 2^15 */
  float xh = (yv - mean_f) * inv_std_f;
  float zp = fmaf(xh, g, b);
  if (res) zp = zp + res[idx];
  if (pre) *pre = zp;
  return zp > 0.0f ? zp : 0.0f;
}

/* Forward: z = ReLU(gamma * xhat + beta [+ res]) in FP32, then Q_a of z (the
 * next layer's activation, role X).  Outputs: z (nullable), zq, its exponent
 * and flags, per-channel mean_f, inv_std_f and the sums [C][2] = S1, S2. */
uint32_t orc_bn_relu_fwd(const int16_t *y, int32_t ey, int64_t N, int64_t C, int64_t HW, const float *gamma,
                         const float *beta, const float *res, float eps, int bits, int rounding, uint64_t seed,
                         float *z, int16_t *zq, int32_t *ez, float *mean_f, float *inv_std_f, int64_t *sums) {
  const int64_t cnt = N * HW, total = N * C * HW;
  float *zz = z ? z : (float *)malloc((size_t)total * sizeof(float));
  for (int64_t c = 0; c < C; ++c) {
    int64_t s1, s2;
    bn_channel_stats(y, N, C, HW, c, &s1, &s2);
    sums[2 * c] = s1;
    sums[2 * c + 1] = s2;
    bn_mean_inv_std(s1, s2, ey, cnt, eps, &mean_f[c], &inv_std_f[c]);
  }
#pragma omp parallel for schedule(static)
  for (int64_t idx = 0; idx < total; ++idx) {
    int64_t c = (idx / HW) % C;
    zz[idx] = bn_relu_elem(y[idx], ey, mean_f[c], inv_std_f[c], gamma[c], beta[c], res, idx, NULL);
  }
  uint32_t flags = orc_quantize(zz, total, bits, rounding, seed, ORC_ROLE_X, zq, ez);
  if (!z) free(zz);
  return flags;
}

/* Backward: dz' = mask * dz (mask: pre-activation > 0, recomputed), dbeta =
 * sum dz', dgamma = sum dz' * xhat taken exactly as inv_std * 2^Edz *
 * (P 2^Ey - mean_f D); a = gamma * inv_std, k1 = fl32(a), k2 = fl32(-a dgamma
 * / n), k3 = fl32(-a dbeta / n) (float64, dgamma and dbeta as FP32);
 * dy = fmaf(k1, dz', fmaf(k2, xhat, k3)) in FP32, then Q_e of dy (role DY).
 * dres (nullable) = dz'.  sums [C][2] = D, P. */
uint32_t orc_bn_relu_bwd(const int16_t *dz, int32_t edz, const int16_t *y, int32_t ey, int64_t N, int64_t C,
                         int64_t HW, const float *gamma, const float *beta, const float *res, const float *mean_f,
                         const float *inv_std_f, int bits, int rounding, uint64_t seed, float *dy, int16_t *dyq,
                         int32_t *edy, float *dgamma, float *dbeta, float *dres, int64_t *sums) {
  const int64_t cnt = N * HW, total = N * C * HW;
  float *dd = dy ? dy : (float *)malloc((size_t)total * sizeof(float));
  float *k = (float *)malloc((size_t)C * 3 * sizeof(float));
#pragma omp parallel for schedule(static)
  for (int64_t c = 0; c < C; ++c) {
    int64_t D = 0, P = 0;
    for (int64_t n = 0; n < N; ++n)
      for (int64_t i = 0; i < HW; ++i) {
        int64_t idx = (n * C + c) * HW + i;
        float pre;
        bn_relu_elem(y[idx], ey, mean_f[c], inv_std_f[c], gamma[c], beta[c], res, idx, &pre);
        int64_t g = pre > 0.0f ? dz[idx] : 0;
        D += g;
        P += g * (int64_t)y[idx];
      }
    sums[2 * c] = D;
    sums[2 * c + 1] = P;
    double db = ldexp((double)D, edz);
    double dg = (double)inv_std_f[c] * ldexp(ldexp((double)P, ey) - (double)mean_f[c] * (double)D, edz);
    dbeta[c] = (float)db;
    dgamma[c] = (float)dg;
    double a = (double)gamma[c] * (double)inv_std_f[c];
    k[3 * c] = (float)a;
    k[3 * c + 1] = (float)(-a * (double)dgamma[c] / (double)cnt);
    k[3 * c + 2] = (float)(-a * (double)dbeta[c] / (double)cnt);
  }
#pragma omp parallel for schedule(static)
  for (int64_t idx = 0; idx < total; ++idx) {
    int64_t c = (idx / HW) % C;
    float pre;
    float yv = ldexpf((float)y[idx], ey);
    float xh = (yv - mean_f[c]) * inv_std_f[c];
    bn_relu_elem(y[idx], ey, mean_f[c], inv_std_f[c], gamma[c], beta[c], res, idx, &pre);
    float dzv = pre > 0.0f ? ldexpf((float)dz[idx], edz) : 0.0f;
    dd[idx] = fmaf(k[3 * c], dzv, fmaf(k[3 * c + 1], xh, k[3 * c + 2]));
    if (dres) dres[idx] = dzv;
  }
  uint32_t flags = orc_quantize(dd, total, bits, rounding, seed, ORC_ROLE_DY, dyq, edy);
  free(k);
  if (!dy) free(dd);
  return flags;
}

/* FP32 SGD with momentum and weight decay on master weights (Fig. 2: the
 * weight gradient is not quantised): g = fmaf(wd, w, dw), v = fmaf(mu, v, g),
 * w = fmaf(-lr, v, w); then Q_w of the new weights (role W). */
uint32_t orc_sgd_quantize(int64_t n, float *w, float *v, const float *dw, float lr, float mu, float wd, int bits,
                          int rounding, uint64_t seed, int16_t *wq, int32_t *ew) {
  for (int64_t i = 0; i < n; ++i) {
    float g = fmaf(wd, w[i], dw[i]);
    v[i] = fmaf(mu, v[i], g);
    w[i] = fmaf(-lr, v[i], w[i]);
  }
  return orc_quantize(w, n, bits, rounding, seed, ORC_ROLE_W, wq, ew);
}
