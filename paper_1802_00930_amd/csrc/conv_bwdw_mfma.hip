// MFMA product path for the backward-weights convolution (WU, Sec. 4.1):
//   dW[k][(c,r,s)] = sum over t = (n*P + p)*Q + q of
//                    dy[n,k,p,q] * x[n, c, p*sh - ph + r, q*sw - pw + s].
// The reduction runs over every output position of the batch (chains beyond a
// million products, Sec. 4.3), so it is split into segments of G chunks that
// run in parallel; each workgroup adds its segment's chunk partials in chunk
// order (FP32) and a second kernel adds the segment sums in segment order, so
// the result does not depend on scheduling.
//
// Operands (same byte-digit split as the forward path, see conv_mfma.hip):
//   A = dy digits blocked by 32 reduction indices, [kb][k][half][32 B],
//       written by a prep kernel in canonical t order;
//   B = x digits as (lo | hi << 8) 16-bit pairs in a zero-padded,
//       channel-major layout XP[c][n*Hpad + row][col] (Hpad = H + 2 ph,
//       row width padded to 8 pairs), also written by a prep kernel.
// For every block of 128 reduction indices a workgroup copies, for each input
// channel its 128 columns touch, the contiguous band of padded rows those
// indices read into LDS, plus a table of each index's row/column offset in
// that band.  A lane owning column (c, r, s) then gathers its 16 operand pairs
// as band[c][offset(t) + r*Wpad + s], which covers padding, strides and image
// boundaries with no branches.
#include <type_traits>

#include "conv_bwdw_mfma.h"

namespace dfp {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kMT = 64;    // output rows (k) per workgroup
constexpr int kNT = 128;   // output columns (c, r, s) per workgroup
constexpr int kSBT = 128;  // reduction indices staged per LDS band

__device__ __forceinline__ uint32_t hi_digit(int32_t a) { return (uint32_t)((a + 128) >> 8) & 0xffu; }
__device__ __forceinline__ uint32_t lo_digit(int32_t a) { return (uint32_t)a & 0xffu; }

// A digits from dy in canonical order: Ad[kb][m][half][16 hi | 16 lo].
// One thread per (kb, m, half), written in that order so a wave's stores are
// contiguous; each thread reads 16 consecutive reduction indices of one plane,
// as two 16-byte loads when they lie in one image and are aligned.  Every
// index fits 32 bits (dy has fewer than 2^31 elements).
struct DyPrep {
  const int16_t* dy;
  uint8_t* ad;
  int32_t K, Mp, PQ, T, KBT;
};
__device__ __forceinline__ void prep_dy_item(const DyPrep& q, int32_t idx) {
  const int16_t* __restrict__ dy = q.dy;
  const int32_t K = q.K, Mp = q.Mp, PQ = q.PQ, T = q.T;
  if (idx >= q.KBT * Mp * 2) return;
  const int32_t half = idx & 1;
  const int32_t m = (idx >> 1) % Mp;
  const int32_t kb = (idx >> 1) / Mp;
  uint32_t hi[4] = {0u, 0u, 0u, 0u}, lo[4] = {0u, 0u, 0u, 0u};
  if (m < K) {
    const int32_t t0 = kb * 32 + half * 16;
    int32_t n = t0 / PQ, pq = t0 - n * PQ;
    const int32_t off = (n * K + m) * PQ + pq;
    if (t0 + 16 <= T && pq + 16 <= PQ && (reinterpret_cast<uintptr_t>(dy + off) & 15) == 0) {
      const uint4* src = reinterpret_cast<const uint4*>(dy + off);
      const uint4 v0 = src[0], v1 = src[1];
      const uint32_t wv[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int32_t v = (int32_t)(int16_t)(wv[i >> 1] >> (16 * (i & 1)));
        hi[i >> 2] |= hi_digit(v) << (8 * (i & 3));
        lo[i >> 2] |= lo_digit(v) << (8 * (i & 3));
      }
    } else {
      int32_t t = t0;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        int32_t v = 0;
        if (t < T) v = dy[(n * K + m) * PQ + pq];
        hi[i >> 2] |= hi_digit(v) << (8 * (i & 3));
        lo[i >> 2] |= lo_digit(v) << (8 * (i & 3));
        ++t;
        if (++pq == PQ) { pq = 0; ++n; }
      }
    }
  }
  uint4* dst = reinterpret_cast<uint4*>(q.ad + (int64_t)idx * 32);
  dst[0] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
  dst[1] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
}
__global__ __launch_bounds__(256) void k_prep_dy(DyPrep q) { prep_dy_item(q, blockIdx.x * 256 + threadIdx.x); }

// XP[c][n*Hpad + u][v] = (lo | hi << 8) of x[n][c][u - ph][v - pw], zero outside.
// Grid (rows of channel c, c): one thread per 8 consecutive pairs of a row
// (Wpad is a multiple of 8), one 16-byte store; consecutive threads read
// consecutive pieces of a source row.
__global__ __launch_bounds__(256) void k_prep_xp(const int16_t* __restrict__ x, uint16_t* __restrict__ xp, int32_t N,
                                                int32_t C, int32_t H, int32_t W, int32_t Hpad, int32_t Wpad,
                                                int32_t ph, int32_t pw) {
  const int32_t c = blockIdx.y;
  const int32_t i = blockIdx.x * 256 + threadIdx.x;  // (n * Hpad + u) * W8 + v8
  const int32_t W8 = Wpad >> 3;
  if (i >= N * Hpad * W8) return;
  const int32_t r = i / W8, v0 = (i - r * W8) * 8;
  const int32_t n = r / Hpad, u = r - n * Hpad;
  const int32_t ih = u - ph;
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  if (ih >= 0 && ih < H) {
    const int16_t* row = x + ((int64_t)(n * C + c) * H + ih) * W;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int32_t iw = v0 + k - pw;
      if (iw >= 0 && iw < W) {
        const int32_t a = row[iw];
        w[k >> 1] |= (lo_digit(a) | (hi_digit(a) << 8)) << (16 * (k & 1));
      }
    }
  }
  reinterpret_cast<uint4*>(xp + ((int64_t)c * N * Hpad * Wpad))[i] = make_uint4(w[0], w[1], w[2], w[3]);
}

// Same layout for rows of a multiple of 8 elements, 16-byte aligned, and a
// column pad PW below 4: each lane loads the two aligned 8-element groups
// around its window (zero outside the row) and takes elements 8-PW .. 15-PW.
template <int PW>
__global__ __launch_bounds__(256) void k_prep_xp_vec(const int16_t* __restrict__ x, uint16_t* __restrict__ xp,
                                                    int32_t N, int32_t C, int32_t H, int32_t W, int32_t Hpad,
                                                    int32_t Wpad, int32_t ph) {
  const int32_t c = blockIdx.y;
  const int32_t i = blockIdx.x * 256 + threadIdx.x;  // (n * Hpad + u) * W8 + v8
  const int32_t W8 = Wpad >> 3;
  if (i >= N * Hpad * W8) return;
  const int32_t r = i / W8, v0 = (i - r * W8) * 8;
  const int32_t n = r / Hpad, u = r - n * Hpad;
  const int32_t ih = u - ph;
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  if (ih >= 0 && ih < H) {
    const int16_t* row = x + ((int64_t)(n * C + c) * H + ih) * W;
    uint32_t g[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};  // elements v0-8 .. v0+7
    if (PW > 0 && v0 >= 8 && v0 - 8 < W) {
      const uint4 q = *reinterpret_cast<const uint4*>(row + v0 - 8);
      g[0] = q.x; g[1] = q.y; g[2] = q.z; g[3] = q.w;
    }
    if (v0 < W) {
      const uint4 q = *reinterpret_cast<const uint4*>(row + v0);
      g[4] = q.x; g[5] = q.y; g[6] = q.z; g[7] = q.w;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int e = 8 - PW + k;
      const int32_t a = (int32_t)(int16_t)(g[e >> 1] >> (16 * (e & 1)));
      w[k >> 1] |= (lo_digit(a) | (hi_digit(a) << 8)) << (16 * (k & 1));
    }
  }
  reinterpret_cast<uint4*>(xp + ((int64_t)c * N * Hpad * Wpad))[i] = make_uint4(w[0], w[1], w[2], w[3]);
}

// Byte mask keeping bytes [lo, hi) of a 16-byte operand.
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

// ((a << 8) + b) << 8) + c as two v_lshl_add_u32.  The shift-adds are plain
// C so the compiler's hazard checks see every read of an MFMA result; the
// empty asm only stops the re-association into shift, shift, add3.
__device__ __forceinline__ uint32_t recombine(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t t = (a << 8) + b;
  asm("" : "+v"(t));
  return (t << 8) + c;
}

// Chunk end: P_j recombined, converted (round to nearest even), added in order.
template <bool PARTIALS>
__device__ __forceinline__ void flush_tile(const Acc3& acc, float (&sum)[16], int64_t j, int32_t* partials,
                                           int64_t O, int64_t col, int64_t CRS, int32_t mrow0, int32_t M,
                                           bool cvalid) {
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const uint32_t p = recombine((uint32_t)acc.hh[v], (uint32_t)acc.xx[v], (uint32_t)acc.ll[v]);
    sum[v] += (float)(int32_t)p;
    if (PARTIALS) {
      const int32_t m = mrow0 + 8 * (v >> 2) + (v & 3);
      if (cvalid && m < M) partials[j * O + (int64_t)m * CRS + col] = (int32_t)p;
    }
  }
}

// Workgroup -> (column tile, row tile, segment).  Workgroup ids are dealt to
// the 8 XCDs in turn (id mod 8), each with its own L2.  The (segment, tile)
// list, segment-major, is cut into 8 contiguous ranges, one per XCD, so the
// tiles of a segment run on one XCD (except where a range ends) and its dy
// digits are fetched into that L2 once for all column tiles.  1-D grid of
// nseg * ntx * nty workgroups.
struct BwdwTile {
  int32_t tx, ty, seg;
};
__device__ __forceinline__ BwdwTile bwdw_tile(const BwdwArgs& a) {
  const int32_t per = a.ntx * a.nty;
  const int32_t W = gridDim.x, b = blockIdx.x, x = b & 7;
  const int32_t l = x * (W >> 3) + min(x, W & 7) + (b >> 3);
  const int32_t seg = l / per, t = l - seg * per;
  return {t % a.ntx, t / a.ntx, seg};
}

template <bool MASKED, bool PARTIALS>
__global__ __launch_bounds__(kThreads, 2) void k_bwdw_mfma(BwdwArgs a) {
  const BwdwTile tl = bwdw_tile(a);
  if (tl.seg >= a.nseg) return;
  extern __shared__ __align__(16) uint8_t smem[];
  uint16_t* band = reinterpret_cast<uint16_t*>(smem);                        // [nch][rows][Wpad]
  int32_t* toff = reinterpret_cast<int32_t*>(smem + a.band_bytes);           // [kSBT]

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int half = lane >> 5;
  const int lc = lane & 31;
  const int32_t RS = a.R * a.S;
  const int64_t CRS = (int64_t)a.C * RS;
  const int64_t col0 = (int64_t)tl.tx * kNT;
  const int64_t col = col0 + wave * 32 + lc;
  const bool cvalid = col < CRS;
  const int64_t colc = cvalid ? col : col0;
  const int32_t c = (int32_t)(colc / RS), rr = (int32_t)((colc % RS) / a.S), ss = (int32_t)(colc % a.S);
  const int32_t c_lo = (int32_t)(col0 / RS);
  const int32_t c_hi = (int32_t)(min(col0 + kNT - 1, CRS - 1) / RS);
  const int32_t nch = c_hi - c_lo + 1;
  const int32_t m0 = tl.ty * kMT;

  // reduction range of this segment
  const int64_t g = tl.seg;
  const int64_t t_seg0 = g * (int64_t)a.G * a.L;
  const int64_t t_seg1 = min(t_seg0 + (int64_t)a.G * a.L, a.T);
  int64_t j = g * (int64_t)a.G;  // first chunk of the segment

  Acc3 acc[2];
  float sum[2][16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      acc[i].hh[v] = 0; acc[i].xx[v] = 0; acc[i].ll[v] = 0;
      sum[i][v] = 0.f;
    }

  const uint8_t* apix = a.ad + ((int64_t)(m0 + lc) * 2 + half) * 32;
  const int64_t a_block_bytes = (int64_t)a.Mp * 64;
  const int32_t Wpad = a.Wpad;
  const int32_t PQ = a.P * a.Q;
  int32_t blk_in_chunk = 0;
  const int32_t chunk_blocks = a.L / 32;

  // first K-block touching the segment, and the block after its last index
  const int64_t kb_begin = t_seg0 / 32;
  const int64_t kb_end = (t_seg1 + 31) / 32;
  for (int64_t sb = kb_begin; sb < kb_end; sb += kSBT / 32) {
    const int64_t sb_end = min(sb + kSBT / 32, kb_end);
    const int64_t t_a = max(sb * 32, t_seg0);
    const int64_t t_b = min(sb_end * 32, t_seg1) - 1;  // last index of the band
    // padded-row span of the band
    const int64_t na = t_a / PQ, pa = (t_a % PQ) / a.Q;
    const int64_t nb = t_b / PQ, pb = (t_b % PQ) / a.Q;
    const int64_t z_a = na * a.Hpad + pa * a.sh;
    const int64_t z_b = nb * a.Hpad + pb * a.sh + a.R - 1;
    const int32_t rows = (int32_t)(z_b - z_a + 1);
    __syncthreads();  // previous band fully consumed
    // offset table: t -> (z(t) - z_a) * Wpad + q * sw, for the band's 128 indices
    if (threadIdx.x < kSBT) {
      const int64_t t = sb * 32 + threadIdx.x;
      int32_t off = 0;
      if (t >= t_a && t <= t_b) {
        const int64_t n = t / PQ, pq = t % PQ;
        const int64_t p = pq / a.Q, q = pq % a.Q;
        off = (int32_t)((n * a.Hpad + p * a.sh - z_a) * Wpad + q * a.sw);
      }
      toff[threadIdx.x] = off;
    }
    // band copy: for each channel, rows [z_a, z_a + rows) of XP are contiguous
    {
      const int32_t vec_per_row = Wpad / 8;  // 16-byte vectors
      const int32_t vec_per_ch = rows * vec_per_row;
      const int32_t total = nch * vec_per_ch;
      for (int32_t i = threadIdx.x; i < total; i += kThreads) {
        const int32_t cc = i / vec_per_ch, rem = i % vec_per_ch;
        const uint4* src = reinterpret_cast<const uint4*>(
            a.xp + (((int64_t)(c_lo + cc) * a.NH + z_a) * Wpad)) + rem;
        reinterpret_cast<uint4*>(band + (int64_t)cc * a.band_ch_stride)[rem] = *src;
      }
    }
    __syncthreads();
    const int32_t lane_base = (c - c_lo) * a.band_ch_stride + rr * Wpad + ss;
    for (int64_t kb = sb; kb < sb_end; ++kb) {
      // ---- B: 16 (lo, hi) pairs of column (c, r, s)
      const int32_t tb = (int32_t)(kb - sb) * 32 + half * 16;
      uint32_t pr[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t p0 = band[lane_base + toff[tb + 2 * i]];
        const uint32_t p1 = band[lane_base + toff[tb + 2 * i + 1]];
        pr[i] = p0 | (p1 << 16);
      }
      v4i bhi, blo;
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        blo[d] = (int)__builtin_amdgcn_perm(pr[2 * d + 1], pr[2 * d], 0x06040200u);
        bhi[d] = (int)__builtin_amdgcn_perm(pr[2 * d + 1], pr[2 * d], 0x07050301u);
      }
      // indices of this block outside the segment (or past T) contribute 0
      const int64_t t0 = kb * 32 + half * 16;
      {
        const int32_t lo_i = (int32_t)min(max(t_seg0 - t0, (int64_t)0), (int64_t)16);
        const int32_t hi_i = (int32_t)min(max(t_seg1 - t0, (int64_t)0), (int64_t)16);
        if (lo_i != 0 || hi_i != 16) {
          const v4i mk = byte_mask16(lo_i, hi_i);
          bhi &= mk;
          blo &= mk;
        }
      }
      // ---- A: two 32-row tiles of dy digits
      v4i ahi[2], alo[2];
      const uint8_t* ap = apix + kb * a_block_bytes;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const uint4* src = reinterpret_cast<const uint4*>(ap + i * 2048);
        const uint4 h4 = src[0], l4 = src[1];
        ahi[i] = (v4i){(int)h4.x, (int)h4.y, (int)h4.z, (int)h4.w};
        alo[i] = (v4i){(int)l4.x, (int)l4.y, (int)l4.z, (int)l4.w};
      }
      if (!MASKED) {
        const bool fresh = blk_in_chunk == 0;
#pragma unroll
        for (int i = 0; i < 2; ++i) mfma_tile(acc[i], ahi[i], alo[i], bhi, blo, fresh);
        ++blk_in_chunk;
        if (blk_in_chunk == chunk_blocks || kb == kb_end - 1) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
            flush_tile<PARTIALS>(acc[i], sum[i], j, a.partials, a.O, colc, CRS, m0 + 32 * i + 4 * half, a.K,
                                 cvalid);
          ++j;
          blk_in_chunk = 0;
        }
      } else {
        const int64_t t_lo = max(kb * 32, t_seg0), t_hi = min(kb * 32 + 32, t_seg1);
        while (true) {
          const int64_t cs = j * (int64_t)a.L;
          const int64_t ce = min(cs + a.L, a.T);
          const int64_t seg_lo = max(t_lo, cs), seg_hi = min(t_hi, ce);
          const v4i mk = byte_mask16((int32_t)min(max(seg_lo - t0, (int64_t)0), (int64_t)16),
                                     (int32_t)min(max(seg_hi - t0, (int64_t)0), (int64_t)16));
          const v4i mhi = bhi & mk, mlo = blo & mk;
          const bool fresh = seg_lo == cs;
#pragma unroll
          for (int i = 0; i < 2; ++i) mfma_tile(acc[i], ahi[i], alo[i], mhi, mlo, fresh);
          if (ce <= t_hi) {
#pragma unroll
            for (int i = 0; i < 2; ++i)
              flush_tile<PARTIALS>(acc[i], sum[i], j, a.partials, a.O, colc, CRS, m0 + 32 * i + 4 * half, a.K,
                                   cvalid);
            ++j;
          }
          if (ce >= t_hi) break;
        }
      }
    }
  }

  // ---- segment sum: scaled result (single segment) or U_g for the ordered reduction
  const int32_t e = a.ea->exp + a.eb->exp;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int32_t m = m0 + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
      if (cvalid && m < a.K) {
        const int64_t o = (int64_t)m * CRS + col;
        if (a.nseg == 1) a.out[o] = ldexpf(sum[i][v], e);
        else a.useg[g * a.O + o] = sum[i][v];
      }
    }
  }
}

// Unit-stride 1x1 layers without padding: x[n][c][p][q] is a C x T matrix of
// the same form as dy (K x T, t = (n*P + p)*Q + q), so both operands are
// prepared by prep_dy_item as digit blocks [KBT][rows][2][16 hi | 16 lo].  In
// that layout a lane's MFMA operand (row lane % 32, indices 16 * (lane / 32)
// .. + 15 of a 32-index block) is one 32-byte piece, and the 64 lanes of a
// wave read 2 KiB of contiguous digits per operand and block, straight into
// registers (the four waves of a workgroup share each row and column piece
// through L1).  Workgroup: a 64 x 64 tile (2 x 2 wave tiles of 32 x 32) of
// one segment; the operands of block kb + 1 are loaded while block kb is
// multiplied.  Chunks are whole blocks (L a multiple of 32) and digits past T
// are zero, so no masking is needed.  Chunk sums and segment output as in the
// kernels above.
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
struct Raw1x1 {
  const int16_t* dy;  // [N][K][PQ]
  const int16_t* x;   // [N][C][PQ]
  int32_t PQ;
};

constexpr int k1x1Threads = 256;
__global__ __launch_bounds__(k1x1Threads, 4) void k_bwdw_1x1(BwdwArgs a, const uint8_t* __restrict__ bd, int32_t Cp) {
  const BwdwTile tl = bwdw_tile(a);
  if (tl.seg >= a.nseg) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5, lc = lane & 31;
  const int32_t m0 = tl.ty * 64 + (wave >> 1) * 32;  // the wave's 32 rows (k)
  const int32_t c0 = tl.tx * 64 + (wave & 1) * 32;   // and 32 columns (c)
  const int64_t t_seg0 = (int64_t)tl.seg * a.G * a.L;
  const int64_t t_seg1 = min(t_seg0 + (int64_t)a.G * a.L, a.T);
  const int64_t kb_begin = t_seg0 / 32, kb_end = (t_seg1 + 31) / 32;
  const int32_t chunk_blocks = a.L / 32;
  const int64_t astep = (int64_t)a.Mp * 64, bstep = (int64_t)Cp * 64;
  const uint4* ap = reinterpret_cast<const uint4*>(a.ad + kb_begin * astep + ((int64_t)(m0 + lc) * 2 + half) * 32);
  const uint4* bp = reinterpret_cast<const uint4*>(bd + kb_begin * bstep + ((int64_t)(c0 + lc) * 2 + half) * 32);
  uint4 ah = ap[0], al = ap[1], bh = bp[0], bl = bp[1];  // digit pieces of the block
  Acc3 acc;
  float sum[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) sum[v] = 0.f;
  int32_t blk = 0;
  for (int64_t kb = kb_begin; kb < kb_end; ++kb) {
    const v4i ahi = (v4i){(int)ah.x, (int)ah.y, (int)ah.z, (int)ah.w};
    const v4i alo = (v4i){(int)al.x, (int)al.y, (int)al.z, (int)al.w};
    const v4i bhi = (v4i){(int)bh.x, (int)bh.y, (int)bh.z, (int)bh.w};
    const v4i blo = (v4i){(int)bl.x, (int)bl.y, (int)bl.z, (int)bl.w};
    if (kb + 1 < kb_end) {
      ap += astep / 16;
      bp += bstep / 16;
      ah = ap[0]; al = ap[1]; bh = bp[0]; bl = bp[1];
    }
    mfma_tile(acc, ahi, alo, bhi, blo, blk == 0);
    if (++blk == chunk_blocks || kb == kb_end - 1) {
      flush_tile<false>(acc, sum, 0, nullptr, a.O, 0, a.C, 0, a.K, false);
      blk = 0;
    }
  }
  const int32_t c = c0 + lc;
  const int32_t e = a.ea->exp + a.eb->exp;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int32_t m = m0 + 8 * (v >> 2) + 4 * half + (v & 3);
    if (c < a.C && m < a.K) {
      const int64_t o = (int64_t)m * a.C + c;
      if (a.nseg == 1) a.out[o] = ldexpf(sum[v], e);
      else a.useg[(int64_t)tl.seg * a.O + o] = sum[v];
    }
  }
}

// 16-byte piece `piece` of row `row` in a 64-byte-per-row operand block,
// swizzled so that the pieces a wave reads fall on distinct LDS banks.
__device__ __forceinline__ int swz(int row, int piece) { return row * 4 + (piece ^ ((row >> 2) & 3)); }

// Unit-stride 1x1 weight gradient from the INT16 tensors through LDS (the
// default when P*Q is a multiple of 4).  Per band of 64 indices (two 32-index
// blocks) the workgroup loads the 64-row slices of dy and x it multiplies with
// coalesced loads, PIECE consecutive elements per lane (16 or 8 bytes, 128
// contiguous bytes per row and band), splits every element into its byte
// digits once, and writes them in the MFMA operand layout: per block and row,
// four 16-byte pieces (hi digits of indices 0-15, 16-31, then lo), swizzled
// across LDS banks as in the forward kernels.  Each of the four waves then
// reads its 32 x 32 tile's operands from LDS.  The loads of band b + 1 are in
// flight while band b is multiplied (two LDS buffers, one barrier per band).
// A piece lies in one image (P*Q a multiple of PIECE); rows past K or C and
// indices past T are zeros.  The loads are buffer loads: per band one offset
// per lane and operand (one division), the row step of the thread's pieces in
// the scalar offset, and rows past K or C or indices past T at an offset past
// the end of the tensor, which reads zeros (both tensors below 2 GiB: checked
// by the launcher).  Chunks, segments and output as in k_bwdw_1x1.
// Raw buffer resource over [p, p + bytes) (offsets past the end read zeros).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
template <int PIECE>
__global__ __launch_bounds__(k1x1Threads, 4) void k_bwdw_1x1s(BwdwArgs a, Raw1x1 raw) {
  constexpr int kLoads = 64 * 64 / PIECE / k1x1Threads;  // pieces per thread and operand per band
  constexpr int kPerRow = 64 / PIECE;                     // pieces per row and band
  __shared__ __align__(16) uint8_t sbuf[2][2][2 * 4096];  // [buffer][operand][block][64 rows x 64 B]
  const BwdwTile tl = bwdw_tile(a);
  if (tl.seg >= a.nseg) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5, lc = lane & 31;
  const int32_t rA0 = tl.ty * 64, rB0 = tl.tx * 64;  // the workgroup's dy rows (k) and x rows (c)
  const int64_t t_seg0 = (int64_t)tl.seg * a.G * a.L;
  const int64_t t_seg1 = min(t_seg0 + (int64_t)a.G * a.L, a.T);
  const int64_t kb_begin = t_seg0 / 32, kb_end = (t_seg1 + 31) / 32;
  const int32_t chunk_blocks = a.L / 32;
  const int32_t PQ = raw.PQ;
  typedef uint32_t vraw __attribute__((ext_vector_type(PIECE / 2)));
  vraw ra[kLoads], rb[kLoads];
  // piece i = j * 256 + thread of the band starting at block kb: row i / kPerRow,
  // indices PIECE (i % kPerRow) .. of the band; i % kPerRow is the same for
  // every j (256 is a multiple of kPerRow), so a thread's pieces share one
  // index range and one image, and piece j lies j * (256 / kPerRow) rows after
  // piece 0
  const int32_t pj = (int32_t)threadIdx.x % kPerRow, row0 = (int32_t)threadIdx.x / kPerRow;
  const __amdgpu_buffer_rsrc_t rs_dy = make_rsrc(raw.dy, (uint32_t)(a.T * a.K * 2));
  const __amdgpu_buffer_rsrc_t rs_x = make_rsrc(raw.x, (uint32_t)(a.T * a.C * 2));
  const int32_t KPQ = a.K * PQ, CPQ = a.C * PQ;
  const int32_t rowA = (rA0 + row0) * PQ, rowB = (rB0 + row0) * PQ;
  const uint32_t jstep = (uint32_t)(k1x1Threads / kPerRow) * (uint32_t)PQ * 2u;
  constexpr uint32_t kOut = 0x80000000u;  // past the end of either tensor
  auto load_band = [&](int64_t kb) {
    const int32_t t = (int32_t)(kb * 32) + PIECE * pj;
    const bool tin = t < (int32_t)a.T;
    const int32_t n = (int32_t)fdiv((uint32_t)(tin ? t : 0), a.div_q), pq = t - n * PQ;
    const uint32_t oa0 = tin ? (uint32_t)(n * KPQ + rowA + pq) * 2u : kOut;
    const uint32_t ob0 = tin ? (uint32_t)(n * CPQ + rowB + pq) * 2u : kOut;
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int32_t row = j * (k1x1Threads / kPerRow) + row0;
      const uint32_t oa = rA0 + row < a.K ? oa0 : kOut;
      const uint32_t ob = rB0 + row < a.C ? ob0 : kOut;
      const uint32_t so = __builtin_amdgcn_readfirstlane((uint32_t)j * jstep);
      if constexpr (PIECE == 8) {
        ra[j] = __builtin_bit_cast(vraw, __builtin_amdgcn_raw_buffer_load_b128(rs_dy, oa, so, 0));
        rb[j] = __builtin_bit_cast(vraw, __builtin_amdgcn_raw_buffer_load_b128(rs_x, ob, so, 0));
      } else {
        ra[j] = __builtin_bit_cast(vraw, __builtin_amdgcn_raw_buffer_load_b64(rs_dy, oa, so, 0));
        rb[j] = __builtin_bit_cast(vraw, __builtin_amdgcn_raw_buffer_load_b64(rs_x, ob, so, 0));
      }
    }
  };
  // digits of the staged pieces into buffer buf
  auto write_band = [&](int buf) {
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int32_t row = j * (k1x1Threads / kPerRow) + row0;
      const int32_t e = PIECE * pj;                       // index within the band
      const int32_t blk = e >> 5, h16 = (e >> 4) & 1, sub = e & 15;
      const int32_t off_hi = blk * 4096 + swz(row, h16) * 16 + sub;
      const int32_t off_lo = blk * 4096 + swz(row, 2 + h16) * 16 + sub;
#pragma unroll
      for (int op = 0; op < 2; ++op) {
        const vraw w = op == 0 ? ra[j] : rb[j];
        uint32_t hi[PIECE / 4], lo[PIECE / 4];
#pragma unroll
        for (int d = 0; d < PIECE / 4; ++d) {
          const uint32_t w0 = w[2 * d], w1 = w[2 * d + 1];
          const uint32_t h0 = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, w0) + (u16x2){128, 128});
          const uint32_t h1 = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, w1) + (u16x2){128, 128});
          lo[d] = __builtin_amdgcn_perm(w1, w0, 0x06040200u);
          hi[d] = __builtin_amdgcn_perm(h1, h0, 0x07050301u);
        }
        uint8_t* base = &sbuf[buf][op][0];
        if (PIECE == 8) {
          *reinterpret_cast<uint2*>(base + off_hi) = make_uint2(hi[0], hi[1]);
          *reinterpret_cast<uint2*>(base + off_lo) = make_uint2(lo[0], lo[1]);
        } else {
          *reinterpret_cast<uint32_t*>(base + off_hi) = hi[0];
          *reinterpret_cast<uint32_t*>(base + off_lo) = lo[0];
        }
      }
    }
  };

  Acc3 acc;
  float sum[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) sum[v] = 0.f;
  const int32_t ra_row = (wave >> 1) * 32 + lc, rb_row = (wave & 1) * 32 + lc;
  const uint32_t oa_hi = swz(ra_row, half) * 16, oa_lo = swz(ra_row, 2 + half) * 16;
  const uint32_t ob_hi = swz(rb_row, half) * 16, ob_lo = swz(rb_row, 2 + half) * 16;
  int32_t blk_in_chunk = 0;
  load_band(kb_begin);
  int buf = 0;
  for (int64_t kb = kb_begin; kb < kb_end; kb += 2, buf ^= 1) {
    write_band(buf);
    __syncthreads();
    if (kb + 2 < kb_end) load_band(kb + 2);
    const int32_t nblk = (int32_t)min((int64_t)2, kb_end - kb);
    for (int32_t b = 0; b < nblk; ++b) {
      const uint8_t* pa = &sbuf[buf][0][b * 4096];
      const uint8_t* pb = &sbuf[buf][1][b * 4096];
      const v4i ahi = *reinterpret_cast<const v4i*>(pa + oa_hi), alo = *reinterpret_cast<const v4i*>(pa + oa_lo);
      const v4i bhi = *reinterpret_cast<const v4i*>(pb + ob_hi), blo = *reinterpret_cast<const v4i*>(pb + ob_lo);
      mfma_tile(acc, ahi, alo, bhi, blo, blk_in_chunk == 0);
      if (++blk_in_chunk == chunk_blocks || kb + b == kb_end - 1) {
        flush_tile<false>(acc, sum, 0, nullptr, a.O, 0, a.C, 0, a.K, false);
        blk_in_chunk = 0;
      }
    }
  }
  const int32_t m0 = rA0 + (wave >> 1) * 32, c = rB0 + (wave & 1) * 32 + lc;
  const int32_t e = a.ea->exp + a.eb->exp;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int32_t m = m0 + 8 * (v >> 2) + 4 * half + (v & 3);
    if (c < a.C && m < a.K) {
      const int64_t o = (int64_t)m * a.C + c;
      if (a.nseg == 1) a.out[o] = ldexpf(sum[v], e);
      else a.useg[(int64_t)tl.seg * a.O + o] = sum[v];
    }
  }
}

// ---------------------------------------------------------------------------
// Band kernel: unit strides, output rows of a multiple of 8, filter width at
// most 4, chunks of whole 32-index blocks.  Reduction indices then come in
// runs of 8 that lie in one output row (t = t0 .. t0+7 are q = q0 .. q0+7 of
// one (n, p)), and for a column (c, r, s) the run's operands are the 8
// consecutive bytes at column q0 + s of padded input row n*Hpad + p + r.  x is
// prepared as separate lo / hi byte planes per padded row, XB[c][z][2][Wpad],
// so a lane reads each run as one 16-byte window at the 8-aligned column q0
// (ds_read2_b64) and extracts its 8 bytes with two byte-aligns by s.
// Per band of 128 indices (4 blocks, 16 runs) the workgroup copies, with
// direct-to-LDS loads into the other half of a double buffer while the
// current band is consumed, the band's dy digits (A, swizzled as in the
// forward kernels) and the padded input rows its runs touch for the
// workgroup's channels; one barrier per band.
constexpr int kBandBlocks = kSBT / 32;               // 4
constexpr int kBandABytes = kBandBlocks * kMT * 64;  // 16 KiB
constexpr int kBandLdsBytes = 76 * 1024;             // two buffers; two workgroups per CU

typedef __attribute__((address_space(3))) void* lds_ptr_t;


__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const uint8_t*)p;
}
// Lane id (0..63) computed afresh at each use: the asm is volatile, so the
// compiler recomputes it rather than keeping it (or values derived from it)
// in a register across a loop.
__device__ __forceinline__ int32_t fresh_lane() {
  int32_t l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}


// XB[c][n*Hpad + u][d][Wpad]: d = 0 lo digits, d = 1 hi digits of
// x[n][c][u - ph][v - pw], zero outside; rows are row_bytes = 2*Wpad + 16 apart
// (the 16 spare bytes shift successive rows across LDS banks).  Column pad PW
// below 4 (same windowing as k_prep_xp_vec).  VEC = 8: rows of a multiple of 8
// elements, read in 16-byte pieces; VEC = 4: rows of a multiple of 4 elements,
// read in 8-byte pieces.  x 16-byte aligned.
template <int PW, int VEC = 8>
__global__ __launch_bounds__(256) void k_prep_xb(const int16_t* __restrict__ x, uint8_t* __restrict__ xb, int32_t N,
                                                int32_t C, int32_t H, int32_t W, int32_t Hpad, int32_t Wpad,
                                                int32_t ph, int32_t row_bytes, DyPrep q) {
  const int32_t c = blockIdx.y;
  if (c >= C) {  // rows of workgroups past the channels prepare the dy digits
    prep_dy_item(q, ((c - C) * gridDim.x + blockIdx.x) * 256 + threadIdx.x);
    return;
  }
  const int32_t i = blockIdx.x * 256 + threadIdx.x;  // (n * Hpad + u) * W8 + v8
  const int32_t W8 = Wpad >> 3;
  if (i >= N * Hpad * W8) return;
  const int32_t r = i / W8, v0 = (i - r * W8) * 8;
  const int32_t n = r / Hpad, u = r - n * Hpad;
  const int32_t ih = u - ph;
  uint32_t lo[2] = {0u, 0u}, hi[2] = {0u, 0u};
  if (ih >= 0 && ih < H) {
    const int16_t* row = x + ((int64_t)(n * C + c) * H + ih) * W;
    uint32_t g[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};  // elements v0-8 .. v0+7
    if (VEC == 8) {
      if (PW > 0 && v0 >= 8 && v0 - 8 < W) {
        const uint4 q = *reinterpret_cast<const uint4*>(row + v0 - 8);
        g[0] = q.x; g[1] = q.y; g[2] = q.z; g[3] = q.w;
      }
      if (v0 < W) {
        const uint4 q = *reinterpret_cast<const uint4*>(row + v0);
        g[4] = q.x; g[5] = q.y; g[6] = q.z; g[7] = q.w;
      }
    } else {
      // elements v0-4 .. v0+7 in pieces of four, each wholly inside or outside the row
      if (PW > 0 && v0 >= 4 && v0 - 4 < W) {
        const uint2 q = *reinterpret_cast<const uint2*>(row + v0 - 4);
        g[2] = q.x; g[3] = q.y;
      }
      if (v0 < W) {
        const uint2 q = *reinterpret_cast<const uint2*>(row + v0);
        g[4] = q.x; g[5] = q.y;
      }
      if (v0 + 4 < W) {
        const uint2 q = *reinterpret_cast<const uint2*>(row + v0 + 4);
        g[6] = q.x; g[7] = q.y;
      }
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int e = 8 - PW + k;
      const int32_t a = (int32_t)(int16_t)(g[e >> 1] >> (16 * (e & 1)));
      lo[k >> 2] |= lo_digit(a) << (8 * (k & 3));
      hi[k >> 2] |= hi_digit(a) << (8 * (k & 3));
    }
  }
  uint8_t* rowp = xb + ((int64_t)c * N * Hpad + r) * row_bytes + v0;
  *reinterpret_cast<uint2*>(rowp) = make_uint2(lo[0], lo[1]);
  *reinterpret_cast<uint2*>(rowp + Wpad) = make_uint2(hi[0], hi[1]);
}

__device__ __forceinline__ void lds_rd128(v4i& d, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1" : "=v"(d) : "v"(addr) : "memory");
}
__device__ __forceinline__ void lds_rd2x64(v4i& d, uint32_t addr) {
  asm volatile("ds_read2_b64 %0, %1 offset1:1" : "=v"(d) : "v"(addr) : "memory");
}
__device__ __forceinline__ void lds_rd64(uint2& d, uint32_t addr) {
  asm volatile("ds_read_b64 %0, %1" : "=v"(d) : "v"(addr) : "memory");
}
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Bytes s .. s+7 of a 16-byte window (s in 0..3), as two dwords.
__device__ __forceinline__ int window8_lo(const v4i& w, uint32_t s) {
  return (int)__builtin_amdgcn_alignbyte((uint32_t)w[1], (uint32_t)w[0], s);
}
__device__ __forceinline__ int window8_hi(const v4i& w, uint32_t s) {
  return (int)__builtin_amdgcn_alignbyte((uint32_t)w[2], (uint32_t)w[1], s);
}

template <bool PARTIALS>
__global__ __launch_bounds__(kThreads, 2) void k_bwdw_band(BwdwArgs a) {
  const BwdwTile tl = bwdw_tile(a);
  if (tl.seg >= a.nseg) return;
  // two buffers, each [B band: nch_max channels x rows_max padded rows x 2 planes x Wpad][A: 16 KiB];
  // a B window read past the last row stays inside the A part that follows it
  __shared__ __align__(16) uint8_t smem[kBandLdsBytes];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int half = lane >> 5;
  const int lc = lane & 31;
  const int32_t RS = a.R * a.S;
  const int32_t CRS = a.C * RS;
  const int32_t col0 = tl.tx * kNT;
  const int32_t col = col0 + wave * 32 + lc;
  const bool cvalid = col < CRS;
  const int32_t colc = cvalid ? col : col0;
  const int32_t c = colc / RS, rr = (colc % RS) / a.S;
  const uint32_t ss = (uint32_t)(colc % a.S);
  const int32_t c_lo = col0 / RS;
  const int32_t m0 = tl.ty * kMT;
  const int32_t g = tl.seg;
  const int32_t seg_len = a.G * a.L;
  const int32_t Ti = (int32_t)a.T;
  const int32_t t_seg0 = g * seg_len;
  const int32_t t_seg1 = min(t_seg0 + seg_len, Ti);
  const int32_t nbands = (t_seg1 - t_seg0 + kSBT - 1) / kSBT;
  const int32_t PQ = a.P * a.Q;
  const int32_t row_bytes = a.row_bytes;
  const int32_t b_region = a.buf_bytes - kBandABytes;
  const int32_t last_kb = t_seg1 / 32 - 1;

  // first padded row read by the band starting at t_b0 (rows_max rows from there fit the tensor)
  auto band_row0 = [&](int32_t t_b0) {
    const int32_t z_first = (t_b0 / PQ) * a.Hpad + (t_b0 % PQ) / a.Q;
    return min(z_first, a.NH - a.rows_max);
  };
  auto issue_band = [&](int32_t b) {
    const int32_t t_b0 = t_seg0 + b * kSBT;
    uint8_t* dstB = smem + (b & 1) * a.buf_bytes;
    uint8_t* dstA = dstB + b_region;
    // A: 4 blocks x 64 rows x 4 pieces of 16 B; slot S holds piece (S & 3) ^ ((row >> 2) & 3) of row S >> 2
    const int32_t kb0 = t_b0 / 32;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int32_t slot = j * 256 + threadIdx.x;
      const int32_t row = slot >> 2;
      const int32_t piece = (slot & 3) ^ ((row >> 2) & 3);
      const int32_t kb = min(kb0 + (row >> 6), last_kb);  // blocks past the segment reload a valid one (unused)
      const uint8_t* src = a.ad + ((int64_t)kb * a.Mp + m0 + (row & 63)) * 64 + piece * 16;
      __builtin_amdgcn_global_load_lds((const void*)src, (lds_ptr_t)(dstA + (j * 256 + wave_u * 64) * 16), 16, 0, 0);
    }
    // B: rows [za, za + rows_max) of each channel, one group of up to 64 pieces per instruction
    const int32_t za = band_row0(t_b0);
    const int32_t ppc = a.rows_max * row_bytes / 16;
    const int32_t nk = (ppc + 63) / 64;
    for (int32_t ii = wave_u; ii < a.nch_max * nk; ii += kThreads / 64) {
      const int32_t cc = ii / nk, k0 = (ii - cc * nk) * 64;
      const int32_t k = k0 + lane;
      if (k < ppc) {
        const int32_t ch = min(c_lo + cc, a.C - 1);
        const uint8_t* src = a.xb + ((int64_t)ch * a.NH + za) * row_bytes + k * 16;
        __builtin_amdgcn_global_load_lds((const void*)src, (lds_ptr_t)(dstB + cc * a.band_ch_stride + k0 * 16), 16,
                                         0, 0);
      }
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
  int32_t j = g * a.G;  // first chunk of the segment
  int32_t blk_in_chunk = 0;
  const int32_t chunk_blocks = a.L / 32;
  const uint32_t smem_base = lds_addr(smem);
  const uint32_t lane_b = (uint32_t)((c - c_lo) * a.band_ch_stride + rr * row_bytes);
  const uint32_t rd_a0 = (uint32_t)(swz(lc, 2 * half) * 16), rd_a1 = (uint32_t)(swz(lc, 2 * half + 1) * 16);

  issue_band(0);
  wait_vmcnt<0>();
  __syncthreads();
  for (int32_t b = 0; b < nbands; ++b) {
    if (b + 1 < nbands) issue_band(b + 1);
    const int32_t t_b0 = t_seg0 + b * kSBT;
    const uint32_t bufB = smem_base + (uint32_t)((b & 1) * a.buf_bytes) + lane_b;
    const uint32_t bufA = smem_base + (uint32_t)((b & 1) * a.buf_bytes + b_region);
    const int32_t nblk = min(kBandBlocks, (t_seg1 - t_b0) / 32);
    // run position (uniform): image n, output row p, column q0 of run t_b0 / 8
    const int32_t za = band_row0(t_b0);
    int32_t rn = t_b0 / PQ, rp = (t_b0 % PQ) / a.Q, rq = t_b0 % a.Q;
    for (int32_t kbl = 0; kbl < nblk; ++kbl) {
      // offsets of the block's four runs; lanes of half h take runs 2h and 2h+1
      int32_t ro[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        ro[u] = (rn * a.Hpad + rp - za) * row_bytes + rq;
        rq += 8;
        if (rq == a.Q) {
          rq = 0;
          if (++rp == a.P) { rp = 0; ++rn; }
        }
      }
      const uint32_t to0 = (uint32_t)(half ? ro[2] : ro[0]), to1 = (uint32_t)(half ? ro[3] : ro[1]);
      v4i ahi[2], alo[2], wl0, wh0, wl1, wh1;
      const uint32_t ab = bufA + (uint32_t)(kbl * 64 * 64);
      lds_rd128(ahi[0], ab + rd_a0);
      lds_rd128(alo[0], ab + rd_a1);
      lds_rd128(ahi[1], ab + rd_a0 + 2048);  // rows 32..63 sit 2048 bytes on at the same swizzle
      lds_rd128(alo[1], ab + rd_a1 + 2048);
      lds_rd2x64(wl0, bufB + to0);
      lds_rd2x64(wh0, bufB + to0 + a.Wpad);
      lds_rd2x64(wl1, bufB + to1);
      lds_rd2x64(wh1, bufB + to1 + a.Wpad);
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(wl0), "+v"(wh0), "+v"(wl1), "+v"(wh1), "+v"(ahi[0]), "+v"(alo[0]), "+v"(ahi[1]),
                     "+v"(alo[1])
                   :
                   : "memory");
      const v4i blo = {window8_lo(wl0, ss), window8_hi(wl0, ss), window8_lo(wl1, ss), window8_hi(wl1, ss)};
      const v4i bhi = {window8_lo(wh0, ss), window8_hi(wh0, ss), window8_lo(wh1, ss), window8_hi(wh1, ss)};
      const bool fresh = blk_in_chunk == 0;
#pragma unroll
      for (int i = 0; i < 2; ++i) mfma_tile(acc[i], ahi[i], alo[i], bhi, blo, fresh);
      if (++blk_in_chunk == chunk_blocks) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
          flush_tile<PARTIALS>(acc[i], sum[i], j, a.partials, a.O, colc, CRS, m0 + 32 * i + 4 * half, a.K, cvalid);
        ++j;
        blk_in_chunk = 0;
      }
    }
    wait_vmcnt<0>();
    __syncthreads();
  }
  if (blk_in_chunk != 0) {  // a segment ending inside a chunk (the last one, at T)
#pragma unroll
    for (int i = 0; i < 2; ++i)
      flush_tile<PARTIALS>(acc[i], sum[i], j, a.partials, a.O, colc, CRS, m0 + 32 * i + 4 * half, a.K, cvalid);
  }

  const int32_t e = a.ea->exp + a.eb->exp;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int32_t m = m0 + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
      if (cvalid && m < a.K) {
        const int32_t o = m * CRS + col;
        if (a.nseg == 1) a.out[o] = ldexpf(sum[i][v], e);
        else a.useg[(int64_t)g * a.O + o] = sum[i][v];
      }
    }
  }
}

// Two-block chunks (L = 64) with every segment a whole number of chunks:
// the two 32-row tiles run one block out of phase (tile 1 consumes block kb-1
// while tile 0 consumes block kb, from operands kept in registers), so each
// chunk conversion of one tile is interleaved with the other tile's MFMAs,
// and the operand reads of a block are in flight during the lagging tile's
// work on the previous one.
__device__ __forceinline__ void interleave_4x16() {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 16, 0);
  }
}

template <bool PARTIALS>
__global__ __launch_bounds__(kThreads, 2) void k_bwdw_band_skew(BwdwArgs a) {
  const BwdwTile tl = bwdw_tile(a);
  if (tl.seg >= a.nseg) return;
  __shared__ __align__(16) uint8_t smem[kBandLdsBytes];
  // byte offset in a band buffer of each of the band's 16 runs of 8 indices
  // (padded row of its output position relative to the band's first row,
  // times the row stride, plus its column), two bands live
  __shared__ __align__(16) int32_t s_ro[2][kSBT / 8];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int half = lane >> 5;
  const int lc = lane & 31;
  const int32_t RS = a.R * a.S;
  const int32_t CRS = a.C * RS;
  const int32_t col0 = tl.tx * kNT;
  const int32_t col = col0 + wave * 32 + lc;
  const bool cvalid = col < CRS;
  const int32_t colc = cvalid ? col : col0;
  const int32_t c = colc / RS, rr = (colc % RS) / a.S;
  const uint32_t ss = (uint32_t)(colc % a.S);
  const int32_t c_lo = col0 / RS;
  const int32_t m0 = tl.ty * kMT;
  const int32_t g = tl.seg;
  const int32_t seg_len = a.G * a.L;
  const int32_t Ti = (int32_t)a.T;
  const int32_t t_seg0 = g * seg_len;
  const int32_t t_seg1 = min(t_seg0 + seg_len, Ti);
  const int32_t nbands = (t_seg1 - t_seg0 + kSBT - 1) / kSBT;
  const int32_t PQ = a.P * a.Q;
  const int32_t row_b = a.row_bytes;
  const int32_t b_region = a.buf_bytes - kBandABytes;
  const int32_t last_kb = t_seg1 / 32 - 1;

  // Band cursor: output position (n, p, q) of the first index of the next band
  // to be copied, advanced without divisions; the copy records each band's
  // position and first padded row for the reads that follow (two bands live).
  int32_t cn = t_seg0 / PQ, cp = (t_seg0 % PQ) / a.Q, cq = t_seg0 % a.Q;
  const int32_t ppc = a.rows_max * row_b / 16;  // 16-byte pieces per channel
  // Every copy below is a buffer load of a per-lane offset fixed for the whole
  // kernel plus a uniform offset, so the address arithmetic stays scalar.
  // A slot j*256 + tid holds piece (tid & 3) ^ ((tid >> 4) & 3) of row tid >> 2
  // of block kb0 + j.
  const __amdgpu_buffer_rsrc_t rs_a = make_rsrc(a.ad, a.ad_bytes);
  const __amdgpu_buffer_rsrc_t rs_b = make_rsrc(a.xb, a.xb_bytes);
  const uint32_t a_block = (uint32_t)a.Mp * 64;
  auto issue_band = [&](int32_t b) {
    const int32_t t_b0 = t_seg0 + b * kSBT;
    uint8_t* dstB = smem + (b & 1) * a.buf_bytes;
    uint8_t* dstA = dstB + b_region;
    const int32_t kb0 = t_b0 / 32;
    // lane values recomputed here rather than held in registers across the band
    const int32_t ln = fresh_lane();
    const int32_t tid = wave_u * 64 + ln;
    const uint32_t a_lane = (uint32_t)((m0 + (tid >> 2)) * 64 + (((tid & 3) ^ ((tid >> 4) & 3)) * 16));
    const uint32_t b_lane = (uint32_t)ln * 16;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int32_t kb = min(kb0 + j, last_kb);  // blocks past the segment reload a valid one (unused)
      const uint32_t so = __builtin_amdgcn_readfirstlane((uint32_t)kb * a_block);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_a, (lds_ptr_t)(dstA + (j * 256 + wave_u * 64) * 16), 16, a_lane, so,
                                               0, 0);
    }
    // B: rows [za, za + rows_max) of each channel (wave w copies channels w, w + 4, ...)
    const int32_t za = __builtin_amdgcn_readfirstlane(min(cn * a.Hpad + cp, a.NH - a.rows_max));
    for (int32_t cc = wave_u; cc < a.nch_max; cc += kThreads / 64) {
      const int32_t ch = min(c_lo + cc, a.C - 1);
      const uint32_t soc = (uint32_t)((ch * a.NH + za) * row_b);
      uint8_t* dstc = dstB + cc * a.band_ch_stride;
      for (int32_t k0 = 0; k0 < ppc; k0 += 64) {
        if (ln < ppc - k0)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rs_b, (lds_ptr_t)(dstc + k0 * 16), 16, b_lane,
                                                   __builtin_amdgcn_readfirstlane(soc + (uint32_t)k0 * 16), 0, 0);
      }
    }
    if ((int32_t)threadIdx.x < kSBT / 8) {  // run u starts at output position (cn, cp, cq + 8u)
      int32_t q = cq + 8 * (int32_t)threadIdx.x, p = cp, n = cn;
      p += q / a.Q;
      q %= a.Q;
      n += p / a.P;
      p %= a.P;
      s_ro[b & 1][threadIdx.x] = (n * a.Hpad + p - za) * row_b + q;
    }
    cq += kSBT;
    while (cq >= a.Q) {
      cq -= a.Q;
      if (++cp == a.P) { cp = 0; ++cn; }
    }
    cn = __builtin_amdgcn_readfirstlane(cn);
    cp = __builtin_amdgcn_readfirstlane(cp);
    cq = __builtin_amdgcn_readfirstlane(cq);
  };

  Acc3 acc0, acc1;
  float sum0[16], sum1[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) { sum0[v] = 0.f; sum1[v] = 0.f; }
  const int32_t j0 = g * a.G;  // first chunk of the segment
  const uint32_t smem_base = lds_addr(smem);
  const uint32_t lane_b = (uint32_t)((c - c_lo) * a.band_ch_stride + rr * row_b);
  const uint32_t rd_a0 = (uint32_t)(swz(lc, 2 * half) * 16), rd_a1 = (uint32_t)(swz(lc, 2 * half + 1) * 16);
  const int32_t mrow0 = m0 + 4 * half, mrow1 = m0 + 32 + 4 * half;

  // Raw operand reads of one block (A rows of both tiles, four B windows), in
  // flight from one block to the next: the reads of block kbs+1 are issued
  // before the conversions and MFMAs of block kbs.
  struct Raw {
    v4i a0h, a0l, a1h, a1l, wl0, wh0, wl1, wh1;
  };
  Raw R0, R1;
  int32_t rkbl = 0, rslot = 0;  // read position (uniform)
  uint32_t rbufA = 0, rbufB = 0;
  auto start_read_band = [&](int32_t bn) {
    rslot = bn & 1;
    rbufB = smem_base + (uint32_t)(rslot * a.buf_bytes) + lane_b;
    rbufA = smem_base + (uint32_t)(rslot * a.buf_bytes + b_region);
    rkbl = 0;
  };
  auto issue_reads = [&](Raw& r) {
    // runs 4 kbl + 2 half and 4 kbl + 2 half + 1 of the band: this lane's 16 indices
    const int2 ro = *reinterpret_cast<const int2*>(&s_ro[rslot][4 * rkbl + 2 * half]);
    const uint32_t to0 = (uint32_t)ro.x, to1 = (uint32_t)ro.y;
    const uint32_t ab = rbufA + (uint32_t)(rkbl * 64 * 64);
    lds_rd128(r.a0h, ab + rd_a0);
    lds_rd128(r.a0l, ab + rd_a1);
    lds_rd128(r.a1h, ab + rd_a0 + 2048);
    lds_rd128(r.a1l, ab + rd_a1 + 2048);
    lds_rd2x64(r.wl0, rbufB + to0);
    lds_rd2x64(r.wh0, rbufB + to0 + a.Wpad);
    lds_rd2x64(r.wl1, rbufB + to1);
    lds_rd2x64(r.wh1, rbufB + to1 + a.Wpad);
    ++rkbl;
  };
  auto wait_raw = [&](Raw& r) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(r.wl0), "+v"(r.wh0), "+v"(r.wl1), "+v"(r.wh1), "+v"(r.a0h), "+v"(r.a0l), "+v"(r.a1h),
                   "+v"(r.a1l)
                 :
                 : "memory");
  };

  const int32_t NB = (t_seg1 - t_seg0) / 32;  // blocks of the segment (even: whole chunks)
  issue_band(0);
  wait_vmcnt<0>();
  __syncthreads();
  if (nbands > 1) issue_band(1);
  start_read_band(0);
  issue_reads(R0);
  v4i ea1h, ea1l, ebh, ebl;  // tile 1's operands of the last even block
  v4i oa1h, oa1l, obh, obl;  // tile 1's operands of the last odd block
  for (int32_t kbs = 0; kbs < NB; kbs += 2) {
    // even block kbs: tile 0 opens chunk kbs/2; tile 1 finishes chunk kbs/2 - 1 on block kbs - 1
    wait_raw(R0);
    issue_reads(R1);  // block kbs + 1, same band (bands hold 4 blocks)
    {
      const v4i bl = {window8_lo(R0.wl0, ss), window8_hi(R0.wl0, ss), window8_lo(R0.wl1, ss), window8_hi(R0.wl1, ss)};
      const v4i bh = {window8_lo(R0.wh0, ss), window8_hi(R0.wh0, ss), window8_lo(R0.wh1, ss), window8_hi(R0.wh1, ss)};
      if (kbs > 0) {
        flush_tile<PARTIALS>(acc0, sum0, j0 + kbs / 2 - 1, a.partials, a.O, colc, CRS, mrow0, a.K, cvalid);
        mfma_tile(acc1, oa1h, oa1l, obh, obl, false);
        interleave_4x16();
      }
      mfma_tile(acc0, R0.a0h, R0.a0l, bh, bl, true);
      ea1h = R0.a1h; ea1l = R0.a1l; ebh = bh; ebl = bl;
    }
    // odd block kbs + 1: tile 0 continues; tile 1 opens chunk kbs/2 on block kbs
    wait_raw(R1);
    if (((kbs + 2) & 3) == 0 && kbs + 2 < NB) {
      // block kbs + 2 opens band nb: every wave has read its last block of band nb - 1,
      // and band nb has landed; then band nb + 1 may overwrite band nb - 1's buffer
      wait_vmcnt<0>();
      __syncthreads();
      const int32_t nb = (kbs + 2) >> 2;
      if (nb + 1 < nbands) issue_band(nb + 1);
      start_read_band(nb);
    }
    if (kbs + 2 < NB) issue_reads(R0);
    {
      const v4i bl = {window8_lo(R1.wl0, ss), window8_hi(R1.wl0, ss), window8_lo(R1.wl1, ss), window8_hi(R1.wl1, ss)};
      const v4i bh = {window8_lo(R1.wh0, ss), window8_hi(R1.wh0, ss), window8_lo(R1.wh1, ss), window8_hi(R1.wh1, ss)};
      if (kbs > 0) flush_tile<PARTIALS>(acc1, sum1, j0 + kbs / 2 - 1, a.partials, a.O, colc, CRS, mrow1, a.K, cvalid);
      mfma_tile(acc0, R1.a0h, R1.a0l, bh, bl, false);
      if (kbs > 0) interleave_4x16();
      mfma_tile(acc1, ea1h, ea1l, ebh, ebl, true);
      oa1h = R1.a1h; oa1l = R1.a1l; obh = bh; obl = bl;
    }
  }
  // last chunk: tile 0 is complete; tile 1 still owes the segment's last block
  flush_tile<PARTIALS>(acc0, sum0, j0 + NB / 2 - 1, a.partials, a.O, colc, CRS, mrow0, a.K, cvalid);
  mfma_tile(acc1, oa1h, oa1l, obh, obl, false);
  interleave_4x16();
  flush_tile<PARTIALS>(acc1, sum1, j0 + NB / 2 - 1, a.partials, a.O, colc, CRS, mrow1, a.K, cvalid);

  const int32_t e = a.ea->exp + a.eb->exp;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int32_t m = m0 + 32 * i + 8 * (v >> 2) + 4 * half + (v & 3);
      if (cvalid && m < a.K) {
        const int32_t o = m * CRS + col;
        const float sv = i == 0 ? sum0[v] : sum1[v];
        if (a.nseg == 1) a.out[o] = ldexpf(sv, e);
        else a.useg[(int64_t)g * a.O + o] = sv;
      }
    }
  }
}

// Eight-wave variant of the band kernel for two-block chunks: the same bands
// and workgroup tile (128 columns x 64 rows), but each wave owns one 32 x 32
// output tile (row tile wave / 4, column group wave % 4), so every wave needs
// at most 128 VGPRs and two workgroups give four waves per SIMD to hide the
// LDS and matrix-core latencies of the per-block chain.  The operands of
// block k + 1 are read while block k is multiplied, then the chunk is
// converted.  Both the operand reads (ds_read_b128 / ds_read2_b64) and the
// band copies are issued from inline assembly and waited for explicitly: the
// reads one block later, the copies before each band's barrier.  The build
// checks in the generated assembly that no instruction touches a read's
// registers before its wait (asm_check.py).
// One 16-byte direct-to-LDS buffer load (lane i writes lds + 16 i) issued from
// inline assembly: the compiler then neither tracks it nor makes its own LDS
// reads wait for it (it cannot tell which buffer a copy targets); the caller
// waits with s_waitcnt vmcnt before a barrier.  M0 carries the LDS address;
// the kernels that use this helper issue no other instruction that reads M0.
__device__ __forceinline__ void dma16(const v4i& rsrc, uint32_t lds, uint32_t voff, uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rsrc), "s"(soff)
               : "memory", "m0");
}
// Raw buffer resource words (uniform) over [p, p + bytes).
__device__ __forceinline__ v4i rsrc_words(const void* p, uint32_t bytes) {
  const uint64_t b = (uint64_t)(uintptr_t)p;
  return v4i{__builtin_amdgcn_readfirstlane((int)(uint32_t)b), __builtin_amdgcn_readfirstlane((int)(uint32_t)(b >> 32)),
             __builtin_amdgcn_readfirstlane((int)bytes), 0x00020000};
}


constexpr int kThreadsW8 = 512;
constexpr int kBandBufBytes = kBandLdsBytes / 2;
// Buffers of the one-workgroup-per-CU build of the eight-wave kernel (wide
// input rows): the second buffer's operand reads still take 16-bit immediate
// offsets (kBandBufBigBytes + 3 * 4096 + 15 < 65536).
constexpr int kBandBufBigBytes = 51 * 1024;

template <int N>
using IC = std::integral_constant<int, N>;

// LDS reads at a lane address plus an immediate byte offset.
template <int OFF>
__device__ __forceinline__ void lds_rd128_at(v4i& d, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(d) : "v"(addr), "n"(OFF) : "memory");
}
template <int OFF8>
__device__ __forceinline__ void lds_rd2x64_at(v4i& d, uint32_t addr) {
  asm volatile("ds_read2_b64 %0, %1 offset0:%2 offset1:%3" : "=v"(d) : "v"(addr), "n"(OFF8), "n"(OFF8 + 1) : "memory");
}
template <int OFF4>
__device__ __forceinline__ void lds_rd2x32_at(v2i& d, uint32_t addr) {
  asm volatile("ds_read2_b32 %0, %1 offset0:%2 offset1:%3" : "=v"(d) : "v"(addr), "n"(OFF4), "n"(OFF4 + 1) : "memory");
}

// Operand registers of one block: A digits (hi, lo) and the B windows of the
// lane's runs, lo and hi digits.  Runs of 8 indices: two 16-byte windows per
// digit; runs of 4: four 8-byte windows per digit.
template <int RUN>
struct BandRaw;
template <>
struct BandRaw<8> {
  v4i ah, al, wl0, wh0, wl1, wh1;
};
template <>
struct BandRaw<4> {
  v4i ah, al;
  v2i wl0, wl1, wl2, wl3, wh0, wh1, wh2, wh3;
};

// Eight-wave band kernel.  Each band buffer holds the band's dy digits first
// (kBandABytes) and then its input rows; the run-offset tables hold offsets
// from the start of the first buffer, so that every operand read is one lane
// register plus an immediate, and a run's hi-digit window lies Wpad bytes
// after its lo-digit window.  The flat-band kernel below takes the 3x3
// same-padding layers; this one the other shapes with runs.  RUN: reduction indices
// per run, consecutive output columns of one output row (8 when the output
// width is a multiple of 8, else 4 for widths that are multiples of 4, such
// as 28); a lane's 16 indices of a block are 16 / RUN runs.  BUFB: bytes per
// band buffer (kBandBufBytes, two workgroups per CU, or kBandBufBigBytes for
// layers whose band needs more, one workgroup per CU: rows of about 200 and more).
template <bool PARTIALS, int RUN = 8, int BUFB = kBandBufBytes>
__global__ __launch_bounds__(kThreadsW8, PARTIALS ? 2 : 4) void k_bwdw_band_w8(BwdwArgs a) {
  static_assert(RUN == 8 || RUN == 4, "runs of 8 or 4 indices");
  static_assert(BUFB + 3 * 4096 + 15 < 65536, "LDS read offsets are 16-bit immediates");
  const BwdwTile tl = bwdw_tile(a);
  if (tl.seg >= a.nseg) return;
  // output scale exponent, read before any copy is in flight (the compiler
  // would otherwise wait for a load still pending, and with it the copies)
  const int32_t e = __builtin_amdgcn_readfirstlane(a.ea->exp + a.eb->exp);
  __shared__ __align__(16) uint8_t sb[2][BUFB];
  // byte offset from sb[0] of each of a band's kSBT / RUN runs, per buffer
  __shared__ __align__(16) int32_t ro[2][kSBT / RUN];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rt = wave >> 2;  // row tile
  const int half = lane >> 5;
  const int lc = lane & 31;
  const int32_t RS = a.R * a.S;
  const int32_t CRS = a.C * RS;
  const int32_t col0 = tl.tx * kNT;
  const int32_t col = col0 + (wave & 3) * 32 + lc;
  const bool cvalid = col < CRS;
  const int32_t colc = cvalid ? col : col0;
  const int32_t c = colc / RS, rr = (colc % RS) / a.S;
  const uint32_t ss = (uint32_t)(colc % a.S);
  const int32_t c_lo = col0 / RS;
  const int32_t m0 = tl.ty * kMT;
  const int32_t g = tl.seg;
  const int32_t seg_len = a.G * a.L;
  const int32_t Ti = (int32_t)a.T;
  const int32_t t_seg0 = g * seg_len;
  const int32_t t_seg1 = min(t_seg0 + seg_len, Ti);
  const int32_t nbands = (t_seg1 - t_seg0 + kSBT - 1) / kSBT;
  const int32_t NB = (t_seg1 - t_seg0) / 32;  // blocks of the segment (whole chunks)
  const int32_t row_b = a.row_bytes;
  const int32_t last_kb = t_seg1 / 32 - 1;

  const int32_t ppc = a.rows_max * row_b / 16;  // 16-byte pieces per channel
  // Copies are buffer loads of a per-lane offset fixed for the kernel plus a
  // uniform offset.  A slot j*512 + tid holds piece (tid & 3) ^ ((tid >> 4) & 3)
  // of row (tid >> 2) & 63 of band block 2j + (tid >> 8).
  const v4i rs_a = rsrc_words(a.ad, a.ad_bytes);
  const v4i rs_b = rsrc_words(a.xb, a.xb_bytes);
  const uint32_t a_block = (uint32_t)a.Mp * 64;
  auto issue_band = [&](int32_t b, int buf_i) __attribute__((always_inline)) {
    const int32_t t_b0 = t_seg0 + b * kSBT;
    // output position (cn, cp, cq) of the band's first index (uniform: scalar arithmetic)
    const int32_t tq = (int32_t)fdiv((uint32_t)t_b0, a.div_q);
    const int32_t cq = __builtin_amdgcn_readfirstlane(t_b0 - tq * a.Q);
    const int32_t cn = __builtin_amdgcn_readfirstlane((int32_t)fdiv((uint32_t)tq, a.div_p));
    const int32_t cp = __builtin_amdgcn_readfirstlane(tq - cn * a.P);
    uint8_t* dstA = sb[buf_i];
    const int32_t kb0 = t_b0 / 32;
    // lane values recomputed here rather than held in registers across the band
    const int32_t ln = fresh_lane();
    const int32_t tid = wave * 64 + ln;
    const uint32_t a_lane = (uint32_t)((m0 + ((tid >> 2) & 63)) * 64 + (((tid & 3) ^ ((tid >> 4) & 3)) * 16));
    const uint32_t b_lane = (uint32_t)ln * 16;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int32_t kb = min(kb0 + 2 * j + (wave >> 2), last_kb);  // blocks past the segment reload a valid one
      const uint32_t so = __builtin_amdgcn_readfirstlane((uint32_t)kb * a_block);
      dma16(rs_a, lds_addr(dstA + (j * 512 + wave * 64) * 16), a_lane, so);
    }
    const int32_t za = __builtin_amdgcn_readfirstlane(min(cn * a.Hpad + cp, a.NH - a.rows_max));
    for (int32_t cc = wave; cc < a.nch_max; cc += kThreadsW8 / 64) {
      const int32_t ch = min(c_lo + cc, a.C - 1);
      const uint32_t soc = (uint32_t)((ch * a.NH + za) * row_b);
      uint8_t* dstc = sb[buf_i] + kBandABytes + cc * a.band_ch_stride;
      for (int32_t k0 = 0; k0 < ppc; k0 += 64) {
        if (ln < ppc - k0)
          dma16(rs_b, lds_addr(dstc + k0 * 16), b_lane, __builtin_amdgcn_readfirstlane(soc + (uint32_t)k0 * 16));
      }
    }
    if (tid < kSBT / RUN) {  // run u starts at output position (cn, cp, cq + RUN u)
      int32_t q = cq + RUN * tid, p = cp, n = cn;
      const int32_t dq = (int32_t)fdiv((uint32_t)q, a.div_q);
      p += dq;
      q -= dq * a.Q;
      const int32_t dp = (int32_t)fdiv((uint32_t)p, a.div_p);
      n += dp;
      p -= dp * a.P;
      ro[buf_i][tid] = buf_i * BUFB + kBandABytes + (n * a.Hpad + p - za) * row_b + q;
    }
  };

  Acc3 acc;
  float sum[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) sum[v] = 0.f;
  const int32_t j0 = g * a.G;  // first chunk of the segment
  // lane parts of the operand addresses, with the base of buffer 0 folded in
  const uint32_t base0 = lds_addr(&sb[0][0]);
  const uint32_t lane_b = base0 + (uint32_t)((c - c_lo) * a.band_ch_stride + rr * row_b);
  const uint32_t rd_a0 = base0 + (uint32_t)(swz(lc, 2 * half) * 16 + rt * 2048);
  const uint32_t rd_a1 = base0 + (uint32_t)(swz(lc, 2 * half + 1) * 16 + rt * 2048);
  const int32_t mrow = m0 + 32 * rt + 4 * half;

  // Operand reads are inline-assembly LDS reads with explicit waits (wait_raw)
  // placed one block after the issue.  Between a read and its wait the
  // compiler takes the destination registers as already written, so it must
  // neither copy nor spill them there: the build checks the generated
  // assembly for exactly that (asm_check.py) and the launcher also requires a
  // build without scratch.
  using Raw = BandRaw<RUN>;
  Raw R0, R1;
  // block K (0..3) of the band in buffer BUF (both compile-time)
  auto read_block = [&](Raw& r, auto bufc, auto kc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value, K = decltype(kc)::value;
    if constexpr (RUN == 8) {
      const int2 o = *reinterpret_cast<const int2*>(&ro[BUF][4 * K + 2 * half]);
      lds_rd128_at<BUF * BUFB + K * 4096>(r.ah, rd_a0);
      lds_rd128_at<BUF * BUFB + K * 4096>(r.al, rd_a1);
      const uint32_t w0 = lane_b + (uint32_t)o.x, w1 = lane_b + (uint32_t)o.y;
      lds_rd2x64_at<0>(r.wl0, w0);
      lds_rd2x64_at<0>(r.wl1, w1);
      lds_rd2x64_at<0>(r.wh0, w0 + a.Wpad);
      lds_rd2x64_at<0>(r.wh1, w1 + a.Wpad);
    } else {
      const v4i o = *reinterpret_cast<const v4i*>(&ro[BUF][8 * K + 4 * half]);
      lds_rd128_at<BUF * BUFB + K * 4096>(r.ah, rd_a0);
      lds_rd128_at<BUF * BUFB + K * 4096>(r.al, rd_a1);
      const uint32_t w0 = lane_b + (uint32_t)o.x, w1 = lane_b + (uint32_t)o.y;
      const uint32_t w2 = lane_b + (uint32_t)o.z, w3 = lane_b + (uint32_t)o.w;
      lds_rd2x32_at<0>(r.wl0, w0);
      lds_rd2x32_at<0>(r.wl1, w1);
      lds_rd2x32_at<0>(r.wl2, w2);
      lds_rd2x32_at<0>(r.wl3, w3);
      lds_rd2x32_at<0>(r.wh0, w0 + a.Wpad);
      lds_rd2x32_at<0>(r.wh1, w1 + a.Wpad);
      lds_rd2x32_at<0>(r.wh2, w2 + a.Wpad);
      lds_rd2x32_at<0>(r.wh3, w3 + a.Wpad);
    }
  };
  auto wait_raw = [&](Raw& r) __attribute__((always_inline)) {
    if constexpr (RUN == 8) {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(r.wl0), "+v"(r.wh0), "+v"(r.wl1), "+v"(r.wh1), "+v"(r.ah), "+v"(r.al)
                   :
                   : "memory");
    } else {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(r.wl0), "+v"(r.wl1), "+v"(r.wl2), "+v"(r.wl3), "+v"(r.wh0), "+v"(r.wh1), "+v"(r.wh2),
                     "+v"(r.wh3), "+v"(r.ah), "+v"(r.al)
                   :
                   : "memory");
    }
  };
  // bytes ss .. ss + 3 of an 8-byte window (ss in 0..3)
  auto win4 = [&](const v2i& w) __attribute__((always_inline)) {
    return (int)__builtin_amdgcn_alignbyte((uint32_t)w.y, (uint32_t)w.x, ss);
  };
  auto operand_hi = [&](const Raw& r) __attribute__((always_inline)) {
    if constexpr (RUN == 8)
      return v4i{window8_lo(r.wh0, ss), window8_hi(r.wh0, ss), window8_lo(r.wh1, ss), window8_hi(r.wh1, ss)};
    else
      return v4i{win4(r.wh0), win4(r.wh1), win4(r.wh2), win4(r.wh3)};
  };
  auto operand_lo = [&](const Raw& r) __attribute__((always_inline)) {
    if constexpr (RUN == 8)
      return v4i{window8_lo(r.wl0, ss), window8_hi(r.wl0, ss), window8_lo(r.wl1, ss), window8_hi(r.wl1, ss)};
    else
      return v4i{win4(r.wl0), win4(r.wl1), win4(r.wl2), win4(r.wl3)};
  };
  // Chunk CH (0 or 1) of band b in buffer CUR: block 2 CH + 1 is read while
  // block 2 CH is multiplied; after the band's last chunk the first block of
  // the next band comes from the other buffer after the band barrier, and the
  // band after next is then copied into this one.
  auto do_chunk = [&](auto curc, auto chc, int32_t b, int32_t nch) __attribute__((always_inline)) {
    constexpr int CUR = decltype(curc)::value, CH = decltype(chc)::value;
    wait_raw(R0);
    read_block(R1, IC<CUR>{}, IC<2 * CH + 1>{});
    mfma_tile(acc, R0.ah, R0.al, operand_hi(R0), operand_lo(R0), true);
    wait_raw(R1);
    if (CH + 1 < nch) {
      read_block(R0, IC<CUR>{}, IC<(2 * CH + 2) & 3>{});
    } else if (b + 1 < nbands) {
      // every wave has read band b and band b + 1 has landed; band b + 2 may
      // then overwrite band b
      wait_vmcnt<0>();
      __syncthreads();
      if (b + 2 < nbands) issue_band(b + 2, CUR);
      read_block(R0, IC<1 - CUR>{}, IC<0>{});
    }
    mfma_tile(acc, R1.ah, R1.al, operand_hi(R1), operand_lo(R1), false);
    flush_tile<PARTIALS>(acc, sum, j0 + 2 * b + CH, a.partials, a.O, colc, CRS, mrow, a.K, cvalid);
  };
  // One band: two chunks, or one at the end of a segment of an odd number of chunk pairs.
  auto do_band = [&](auto curc, int32_t b) __attribute__((always_inline)) {
    const int32_t nch = min(2, (NB - 4 * b) >> 1);
    do_chunk(curc, IC<0>{}, b, nch);
    if (nch > 1) do_chunk(curc, IC<1>{}, b, nch);
  };

  issue_band(0, 0);
  wait_vmcnt<0>();
  __syncthreads();
  if (nbands > 1) issue_band(1, 1);
  read_block(R0, IC<0>{}, IC<0>{});
  for (int32_t b = 0; b < nbands; b += 2) {
    do_band(IC<0>{}, b);
    if (b + 1 < nbands) do_band(IC<1>{}, b + 1);
  }

  const int32_t ln = fresh_lane();
  const int32_t ocol = col0 + (wave & 3) * 32 + (ln & 31);
  const int32_t orow = m0 + 32 * rt + 4 * (ln >> 5);
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int32_t m = orow + 8 * (v >> 2) + (v & 3);
    if (ocol < CRS && m < a.K) {
      const int32_t o = m * CRS + ocol;
      if (a.nseg == 1) a.out[o] = ldexpf(sum[v], e);
      else a.useg[(int64_t)g * a.O + o] = sum[v];
    }
  }
}

// ---------------------------------------------------------------------------
// Flat-band kernel: 3x3 filters with unit stride and one pixel of padding.
// There H = P and W = Q, so the input pixel that column (c, r, s) pairs with
// reduction index t = (n*P + p)*Q + q, x[n][c][p + r - 1][q + s - 1], sits
// at index t + delta(r, s) of channel c's pixels laid out in t order
// (delta = (r - 1)*W + s - 1), unless p + r - 1 or q + s - 1 falls outside
// the image, where the product must vanish (the index t + delta then lands on
// a neighbouring row or image).  A lane therefore reads its 16 indices of a
// block as one window at a fixed distance from the band start, whatever the
// image width, and zeroes the bytes of invalid pairs: v_perm_b32 does both
// per dword, with selector byte a + k for byte k of a valid index (a = the
// window's byte misalignment, fixed per (r, s)) and 12 (the constant 0)
// otherwise.  The selectors depend only on t and (r, s): the preparation
// pass writes them for every group of 64 indices, TAB[t / 64][r*3 + s][4
// pieces of 16 indices][4 dwords], and each band copies its two groups beside
// the operands.  The input is prepared as byte planes in t order,
// XF[c][d][HALO + t] (d = 0 lo digits, 1 hi digits; HALO >= W + 1 zero bytes
// before t = 0 and zeros past T); a band of 128 indices copies plane bytes
// t_b0 .. t_b0 + kPlane - 1 (from HALO indices before the band to HALO + 16
// after it).  The dy digits, the workgroup tiles, the band double buffer and
// the chunk / segment order are those of the eight-wave kernel above.
constexpr int kFlatRS = 9;                            // 3 x 3 filters
constexpr int kFlatNch = (kNT - 1) / kFlatRS + 2;     // channels a column tile touches (16)
constexpr int kFlatTabBytes = 2 * kFlatRS * 64;       // selectors of the band's two groups
template <int HALO>
struct FlatGeo {
  static_assert(HALO % 16 == 0, "16-byte copy pieces");
  static constexpr int kPlane = 2 * HALO + kSBT + 16;  // band bytes per digit plane
  static constexpr int kChStride = 2 * kPlane;         // both planes of a channel
  // the planes' copy in wave instructions of 64 pieces (1 KiB); the last one
  // partly fills padding, so that the selector groups start on an instruction
  static constexpr int kXInstr = (kFlatNch * kChStride / 16 + 63) / 64;
  static constexpr int kXBytes = kXInstr * 1024;
  static constexpr int kInstr = kXInstr + 2;  // + the selector groups (64 + 8 pieces)
  static constexpr int kPerWave = (kInstr + 7) / 8;
  static constexpr int kBuf = kBandABytes + kXBytes + kFlatTabBytes;
  static_assert(kBuf + 3 * 4096 + 15 < 65536, "LDS read offsets are 16-bit immediates");
  static_assert(kPlane / 4 + 3 * 8 + 4 < 256, "ds_read2_b32 dword offsets are 8-bit");
};

// The preparation pass: workgroups [0, nbx) write XF, [nbx, nbx + nbt) the
// selector table, the rest the dy digits.
struct FlatPrep {
  const int16_t* x;
  uint8_t* xf;
  int32_t C, P, Q, PQ, T, plane, halo, ngroups;
  uint32_t tab;
  bool vec8;  // P*Q a multiple of 8 and x 16-byte aligned: 8 plane bytes per thread
};
__global__ __launch_bounds__(256) void k_prep_flat(FlatPrep f, DyPrep q, int32_t nbx, int32_t nbt) {
  const int32_t b = blockIdx.x;
  if (b >= nbx + nbt) {
    prep_dy_item(q, (b - nbx - nbt) * 256 + threadIdx.x);
    return;
  }
  if (b >= nbx) {  // one thread per selector dword (group, r*3 + s, piece, dword)
    const int32_t i = (b - nbx) * 256 + threadIdx.x;
    if (i >= f.ngroups * kFlatRS * 16) return;
    const int32_t gi = i / (kFlatRS * 16), rem = i - gi * (kFlatRS * 16);
    const int32_t rsv = rem >> 4, r = rsv / 3, s = rsv - 3 * r;
    // the window's misalignment: HALO is a multiple of 4, so delta mod 4
    const uint32_t a = (uint32_t)(16 + (r - 1) * f.Q + (s - 1)) & 3u;
    const int32_t t0 = gi * 64 + (rem & 15) * 4;
    uint32_t sel = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int32_t t = t0 + k;
      bool valid = false;
      if (t < f.T) {
        const int32_t n = t / f.PQ, pq = t - n * f.PQ;
        const int32_t p = pq / f.Q, qq = pq - p * f.Q;
        valid = (uint32_t)(p + r - 1) < (uint32_t)f.P && (uint32_t)(qq + s - 1) < (uint32_t)f.Q;
      }
      sel |= (valid ? a + (uint32_t)k : 12u) << (8 * k);
    }
    reinterpret_cast<uint32_t*>(f.xf + f.tab)[i] = sel;
    return;
  }
  if (f.vec8) {
    // one thread per 8 bytes of channel c's two planes: P*Q a multiple of 8
    // and x 16-byte aligned, so the 8 indices from a multiple of 8 lie in one
    // image and are one 16-byte load
    const int32_t per = f.plane >> 3;
    const int32_t i = b * 256 + threadIdx.x;
    if (i >= f.C * per) return;
    const int32_t c = i / per, u = (i - c * per) * 8;
    const int32_t t = u - f.halo;
    uint32_t lo[2] = {0u, 0u}, hi[2] = {0u, 0u};
    if (t >= 0 && t < f.T) {
      const int32_t n = t / f.PQ, pq = t - n * f.PQ;
      const uint4 v = *reinterpret_cast<const uint4*>(f.x + ((int64_t)n * f.C + c) * f.PQ + pq);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int32_t a = (int32_t)(int16_t)(w[k >> 1] >> (16 * (k & 1)));
        lo[k >> 2] |= lo_digit(a) << (8 * (k & 3));
        hi[k >> 2] |= hi_digit(a) << (8 * (k & 3));
      }
    }
    uint8_t* row = f.xf + (int64_t)c * 2 * f.plane + u;
    *reinterpret_cast<uint2*>(row) = make_uint2(lo[0], lo[1]);
    *reinterpret_cast<uint2*>(row + f.plane) = make_uint2(hi[0], hi[1]);
    return;
  }
  // one thread per 4 bytes of channel c's two planes
  const int32_t per = f.plane >> 2;
  const int32_t i = b * 256 + threadIdx.x;
  if (i >= f.C * per) return;
  const int32_t c = i / per, u = (i - c * per) * 4;
  uint32_t lo = 0, hi = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int32_t t = u + k - f.halo;
    if (t >= 0 && t < f.T) {
      const int32_t n = t / f.PQ, pq = t - n * f.PQ;
      const int32_t v = f.x[((int64_t)n * f.C + c) * f.PQ + pq];
      lo |= lo_digit(v) << (8 * k);
      hi |= hi_digit(v) << (8 * k);
    }
  }
  uint8_t* row = f.xf + (int64_t)c * 2 * f.plane + u;
  *reinterpret_cast<uint32_t*>(row) = lo;
  *reinterpret_cast<uint32_t*>(row + f.plane) = hi;
}

// Two dwords at independent immediate dword offsets.
template <int O0, int O1>
__device__ __forceinline__ void lds_rd2x32_o(v2i& d, uint32_t addr) {
  asm volatile("ds_read2_b32 %0, %1 offset0:%2 offset1:%3" : "=v"(d) : "v"(addr), "n"(O0), "n"(O1) : "memory");
}

struct FlatRaw {
  v4i ah, al;
  v2i l01, l23, h01, h23, x4;  // lo / hi window dwords 0..3, and dword 4 of both
  v4i sel;
};

// PARTIALS (test and verification runs): the same kernel also stores every
// chunk partial, built for two waves per SIMD (the partial stores need more
// than 128 VGPRs).
template <int HALO, bool PARTIALS = false>
__global__ __launch_bounds__(kThreadsW8, PARTIALS ? 2 : 4) void k_bwdw_flat(BwdwArgs a) {
  using F = FlatGeo<HALO>;
  const BwdwTile tl = bwdw_tile(a);
  if (tl.seg >= a.nseg) return;
  const int32_t e = __builtin_amdgcn_readfirstlane(a.ea->exp + a.eb->exp);
  __shared__ __align__(16) uint8_t sb[2][F::kBuf];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int rt = wave >> 2;  // row tile
  const int half = lane >> 5;
  const int lc = lane & 31;
  const int32_t CRS = a.C * kFlatRS;
  const int32_t col0 = tl.tx * kNT;
  const int32_t col = col0 + (wave & 3) * 32 + lc;
  const bool cvalid = col < CRS;
  const int32_t colc = cvalid ? col : col0;
  const int32_t c = colc / kFlatRS, rs = colc - c * kFlatRS;
  const int32_t r = rs / 3, s = rs - 3 * r;
  const int32_t c_lo = col0 / kFlatRS;
  const int32_t m0 = tl.ty * kMT;
  const int32_t g = tl.seg;
  const int32_t seg_len = a.G * a.L;
  const int32_t Ti = (int32_t)a.T;
  const int32_t t_seg0 = g * seg_len;
  const int32_t t_seg1 = min(t_seg0 + seg_len, Ti);
  const int32_t nbands = (t_seg1 - t_seg0 + kSBT - 1) / kSBT;
  const int32_t NB = (t_seg1 - t_seg0) / 32;  // blocks of the segment (whole chunks)
  const int32_t last_kb = t_seg1 / 32 - 1;

  const v4i rs_a = rsrc_words(a.ad, a.ad_bytes);
  const v4i rs_b = rsrc_words(a.xb, a.xb_bytes);
  const uint32_t a_block = (uint32_t)a.Mp * 64;
  // Per-lane source offsets of the band copies, the same for every band (the
  // band start goes into the uniform offset).  A slot j*512 + tid of the dy
  // region holds piece (tid & 3) ^ ((tid >> 4) & 3) of row (tid >> 2) & 63 of
  // band block 2j + (tid >> 8).  Wave w issues the plane / selector copy
  // instructions w, w + 8, ...: instruction q < kXInstr copies plane pieces
  // 64q .. 64q + 63 (piece i: channel i / (kChStride / 16), its plane and
  // 16-byte piece; pieces past the 16 channels reload piece 0 into padding),
  // the next two the 72 selector pieces of the band's two groups.
  const uint32_t a_lane =
      (uint32_t)((m0 + ((threadIdx.x >> 2) & 63)) * 64 + (((threadIdx.x & 3) ^ ((threadIdx.x >> 4) & 3)) * 16));
  uint32_t vo[F::kPerWave];
#pragma unroll
  for (int u = 0; u < F::kPerWave; ++u) {
    const int32_t q = u * 8 + wave;
    if (q < F::kXInstr) {
      int32_t i = q * 64 + lane;
      if (i >= kFlatNch * F::kChStride / 16) i = 0;
      const int32_t cc = i / (F::kChStride / 16), pi = i - cc * (F::kChStride / 16);
      const int32_t d = pi >= F::kPlane / 16 ? 1 : 0;
      const int32_t k = pi - d * (F::kPlane / 16);
      const int32_t ch = min(c_lo + cc, a.C - 1);
      vo[u] = (uint32_t)(ch * 2 + d) * (uint32_t)a.flat_plane + (uint32_t)(k * 16);
    } else {
      vo[u] = a.flat_tab + (uint32_t)((q - F::kXInstr) * 64 + lane) * 16;
    }
  }
  auto issue_band = [&](int32_t b, int buf_i) __attribute__((always_inline)) {
    const int32_t t_b0 = t_seg0 + b * kSBT;
    uint8_t* dst = sb[buf_i];
    const int32_t kb0 = t_b0 / 32;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int32_t kb = min(kb0 + 2 * j + (wave >> 2), last_kb);  // blocks past the segment reload a valid one
      const uint32_t so = __builtin_amdgcn_readfirstlane((uint32_t)kb * a_block);
      dma16(rs_a, lds_addr(dst + (j * 512 + wave * 64) * 16), a_lane, so);
    }
    // a band's planes start t_b0 bytes into each plane, its selector groups
    // (t_b0 / 64) * 576 = 9 * t_b0 bytes into the table
    const uint32_t so_x = __builtin_amdgcn_readfirstlane((uint32_t)t_b0);
#pragma unroll
    for (int u = 0; u < F::kPerWave; ++u) {
      const int32_t q = u * 8 + wave;
      if (q < F::kXInstr)
        dma16(rs_b, lds_addr(dst + kBandABytes + q * 1024), vo[u], so_x);
      else if (q < F::kInstr && (q == F::kXInstr || lane < kFlatTabBytes / 16 - 64))
        dma16(rs_b, lds_addr(dst + kBandABytes + q * 1024), vo[u], so_x * (uint32_t)kFlatRS);
    }
  };

  Acc3 acc;
  float sum[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) sum[v] = 0.f;
  const int32_t j0 = g * a.G;  // first chunk of the segment
  const uint32_t base0 = lds_addr(&sb[0][0]);
  const uint32_t rd_a0 = base0 + (uint32_t)(swz(lc, 2 * half) * 16 + rt * 2048);
  const uint32_t rd_a1 = base0 + (uint32_t)(swz(lc, 2 * half + 1) * 16 + rt * 2048);
  // window start: byte HALO + delta of the lane's 16 indices, rounded down to a dword
  const uint32_t wofs = (uint32_t)(HALO + (r - 1) * a.Q + (s - 1)) & ~3u;
  const uint32_t xw0 = base0 + (uint32_t)(kBandABytes + (c - c_lo) * F::kChStride + half * 16) + wofs;
  const uint32_t xw1 = xw0 + F::kBuf;
  const uint32_t selw = base0 + (uint32_t)(kBandABytes + F::kXBytes + rs * 64 + half * 16);
  const int32_t mrow = m0 + 32 * rt + 4 * half;

  // Operand reads are inline-assembly LDS reads with explicit waits one block
  // after the issue (checked in the generated assembly by asm_check.py, and
  // the launcher requires a build without scratch).
  FlatRaw R0, R1;
  auto read_block = [&](FlatRaw& q, auto bufc, auto kc) __attribute__((always_inline)) {
    constexpr int BUF = decltype(bufc)::value, K = decltype(kc)::value;
    lds_rd128_at<BUF * F::kBuf + K * 4096>(q.ah, rd_a0);
    lds_rd128_at<BUF * F::kBuf + K * 4096>(q.al, rd_a1);
    const uint32_t xw = BUF ? xw1 : xw0;
    constexpr int D = K * 8, H = F::kPlane / 4;  // dword offsets of the block and of the hi plane
    lds_rd2x32_o<D, D + 1>(q.l01, xw);
    lds_rd2x32_o<D + 2, D + 3>(q.l23, xw);
    lds_rd2x32_o<H + D, H + D + 1>(q.h01, xw);
    lds_rd2x32_o<H + D + 2, H + D + 3>(q.h23, xw);
    lds_rd2x32_o<D + 4, H + D + 4>(q.x4, xw);
    lds_rd128_at<BUF * F::kBuf + (K >> 1) * (kFlatRS * 64) + (K & 1) * 32>(q.sel, selw);
  };
  auto wait_raw = [&](FlatRaw& q) __attribute__((always_inline)) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(q.ah), "+v"(q.al), "+v"(q.l01), "+v"(q.l23), "+v"(q.h01), "+v"(q.h23), "+v"(q.x4),
                   "+v"(q.sel)
                 :
                 : "memory");
  };
  auto pm = [](int hi, int lo, int sel) __attribute__((always_inline)) {
    return (int)__builtin_amdgcn_perm((uint32_t)hi, (uint32_t)lo, (uint32_t)sel);
  };
  auto operand_lo = [&](const FlatRaw& q) __attribute__((always_inline)) {
    return v4i{pm(q.l01.y, q.l01.x, q.sel.x), pm(q.l23.x, q.l01.y, q.sel.y), pm(q.l23.y, q.l23.x, q.sel.z),
               pm(q.x4.x, q.l23.y, q.sel.w)};
  };
  auto operand_hi = [&](const FlatRaw& q) __attribute__((always_inline)) {
    return v4i{pm(q.h01.y, q.h01.x, q.sel.x), pm(q.h23.x, q.h01.y, q.sel.y), pm(q.h23.y, q.h23.x, q.sel.z),
               pm(q.x4.y, q.h23.y, q.sel.w)};
  };
  auto do_chunk = [&](auto curc, auto chc, int32_t b, int32_t nch) __attribute__((always_inline)) {
    constexpr int CUR = decltype(curc)::value, CH = decltype(chc)::value;
    wait_raw(R0);
    read_block(R1, IC<CUR>{}, IC<2 * CH + 1>{});
    mfma_tile(acc, R0.ah, R0.al, operand_hi(R0), operand_lo(R0), true);
    wait_raw(R1);
    if (CH + 1 < nch) {
      read_block(R0, IC<CUR>{}, IC<(2 * CH + 2) & 3>{});
    } else if (b + 1 < nbands) {
      wait_vmcnt<0>();
      __syncthreads();
      if (b + 2 < nbands) issue_band(b + 2, CUR);
      read_block(R0, IC<1 - CUR>{}, IC<0>{});
    }
    mfma_tile(acc, R1.ah, R1.al, operand_hi(R1), operand_lo(R1), false);
    flush_tile<PARTIALS>(acc, sum, j0 + 2 * b + CH, a.partials, a.O, colc, CRS, mrow, a.K, cvalid);
  };
  auto do_band = [&](auto curc, int32_t b) __attribute__((always_inline)) {
    const int32_t nch = min(2, (NB - 4 * b) >> 1);
    do_chunk(curc, IC<0>{}, b, nch);
    if (nch > 1) do_chunk(curc, IC<1>{}, b, nch);
  };

  issue_band(0, 0);
  wait_vmcnt<0>();
  __syncthreads();
  if (nbands > 1) issue_band(1, 1);
  read_block(R0, IC<0>{}, IC<0>{});
  for (int32_t b = 0; b < nbands; b += 2) {
    do_band(IC<0>{}, b);
    if (b + 1 < nbands) do_band(IC<1>{}, b + 1);
  }

  // Stores: a 64-bit base per workgroup, the lane's column and half in the
  // vector offset and each value's row in the uniform one (whole 64-row
  // tiles); the ragged last tile checks its rows.
  const int32_t ln = fresh_lane();
  const int32_t ocol = col0 + (wave & 3) * 32 + (ln & 31);
  const int32_t orow = m0 + 32 * rt + 4 * (ln >> 5);
  if (ocol < CRS) {
    float* dst = a.nseg == 1 ? a.out : a.useg + (int64_t)g * a.O;
    if (m0 + kMT <= a.K) {
      const __amdgpu_buffer_rsrc_t rs_o = make_rsrc(dst, (uint32_t)a.O * 4u);
      const uint32_t lane_off = (uint32_t)(4 * (ln >> 5) * CRS + ocol) * 4u;
      const uint32_t row0 = (uint32_t)(m0 + 32 * rt);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float y = a.nseg == 1 ? ldexpf(sum[v], e) : sum[v];
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(y), rs_o, lane_off,
                                              (row0 + (uint32_t)(8 * (v >> 2) + (v & 3))) * (uint32_t)CRS * 4u, 0);
      }
    } else {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int32_t m = orow + 8 * (v >> 2) + (v & 3);
        if (m < a.K) dst[m * CRS + ocol] = a.nseg == 1 ? ldexpf(sum[v], e) : sum[v];
      }
    }
  }
}

// dW = 2^e * (((U_0 + U_1) + U_2) + ...), segment order.
__global__ __launch_bounds__(64) void k_seg_reduce(const float* __restrict__ useg, float* __restrict__ out, int64_t O,
                                                  int32_t nseg, const dfp_scale* ea, const dfp_scale* eb) {
  const int64_t o = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (o >= O) return;
  float s = 0.f;
  int32_t g = 0;
  for (; g + 32 <= nseg; g += 32) {  // 32 loads in flight per lane
    float v[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) v[i] = useg[(int64_t)(g + i) * O + o];
#pragma unroll
    for (int i = 0; i < 32; ++i) s += v[i];
  }
  for (; g + 8 <= nseg; g += 8) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = useg[(int64_t)(g + i) * O + o];
#pragma unroll
    for (int i = 0; i < 8; ++i) s += v[i];
  }
  for (; g < nseg; ++g) s += useg[(int64_t)g * O + o];
  out[o] = ldexpf(s, ea->exp + eb->exp);
}

inline int64_t align256(int64_t v) { return (v + 255) & ~(int64_t)255; }

// 1-D grid of bwdw_tile; sets the tile counts in args.
dim3 bwdw_grid(BwdwArgs& args, const BwdwPlan& p) {
  args.ntx = (int32_t)((args.O / args.K + kNT - 1) / kNT);
  args.nty = p.Mp / kMT;
  return dim3((unsigned)(p.nseg * args.ntx * args.nty));
}

}  // namespace

// The band kernels read LDS with inline assembly and wait for the reads
// explicitly (see no_scratch): a band kernel is used only if its build has no
// scratch, else the general kernel (ordinary LDS reads) runs.
// The build also checks the assembly of these kernels (asm_check.py: no
// instruction names a register of an LDS read before the wait that completes
// it) and defines DFP_ASM_UNSAFE_* = 1 for a kernel that fails.
#ifndef DFP_ASM_UNSAFE_BAND_W8
#define DFP_ASM_UNSAFE_BAND_W8 0
#endif
#ifndef DFP_ASM_UNSAFE_BAND_W8_PARTIALS
#define DFP_ASM_UNSAFE_BAND_W8_PARTIALS 0
#endif
#ifndef DFP_ASM_UNSAFE_BAND_SKEW
#define DFP_ASM_UNSAFE_BAND_SKEW 0
#endif
#ifndef DFP_ASM_UNSAFE_BAND_SKEW_PARTIALS
#define DFP_ASM_UNSAFE_BAND_SKEW_PARTIALS 0
#endif
#ifndef DFP_ASM_UNSAFE_BAND
#define DFP_ASM_UNSAFE_BAND 0
#endif
#ifndef DFP_ASM_UNSAFE_BAND_FLAT
#define DFP_ASM_UNSAFE_BAND_FLAT 0
#endif
#ifndef DFP_ASM_UNSAFE_BAND_PARTIALS
#define DFP_ASM_UNSAFE_BAND_PARTIALS 0
#endif
struct BandKernelsSafe {
  bool w8, w8_t, skew_t, skew_f, band_t, band_f, w8_r4, w8_big, flat, flat_t;
};
static const BandKernelsSafe& band_kernels_safe() {
  static const BandKernelsSafe safe{
      !DFP_ASM_UNSAFE_BAND_W8 && no_scratch(reinterpret_cast<const void*>(&k_bwdw_band_w8<false>)),
      !DFP_ASM_UNSAFE_BAND_W8_PARTIALS && no_scratch(reinterpret_cast<const void*>(&k_bwdw_band_w8<true>)),
      !DFP_ASM_UNSAFE_BAND_SKEW_PARTIALS && no_scratch(reinterpret_cast<const void*>(&k_bwdw_band_skew<true>)),
      !DFP_ASM_UNSAFE_BAND_SKEW && no_scratch(reinterpret_cast<const void*>(&k_bwdw_band_skew<false>)),
      !DFP_ASM_UNSAFE_BAND_PARTIALS && no_scratch(reinterpret_cast<const void*>(&k_bwdw_band<true>)),
      !DFP_ASM_UNSAFE_BAND && no_scratch(reinterpret_cast<const void*>(&k_bwdw_band<false>)),
      !DFP_ASM_UNSAFE_BAND_W8 && no_scratch(reinterpret_cast<const void*>(&k_bwdw_band_w8<false, 4>)),
      !DFP_ASM_UNSAFE_BAND_W8 &&
          no_scratch(reinterpret_cast<const void*>(&k_bwdw_band_w8<false, 8, kBandBufBigBytes>)),
      !DFP_ASM_UNSAFE_BAND_FLAT && no_scratch(reinterpret_cast<const void*>(&k_bwdw_flat<16>)) &&
          no_scratch(reinterpret_cast<const void*>(&k_bwdw_flat<32>)) &&
          no_scratch(reinterpret_cast<const void*>(&k_bwdw_flat<64>)) &&
          no_scratch(reinterpret_cast<const void*>(&k_bwdw_flat<128>)) &&
          no_scratch(reinterpret_cast<const void*>(&k_bwdw_flat<240>)),
      !DFP_ASM_UNSAFE_BAND_FLAT && no_scratch(reinterpret_cast<const void*>(&k_bwdw_flat<16, true>)) &&
          no_scratch(reinterpret_cast<const void*>(&k_bwdw_flat<32, true>)) &&
          no_scratch(reinterpret_cast<const void*>(&k_bwdw_flat<64, true>)) &&
          no_scratch(reinterpret_cast<const void*>(&k_bwdw_flat<128, true>)) &&
          no_scratch(reinterpret_cast<const void*>(&k_bwdw_flat<240, true>))};
  return safe;
}

// A 1x1 convolution without padding and with stride (sh, sw) reads input
// pixel (p*sh, q*sw) for output pixel (p, q), so its weight gradient is the
// unit-stride one over the subsampled input x[:, :, ::sh, ::sw] (N x C x P x
// Q), with the same reduction index t = (n*P + p)*Q + q and hence the same
// chunks and segments.  The subsampled input is gathered into the workspace
// and the unit-stride kernels run on it (their input band then spans P*Q
// pixels per image instead of H*W).
static bool strided_1x1(const Geom& g) {
  // (k_subsample indexes a plane and sizes its grid with 32 bits)
  return g.r == 1 && g.s == 1 && g.ph == 0 && g.pw == 0 && (g.sh > 1 || g.sw > 1) &&
         (int64_t)g.h * g.w < (1ll << 31) - 256;
}
// Unit-stride 1x1 layers without padding (x is then a C x T matrix like dy).
static bool unit_1x1(const Geom& g) {
  return g.r == 1 && g.s == 1 && g.ph == 0 && g.pw == 0 && g.sh == 1 && g.sw == 1;
}
static Geom subsampled(const Geom& g) {
  Geom u = g;
  u.h = g.p;
  u.w = g.q;
  u.sh = u.sw = 1;
  return u;
}

namespace {
// Thread (x, y): in-plane position pq of every subsampled plane (n, c) =
// y, y + gridDim.y, ...; its source offset in the plane is computed once.
__global__ __launch_bounds__(256) void k_subsample(const int16_t* __restrict__ x, int16_t* __restrict__ xs,
                                                   int64_t planes, int32_t H, int32_t W, int32_t P, int32_t Q,
                                                   int32_t sh, int32_t sw) {
  const int32_t pq = blockIdx.x * 256 + threadIdx.x;
  if (pq >= P * Q) return;
  const int32_t pp = pq / Q, qq = pq - pp * Q;
  const int32_t off = pp * sh * W + qq * sw;
  for (int64_t nc = blockIdx.y; nc < planes; nc += gridDim.y) xs[nc * P * Q + pq] = x[nc * H * W + off];
}
}  // namespace

// Layers the flat-band kernel takes: 3x3 filters with unit stride and one
// pixel of padding (so H = P and W = Q) on images up to 239 wide, chunks of 64
// indices and whole chunks only.  Its workspace (in the x-operand region): the
// planes XF[C][2][plane] with halo bytes before t = 0 (the smallest built
// halo of at least W + 1) and, from byte tab on, the selector table of
// T / 64 + 2 groups (a band reads the group after its last one).
struct FlatLayout {
  int32_t halo, plane, ngroups;
  int64_t tab, bytes;
};
static int32_t flat_halo(int32_t w) {
  for (int32_t h : {16, 32, 64, 128, 240})
    if (w + 1 <= h) return h;
  return 0;
}
static bool flat_geom(const Geom& g) {
  const int64_t T = (int64_t)g.n * g.p * g.q;
  return g.r == 3 && g.s == 3 && g.ph == 1 && g.pw == 1 && g.sh == 1 && g.sw == 1 && g.h == g.p && g.w == g.q &&
         flat_halo(g.q) > 0 && g.L == 64 && T % 64 == 0 && T + 1024 < (1ll << 31);
}
static FlatLayout flat_layout(const Geom& g) {
  const int64_t T = (int64_t)g.n * g.p * g.q;
  FlatLayout f{};
  f.halo = flat_halo(g.q);
  // a band starts at t_b0 <= T - 64 and reads plane bytes t_b0 .. t_b0 + 2 halo + 143
  f.plane = (int32_t)((T - 64 + 2 * f.halo + kSBT + 16 + 15) / 16 * 16);
  f.ngroups = (int32_t)(T / 64 + 2);
  f.tab = align256((int64_t)g.c * 2 * f.plane);
  f.bytes = f.tab + (int64_t)f.ngroups * kFlatRS * 64;
  return f;
}

BwdwPlan plan_bwdw_mfma(const Geom& g) {
  if (strided_1x1(g)) {
    BwdwPlan p = plan_bwdw_mfma(subsampled(g));
    p.sub_bytes = align256((int64_t)g.n * g.c * g.p * g.q * 2);
    p.bytes += p.sub_bytes;
    return p;
  }
  BwdwPlan p{};
  p.T = (int64_t)g.n * g.p * g.q;
  p.KBT = (p.T + 31) / 32;
  p.Mp = (g.k + kMT - 1) / kMT * kMT;
  p.Hpad = g.h + 2 * g.ph;
  p.Wpad = (g.w + 2 * g.pw + 7) / 8 * 8;
  const int64_t J = (p.T + g.L - 1) / g.L;
  p.nseg = (int32_t)((J + g.G - 1) / g.G);
  // largest band (padded rows touched by kSBT consecutive indices of a segment)
  const int64_t PQ = (int64_t)g.p * g.q;
  int64_t rows_max = 0;
  const int64_t seg_len = (int64_t)g.G * g.L;
  for (int64_t s = 0; s < p.nseg; ++s) {
    const int64_t t0 = s * seg_len, t1 = std::min(t0 + seg_len, p.T);
    for (int64_t sb = t0 / 32; sb < (t1 + 31) / 32; sb += kSBT / 32) {
      const int64_t ta = std::max(sb * 32, t0), tb = std::min((sb + kSBT / 32) * 32, t1) - 1;
      const int64_t za = (ta / PQ) * p.Hpad + ((ta % PQ) / g.q) * g.sh;
      const int64_t zb = (tb / PQ) * p.Hpad + ((tb % PQ) / g.q) * g.sh + g.r - 1;
      rows_max = std::max(rows_max, zb - za + 1);
    }
  }
  const int64_t RS = (int64_t)g.r * g.s;
  p.nch_max = (int32_t)std::min<int64_t>(g.c, (kNT - 1) / RS + 2);
  p.rows_max = (int32_t)rows_max;
  p.band_ch_stride = (int32_t)(rows_max * p.Wpad);
  p.band_bytes = align256((int64_t)p.nch_max * p.band_ch_stride * 2);
  p.smem_bytes = p.band_bytes + kSBT * 4;
  p.ad_bytes = align256(p.KBT * p.Mp * 64);
  // pair layout [C][N*Hpad][Wpad] u16, or the band kernel's byte planes with 16 spare bytes per row
  p.xp_bytes = align256((int64_t)g.c * g.n * p.Hpad * (2 * p.Wpad + 16));
  if (unit_1x1(g)) p.xp_bytes = std::max<int64_t>(p.xp_bytes, align256(p.KBT * ((g.c + 63) / 64 * 64) * 64));
  if (flat_geom(g)) p.xp_bytes = std::max<int64_t>(p.xp_bytes, align256(flat_layout(g).bytes));
  p.u_bytes = p.nseg > 1 ? align256((int64_t)p.nseg * g.k * g.c * RS * 4) : 0;
  p.bytes = p.ad_bytes + p.xp_bytes + p.u_bytes;
  return p;
}

// Band kernel geometry: row stride, channel stride (bytes), bytes per buffer
// and run length (reduction indices per run: 8 when output and input widths
// are multiples of 8, 4 when they are multiples of 4, which only the
// eight-wave kernel reads); buf_bytes = 0 when the layer does not meet the
// kernels' conditions.
struct BandLayout {
  int32_t row_bytes, ch_stride, buf_bytes, run;
  bool big;  // buffers beyond two workgroups' share of LDS: the eight-wave kernel's one-workgroup build only
};
static BandLayout band_layout(const Geom& g, const BwdwPlan& p) {
  BandLayout bl{0, 0, 0, 0, false};
  const int32_t run = (g.q % 8) == 0 && (g.w % 8) == 0 ? 8 : (g.q % 4) == 0 && (g.w % 4) == 0 ? 4 : 0;
  if (run == 0 || g.sh != 1 || g.sw != 1 || g.s > 4 || g.pw >= 4 || (g.L % 32) != 0 || (p.T % 32) != 0 ||
      p.T >= (1ll << 31))
    return bl;
  bl.row_bytes = 2 * p.Wpad + 16;
  // channel stride congruent to 64 mod 256: with the odd row stride above, the
  // (channel, filter row) pairs of a wave fall on distinct LDS bank groups
  int64_t chs = (int64_t)p.rows_max * bl.row_bytes;
  chs += (64 - chs % 256 + 256) % 256;
  const int64_t buf = kBandABytes + p.nch_max * chs;
  if (buf > kBandBufBigBytes) return bl;
  bl.big = 2 * buf > kBandLdsBytes;
  bl.ch_stride = (int32_t)chs;
  bl.buf_bytes = (int32_t)buf;
  bl.run = run;
  return bl;
}

bool bwdw_mfma_supported(const Geom& g) {
  const BwdwPlan p = plan_bwdw_mfma(g);
  return p.smem_bytes <= 64 * 1024;
}

dfp_status launch_bwdw_mfma(const Geom& g, const int16_t* x, const dfp_scale* sx, const int16_t* dy,
                            const dfp_scale* sdy, float* dw, int32_t* partials, void* ws, hipStream_t st) {
  if (strided_1x1(g)) {
    const BwdwPlan p = plan_bwdw_mfma(g);
    int16_t* xs = reinterpret_cast<int16_t*>(reinterpret_cast<uint8_t*>(ws) + (p.bytes - p.sub_bytes));
    const int64_t planes = (int64_t)g.n * g.c;
    const int32_t gx = (g.p * g.q + 255) / 256;
    const int64_t gy = std::max<int64_t>(1, std::min<int64_t>(planes, std::max(1, 16384 / gx)));
    DFP_LAUNCH(K_XPREP, k_subsample, dim3((unsigned)gx, (unsigned)gy), dim3(256), 0, st, x, xs, planes, g.h, g.w,
               g.p, g.q, g.sh, g.sw);
    // the subsampled plan's workspace ends where xs begins
    return launch_bwdw_mfma(subsampled(g), xs, sx, dy, sdy, dw, partials, ws, st);
  }
  const BwdwPlan p = plan_bwdw_mfma(g);
  uint8_t* base = reinterpret_cast<uint8_t*>(ws);
  uint8_t* ad = base;
  uint16_t* xp = reinterpret_cast<uint16_t*>(base + p.ad_bytes);
  float* useg = reinterpret_cast<float*>(base + p.ad_bytes + p.xp_bytes);
  const DyPrep dq{dy, ad, g.k, p.Mp, g.p * g.q, (int32_t)p.T, (int32_t)p.KBT};
  const int64_t dy_blocks = (p.KBT * p.Mp * 2 + 255) / 256;
  // unit-stride 1x1 without partials: both operands as digit blocks (the
  // digit preparation indexes elements with 32 bits)
  if (unit_1x1(g) && !partials && (g.L % 32) == 0 && (int64_t)g.n * std::max(g.c, g.k) * g.p * g.q < (1ll << 31)) {
    const int32_t Cp = (g.c + 63) / 64 * 64;
    uint8_t* bd = reinterpret_cast<uint8_t*>(xp);
    const int32_t PQ = g.p * g.q;
    // P*Q a multiple of 4: the INT16 tensors are read directly (staged through
    // LDS, buffer loads over tensors below 2 GiB)
    const bool direct = PQ % 4 == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                        (reinterpret_cast<uintptr_t>(dy) & 15) == 0 &&
                        p.T * std::max(g.c, g.k) * 2 < (1ll << 31);
    if (!direct) {
      const DyPrep dqx{x, bd, g.c, Cp, PQ, (int32_t)p.T, (int32_t)p.KBT};
      DFP_LAUNCH(K_WPREP, k_prep_dy, dim3((unsigned)dy_blocks), dim3(256), 0, st, dq);
      DFP_LAUNCH(K_XPREP, k_prep_dy, dim3((unsigned)((p.KBT * Cp * 2 + 255) / 256)), dim3(256), 0, st, dqx);
    }
    const Raw1x1 raw{dy, x, PQ};
    BwdwArgs args{};
    args.ad = ad;
    args.ea = sx;
    args.eb = sdy;
    args.out = dw;
    args.useg = useg;
    args.T = p.T;
    args.O = (int64_t)g.k * g.c;
    args.K = g.k; args.Mp = p.Mp; args.C = g.c; args.R = 1; args.S = 1;
    args.L = g.L; args.G = g.G; args.nseg = p.nseg;
    args.ntx = Cp / 64;
    args.nty = p.Mp / 64;
    const dim3 grid1((unsigned)(p.nseg * args.ntx * args.nty));
    args.div_q = make_fastdiv((uint32_t)PQ);  // the direct kernels: image of an index
    if (direct && PQ % 8 == 0) DFP_LAUNCH(K_BWDW_MFMA, k_bwdw_1x1s<8>, grid1, dim3(k1x1Threads), 0, st, args, raw);
    else if (direct) DFP_LAUNCH(K_BWDW_MFMA, k_bwdw_1x1s<4>, grid1, dim3(k1x1Threads), 0, st, args, raw);
    else DFP_LAUNCH(K_BWDW_MFMA, k_bwdw_1x1, grid1, dim3(k1x1Threads), 0, st, args, bd, Cp);
    if (p.nseg > 1)
      DFP_LAUNCH(K_BWDW_REDUCE, k_seg_reduce, dim3((unsigned)((args.O + 63) / 64)), dim3(64), 0, st, useg, dw,
                 args.O, p.nseg, sx, sdy);
    return DFP_OK;
  }
  const BandLayout bl = band_layout(g, p);
  // the band kernels address both digit tensors with 32-bit buffer offsets
  const BandKernelsSafe& safe = band_kernels_safe();
  if (flat_geom(g) && (partials ? safe.flat_t : safe.flat) && p.ad_bytes < (1ll << 31) &&
      flat_layout(g).bytes < (1ll << 31) && (int64_t)g.k * g.c * 9 * 4 < (1ll << 32)) {
    // 3x3 same-padding layers: the flat-band kernel (also where the band
    // kernels' runs apply: it takes no per-band run table and reads every
    // operand at an immediate offset), after one preparation launch for the
    // t-ordered planes, the selector table and the dy digits
    const FlatLayout fl = flat_layout(g);
    uint8_t* xf = reinterpret_cast<uint8_t*>(xp);
    const bool vec8 = (g.p * g.q) % 8 == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0;
    const FlatPrep f{x, xf, g.c, g.p, g.q, g.p * g.q, (int32_t)p.T, fl.plane, fl.halo, fl.ngroups, (uint32_t)fl.tab,
                     vec8};
    const int32_t nbx = (int32_t)(((int64_t)g.c * (fl.plane / (vec8 ? 8 : 4)) + 255) / 256);
    const int32_t nbt = (fl.ngroups * kFlatRS * 16 + 255) / 256;
    DFP_LAUNCH(K_XPREP, k_prep_flat, dim3((unsigned)(nbx + nbt + dy_blocks)), dim3(256), 0, st, f, dq, nbx, nbt);
    BwdwArgs args{};
    args.ad = ad;
    args.xb = xf;
    args.ea = sx;
    args.eb = sdy;
    args.out = dw;
    args.useg = useg;
    args.partials = partials;
    args.T = p.T;
    args.O = (int64_t)g.k * g.c * 9;
    args.K = g.k; args.Mp = p.Mp; args.C = g.c; args.R = 3; args.S = 3;
    args.P = g.p; args.Q = g.q; args.sh = 1; args.sw = 1;
    args.L = g.L; args.G = g.G; args.nseg = p.nseg;
    args.ad_bytes = (uint32_t)p.ad_bytes;
    args.xb_bytes = (uint32_t)fl.bytes;
    args.flat_plane = fl.plane;
    args.flat_tab = (uint32_t)fl.tab;
    const dim3 grid = bwdw_grid(args, p);
#define DFP_FLAT(H)                                                                                  \
  do {                                                                                               \
    if (partials) DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_flat<H, true>), grid, dim3(kThreadsW8), 0, st, args); \
    else DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_flat<H, false>), grid, dim3(kThreadsW8), 0, st, args);         \
  } while (0)
    switch (fl.halo) {
      case 16: DFP_FLAT(16); break;
      case 32: DFP_FLAT(32); break;
      case 64: DFP_FLAT(64); break;
      case 128: DFP_FLAT(128); break;
      default: DFP_FLAT(240); break;
    }
#undef DFP_FLAT
    if (p.nseg > 1)
      DFP_LAUNCH(K_BWDW_REDUCE, k_seg_reduce, dim3((unsigned)((args.O + 63) / 64)), dim3(64), 0, st, useg, dw,
                 args.O, p.nseg, sx, sdy);
    return DFP_OK;
  }
  const bool l64 = g.L == 64 && (p.T % 64) == 0;  // every segment a whole number of two-block chunks
  // runs of 4 and big buffers: the eight-wave kernel only (L = 64, no partials)
  const bool band_ok = bl.big ? (bl.run == 8 && l64 && !partials && safe.w8_big)
                       : bl.run == 8 ? (l64 ? (partials ? safe.skew_t : (safe.w8 || safe.skew_f))
                                            : (partials ? safe.band_t : safe.band_f))
                                     : (l64 && !partials && safe.w8_r4);
  if (band_ok && bl.buf_bytes > 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 && p.ad_bytes < (1ll << 31) &&
      p.xp_bytes < (1ll << 31)) {
    uint8_t* xb = reinterpret_cast<uint8_t*>(xp);  // same workspace region as the pair layout
    // one launch prepares both operands: rows of workgroups 0 .. C-1 the x
    // planes, the rows after them the dy digits
    const int64_t per_c = (int64_t)g.n * p.Hpad * (p.Wpad / 8);
    const int64_t gx = (per_c + 255) / 256;
    const int64_t gy_dy = (dy_blocks + gx - 1) / gx;
    const bool merged = g.c + gy_dy <= 65535;  // grid y limit; else dy gets its own launch
    if (!merged) DFP_LAUNCH(K_WPREP, k_prep_dy, dim3((unsigned)dy_blocks), dim3(256), 0, st, dq);
    const dim3 grid_xb((unsigned)gx, (unsigned)(g.c + (merged ? gy_dy : 0)));
#define DFP_PREP_XB(PW, VEC)                                                                                  \
  DFP_LAUNCH(K_XPREP, (k_prep_xb<PW, VEC>), grid_xb, dim3(256), 0, st, x, xb, g.n, g.c, g.h, g.w, p.Hpad, p.Wpad, \
             g.ph, bl.row_bytes, dq)
    if (bl.run == 8) {
      if (g.pw == 0) DFP_PREP_XB(0, 8);
      else if (g.pw == 1) DFP_PREP_XB(1, 8);
      else if (g.pw == 2) DFP_PREP_XB(2, 8);
      else DFP_PREP_XB(3, 8);
    } else {
      if (g.pw == 0) DFP_PREP_XB(0, 4);
      else if (g.pw == 1) DFP_PREP_XB(1, 4);
      else if (g.pw == 2) DFP_PREP_XB(2, 4);
      else DFP_PREP_XB(3, 4);
    }
#undef DFP_PREP_XB
    BwdwArgs args{};
    args.ad = ad;
    args.xb = xb;
    args.ea = sx;
    args.eb = sdy;
    args.out = dw;
    args.useg = useg;
    args.partials = partials;
    args.T = p.T;
    args.O = (int64_t)g.k * g.c * g.r * g.s;
    args.K = g.k; args.Mp = p.Mp; args.C = g.c; args.R = g.r; args.S = g.s;
    args.P = g.p; args.Q = g.q; args.sh = 1; args.sw = 1;
    args.Hpad = p.Hpad; args.Wpad = p.Wpad; args.NH = g.n * p.Hpad;
    args.L = g.L; args.G = g.G; args.nseg = p.nseg;
    args.rows_max = p.rows_max;
    args.nch_max = p.nch_max;
    args.band_ch_stride = bl.ch_stride;
    args.buf_bytes = bl.buf_bytes;
    args.row_bytes = bl.row_bytes;
    args.ad_bytes = (uint32_t)p.ad_bytes;
    args.div_q = make_fastdiv((uint32_t)g.q);
    args.div_p = make_fastdiv((uint32_t)g.p);
    args.xb_bytes = (uint32_t)p.xp_bytes;
    const dim3 grid = bwdw_grid(args, p);
    if (bl.big) {
      DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_band_w8<false, 8, kBandBufBigBytes>), grid, dim3(kThreadsW8), 0, st, args);
    } else if (bl.run == 4) {
      DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_band_w8<false, 4>), grid, dim3(kThreadsW8), 0, st, args);
    } else if (l64) {
      // partials: the eight-wave kernel built for two waves per SIMD (its
      // partial stores need more than 128 VGPRs), else the two-tile kernel
      // (same chunks, same order of additions)
      if (partials && safe.w8_t) DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_band_w8<true>), grid, dim3(kThreadsW8), 0, st, args);
      else if (partials) DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_band_skew<true>), grid, dim3(kThreads), 0, st, args);
      else if (safe.w8) DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_band_w8<false>), grid, dim3(kThreadsW8), 0, st, args);
      else DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_band_skew<false>), grid, dim3(kThreads), 0, st, args);
    } else {
      if (partials) DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_band<true>), grid, dim3(kThreads), 0, st, args);
      else DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_band<false>), grid, dim3(kThreads), 0, st, args);
    }
    if (p.nseg > 1) {
      DFP_LAUNCH(K_BWDW_REDUCE, k_seg_reduce, dim3((unsigned)((args.O + 63) / 64)), dim3(64), 0, st, useg, dw,
                 args.O, p.nseg, sx, sdy);
    }
    return DFP_OK;
  }
  DFP_LAUNCH(K_WPREP, k_prep_dy, dim3((unsigned)dy_blocks), dim3(256), 0, st, dq);
  {
    const int64_t per_c = (int64_t)g.n * p.Hpad * (p.Wpad / 8);
    const dim3 grid_xp((unsigned)((per_c + 255) / 256), (unsigned)g.c);
    const bool vec = (g.w % 8) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 && g.pw < 4;
    if (vec && g.pw == 0)
      DFP_LAUNCH(K_XPREP, k_prep_xp_vec<0>, grid_xp, dim3(256), 0, st, x, xp, g.n, g.c, g.h, g.w, p.Hpad, p.Wpad, g.ph);
    else if (vec && g.pw == 1)
      DFP_LAUNCH(K_XPREP, k_prep_xp_vec<1>, grid_xp, dim3(256), 0, st, x, xp, g.n, g.c, g.h, g.w, p.Hpad, p.Wpad, g.ph);
    else if (vec && g.pw == 2)
      DFP_LAUNCH(K_XPREP, k_prep_xp_vec<2>, grid_xp, dim3(256), 0, st, x, xp, g.n, g.c, g.h, g.w, p.Hpad, p.Wpad, g.ph);
    else if (vec)
      DFP_LAUNCH(K_XPREP, k_prep_xp_vec<3>, grid_xp, dim3(256), 0, st, x, xp, g.n, g.c, g.h, g.w, p.Hpad, p.Wpad, g.ph);
    else
      DFP_LAUNCH(K_XPREP, k_prep_xp, grid_xp, dim3(256), 0, st, x, xp, g.n, g.c, g.h, g.w, p.Hpad, p.Wpad, g.ph, g.pw);
  }
  BwdwArgs args{};
  args.ad = ad;
  args.xp = xp;
  args.ea = sx;
  args.eb = sdy;
  args.out = dw;
  args.useg = useg;
  args.partials = partials;
  args.T = p.T;
  args.O = (int64_t)g.k * g.c * g.r * g.s;
  args.K = g.k; args.Mp = p.Mp; args.C = g.c; args.R = g.r; args.S = g.s;
  args.P = g.p; args.Q = g.q; args.sh = g.sh; args.sw = g.sw;
  args.Hpad = p.Hpad; args.Wpad = p.Wpad; args.NH = g.n * p.Hpad;
  args.L = g.L; args.G = g.G; args.nseg = p.nseg;
  args.band_bytes = (int32_t)p.band_bytes;
  args.band_ch_stride = p.band_ch_stride;
  const dim3 grid = bwdw_grid(args, p);
  const bool masked = (g.L % 32) != 0;
  const size_t smem = (size_t)p.smem_bytes;
  if (masked) {
    if (partials) DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_mfma<true, true>), grid, dim3(kThreads), smem, st, args);
    else DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_mfma<true, false>), grid, dim3(kThreads), smem, st, args);
  } else {
    if (partials) DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_mfma<false, true>), grid, dim3(kThreads), smem, st, args);
    else DFP_LAUNCH(K_BWDW_MFMA, (k_bwdw_mfma<false, false>), grid, dim3(kThreads), smem, st, args);
  }
  if (p.nseg > 1) {
    DFP_LAUNCH(K_BWDW_REDUCE, k_seg_reduce, dim3((unsigned)((args.O + 63) / 64)), dim3(64), 0, st, useg, dw,
               args.O, p.nseg, sx, sdy);
  }
  return DFP_OK;
}

}  // namespace dfp
