// Internal interface of the backward-weights MFMA kernels.
#pragma once

#include <algorithm>

#include "dfp_internal.h"

namespace dfp {

struct BwdwPlan {
  int64_t T, KBT;                       // reduction length, blocks of 32
  int32_t Mp, Hpad, Wpad, nseg;         // padded rows of dy digits, padded x rows / row width, segments
  int32_t nch_max, rows_max, band_ch_stride;
  int64_t band_bytes, smem_bytes;       // LDS band (all channels of a column tile) + offset table
  int64_t ad_bytes, xp_bytes, u_bytes, bytes;
  int64_t sub_bytes;                    // strided 1x1: the subsampled input, at the end of the workspace
};

struct BwdwArgs {
  const uint8_t* ad;      // dy digits [KBT][Mp][2][32]
  const uint16_t* xp;     // x digit pairs [C][N*Hpad][Wpad]
  const uint8_t* xb;      // x digit planes [C][N*Hpad][2][Wpad] (band kernel)
  const dfp_scale* ea;    // x scale
  const dfp_scale* eb;    // dy scale
  float* out;             // dW [K][C][R][S]
  float* useg;            // segment sums [nseg][K*C*R*S]
  int32_t* partials;
  int64_t T, O;
  int32_t K, Mp, C, R, S, P, Q, sh, sw, Hpad, Wpad, NH, L, G, nseg, band_bytes, band_ch_stride;
  int32_t rows_max, nch_max, buf_bytes, row_bytes;  // band kernel: rows / channels per band, buffer and row bytes
  int32_t ntx, nty;  // column tiles and row tiles per segment (the grid is 1-D, see bwdw_grid)
  uint32_t ad_bytes, xb_bytes;  // sizes of the two digit tensors (band kernels: buffer bounds)
  FastDiv div_q, div_p;         // division by Q and by P (band-table positions)
  int32_t flat_plane;           // flat-band kernel: bytes per digit plane of the t-ordered input
  uint32_t flat_tab;            // flat-band kernel: byte offset of the selector table after the planes
};

BwdwPlan plan_bwdw_mfma(const Geom& g);
bool bwdw_mfma_supported(const Geom& g);
dfp_status launch_bwdw_mfma(const Geom& g, const int16_t* x, const dfp_scale* sx, const int16_t* dy,
                            const dfp_scale* sdy, float* dw, int32_t* partials, void* ws, hipStream_t st);

}  // namespace dfp
