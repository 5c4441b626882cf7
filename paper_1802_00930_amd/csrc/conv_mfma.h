// Internal interface of the MFMA convolution kernels.
#pragma once

#include "dfp_internal.h"

namespace dfp {

// Workspace plan of the forward / backward-data MFMA path.
struct ConvMfmaPlan {
  int32_t M, Mp, Cin, T, KB, CG;   // output channels (padded), reduction channels, T, 32-blocks, 16-groups
  int32_t Hp, Wp, top, left, dil_h, dil_w;  // channels-last digit tensor geometry
  int32_t Po, Qo;                  // output spatial size
  int64_t ws_a_bytes, ws_b_bytes, ws_t_bytes, bytes;
};

struct ConvMfmaArgs {
  const uint8_t* xs;    // B digits [n][Hp][Wp][CG][32]
  const uint8_t* wsa;   // A digits [KB][Mp][2][32]
  const int2* boff;     // per block: byte offsets into xs of its two 16-channel halves (tap and group)
  const dfp_scale* ea;  // exponent of the B-source tensor
  const dfp_scale* eb;  // exponent of the filter
  float* out;
  dfp_scale* so;
  int32_t* partials;
  int64_t NP, O;
  int32_t M, Mp, Cin, S, T, KB, L, CG, Hp, Wp, Po, Qo;
  int32_t ustride_h, ustride_w, rsign, roff_h, roff_w;
  // Blocked-DFP (nullable): int8 exponents [nb][M] of the A rows and [nb][NP]
  // of the B columns, one per block of bk reduction indices (bk a multiple of L)
  const int8_t* exa;
  const int8_t* exb;
  int32_t bk, nb;
  // 1: xs is in the plane layout [n][Hp][Cin/32][digit][half][Wp][16 B] (the
  // 16 channels of one half-block and one digit of consecutive columns are
  // adjacent), written for the four-waves-per-SIMD kernel; 0: [n][Hp][Wp][CG][32 B]
  int32_t plane;
  FastDiv div_pq, div_q;  // n / (Po*Qo) and n / Qo for output pixel indices
  // four-waves-per-SIMD kernel: filter blocks kb0 .. kb0 + kbn - 1 in this launch;
  // phase_flags bit 0: first phase (sums start at 0), bit 1: last (scale, store, max)
  int32_t kb0, kbn, phase_flags;
};

// The plane layout and its kernel serve 32-channel blocks (Cin a multiple of
// 32) and full chunks of two blocks (T a multiple of 64): at L = 64 any number
// of blocks, in phases of at most 36 resident blocks; one chunk over the whole
// reduction (INT32 outputs) at most 36 blocks.
bool conv_w16_eligible(int32_t Cin, int32_t T, int32_t L, bool i32);

// Largest exponent-block count the blocked matrix-core kernel stages in LDS.
constexpr int32_t kBlockedMaxBlocks = 80;

// Output rows per workgroup tile of the main kernels (A digits are padded to it).
constexpr int32_t kMfmaRowTile = 64;

ConvMfmaPlan plan_conv_mfma(const Geom& g, int32_t dir);
// Picks and launches the main kernel for prepared digit operands (args.L,
// args.partials and i32 select it); ws_b_bytes is the size of args.xs.
dfp_status launch_mfma_main(ConvMfmaArgs& args, int64_t ws_b_bytes, int kid, int kid32, bool i32, hipStream_t st);
// The B prep kernel stages one source row of at least 16 channels in LDS.
bool conv_mfma_supported(const Geom& g, int32_t dir);
dfp_status launch_conv_mfma(int32_t dir, const Geom& g, const int16_t* a, const dfp_scale* sa, const int16_t* b,
                            const dfp_scale* sb, float* out, dfp_scale* so, int32_t* partials, void* ws,
                            hipStream_t st, bool i32 = false,
                            bool prefer_w16 = false, bool so_reset = true);
// Strided 1x1 backward-data without padding through the unit-stride grid:
// workspace bytes it needs (0 if the layer does not qualify), and the launch.
int64_t conv_bwd_data_sub_bytes(const Geom& g);
// Strided backward-data split by output phase into unit-stride problems over
// the undilated dy (K a multiple of the chunk length): workspace bytes (0 if
// the layer does not qualify), and the launch.
int64_t conv_bwd_data_phase_bytes(const Geom& g);
dfp_status launch_conv_bwd_data_phases(const Geom& g, const int16_t* dy, const dfp_scale* sdy, const int16_t* w,
                                       const dfp_scale* sw, float* dx, dfp_scale* so, void* ws, hipStream_t st,
                                       bool prefer_w16);
dfp_status launch_conv_bwd_data_sub(const Geom& g, const int16_t* dy, const dfp_scale* sdy, const int16_t* w,
                                    const dfp_scale* sw, float* dx, dfp_scale* so, void* ws, hipStream_t st,
                                    bool prefer_w16);

}  // namespace dfp
