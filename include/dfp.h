/*
 * dfp.h -- C ABI of libdfp: Dynamic Fixed Point (DFP) INT16 convolution for
 * AMD Instinct MI355X (gfx950).
 *
 * Method: Das et al., "Mixed Precision Training of Convolutional Neural
 * Networks using Integer Operations", ICLR 2018.
 *   - A DFP tensor is an integer tensor I with one shared exponent Es; element
 *     n stands for i_n * 2^Es (Sec. 3, Eq. 3).
 *   - Es comes from the tensor-wide max magnitude: Es = E(max|f|) - (P - 2)
 *     with P the integer width (Sec. 3.1, Eq. 1-2); stored as an 8-bit signed
 *     value (Sec. 3).
 *   - FP (forward), BP (backward-data) and WU (backward-weights) convolutions
 *     take two DFP16 tensors and produce FP32 (Sec. 4.1).  Products are
 *     INT16 x INT16 summed into INT32 over short chains; each chain's INT32
 *     partial is converted to FP32 and accumulated with the scale 2^(Ea+Eb)
 *     (Sec. 4.2 Algorithm 2, Sec. 4.3, Eq. 4).
 *   - FP32 outputs are down-converted to DFP16 using the max of the current
 *     output and nearest, stochastic or biased rounding (Sec. 1, Sec. 4.1).
 *
 * Conventions shared by every entry point
 *   - Tensor pointers are DEVICE pointers owned by the caller.  Activations and
 *     gradients are NCHW, filters KCRS, all densely packed.  The library
 *     allocates no device memory: scratch space is the caller's `workspace`.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Every call only
 *     enqueues work on that stream and returns; nothing synchronises.
 *   - Return codes report argument errors detected on the host before any
 *     HIP call (nothing is enqueued then), or a failed launch (DFP_ERR_HIP).
 *     Conditions that depend on the data are reported in the device-side
 *     dfp_scale.flags word, readable after the stream has finished.
 *   - Outputs are overwritten, never accumulated into.
 *   - Not re-entrant on one dfp_scale: two calls in flight that write the
 *     same dfp_scale race.  Otherwise stateless and thread-safe (the optional
 *     profiler below is process-global).
 *
 * Numerics (identical in the CPU oracle used by the tests)
 *   - E(.) = floor(log2 |.|) (subnormals included).  Es = E(max|f|) - (P-2),
 *     clamped below at -128 (flag EXP_CLAMPED).  All-zero tensor: Es = 0,
 *     flag ZERO_TENSOR.  Any NaN/Inf: all integers 0, Es = 0, flag NONFINITE.
 *   - P = bits in {15, 16}.  15 is the paper's experimental setting (inputs
 *     shifted by one bit, "DFP15", Sec. 4.3): integers in [-2^14, 2^14], never
 *     saturating.  P = 16 clamps to [-32767, 32767] (flag SATURATED).
 *     Convolution operands are integers of the descriptor's P: at P = 15
 *     |i| <= 2^14 (what dfp_quantize writes), which the matrix-core path
 *     relies on (its byte digits hold |i| < 32640); larger magnitudes at P = 15
 *     give unspecified outputs.  P = 16 takes the full INT16 range.
 *   - Rounding of x = f * 2^-Es: NEAREST = ties to even; BIASED = ties toward
 *     +inf, floor(x + 1/2); STOCHASTIC = floor(x) + (U < F) with
 *     F = floor(frac(x) * 2^32) and U a Philox4x32-10 word (Salmon et al.,
 *     SC'11): key = seed, counter = (q mod 2^32, q div 2^32, role, 0),
 *     q = idx / 4, U = word idx % 4 of the block, idx = the element's flat
 *     index; DOWN = floor(x) (the plain right shift of Eq. 6).
 *   - Reduction order and chunks: chunk j holds the L consecutive reduction
 *     indices t in [jL, min(T, (j+1)L)) of
 *        forward         t = (r*S + s)*C + c      (T = C*R*S)
 *        backward-data   t = (r*S + s)*K + k      (T = K*R*S)
 *        backward-weight t = (n*P + p)*Q + q      (T = N*P*Q)
 *     Padding taps and stride holes contribute 0 and keep their slot.
 *     P_j = sum of the chunk's products modulo 2^32 (two's-complement wrap).
 *   - FP32: F_j = (float)P_j (round to nearest even).  Forward and
 *     backward-data add F_0, F_1, ... strictly in order.  Backward-weights
 *     adds chunks in order inside segments of G = seg_chunks chunks, then adds
 *     the segment sums in order.  The result is scaled once by 2^(Ea+Eb)
 *     (single rounding, gradual underflow; +-inf on overflow, flag OUTPUT_INF).
 */
#ifndef DFP_H_
#define DFP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum dfp_status {
  DFP_OK = 0,
  DFP_ERR_NULL = 1,      /* a required pointer is NULL                        */
  DFP_ERR_SHAPE = 2,     /* a dimension < 1, pad < 0, stride < 1, output < 1, or
                            an element count beyond 2^40                       */
  DFP_ERR_PARAM = 3,     /* bits, rounding, role, chunk_len, seg_chunks or path */
  DFP_ERR_ALIGN = 4,     /* FP32 src not 16-byte aligned or INT16 dst not 8-byte */
  DFP_ERR_WORKSPACE = 5, /* workspace NULL or smaller than dfp_workspace_bytes() */
  DFP_ERR_HIP = 6,       /* a HIP launch or runtime call failed                 */
  DFP_ERR_SCRATCH_LIMIT = 7 /* dfp_conv_bwd_weights_noalloc: the layer needs more
                               than DFP_NOALLOC_SCRATCH_BYTES of scratch        */
} dfp_status;

typedef enum dfp_rounding {
  DFP_ROUND_NEAREST = 0,
  DFP_ROUND_STOCHASTIC = 1,
  DFP_ROUND_BIASED = 2,
  DFP_ROUND_DOWN = 3
} dfp_rounding;

/* Role of a tensor: selects its logical shape from the descriptor
 * (X, DX: N,C,H,W;  W: K,C,R,S;  DY, Y: N,K,P,Q) and is word 2 of the Philox
 * counter, so the five tensors of a layer draw independent streams. */
typedef enum dfp_role {
  DFP_ROLE_X = 0,
  DFP_ROLE_W = 1,
  DFP_ROLE_DY = 2,
  DFP_ROLE_Y = 3,
  DFP_ROLE_DX = 4
} dfp_role;

typedef enum dfp_direction { DFP_FWD = 0, DFP_BWD_DATA = 1, DFP_BWD_WT = 2 } dfp_direction;

/* Integer-product path (the measured choice is the default).  AUTO and MFMA
 * both build exact INT16 products from int8 MFMA on byte digits and give the
 * same results; AUTO also weighs the work size when it picks the kernel (a
 * filter of more than 36 blocks of 32 reduction indices takes the
 * four-waves-per-SIMD kernel in phases only when the layer has enough output
 * pixels), MFMA takes that kernel whenever its operand layout fits. */
typedef enum dfp_path {
  DFP_PATH_AUTO = 0, /* byte-split int8 MFMA, kernel by shape and work size     */
  DFP_PATH_MFMA = 1, /* byte-split int8 MFMA, four-waves-per-SIMD kernel first  */
  DFP_PATH_VALU = 2  /* one lane per output, VALU integer multiply-add          */
} dfp_path;

#define DFP_FLAG_NONFINITE 1u    /* input held NaN or Inf                     */
#define DFP_FLAG_EXP_CLAMPED 2u  /* Es fell below -128 and was clamped        */
#define DFP_FLAG_SATURATED 4u    /* P = 16 only: an integer clamped to +-32767 */
#define DFP_FLAG_ZERO_TENSOR 8u  /* every element was zero                    */
#define DFP_FLAG_OUTPUT_INF 16u  /* a convolution output overflowed FP32      */

/* Host-side layer descriptor, read only during the call. */
typedef struct dfp_desc {
  int32_t n, c, h, w;       /* activations NCHW                                */
  int32_t k, r, s;          /* filters KCRS                                     */
  int32_t stride_h, stride_w;
  int32_t pad_h, pad_w;     /* output P = (H + 2 pad_h - R)/stride_h + 1, same Q */
  int32_t chunk_len;        /* L >= 1: products per INT32 partial               */
  int32_t seg_chunks;       /* backward-weights segment size G in chunks;
                               0 -> max(1, 4096 / L)                            */
  int32_t bits;             /* P in {15, 16}                                    */
  int32_t rounding;         /* dfp_rounding, for quantise / down-convert        */
  int32_t path;             /* dfp_path                                         */
  uint64_t seed;            /* Philox key for stochastic rounding               */
} dfp_desc;

/* Device-resident scale of one DFP tensor (16 bytes, caller-allocated). */
typedef struct dfp_scale {
  uint32_t amax_bits; /* max over elements of (bit pattern & 0x7fffffff)      */
  int32_t exp;        /* shared exponent Es (int8 range)                      */
  uint32_t flags;     /* DFP_FLAG_* bits                                      */
  uint32_t reserved;
} dfp_scale;

/* Quantise an FP32 tensor to DFP (Sec. 3.1 Eq. 1-3; the quantisers Q_a, Q_w,
 * Q_e of Sec. 4.1).  src: FP32 [numel(role)], 16-byte aligned; dst: INT16
 * [numel(role)], 8-byte aligned; s: receives amax_bits, exp and flags.
 * Enqueues a max-magnitude reduction followed by the rounding pass; the
 * reduction keeps its per-workgroup maxima in dst until the rounding pass
 * overwrites it, so dst must not alias src. */
dfp_status dfp_quantize(const dfp_desc* d, int32_t role, const float* src, int16_t* dst,
                        dfp_scale* s, void* stream);

/* Forward convolution FP (Algorithm 2, Sec. 4.3).  x: INT16 [N,C,H,W] with
 * scale sx; w: INT16 [K,C,R,S] with scale sw; y: FP32 [N,K,P,Q].
 * sy (nullable): receives max|y| in amax_bits and OUTPUT_INF, ready for
 * dfp_downconvert(..., amax_ready = 1).  partials (nullable, for tests):
 * INT32 [J][N*K*P*Q], every chunk partial P_j.  workspace: device scratch of
 * at least dfp_workspace_bytes(d, DFP_FWD) bytes, 256-byte aligned. */
dfp_status dfp_conv_fwd(const dfp_desc* d, const int16_t* x, const dfp_scale* sx, const int16_t* w,
                        const dfp_scale* sw, float* y, dfp_scale* sy, void* workspace,
                        size_t ws_bytes, int32_t* partials, void* stream);

/* Backward-data convolution BP (Sec. 4.1, the adjoint of FP):
 * dx[n,c,h,w] = sum over (r,s,k) of dy[n,k,p,q] * w[k,c,r,s] with
 * p = (h + pad_h - r)/stride_h, q = (w + pad_w - s)/stride_w when both are
 * integers in range.  dy: INT16 [N,K,P,Q]; w: INT16 [K,C,R,S];
 * dx: FP32 [N,C,H,W]; sdx, partials, workspace as for the forward call. */
dfp_status dfp_conv_bwd_data(const dfp_desc* d, const int16_t* dy, const dfp_scale* sdy,
                             const int16_t* w, const dfp_scale* sw, float* dx, dfp_scale* sdx,
                             void* workspace, size_t ws_bytes, int32_t* partials, void* stream);

/* Backward-weights convolution WU (Sec. 4.1; chains longer than a million
 * products, Sec. 4.3): dw[k,c,r,s] = sum over (n,p,q) of dy[n,k,p,q] *
 * x[n,c,p*stride_h-pad_h+r, q*stride_w-pad_w+s].  x: INT16 [N,C,H,W];
 * dy: INT16 [N,K,P,Q]; dw: FP32 [K,C,R,S] (not quantised, Fig. 2 caption).
 * workspace: at least dfp_workspace_bytes(d, DFP_BWD_WT) bytes. */
dfp_status dfp_conv_bwd_weights(const dfp_desc* d, const int16_t* x, const dfp_scale* sx,
                                const int16_t* dy, const dfp_scale* sdy, float* dw, void* workspace,
                                size_t ws_bytes, int32_t* partials, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * backward-weights convolution of dfp_conv_bwd_weights, with the same
 * operands, numerics and argument errors, no partials, and no workspace
 * argument.  Its scratch (digit planes of x and dy, the per-segment FP32
 * sums) lives in a static device array of DFP_NOALLOC_SCRATCH_BYTES bytes
 * inside the library: every GPU the call runs on holds one such array from
 * the library's first use on it until the process ends.  A layer whose
 * workspace, dfp_workspace_bytes(d, DFP_BWD_WT), exceeds that size returns
 * DFP_ERR_SCRATCH_LIMIT before any HIP call.  stream (NULL = the default
 * stream) must belong to the current device, else DFP_ERR_PARAM.  Nothing in
 * the scratch needs to start at zero; the array keeps the last call's
 * contents.  Calls in flight at the same time on one GPU share the array and
 * race: order them (one stream, or events).  The call allocates nothing: no
 * hipMalloc, hipFree or allocating library routine (with the optional
 * launch profiler below switched on, it records HIP events). */
#define DFP_NOALLOC_SCRATCH_BYTES (64u << 20)
dfp_status dfp_conv_bwd_weights_noalloc(const dfp_desc* d, const int16_t* x, const dfp_scale* sx,
                                        const int16_t* dy, const dfp_scale* sdy, float* dw, void* stream);

/* Down-convert an FP32 convolution output to DFP (Sec. 1: scale from the max
 * of the current output; Sec. 4.1: Q_a after FP, Q_e after BP).  role is
 * DFP_ROLE_Y or DFP_ROLE_DX (sets the shape and the Philox stream).
 * amax_ready = 1: s->amax_bits (and flags) were produced by the convolution
 * that wrote src (its sy / sdx), so the max pass is skipped; 0: recompute
 * (dst is scratch for the max pass, as in dfp_quantize). */
dfp_status dfp_downconvert(const dfp_desc* d, int32_t role, const float* src, int16_t* dst,
                           dfp_scale* s, int32_t amax_ready, void* stream);

/* Single-chunk DFP-32 outputs (Alg. 2 with one chunk over the whole reduction,
 * Sec. 4.3: the INT32 accumulator itself, with exponent Ex + Ew).  The
 * descriptor's chunk_len must be at least the reduction length (C*R*S
 * forward, K*R*S backward-data), else DFP_ERR_PARAM.  y / dx: INT32 in the
 * layout of dfp_conv_fwd's y / dfp_conv_bwd_data's dx, each element the
 * wrapped (mod 2^32) sum of its products.  sy / sdx (required, 16-byte
 * aligned): receives exp = Ex + Ew (or Edy + Ew) and amax_bits = max |i| as an
 * unsigned integer (2^31 for -2^31), ready for dfp_downconvert_i32(...,
 * amax_ready = 1).  workspace: as for the FP32-output call of the same
 * direction. */
dfp_status dfp_conv_fwd_i32(const dfp_desc* d, const int16_t* x, const dfp_scale* sx, const int16_t* w,
                            const dfp_scale* sw, int32_t* y, dfp_scale* sy, void* workspace,
                            size_t ws_bytes, void* stream);
dfp_status dfp_conv_bwd_data_i32(const dfp_desc* d, const int16_t* dy, const dfp_scale* sdy,
                                 const int16_t* w, const dfp_scale* sw, int32_t* dx, dfp_scale* sdx,
                                 void* workspace, size_t ws_bytes, void* stream);

/* Integer down-conversion of a DFP-32 tensor <I, E_in> to DFP (Eq. 6, with the
 * shift count read so that the max lands at bit P-2 as Eq. 2 places it):
 * Rs = floor(log2 max|I|) - (P - 2) (negative Rs is an exact left shift), new
 * exponent E_in + Rs (clamped at -128 by raising Rs, flag EXP_CLAMPED), each
 * integer rounded from I * 2^-Rs in the descriptor's mode (the stochastic
 * stream of `role`, DFP_ROLE_Y or DFP_ROLE_DX); P = 16 saturates at +-32767.
 * src: INT32 [numel(role)], 16-byte aligned.  sin: exp = E_in; with
 * amax_ready = 1 also amax_bits = max |I| (the sy / sdx of the _i32
 * convolutions); amax_ready = 0 recomputes the max, using dst as scratch.
 * dst: INT16, 8-byte aligned.  sout (not sin): receives amax_bits, exp and
 * flags (ZERO_TENSOR for an all-zero tensor, exponent 0). */
dfp_status dfp_downconvert_i32(const dfp_desc* d, int32_t role, const int32_t* src, const dfp_scale* sin,
                               int16_t* dst, dfp_scale* sout, int32_t amax_ready, void* stream);

/* Device workspace needed by a convolution direction (bytes, 0 if none);
 * 0 also for an invalid descriptor. */
size_t dfp_workspace_bytes(const dfp_desc* d, int32_t direction);

/* Number of chunks J = ceil(T / L) of a direction; -1 for an invalid descriptor. */
int64_t dfp_num_chunks(const dfp_desc* d, int32_t direction);

/* ---------------------------------------------------------------- GEMM --
 * The paper's INT16 kernels serve "convolutions and GEMM" (Sec. 4); its FC
 * layers stayed FP32 in the experiments.  dfp_gemm computes
 *   D[i][j] = 2^(Ea+Eb) * fold over chunks c of fl32(P_c[i][j]),
 *   P_c[i][j] = sum over t in [cL, min(k, (c+1)L)) of opA[i][t] * opB[t][j]
 * (mod 2^32), the fold adding in chunk order in FP32 with the scale applied
 * once: the forward convolution's contract (Alg. 2, Sec. 4.3).  Layouts,
 * all row-major: opA[i][t] = a[i*k + t] (trans_a = 0) or a[t*m + i]
 * (trans_a = 1); opB[t][j] = b[t*n + j] (trans_b = 0) or b[j*k + t]
 * (trans_b = 1); D is [m][n].  A fully connected layer y = x W^T with
 * x [batch][in], W [out][in] is (m, n, k) = (batch, out, in), trans_b = 1;
 * its backward-data dx = dy W is (batch, in, out), no transposes; its
 * backward-weights dW = dy^T x is (out, in, batch), trans_a = 1. */
typedef struct dfp_gemm_desc {
  int32_t m, n, k;          /* >= 1; m*n, m*k, k*n at most 2^40                */
  int32_t trans_a, trans_b; /* 0 or 1, as above                                  */
  int32_t chunk_len;        /* L >= 1                                            */
  int32_t bits;             /* P of the operands, 15 or 16 (16: VALU path)       */
  int32_t path;             /* dfp_path                                          */
} dfp_gemm_desc;

/* a, b: INT16 operands of P = bits (at P = 15 |i| <= 2^14); sa, sb: their
 * scales (exp read on the device), 16-byte aligned.  out: FP32 [m][n].
 * sd (nullable, 16-byte aligned): cleared, then receives max |D| as FP32 bits
 * and OUTPUT_INF, ready for dfp_downconvert_tensor(..., amax_ready = 1).
 * partials (nullable): INT32 [J][m*n], every chunk partial.  workspace: at
 * least dfp_gemm_workspace_bytes(d) bytes, 256-byte aligned (the operands'
 * digit planes).  Errors as for the convolutions. */
dfp_status dfp_gemm(const dfp_gemm_desc* d, const int16_t* a, const dfp_scale* sa, const int16_t* b,
                    const dfp_scale* sb, float* out, dfp_scale* sd, void* workspace, size_t ws_bytes,
                    int32_t* partials, void* stream);
/* Workspace bytes of dfp_gemm (0 on the VALU path or for an invalid descriptor). */
size_t dfp_gemm_workspace_bytes(const dfp_gemm_desc* d);
/* J = ceil(k / L); -1 for an invalid descriptor. */
int64_t dfp_gemm_num_chunks(const dfp_gemm_desc* d);

/* dfp_quantize / dfp_downconvert for a flat tensor of n elements (GEMM
 * operands and outputs): the same numerics, bits in {15, 16}, rounding a
 * dfp_rounding, role (any dfp_role) selecting the stochastic stream.
 * Alignment, scratch use of dst and errors as for dfp_quantize. */
dfp_status dfp_quantize_tensor(int64_t n, int32_t bits, int32_t rounding, uint64_t seed, int32_t role,
                               const float* src, int16_t* dst, dfp_scale* s, void* stream);
dfp_status dfp_downconvert_tensor(int64_t n, int32_t bits, int32_t rounding, uint64_t seed, int32_t role,
                                  const float* src, int16_t* dst, dfp_scale* s, int32_t amax_ready,
                                  void* stream);

/* ----------------------------------------------------------- Blocked-DFP --
 * Several exponents per tensor, each shared by a small block of integers
 * (Sec. 3, "Blocked-DFP").  dfp_quantize_blocked splits each row of src
 * [rows][cols] (FP32, row-major) into blocks of `block` consecutive elements
 * (the last one of a row possibly shorter) and quantises every block like a
 * tensor of its own (Eq. 1-3: its own max, exponent clamp at -128, zero and
 * non-finite rules, P = 16 saturation); the stochastic word of an element is
 * that of its flat index, as in dfp_quantize.  dst: INT16 [rows][cols].
 * exps: int8 [nb][rows], nb = ceil(cols / block), block-major.  s: amax_bits
 * = max |f| of the tensor, exp = 0, flags = NONFINITE / EXP_CLAMPED /
 * SATURATED if any block has them, ZERO_TENSOR if every block is zero. */
dfp_status dfp_quantize_blocked(int64_t rows, int64_t cols, int64_t block, int32_t bits, int32_t rounding,
                                uint64_t seed, int32_t role, const float* src, int16_t* dst, int8_t* exps,
                                dfp_scale* s, void* stream);

/* Blocked-DFP GEMM: D[i][j] = fold over chunks c, in chunk order in FP32, of
 * fl32(P_c[i][j]) * 2^(ea[blk][i] + eb[blk][j]), blk = cL / block_k (Alg. 2
 * scaling each partial; chunks lie inside blocks).  Operands with the
 * reduction contiguous, as dfp_quantize_blocked writes them: a [m][k], b
 * [n][k] (the descriptor must say trans_a = 0, trans_b = 1), ea int8 [nb][m],
 * eb int8 [nb][n], nb = ceil(k / block_k).  block_k must be a multiple of
 * chunk_len.  out, sd, partials as for dfp_gemm (no final scale: every chunk
 * carries its own).  workspace: dfp_gemm_blocked_workspace_bytes(d, block_k)
 * bytes (0 when the call runs on the VALU path: P = 16, chunk_len not a
 * multiple of 32, or more than 80 blocks). */
dfp_status dfp_gemm_blocked(const dfp_gemm_desc* d, int32_t block_k, const int16_t* a, const int8_t* ea,
                            const int16_t* b, const int8_t* eb, float* out, dfp_scale* sd, void* workspace,
                            size_t ws_bytes, int32_t* partials, void* stream);
size_t dfp_gemm_blocked_workspace_bytes(const dfp_gemm_desc* d, int32_t block_k);

/* ------------------------------------------------ around the convolutions --
 * The FP32 steps either side of a layer's convolutions in a DFP16 training
 * step (Sec. 4.1, Fig. 2): batch normalisation reads DFP16 tensors and
 * up-converts them, works in FP32 and feeds Q_a (forward) or Q_e (backward)
 * with its outputs; the weight update is FP32 SGD on master weights followed
 * by Q_w.  Operation orders (every step a single IEEE rounding, no
 * contraction):
 *   statistics   S1 = sum i, S2 = sum i^2 over a channel's N*HW integers,
 *                exact in 64-bit integers; mean = fl64(S1 2^E / cnt),
 *                var = max(0, fl64(S2 2^2E / cnt) - mean*mean) in float64;
 *                mean_f = fl32(mean), inv_std = 1 / sqrt(fl32(var) + eps) in
 *                FP32;
 *   forward      v = i 2^E, xhat = (v - mean_f) * inv_std,
 *                pre = fma(xhat, gamma, beta) [+ res], z = pre > 0 ? pre : 0,
 *                then Q_a of z (role X: the next layer's input);
 *   backward     g = dz' = (pre > 0 ? dz 2^Edz : 0) with pre recomputed;
 *                D = sum of the masked dz integers, Pd = sum of masked dz * y
 *                integers (exact); dbeta = fl32(D 2^Edz), dgamma =
 *                fl32(inv_std (Pd 2^Ey - mean_f D) 2^Edz); a = gamma inv_std,
 *                k1 = fl32(a), k2 = fl32(-a dgamma / cnt), k3 = fl32(-a dbeta
 *                / cnt) in float64; dy = fma(k1, g, fma(k2, xhat, k3)), then
 *                Q_e of dy (role DY); dres = g.
 * Tensors are [n][c][hw] (NCHW with hw = H*W), at most 2^31 - 1 elements;
 * per-channel arrays are FP32 [c]; every pointer is device memory. */
typedef struct dfp_bn_desc {
  int32_t n, c, hw; /* >= 1, n*c*hw < 2^31                                     */
  int32_t bits;     /* P of the quantised output, 15 or 16                      */
  int32_t rounding; /* dfp_rounding of Q_a / Q_e                                */
  float eps;        /* finite, >= 0                                             */
  uint64_t seed;    /* Philox key of stochastic rounding                        */
} dfp_bn_desc;

/* Batch normalisation + optional residual add + ReLU forward on a DFP16
 * tensor y (INT16 [n][c][hw], exponent sy->exp), then Q_a of the result.
 * gamma, beta: FP32 [c].  res (nullable): FP32 [n][c][hw] added before the
 * ReLU.  z (nullable): receives the FP32 result.  zq: INT16 result of Q_a,
 * its scale in sz (exp, amax_bits, flags as dfp_quantize).  mean, inv_std:
 * FP32 [c] (the backward call's inputs).  sums (nullable): int64 [c][2] =
 * S1, S2.  workspace: dfp_bn_workspace_bytes(d) bytes, 256-byte aligned.
 * Without res the output max comes from each channel's smallest and largest
 * integer (z is monotone in i per channel), so the tensor is read twice;
 * with res a max pass over z runs before the rounding pass and uses zq as
 * scratch.  zq, z must not alias y or res.  Pointers to FP32 and INT16
 * tensors 16-byte aligned, scales 16-byte aligned. */
dfp_status dfp_bn_relu_fwd(const dfp_bn_desc* d, const int16_t* y, const dfp_scale* sy, const float* gamma,
                           const float* beta, const float* res, float* z, int16_t* zq, dfp_scale* sz,
                           float* mean, float* inv_std, int64_t* sums, void* workspace, size_t ws_bytes,
                           void* stream);

/* Backward of dfp_bn_relu_fwd: dz (INT16 [n][c][hw], exponent sdz->exp) is
 * the gradient at z; y, sy, gamma, beta, res, mean, inv_std as given to and
 * returned by the forward call.  dyq: INT16 Q_e of the gradient at y, scale
 * in sdy (a max pass first, with dyq as scratch).  dy (nullable): the FP32
 * gradient at y.  dgamma, dbeta: FP32 [c].  dres (nullable): the FP32
 * gradient at res (the masked dz').  sums (nullable): int64 [c][2] = D, Pd.
 * workspace as for the forward call. */
dfp_status dfp_bn_relu_bwd(const dfp_bn_desc* d, const int16_t* dz, const dfp_scale* sdz, const int16_t* y,
                           const dfp_scale* sy, const float* gamma, const float* beta, const float* res,
                           const float* mean, const float* inv_std, float* dy, int16_t* dyq, dfp_scale* sdy,
                           float* dgamma, float* dbeta, float* dres, int64_t* sums, void* workspace,
                           size_t ws_bytes, void* stream);

/* Workspace bytes of dfp_bn_relu_fwd / _bwd; 0 for an invalid descriptor. */
size_t dfp_bn_workspace_bytes(const dfp_bn_desc* d);

/* One FP32 SGD step with momentum mu and weight decay wd on n master weights,
 * in place (Fig. 2: the weight gradient is not quantised):
 *   g = fma(wd, w, dw);  v = fma(mu, v, g);  w = fma(-lr, v, w);
 * then Q_w of the new w (dfp_quantize numerics, role W): wq INT16 [n] with
 * scale sw.  w, v, dw: FP32 [n], 16-byte aligned; wq: 8-byte aligned, also
 * the max pass's scratch. */
dfp_status dfp_sgd_quantize(int64_t n, float lr, float mu, float wd, int32_t bits, int32_t rounding,
                            uint64_t seed, float* w, float* v, const float* dw, int16_t* wq, dfp_scale* sw,
                            void* stream);

/* Output height and width of the forward convolution; DFP_ERR_SHAPE if < 1. */
dfp_status dfp_output_dims(const dfp_desc* d, int32_t* p, int32_t* q);

/* Static text for a status code. */
const char* dfp_status_str(int32_t status);

/* ---- optional launch profiler (process-global, for benchmarks) ----------
 * dfp_profile_start(cap): from now on every kernel the library launches is
 * bracketed by a pair of HIP events on its stream, up to cap launches.
 * dfp_profile_stop(ids, ms, cap): waits for the recorded events, writes the
 * kernel id and duration (ms) of each launch, returns how many were written
 * and stops recording.  dfp_kernel_name(id): static name of a kernel id. */
dfp_status dfp_profile_start(int32_t capacity);
int32_t dfp_profile_stop(int32_t* kernel_ids, float* ms, int32_t capacity);
const char* dfp_kernel_name(int32_t kernel_id);

#ifdef __cplusplus
}
#endif

#endif /* DFP_H_ */
