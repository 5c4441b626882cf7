// Internal declarations shared by the libdfp translation units (host + device).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dfp.h"

namespace dfp {

// Kernel ids reported by the launch profiler (dfp_profile_*).
enum KernelId : int32_t {
  K_SCALE_RESET = 0,
  K_AMAX = 1,
  K_QUANT = 2,
  K_FWD_VALU = 3,
  K_BWDD_VALU = 4,
  K_BWDW_VALU = 5,
  K_WPREP = 6,
  K_FWD_MFMA = 7,
  K_BWDD_MFMA = 8,
  K_BWDW_MFMA = 9,
  K_BWDW_REDUCE = 10,
  K_XPREP = 11,
  K_FWD_I32 = 12,
  K_BWDD_I32 = 13,
  K_DC_I32 = 14,
  K_GEMM_PREP = 15,
  K_GEMM = 16,
  K_QUANT_BLOCKED = 17,
  K_GEMM_BLOCKED = 18,
  K_BN_STATS = 19,
  K_BN_FINAL = 20,
  K_BN_AMAX = 21,
  K_BN_CONVERT = 22,
  K_SGD = 23,
  K_NUM_KERNELS = 24
};

// n / d for 0 <= n < 2^32 by multiply-high (round-up method, l = ceil(log2 d),
// m = floor(2^32 (2^l - d) / d) + 1, q = (mulhi(m, n) + n) >> l).
struct FastDiv {
  uint32_t m, l;
};
inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  const uint64_t m = ((((uint64_t)1 << 32) * (((uint64_t)1 << l) - d)) / d) + 1;
  return {(uint32_t)m, l};
}
__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv f) {
  return (uint32_t)(((uint64_t)__umulhi(n, f.m) + n) >> f.l);
}

// True if the kernel's build uses no scratch (private segment).  Kernels that
// read LDS with inline assembly and wait for the reads in a later statement
// need the compiler neither to copy nor to spill a register such a read is
// still filling between the two.  The build verifies that on the generated
// assembly (asm_check.py, which takes a failing kernel out of use); a kernel
// whose build has scratch is not launched either.
inline bool no_scratch(const void* kernel) {
  hipFuncAttributes attr{};
  return hipFuncGetAttributes(&attr, kernel) == hipSuccess && attr.localSizeBytes == 0;
}

// Convolution geometry handed to kernels by value.
struct Geom {
  int32_t n, c, h, w;   // activations NCHW
  int32_t k, r, s;      // filters KCRS
  int32_t sh, sw, ph, pw;
  int32_t p, q;         // forward output height / width
  int32_t L;            // chunk length (products per INT32 partial)
  int32_t G;            // backward-weights segment size in chunks
};

// Profiler hooks (api.hip). prof_begin returns a record slot or -1.
int prof_begin(int32_t id, hipStream_t st);
void prof_end(int slot, hipStream_t st);

// Launch with profiling and error capture; used inside functions returning dfp_status.
#define DFP_LAUNCH(ID, KERNEL, GRID, BLOCK, SHMEM, STREAM, ...)                 \
  do {                                                                          \
    int _slot = ::dfp::prof_begin((ID), (STREAM));                              \
    hipLaunchKernelGGL(KERNEL, (GRID), (BLOCK), (SHMEM), (STREAM), __VA_ARGS__); \
    hipError_t _err = hipGetLastError();                                        \
    ::dfp::prof_end(_slot, (STREAM));                                           \
    if (_err != hipSuccess) return DFP_ERR_HIP;                                 \
  } while (0)

// ---- launchers (one per translation unit) ----
// quantize.hip
dfp_status launch_scale_reset(dfp_scale* s, hipStream_t st);
// Writes amax_bits and clears flags; scratch (the destination INT16 buffer of
// n elements) holds partial maxima until the rounding pass overwrites it.
dfp_status launch_amax(const float* src, int64_t n, int16_t* scratch, dfp_scale* s, hipStream_t st);
// Reduces part[0 .. nparts) (per-workgroup maxima of |.| bits) into
// s->amax_bits and clears s->flags.
dfp_status launch_amax_final(const uint32_t* part, int32_t nparts, dfp_scale* s, hipStream_t st);
// Max pass + rounding pass, or one launch for a small P = 15 tensor.
dfp_status launch_quantize(const float* src, int16_t* dst, int64_t n, dfp_scale* s, int32_t bits, int32_t rounding,
                           uint64_t seed, uint32_t role, hipStream_t st);
dfp_status launch_quant_convert(const float* src, int16_t* dst, int64_t n, dfp_scale* s, int32_t bits,
                                int32_t rounding, uint64_t seed, uint32_t role, hipStream_t st);

// DFP-32 -> DFP (Eq. 6): sin carries E_in (and the max |src| when amax_ready);
// sout receives amax_bits, the new exponent and flags; dst is also the max
// pass's scratch.
dfp_status launch_downconvert_i32(const int32_t* src, int64_t n, const dfp_scale* sin, int16_t* dst, dfp_scale* sout,
                                  bool amax_ready, int32_t bits, int32_t rounding, uint64_t seed, uint32_t role,
                                  hipStream_t st);

// Blocked-DFP: blocks of B consecutive elements along each row of src
// [rows][cols]; exps [nb][rows]; s receives the tensor max and flags.
dfp_status launch_quantize_blocked(const float* src, int16_t* dst, int8_t* exps, int64_t rows, int64_t cols,
                                   int64_t B, dfp_scale* s, int32_t bits, int32_t rounding, uint64_t seed,
                                   uint32_t role, hipStream_t st);

// conv_valu.hip: one lane per output, VALU integer multiply-add.
// i32: single-chunk DFP-32 output (forward / backward-data), out holds INT32.
dfp_status launch_conv_valu(int32_t dir, const Geom& g, const int16_t* a, const dfp_scale* sa,
                            const int16_t* b, const dfp_scale* sb, float* out, dfp_scale* so,
                            int32_t* partials, hipStream_t st, bool i32 = false);

// gemm.hip: D[m][n] = opA opB with the forward convolution's chunked contract.
struct GemmPlan {
  int32_t KB, G16, Mp;                          // 32-blocks and 16-groups of the padded reduction, padded rows
  int64_t a_bytes, b_bytes, t_bytes, bytes;     // A digits, B digits, B offset table, total workspace
};
GemmPlan plan_gemm(int32_t m, int32_t n, int32_t k);
// exa / exb (nullable): Blocked-DFP exponent tables [nb][m] and [nb][n] per
// block of bk reduction indices (then sa / sb are unused).
dfp_status launch_gemm_mfma(int32_t m, int32_t n, int32_t k, int32_t trans_a, int32_t trans_b, int32_t L,
                            const int16_t* a, const dfp_scale* sa, const int16_t* b, const dfp_scale* sb,
                            float* d, dfp_scale* so, int32_t* partials, void* ws, hipStream_t st,
                            const int8_t* exa = nullptr, const int8_t* exb = nullptr, int32_t bk = 0);
// so (nullable) must be cleared by the caller.
dfp_status launch_gemm_blocked_valu(int32_t m, int32_t n, int32_t k, int32_t L, int32_t bk, const int16_t* a,
                                    const int8_t* ea, const int16_t* b, const int8_t* eb, float* d, dfp_scale* so,
                                    int32_t* partials, hipStream_t st);
// so (nullable) must be cleared by the caller.
dfp_status launch_gemm_valu(int32_t m, int32_t n, int32_t k, int32_t trans_a, int32_t trans_b, int32_t L,
                            const int16_t* a, const dfp_scale* sa, const int16_t* b, const dfp_scale* sb,
                            float* d, dfp_scale* so, int32_t* partials, hipStream_t st);

// train.hip: the steps either side of the convolutions in a training step.
dfp_status launch_bn_relu_fwd(const dfp_bn_desc& d, const int16_t* y, const dfp_scale* sy, const float* gamma,
                              const float* beta, const float* res, float* z, int16_t* zq, dfp_scale* sz, float* mean,
                              float* inv_std, int64_t* sums, void* ws, hipStream_t st);
dfp_status launch_bn_relu_bwd(const dfp_bn_desc& d, const int16_t* dz, const dfp_scale* sdz, const int16_t* y,
                              const dfp_scale* sy, const float* gamma, const float* beta, const float* res,
                              const float* mean, const float* inv_std, float* dy, int16_t* dyq, dfp_scale* sdy,
                              float* dgamma, float* dbeta, float* dres, int64_t* sums, void* ws, hipStream_t st);
size_t bn_workspace_bytes(const dfp_bn_desc& d);
dfp_status launch_sgd_quantize(int64_t n, float lr, float mu, float wd, int32_t bits, int32_t rounding,
                               uint64_t seed, float* w, float* v, const float* dw, int16_t* wq, dfp_scale* sw,
                               hipStream_t st);

}  // namespace dfp
