// C ABI of libdfp: host-side validation and dispatch.  Every argument check
// runs before the first HIP call, so an invalid call enqueues nothing.
#include <algorithm>
#include <mutex>
#include <vector>

#include "dfp_internal.h"
#include "conv_mfma.h"
#include "conv_bwdw_mfma.h"

namespace dfp {

// ----------------------------------------------------------------- profiler
namespace {
struct ProfRec {
  int32_t id;
  hipEvent_t start, stop;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
int32_t g_prof_cap = 0;
std::vector<ProfRec> g_prof;
std::vector<hipEvent_t> g_event_pool;

hipEvent_t pooled_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

int prof_begin(int32_t id, hipStream_t st) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof_on || (int32_t)g_prof.size() >= g_prof_cap) return -1;
  ProfRec rec{id, pooled_event(), pooled_event()};
  if (!rec.start || !rec.stop) return -1;
  (void)hipEventRecord(rec.start, st);
  g_prof.push_back(rec);
  return (int)g_prof.size() - 1;
}

void prof_end(int slot, hipStream_t st) {
  if (slot < 0) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  (void)hipEventRecord(g_prof[slot].stop, st);
}

// ---------------------------------------------------- no-allocation scratch
// The scratch of dfp_conv_bwd_weights_noalloc.  In host code `scratch` only
// names the symbol; its device address on a GPU comes from
// hipGetSymbolAddress, taken once per device with that device current.
static __device__ __align__(256) uint8_t scratch[DFP_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on device `dev` (the current device), or null.
void* scratch_on_device(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}
}  // namespace

// ------------------------------------------------------------- validation
namespace {

bool geom_from_desc(const dfp_desc* d, Geom* g) {
  if (d->n < 1 || d->c < 1 || d->h < 1 || d->w < 1 || d->k < 1 || d->r < 1 || d->s < 1) return false;
  if (d->stride_h < 1 || d->stride_w < 1 || d->pad_h < 0 || d->pad_w < 0) return false;
  const int64_t hp = (int64_t)d->h + 2 * (int64_t)d->pad_h - d->r;
  const int64_t wp = (int64_t)d->w + 2 * (int64_t)d->pad_w - d->s;
  if (hp < 0 || wp < 0) return false;
  const int64_t p = hp / d->stride_h + 1, q = wp / d->stride_w + 1;
  if (p < 1 || q < 1 || p > (1 << 30) || q > (1 << 30)) return false;
  const int64_t lim = (int64_t)1 << 40;
  const int64_t xs = (int64_t)d->n * d->c * d->h * d->w;
  const int64_t ys = (int64_t)d->n * d->k * p * q;
  const int64_t ws = (int64_t)d->k * d->c * d->r * d->s;
  if (xs > lim || ys > lim || ws > lim) return false;
  g->n = d->n; g->c = d->c; g->h = d->h; g->w = d->w;
  g->k = d->k; g->r = d->r; g->s = d->s;
  g->sh = d->stride_h; g->sw = d->stride_w; g->ph = d->pad_h; g->pw = d->pad_w;
  g->p = (int32_t)p; g->q = (int32_t)q;
  g->L = d->chunk_len;
  g->G = d->seg_chunks > 0 ? d->seg_chunks : ((4096 / (d->chunk_len > 0 ? d->chunk_len : 1)) > 1 ? 4096 / d->chunk_len : 1);
  return true;
}

bool params_ok(const dfp_desc* d) {
  if (d->bits != 15 && d->bits != 16) return false;
  if (d->rounding < 0 || d->rounding > 3) return false;
  if (d->chunk_len < 1 || d->seg_chunks < 0) return false;
  if (d->path < DFP_PATH_AUTO || d->path > DFP_PATH_VALU) return false;
  return true;
}

int64_t role_numel(const Geom& g, int32_t role) {
  switch (role) {
    case DFP_ROLE_X:
    case DFP_ROLE_DX: return (int64_t)g.n * g.c * g.h * g.w;
    case DFP_ROLE_W: return (int64_t)g.k * g.c * g.r * g.s;
    case DFP_ROLE_DY:
    case DFP_ROLE_Y: return (int64_t)g.n * g.k * g.p * g.q;
    default: return -1;
  }
}

int64_t reduction_len(const Geom& g, int32_t dir) {
  if (dir == DFP_FWD) return (int64_t)g.c * g.r * g.s;
  if (dir == DFP_BWD_DATA) return (int64_t)g.k * g.r * g.s;
  return (int64_t)g.n * g.p * g.q;
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

// Common checks for the three convolutions.
dfp_status conv_checks(const dfp_desc* d, Geom* g, const void* a, const void* sa, const void* b,
                       const void* sb, const void* out) {
  if (!d || !a || !sa || !b || !sb || !out) return DFP_ERR_NULL;
  if (!params_ok(d)) return DFP_ERR_PARAM;
  if (!geom_from_desc(d, g)) return DFP_ERR_SHAPE;
  return DFP_OK;
}

// The byte-digit split is exact for integers in [-32768, 32639], which holds
// for every DFP15 tensor; 16-bit tensors (up to +-32767) take the VALU path.
bool use_mfma(const Geom& g, int32_t path, int32_t bits, int32_t dir) {
  if (path == DFP_PATH_VALU || bits != 15) return false;
  if (dir == DFP_BWD_WT) return bwdw_mfma_supported(g);
  return conv_mfma_supported(g, dir);
}

size_t workspace_bytes(const Geom& g, int32_t dir, int32_t path, int32_t bits) {
  if (!use_mfma(g, path, bits, dir)) return 0;
  if (dir == DFP_BWD_DATA)  // room for either route (partials take the general one)
    return (size_t)std::max(std::max<int64_t>(plan_conv_mfma(g, dir).bytes, conv_bwd_data_sub_bytes(g)),
                            conv_bwd_data_phase_bytes(g));
  if (dir == DFP_FWD) return (size_t)plan_conv_mfma(g, dir).bytes;
  return (size_t)plan_bwdw_mfma(g).bytes;
}

dfp_status ws_check(const Geom& g, int32_t dir, int32_t path, int32_t bits, const void* ws, size_t ws_bytes) {
  const size_t need = workspace_bytes(g, dir, path, bits);
  if (need == 0) return DFP_OK;
  if (!ws || ws_bytes < need || !aligned(ws, 256)) return DFP_ERR_WORKSPACE;
  return DFP_OK;
}

// GEMM descriptor and flat-tensor checks.
dfp_status gemm_desc_check(const dfp_gemm_desc* d) {
  if (!d) return DFP_ERR_NULL;
  if (d->m < 1 || d->n < 1 || d->k < 1) return DFP_ERR_SHAPE;
  if ((int64_t)d->m * d->n > ((int64_t)1 << 40) || (int64_t)d->m * d->k > ((int64_t)1 << 40) ||
      (int64_t)d->k * d->n > ((int64_t)1 << 40))
    return DFP_ERR_SHAPE;
  if ((d->trans_a != 0 && d->trans_a != 1) || (d->trans_b != 0 && d->trans_b != 1)) return DFP_ERR_PARAM;
  if (d->chunk_len < 1 || (d->bits != 15 && d->bits != 16)) return DFP_ERR_PARAM;
  if (d->path < DFP_PATH_AUTO || d->path > DFP_PATH_VALU) return DFP_ERR_PARAM;
  return DFP_OK;
}
bool gemm_use_mfma(const dfp_gemm_desc* d) {
  // grid rows of 64-row tiles must fit a launch dimension
  return d->path != DFP_PATH_VALU && d->bits == 15 && (d->m + 63) / 64 <= 65535;
}
// Blocked-DFP GEMM on matrix cores: P = 15, chunks of whole 32-blocks, the
// workgroup's exponent tables small enough for LDS, 32-bit output indices.
bool gemm_blocked_use_mfma(const dfp_gemm_desc* d, int32_t block_k) {
  const int64_t nb = ((int64_t)d->k + block_k - 1) / block_k;
  return gemm_use_mfma(d) && d->chunk_len % 32 == 0 && nb <= kBlockedMaxBlocks &&
         (int64_t)d->m * d->n < ((int64_t)1 << 31) && plan_gemm(d->m, d->n, d->k).b_bytes < ((int64_t)1 << 31);
}
bool flat_params_ok(int64_t n, int32_t bits, int32_t rounding, int32_t role) {
  return n >= 1 && n <= ((int64_t)1 << 40) && (bits == 15 || bits == 16) && rounding >= 0 && rounding <= 3 &&
         role >= DFP_ROLE_X && role <= DFP_ROLE_DX;
}

// Batch-norm descriptor checks: sizes, parameters, then the workspace.
dfp_status bn_desc_check(const dfp_bn_desc* d) {
  if (d->n < 1 || d->c < 1 || d->hw < 1) return DFP_ERR_SHAPE;
  if ((int64_t)d->n * d->c * d->hw >= ((int64_t)1 << 31)) return DFP_ERR_SHAPE;
  if (d->bits != 15 && d->bits != 16) return DFP_ERR_PARAM;
  if (d->rounding < 0 || d->rounding > 3) return DFP_ERR_PARAM;
  if (!(d->eps >= 0.0f) || d->eps == __builtin_inff()) return DFP_ERR_PARAM;
  return DFP_OK;
}
}  // namespace
}  // namespace dfp

using namespace dfp;

extern "C" {

const char* dfp_status_str(int32_t status) {
  switch (status) {
    case DFP_OK: return "ok";
    case DFP_ERR_NULL: return "null pointer";
    case DFP_ERR_SHAPE: return "invalid shape";
    case DFP_ERR_PARAM: return "invalid parameter";
    case DFP_ERR_ALIGN: return "misaligned pointer";
    case DFP_ERR_WORKSPACE: return "workspace missing or too small";
    case DFP_ERR_HIP: return "HIP error";
    case DFP_ERR_SCRATCH_LIMIT: return "layer needs more than the no-allocation scratch (64 MiB)";
    default: return "unknown status";
  }
}

dfp_status dfp_output_dims(const dfp_desc* d, int32_t* p, int32_t* q) {
  if (!d || !p || !q) return DFP_ERR_NULL;
  Geom g;
  if (!geom_from_desc(d, &g)) return DFP_ERR_SHAPE;
  *p = g.p;
  *q = g.q;
  return DFP_OK;
}

int64_t dfp_num_chunks(const dfp_desc* d, int32_t direction) {
  Geom g;
  if (!d || d->chunk_len < 1 || direction < 0 || direction > 2 || !geom_from_desc(d, &g)) return -1;
  const int64_t T = reduction_len(g, direction);
  return (T + d->chunk_len - 1) / d->chunk_len;
}

size_t dfp_workspace_bytes(const dfp_desc* d, int32_t direction) {
  Geom g;
  if (!d || !params_ok(d) || direction < 0 || direction > 2 || !geom_from_desc(d, &g)) return 0;
  return workspace_bytes(g, direction, d->path, d->bits);
}

dfp_status dfp_quantize(const dfp_desc* d, int32_t role, const float* src, int16_t* dst, dfp_scale* s,
                        void* stream) {
  if (!d || !src || !dst || !s) return DFP_ERR_NULL;
  if (!params_ok(d) || role < DFP_ROLE_X || role > DFP_ROLE_DX) return DFP_ERR_PARAM;
  Geom g;
  if (!geom_from_desc(d, &g)) return DFP_ERR_SHAPE;
  if (!aligned(src, 16) || !aligned(dst, 8) || !aligned(s, 16)) return DFP_ERR_ALIGN;
  const int64_t n = role_numel(g, role);
  hipStream_t st = (hipStream_t)stream;
  return launch_quantize(src, dst, n, s, d->bits, d->rounding, d->seed, (uint32_t)role, st);
}

dfp_status dfp_downconvert(const dfp_desc* d, int32_t role, const float* src, int16_t* dst, dfp_scale* s,
                           int32_t amax_ready, void* stream) {
  if (!d || !src || !dst || !s) return DFP_ERR_NULL;
  if (!params_ok(d) || (role != DFP_ROLE_Y && role != DFP_ROLE_DX) || (amax_ready != 0 && amax_ready != 1))
    return DFP_ERR_PARAM;
  Geom g;
  if (!geom_from_desc(d, &g)) return DFP_ERR_SHAPE;
  if (!aligned(src, 16) || !aligned(dst, 8) || !aligned(s, 16)) return DFP_ERR_ALIGN;
  const int64_t n = role_numel(g, role);
  hipStream_t st = (hipStream_t)stream;
  dfp_status rc;
  if (!amax_ready && (rc = launch_amax(src, n, dst, s, st)) != DFP_OK) return rc;
  return launch_quant_convert(src, dst, n, s, d->bits, d->rounding, d->seed, (uint32_t)role, st);
}

static dfp_status conv_common(int32_t dir, const dfp_desc* d, const int16_t* a, const dfp_scale* sa,
                              const int16_t* b, const dfp_scale* sb, float* out, dfp_scale* so, void* ws,
                              size_t ws_bytes, int32_t* partials, void* stream) {
  Geom g;
  dfp_status rc = conv_checks(d, &g, a, sa, b, sb, out);
  if (rc != DFP_OK) return rc;
  if ((rc = ws_check(g, dir, d->path, d->bits, ws, ws_bytes)) != DFP_OK) return rc;
  if (so && !aligned(so, 16)) return DFP_ERR_ALIGN;
  hipStream_t st = (hipStream_t)stream;
  if (use_mfma(g, d->path, d->bits, dir)) {
    if (dir == DFP_BWD_WT) return launch_bwdw_mfma(g, a, sa, b, sb, out, partials, ws, st);
    if (dir == DFP_BWD_DATA && !partials && conv_bwd_data_sub_bytes(g) > 0)
      return launch_conv_bwd_data_sub(g, a, sa, b, sb, out, so, ws, st, d->path == DFP_PATH_MFMA);
    if (dir == DFP_BWD_DATA && !partials && conv_bwd_data_phase_bytes(g) > 0)
      return launch_conv_bwd_data_phases(g, a, sa, b, sb, out, so, ws, st, d->path == DFP_PATH_MFMA);
    // the filter prep kernel clears so before the main kernel raises it
    return launch_conv_mfma(dir, g, a, sa, b, sb, out, so, partials, ws, st, false, d->path == DFP_PATH_MFMA);
  }
  if (so && (rc = launch_scale_reset(so, st)) != DFP_OK) return rc;
  return launch_conv_valu(dir, g, a, sa, b, sb, out, so, partials, st);
}

// Single-chunk DFP-32 output (forward or backward-data): chunk_len must cover
// the whole reduction, so the one INT32 partial is the output.
static dfp_status conv_i32_common(int32_t dir, const dfp_desc* d, const int16_t* a, const dfp_scale* sa,
                                  const int16_t* b, const dfp_scale* sb, int32_t* out, dfp_scale* so, void* ws,
                                  size_t ws_bytes, void* stream) {
  Geom g;
  dfp_status rc = conv_checks(d, &g, a, sa, b, sb, out);
  if (rc != DFP_OK) return rc;
  if (!so) return DFP_ERR_NULL;
  if (d->chunk_len < reduction_len(g, dir)) return DFP_ERR_PARAM;
  if ((rc = ws_check(g, dir, d->path, d->bits, ws, ws_bytes)) != DFP_OK) return rc;
  if (!aligned(so, 16)) return DFP_ERR_ALIGN;
  hipStream_t st = (hipStream_t)stream;
  float* outf = reinterpret_cast<float*>(out);
  if (use_mfma(g, d->path, d->bits, dir))  // the filter prep kernel clears so
    return launch_conv_mfma(dir, g, a, sa, b, sb, outf, so, nullptr, ws, st, true);
  if ((rc = launch_scale_reset(so, st)) != DFP_OK) return rc;
  return launch_conv_valu(dir, g, a, sa, b, sb, outf, so, nullptr, st, true);
}

dfp_status dfp_conv_fwd_i32(const dfp_desc* d, const int16_t* x, const dfp_scale* sx, const int16_t* w,
                            const dfp_scale* sw, int32_t* y, dfp_scale* sy, void* workspace, size_t ws_bytes,
                            void* stream) {
  return conv_i32_common(DFP_FWD, d, x, sx, w, sw, y, sy, workspace, ws_bytes, stream);
}

dfp_status dfp_conv_bwd_data_i32(const dfp_desc* d, const int16_t* dy, const dfp_scale* sdy, const int16_t* w,
                                 const dfp_scale* sw, int32_t* dx, dfp_scale* sdx, void* workspace, size_t ws_bytes,
                                 void* stream) {
  return conv_i32_common(DFP_BWD_DATA, d, dy, sdy, w, sw, dx, sdx, workspace, ws_bytes, stream);
}

dfp_status dfp_downconvert_i32(const dfp_desc* d, int32_t role, const int32_t* src, const dfp_scale* sin,
                               int16_t* dst, dfp_scale* sout, int32_t amax_ready, void* stream) {
  if (!d || !src || !sin || !dst || !sout) return DFP_ERR_NULL;
  if (!params_ok(d) || (role != DFP_ROLE_Y && role != DFP_ROLE_DX) || (amax_ready != 0 && amax_ready != 1) ||
      sin == sout)
    return DFP_ERR_PARAM;
  Geom g;
  if (!geom_from_desc(d, &g)) return DFP_ERR_SHAPE;
  if (!aligned(src, 16) || !aligned(dst, 8) || !aligned(sin, 16) || !aligned(sout, 16)) return DFP_ERR_ALIGN;
  const int64_t n = role_numel(g, role);
  return launch_downconvert_i32(src, n, sin, dst, sout, amax_ready != 0, d->bits, d->rounding, d->seed,
                                (uint32_t)role, (hipStream_t)stream);
}

// ------------------------------------------------------------------ GEMM
size_t dfp_gemm_workspace_bytes(const dfp_gemm_desc* d) {
  if (gemm_desc_check(d) != DFP_OK || !gemm_use_mfma(d)) return 0;
  return (size_t)plan_gemm(d->m, d->n, d->k).bytes;
}

int64_t dfp_gemm_num_chunks(const dfp_gemm_desc* d) {
  if (gemm_desc_check(d) != DFP_OK) return -1;
  return ((int64_t)d->k + d->chunk_len - 1) / d->chunk_len;
}

dfp_status dfp_gemm(const dfp_gemm_desc* d, const int16_t* a, const dfp_scale* sa, const int16_t* b,
                    const dfp_scale* sb, float* out, dfp_scale* sd, void* workspace, size_t ws_bytes,
                    int32_t* partials, void* stream) {
  dfp_status rc = gemm_desc_check(d);
  if (rc != DFP_OK) return rc;
  if (!a || !sa || !b || !sb || !out) return DFP_ERR_NULL;
  if (!aligned(a, 2) || !aligned(b, 2) || !aligned(out, 4) || (sd && !aligned(sd, 16)) ||
      (partials && !aligned(partials, 4)) || !aligned(sa, 16) || !aligned(sb, 16))
    return DFP_ERR_ALIGN;
  hipStream_t st = (hipStream_t)stream;
  if (gemm_use_mfma(d)) {
    const size_t need = (size_t)plan_gemm(d->m, d->n, d->k).bytes;
    if (!workspace || ws_bytes < need || !aligned(workspace, 256)) return DFP_ERR_WORKSPACE;
    return launch_gemm_mfma(d->m, d->n, d->k, d->trans_a, d->trans_b, d->chunk_len, a, sa, b, sb, out, sd,
                            partials, workspace, st);
  }
  if (sd && (rc = launch_scale_reset(sd, st)) != DFP_OK) return rc;
  return launch_gemm_valu(d->m, d->n, d->k, d->trans_a, d->trans_b, d->chunk_len, a, sa, b, sb, out, sd,
                          partials, st);
}

dfp_status dfp_quantize_blocked(int64_t rows, int64_t cols, int64_t block, int32_t bits, int32_t rounding,
                                uint64_t seed, int32_t role, const float* src, int16_t* dst, int8_t* exps,
                                dfp_scale* s, void* stream) {
  if (!src || !dst || !exps || !s) return DFP_ERR_NULL;
  if (rows < 1 || cols < 1 || rows * cols > ((int64_t)1 << 40)) return DFP_ERR_SHAPE;
  if (block < 1 || !flat_params_ok(rows * cols, bits, rounding, role)) return DFP_ERR_PARAM;
  if (!aligned(src, 4) || !aligned(dst, 2) || !aligned(s, 16)) return DFP_ERR_ALIGN;
  return launch_quantize_blocked(src, dst, exps, rows, cols, block, s, bits, rounding, seed, (uint32_t)role,
                                 (hipStream_t)stream);
}

size_t dfp_gemm_blocked_workspace_bytes(const dfp_gemm_desc* d, int32_t block_k) {
  if (gemm_desc_check(d) != DFP_OK || !gemm_blocked_use_mfma(d, block_k)) return 0;
  return (size_t)plan_gemm(d->m, d->n, d->k).bytes;
}

dfp_status dfp_gemm_blocked(const dfp_gemm_desc* d, int32_t block_k, const int16_t* a, const int8_t* ea,
                            const int16_t* b, const int8_t* eb, float* out, dfp_scale* sd, void* workspace,
                            size_t ws_bytes, int32_t* partials, void* stream) {
  dfp_status rc = gemm_desc_check(d);
  if (rc != DFP_OK) return rc;
  if (!a || !ea || !b || !eb || !out) return DFP_ERR_NULL;
  if (d->trans_a != 0 || d->trans_b != 1 || block_k < 1 || block_k % d->chunk_len != 0) return DFP_ERR_PARAM;
  if (!aligned(a, 2) || !aligned(b, 2) || !aligned(out, 4) || (sd && !aligned(sd, 16)) ||
      (partials && !aligned(partials, 4)))
    return DFP_ERR_ALIGN;
  hipStream_t st = (hipStream_t)stream;
  if (gemm_blocked_use_mfma(d, block_k)) {
    const size_t need = (size_t)plan_gemm(d->m, d->n, d->k).bytes;
    if (!workspace || ws_bytes < need || !aligned(workspace, 256)) return DFP_ERR_WORKSPACE;
    return launch_gemm_mfma(d->m, d->n, d->k, 0, 1, d->chunk_len, a, nullptr, b, nullptr, out, sd, partials,
                            workspace, st, ea, eb, block_k);
  }
  if (sd && (rc = launch_scale_reset(sd, st)) != DFP_OK) return rc;
  return launch_gemm_blocked_valu(d->m, d->n, d->k, d->chunk_len, block_k, a, ea, b, eb, out, sd, partials, st);
}

dfp_status dfp_quantize_tensor(int64_t n, int32_t bits, int32_t rounding, uint64_t seed, int32_t role,
                               const float* src, int16_t* dst, dfp_scale* s, void* stream) {
  if (!src || !dst || !s) return DFP_ERR_NULL;
  if (!flat_params_ok(n, bits, rounding, role)) return DFP_ERR_PARAM;
  if (!aligned(src, 16) || !aligned(dst, 8) || !aligned(s, 16)) return DFP_ERR_ALIGN;
  hipStream_t st = (hipStream_t)stream;
  return launch_quantize(src, dst, n, s, bits, rounding, seed, (uint32_t)role, st);
}

dfp_status dfp_downconvert_tensor(int64_t n, int32_t bits, int32_t rounding, uint64_t seed, int32_t role,
                                  const float* src, int16_t* dst, dfp_scale* s, int32_t amax_ready,
                                  void* stream) {
  if (!src || !dst || !s) return DFP_ERR_NULL;
  if (!flat_params_ok(n, bits, rounding, role) || (amax_ready != 0 && amax_ready != 1)) return DFP_ERR_PARAM;
  if (!aligned(src, 16) || !aligned(dst, 8) || !aligned(s, 16)) return DFP_ERR_ALIGN;
  hipStream_t st = (hipStream_t)stream;
  dfp_status rc;
  if (!amax_ready && (rc = launch_amax(src, n, dst, s, st)) != DFP_OK) return rc;
  return launch_quant_convert(src, dst, n, s, bits, rounding, seed, (uint32_t)role, st);
}

size_t dfp_bn_workspace_bytes(const dfp_bn_desc* d) {
  if (!d || bn_desc_check(d) != DFP_OK) return 0;
  return bn_workspace_bytes(*d);
}

dfp_status dfp_bn_relu_fwd(const dfp_bn_desc* d, const int16_t* y, const dfp_scale* sy, const float* gamma,
                           const float* beta, const float* res, float* z, int16_t* zq, dfp_scale* sz, float* mean,
                           float* inv_std, int64_t* sums, void* workspace, size_t ws_bytes, void* stream) {
  if (!d || !y || !sy || !gamma || !beta || !zq || !sz || !mean || !inv_std) return DFP_ERR_NULL;
  dfp_status rc;
  if ((rc = bn_desc_check(d)) != DFP_OK) return rc;
  if (!aligned(y, 16) || !aligned(zq, 16) || (res && !aligned(res, 16)) || (z && !aligned(z, 16)) ||
      !aligned(sy, 16) || !aligned(sz, 16) || (sums && !aligned(sums, 8)))
    return DFP_ERR_ALIGN;
  if (!workspace || ws_bytes < bn_workspace_bytes(*d) || !aligned(workspace, 256)) return DFP_ERR_WORKSPACE;
  return launch_bn_relu_fwd(*d, y, sy, gamma, beta, res, z, zq, sz, mean, inv_std, sums, workspace,
                            (hipStream_t)stream);
}

dfp_status dfp_bn_relu_bwd(const dfp_bn_desc* d, const int16_t* dz, const dfp_scale* sdz, const int16_t* y,
                           const dfp_scale* sy, const float* gamma, const float* beta, const float* res,
                           const float* mean, const float* inv_std, float* dy, int16_t* dyq, dfp_scale* sdy,
                           float* dgamma, float* dbeta, float* dres, int64_t* sums, void* workspace, size_t ws_bytes,
                           void* stream) {
  if (!d || !dz || !sdz || !y || !sy || !gamma || !beta || !mean || !inv_std || !dyq || !sdy || !dgamma || !dbeta)
    return DFP_ERR_NULL;
  dfp_status rc;
  if ((rc = bn_desc_check(d)) != DFP_OK) return rc;
  if (!aligned(dz, 16) || !aligned(y, 16) || !aligned(dyq, 16) || (res && !aligned(res, 16)) ||
      (dy && !aligned(dy, 16)) || (dres && !aligned(dres, 16)) || !aligned(sdz, 16) || !aligned(sy, 16) ||
      !aligned(sdy, 16) || (sums && !aligned(sums, 8)))
    return DFP_ERR_ALIGN;
  if (!workspace || ws_bytes < bn_workspace_bytes(*d) || !aligned(workspace, 256)) return DFP_ERR_WORKSPACE;
  return launch_bn_relu_bwd(*d, dz, sdz, y, sy, gamma, beta, res, mean, inv_std, dy, dyq, sdy, dgamma, dbeta, dres,
                            sums, workspace, (hipStream_t)stream);
}

dfp_status dfp_sgd_quantize(int64_t n, float lr, float mu, float wd, int32_t bits, int32_t rounding, uint64_t seed,
                            float* w, float* v, const float* dw, int16_t* wq, dfp_scale* sw, void* stream) {
  if (!w || !v || !dw || !wq || !sw) return DFP_ERR_NULL;
  if (!flat_params_ok(n, bits, rounding, DFP_ROLE_W)) return DFP_ERR_PARAM;
  if (!aligned(w, 16) || !aligned(v, 16) || !aligned(dw, 16) || !aligned(wq, 8) || !aligned(sw, 16))
    return DFP_ERR_ALIGN;
  return launch_sgd_quantize(n, lr, mu, wd, bits, rounding, seed, w, v, dw, wq, sw, (hipStream_t)stream);
}

dfp_status dfp_conv_fwd(const dfp_desc* d, const int16_t* x, const dfp_scale* sx, const int16_t* w,
                        const dfp_scale* sw, float* y, dfp_scale* sy, void* workspace, size_t ws_bytes,
                        int32_t* partials, void* stream) {
  return conv_common(DFP_FWD, d, x, sx, w, sw, y, sy, workspace, ws_bytes, partials, stream);
}

dfp_status dfp_conv_bwd_data(const dfp_desc* d, const int16_t* dy, const dfp_scale* sdy, const int16_t* w,
                             const dfp_scale* sw, float* dx, dfp_scale* sdx, void* workspace, size_t ws_bytes,
                             int32_t* partials, void* stream) {
  return conv_common(DFP_BWD_DATA, d, dy, sdy, w, sw, dx, sdx, workspace, ws_bytes, partials, stream);
}

dfp_status dfp_conv_bwd_weights(const dfp_desc* d, const int16_t* x, const dfp_scale* sx, const int16_t* dy,
                                const dfp_scale* sdy, float* dw, void* workspace, size_t ws_bytes,
                                int32_t* partials, void* stream) {
  return conv_common(DFP_BWD_WT, d, x, sx, dy, sdy, dw, nullptr, workspace, ws_bytes, partials, stream);
}

dfp_status dfp_conv_bwd_weights_noalloc(const dfp_desc* d, const int16_t* x, const dfp_scale* sx,
                                        const int16_t* dy, const dfp_scale* sdy, float* dw, void* stream) {
  Geom g;
  dfp_status rc = conv_checks(d, &g, x, sx, dy, sdy, dw);
  if (rc != DFP_OK) return rc;
  const size_t need = workspace_bytes(g, DFP_BWD_WT, d->path, d->bits);
  if (need > (size_t)DFP_NOALLOC_SCRATCH_BYTES) return DFP_ERR_SCRATCH_LIMIT;
  hipStream_t st = (hipStream_t)stream;
  if (!use_mfma(g, d->path, d->bits, DFP_BWD_WT)) return launch_conv_valu(DFP_BWD_WT, g, x, sx, dy, sdy, dw, nullptr,
                                                                            nullptr, st);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return DFP_ERR_HIP;
  if (st) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(st, &sdev) != hipSuccess) return DFP_ERR_HIP;
    if ((int)sdev != dev) return DFP_ERR_PARAM;
  }
  void* ws = scratch_on_device(dev);
  if (!ws) return DFP_ERR_HIP;
  return launch_bwdw_mfma(g, x, sx, dy, sdy, dw, nullptr, ws, st);
}

dfp_status dfp_profile_start(int32_t capacity) {
  if (capacity < 0) return DFP_ERR_PARAM;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& r : g_prof) {
    g_event_pool.push_back(r.start);
    g_event_pool.push_back(r.stop);
  }
  g_prof.clear();
  g_prof.reserve(capacity);
  g_prof_cap = capacity;
  g_prof_on = true;
  return DFP_OK;
}

int32_t dfp_profile_stop(int32_t* kernel_ids, float* ms, int32_t capacity) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_on = false;
  int32_t n = 0;
  for (auto& r : g_prof) {
    if (n < capacity && kernel_ids && ms) {
      float t = -1.f;
      if (hipEventSynchronize(r.stop) == hipSuccess && hipEventElapsedTime(&t, r.start, r.stop) == hipSuccess) {
        kernel_ids[n] = r.id;
        ms[n] = t;
        ++n;
      }
    }
    g_event_pool.push_back(r.start);
    g_event_pool.push_back(r.stop);
  }
  g_prof.clear();
  return n;
}

const char* dfp_kernel_name(int32_t id) {
  static const char* names[K_NUM_KERNELS] = {
      "scale_reset", "amax", "quant_convert", "conv_fwd_valu", "conv_bwd_data_valu", "conv_bwd_wt_valu",
      "weight_prep", "conv_fwd_mfma", "conv_bwd_data_mfma", "conv_bwd_wt_mfma", "bwd_wt_segment_reduce",
      "act_prep", "conv_fwd_i32", "conv_bwd_data_i32", "downconvert_i32", "gemm_prep", "gemm", "quant_blocked", "gemm_blocked",
      "bn_stats", "bn_finalize", "bn_amax", "bn_convert", "sgd"};
  if (id < 0 || id >= K_NUM_KERNELS) return "unknown";
  return names[id];
}

}  // extern "C"
