// Measured ceilings of the units the DFP convolution path runs on (gfx950),
// for the benchmark's roofline context.  Not part of libdfp: built into
// libpeaks.so and called by `bench.py --peaks`.
//
//   peaks_mfma_i8      dependency-free v_mfma_i32_32x32x32_i8 (shape 0) or
//                      v_mfma_i32_16x16x64_i8 (shape 1) on every SIMD
//   peaks_dot2_i16     dependency-free v_dot2_i32_i16 (two INT16 products per
//                      lane and instruction), the packed-INT16 VALU path
//   peaks_chunk_loop   the byte-split inner loop of one 32x32 output tile at
//                      chunk length 64 with registers as operands: 8 MFMAs
//                      (hi*hi, lo*lo and both cross products over two
//                      32-index blocks) then the chunk conversion of 16
//                      outputs per lane (two shift-adds, int -> float, add),
//                      four waves per SIMD; the method's attainable rate
//                      with no operand traffic at all
//   peaks_hbm_read     grid-stride 16-byte loads over a buffer, summed
//   peaks_hbm_copy     grid-stride 16-byte copy
// Each returns the kernel time in milliseconds of the second of two launches
// (HIP events on the null stream), or a negative value on a HIP error.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef short v2s __attribute__((ext_vector_type(2)));

namespace {

template <int SHAPE>
__global__ __launch_bounds__(256, 2) void k_mfma(int* out, int iters, int seed) {
  v4i a = {seed, seed + 1, seed + 2, seed + 3}, b = a + 7;
  if (SHAPE == 0) {
    v16i c0 = {0}, c1 = {0}, c2 = {0}, c3 = {0};
    for (int i = 0; i < iters; ++i) {
      c0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b, a, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, a, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b, b, c3, 0, 0, 0);
    }
    int s = 0;
    for (int v = 0; v < 16; ++v) s += c0[v] + c1[v] + c2[v] + c3[v];
    out[blockIdx.x * 256 + threadIdx.x] = s;
  } else {
    v4i c0 = {0}, c1 = {0}, c2 = {0}, c3 = {0};
    for (int i = 0; i < iters; ++i) {
      // two 16x16x64 per 32x32x32 in work: eight per iteration
      c0 = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_i32_16x16x64_i8(b, a, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, a, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_i32_16x16x64_i8(b, b, c3, 0, 0, 0);
      c0 = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_i32_16x16x64_i8(b, a, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, a, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_i32_16x16x64_i8(b, b, c3, 0, 0, 0);
    }
    out[blockIdx.x * 256 + threadIdx.x] = c0[0] + c1[1] + c2[2] + c3[3];
  }
}

__global__ __launch_bounds__(256) void k_dot2(int* out, int iters, int seed) {
  int s[8];
  for (int j = 0; j < 8; ++j) s[j] = seed + j;
  const int ai = seed * 3 + (int)threadIdx.x, bi = seed * 5 + 1;
  v2s a = {(short)ai, (short)(ai >> 3)}, b = {(short)bi, (short)(bi >> 2)};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < 8; ++j) s[j] = __builtin_amdgcn_sdot2(a, b, s[j], false);
  }
  int t = 0;
  for (int j = 0; j < 8; ++j) t += s[j];
  out[blockIdx.x * 256 + threadIdx.x] = t;
}

__global__ __launch_bounds__(256, 4) void k_chunk_loop(float* out, int iters, int seed) {
  v4i ah = {seed, seed + 1, seed + 2, seed + 3}, al = ah + 5, bh = ah + 7, bl = ah + 9;
  v16i hh = {0}, xx = {0}, ll = {0};
  float s[16];
  for (int v = 0; v < 16; ++v) s[v] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      hh = __builtin_amdgcn_mfma_i32_32x32x32_i8(ah, bh, blk ? hh : v16i{0}, 0, 0, 0);
      ll = __builtin_amdgcn_mfma_i32_32x32x32_i8(al, bl, blk ? ll : v16i{0}, 0, 0, 0);
      xx = __builtin_amdgcn_mfma_i32_32x32x32_i8(ah, bl, blk ? xx : v16i{0}, 0, 0, 0);
      xx = __builtin_amdgcn_mfma_i32_32x32x32_i8(al, bh, xx, 0, 0, 0);
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      // the product kernels' four operations per output: two shift-adds
      // (kept as such: the compiler would otherwise form two shifts and an
      // add3), int -> float, add
      uint32_t t = ((uint32_t)hh[v] << 8) + (uint32_t)xx[v];
      asm("" : "+v"(t));
      const uint32_t p = (t << 8) + (uint32_t)ll[v];
      s[v] += (float)(int32_t)p;
    }
    ah += 1;
    bl += 1;
  }
  float acc = 0.f;
  for (int v = 0; v < 16; ++v) acc += s[v];
  out[blockIdx.x * 256 + threadIdx.x] = acc;
}

__global__ __launch_bounds__(256) void k_read(const uint4* __restrict__ src, int64_t n16, uint32_t* out) {
  uint32_t acc = 0;
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n16; i += stride) {
    const uint4 a = src[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  out[blockIdx.x * 256 + threadIdx.x] = acc;
}

__global__ __launch_bounds__(256) void k_copy(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n16) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += stride) dst[i] = src[i];
}

template <typename F>
float time2(F launch) {
  hipEvent_t a, b;
  if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) return -1.f;
  launch();
  (void)hipEventRecord(a, nullptr);
  launch();
  (void)hipEventRecord(b, nullptr);
  float ms = -1.f;
  if (hipGetLastError() != hipSuccess || hipEventSynchronize(b) != hipSuccess ||
      hipEventElapsedTime(&ms, a, b) != hipSuccess)
    ms = -1.f;
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  return ms;
}

}  // namespace

extern "C" {

// blocks of 256 threads (4 waves); each wave issues 4 * iters MFMAs
// (32x32x32) or 8 * iters (16x16x64): 4 * 32768 int8 MACs per iteration.
float peaks_mfma_i8(int shape, int blocks, int iters) {
  int* out = nullptr;
  if (blocks < 1 || iters < 1 || hipMalloc(&out, (size_t)blocks * 256 * 4) != hipSuccess) return -1.f;
  const float ms = time2([&] {
    if (shape == 0) hipLaunchKernelGGL(k_mfma<0>, dim3(blocks), dim3(256), 0, nullptr, out, iters, 1);
    else hipLaunchKernelGGL(k_mfma<1>, dim3(blocks), dim3(256), 0, nullptr, out, iters, 1);
  });
  (void)hipFree(out);
  return ms;
}

// each lane issues 8 * iters v_dot2_i32_i16 (2 INT16 MACs each)
float peaks_dot2_i16(int blocks, int iters) {
  int* out = nullptr;
  if (blocks < 1 || iters < 1 || hipMalloc(&out, (size_t)blocks * 256 * 4) != hipSuccess) return -1.f;
  const float ms = time2([&] { hipLaunchKernelGGL(k_dot2, dim3(blocks), dim3(256), 0, nullptr, out, iters, 1); });
  (void)hipFree(out);
  return ms;
}

// each wave runs iters chunks of 64 on one 32x32 tile: 8 MFMAs (8 * 32768
// int8 MACs = 32x32x64 INT16-equivalent MACs) and the conversion of 1024 outputs
float peaks_chunk_loop(int blocks, int iters) {
  float* out = nullptr;
  if (blocks < 1 || iters < 1 || hipMalloc(&out, (size_t)blocks * 256 * 4) != hipSuccess) return -1.f;
  const float ms =
      time2([&] { hipLaunchKernelGGL(k_chunk_loop, dim3(blocks), dim3(256), 0, nullptr, out, iters, 1); });
  (void)hipFree(out);
  return ms;
}

// bytes: buffer size (a multiple of 16)
float peaks_hbm_read(int64_t bytes, int blocks) {
  uint4* src = nullptr;
  uint32_t* out = nullptr;
  if (bytes < 16 || blocks < 1 || hipMalloc(&src, (size_t)bytes) != hipSuccess) return -1.f;
  if (hipMalloc(&out, (size_t)blocks * 256 * 4) != hipSuccess || hipMemset(src, 1, (size_t)bytes) != hipSuccess) {
    (void)hipFree(src);
    return -1.f;
  }
  const float ms =
      time2([&] { hipLaunchKernelGGL(k_read, dim3(blocks), dim3(256), 0, nullptr, src, bytes / 16, out); });
  (void)hipFree(src);
  (void)hipFree(out);
  return ms;
}

float peaks_hbm_copy(int64_t bytes, int blocks) {
  uint4 *src = nullptr, *dst = nullptr;
  if (bytes < 16 || blocks < 1 || hipMalloc(&src, (size_t)bytes) != hipSuccess) return -1.f;
  if (hipMalloc(&dst, (size_t)bytes) != hipSuccess || hipMemset(src, 1, (size_t)bytes) != hipSuccess) {
    (void)hipFree(src);
    return -1.f;
  }
  const float ms =
      time2([&] { hipLaunchKernelGGL(k_copy, dim3(blocks), dim3(256), 0, nullptr, src, dst, bytes / 16); });
  (void)hipFree(src);
  (void)hipFree(dst);
  return ms;
}

}  // extern "C"
