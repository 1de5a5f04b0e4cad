// Measured-peak microbenchmarks of the GPU the library runs on: a plain
// device copy (the HBM roof every bandwidth fraction is quoted against) and
// a loop of independent bf16 matrix-core products (the MFMA roof of the
// attention kernel).  Diagnostics only; the layer never calls them.
#include "common.h"
#include "kernels.h"

namespace scope {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// Grid-stride copy, four 16-byte loads in flight per lane before the
// stores; count16 = bytes / 16.
__global__ __launch_bounds__(256) void peak_copy_kernel(const u32x4 *__restrict__ src,
                                                        u32x4 *__restrict__ dst, size_t count16) {
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < count16; i += 4 * stride) {
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(&src[i + u * stride]);
#pragma unroll
    for (int u = 0; u < 4; ++u) __builtin_nontemporal_store(v[u], &dst[i + u * stride]);
  }
  for (; i < count16; i += stride) dst[i] = src[i];
}

// Eight independent 32x32x16 bf16 accumulation chains per wave, operands
// held in registers: each iteration issues 8 MFMAs (8 * 32768 flops).  The
// accumulators' sum is written per lane so the work cannot be dropped.
__global__ __launch_bounds__(256) void peak_mfma_kernel(float *out, int iters, float seed) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    a[j] = static_cast<__bf16>(seed * static_cast<float>(lane + j));
    b[j] = static_cast<__bf16>(seed * static_cast<float>(lane - j));
  }
  f32x16 acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.0f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < 8; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  out[static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x] = s;
}

}  // namespace

hipError_t peak_copy(const void *src, void *dst, size_t bytes, hipStream_t s) {
  const size_t n16 = bytes / 16;
  if (n16 == 0) return hipSuccess;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const size_t want = (n16 + 255) / 256;
  const unsigned blocks = static_cast<unsigned>(want < static_cast<size_t>(cus) * 8 ? want : static_cast<size_t>(cus) * 8);
  hipLaunchKernelGGL(peak_copy_kernel, dim3(blocks), dim3(256), 0, s,
                     static_cast<const u32x4 *>(src), static_cast<u32x4 *>(dst), n16);
  return hipGetLastError();
}

int peak_mfma_threads(int blocks) { return blocks * 256; }

hipError_t peak_mfma(float *out, int blocks, int iters, hipStream_t s) {
  hipLaunchKernelGGL(peak_mfma_kernel, dim3(blocks), dim3(256), 0, s, out, iters, 1.0f / 1024.0f);
  return hipGetLastError();
}

}  // namespace scope
