// Streaming-read and copy kernels for measurement (see comem_probe.h).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "comem_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void read_kernel(const u32x4* __restrict__ src, size_t n16, uint32_t* sink) {
  const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const size_t lo = blockIdx.x * per;
  const size_t hi = lo + per < n16 ? lo + per : n16;
  uint32_t acc = 0;
  size_t i = lo + threadIdx.x;
  for (; i + 7 * 256 < hi; i += 8 * 256) {
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(&src[i + u * 256]);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < hi; i += 256) {
    const u32x4 v = __builtin_nontemporal_load(&src[i]);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (acc == 0x7fc00001u) sink[blockIdx.x * 256 + threadIdx.x] = acc;  // a NaN payload finite data never XORs to
}

__global__ __launch_bounds__(256) void copy_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst, size_t n16) {
  for (size_t i = blockIdx.x * 256 + threadIdx.x; i < n16; i += static_cast<size_t>(gridDim.x) * 256) dst[i] = src[i];
}

}  // namespace

extern "C" int comem_probe_read(const void* src, size_t bytes, uint32_t* sink, int blocks, void* hip_stream) {
  if (src == nullptr || sink == nullptr || blocks <= 0 || bytes % 16 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(read_kernel, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(hip_stream),
                     static_cast<const u32x4*>(src), bytes / 16, sink);
  return hipGetLastError();
}

extern "C" int comem_probe_copy(const void* src, void* dst, size_t bytes, int blocks, void* hip_stream) {
  if (src == nullptr || dst == nullptr || blocks <= 0 || bytes % 16 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(hip_stream),
                     static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), bytes / 16);
  return hipGetLastError();
}
