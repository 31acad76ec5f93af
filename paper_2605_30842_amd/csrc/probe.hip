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

// One 32-token tile of a KV head as the decode kernel's lane (c, g) reads it:
// per 16-row half, K row c at 16 g + 64 kk (bf16) or 32 g + 16 i (FP8), and
// V rows 4 g + r at 16 c (bf16) or 8 c (FP8).
template <int HB>
struct KvTile {
  static constexpr int KL = HB == 256 ? 4 : 2;  // K loads of 16 bytes per half
  u32x4 k[2][KL];
  u32x4 v[2][4];  // FP8: the low two words only
};

__device__ inline __amdgpu_buffer_rsrc_t probe_rsrc(const char* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), 0, bytes, 0x00020000);
}

template <int HB>
__device__ inline void load_kv_tile(KvTile<HB>& t, const char* kh, const char* vh, int64_t tok, int64_t stride,
                                    int c, int g) {
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const uint32_t bytes = static_cast<uint32_t>(15 * stride + HB);
    const __amdgpu_buffer_rsrc_t rk = probe_rsrc(kh + (tok + 16 * s) * stride, bytes);
    const __amdgpu_buffer_rsrc_t rv = probe_rsrc(vh + (tok + 16 * s) * stride, bytes);
#pragma unroll
    for (int i = 0; i < KvTile<HB>::KL; ++i) {
      const uint32_t off = static_cast<uint32_t>(c * stride) + (HB == 256 ? 16 * g + 64 * i : 32 * g + 16 * i);
      t.k[s][i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, 0));
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint32_t off = static_cast<uint32_t>((4 * g + r) * stride) + (HB == 256 ? 16 * c : 8 * c);
      if constexpr (HB == 256) {
        t.v[s][r] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, 2));
      } else {
        const uint64_t w = __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(rv, off, 0, 2));
        t.v[s][r] = u32x4{static_cast<uint32_t>(w), static_cast<uint32_t>(w >> 32), 0u, 0u};
      }
    }
  }
}

template <int HB>
__device__ inline uint32_t fold_kv_tile(const KvTile<HB>& t) {
  uint32_t a = 0;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int i = 0; i < KvTile<HB>::KL; ++i) a ^= t.k[s][i].x ^ t.k[s][i].y ^ t.k[s][i].z ^ t.k[s][i].w;
#pragma unroll
    for (int r = 0; r < 4; ++r) a ^= t.v[s][r].x ^ t.v[s][r].y ^ t.v[s][r].z ^ t.v[s][r].w;
  }
  return a;
}

template <int HB>
__global__ __launch_bounds__(256) void read_kv_heads_kernel(const char* k, const char* v, int64_t stride, int chunk,
                                                            uint32_t* sink) {
  const uint32_t lin = blockIdx.x + gridDim.x * blockIdx.y;
  const int h = static_cast<int>(lin % gridDim.y), j = static_cast<int>(lin / gridDim.y);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, c = lane & 15, g = lane >> 4;
  const char* kh = k + static_cast<int64_t>(h) * HB;
  const char* vh = v + static_cast<int64_t>(h) * HB;
  const int64_t t0 = static_cast<int64_t>(j) * chunk;
  const int ntiles = chunk / 32;
  uint32_t acc = 0;
  KvTile<HB> A, B;
  int t = w;
  load_kv_tile<HB>(A, kh, vh, t0 + 32 * t, stride, c, g);
  for (;;) {
    int nx = t + 4;
    load_kv_tile<HB>(B, kh, vh, t0 + 32 * (nx < ntiles ? nx : t), stride, c, g);
    __builtin_amdgcn_sched_barrier(0);
    acc ^= fold_kv_tile<HB>(A);
    if (nx >= ntiles) break;
    t = nx;
    nx = t + 4;
    load_kv_tile<HB>(A, kh, vh, t0 + 32 * (nx < ntiles ? nx : t), stride, c, g);
    __builtin_amdgcn_sched_barrier(0);
    acc ^= fold_kv_tile<HB>(B);
    if (nx >= ntiles) break;
    t = nx;
  }
  if (acc == 0x7fc00001u) sink[threadIdx.x] = acc;  // as in read_kernel
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

extern "C" int comem_probe_read_kv_heads(const void* k, const void* v, int64_t tokens, int kv_heads, int head_bytes,
                                         int64_t stride_token, int chunk, uint32_t* sink, void* hip_stream) {
  if (k == nullptr || v == nullptr || sink == nullptr) return hipErrorInvalidValue;
  if (head_bytes != 128 && head_bytes != 256) return hipErrorInvalidValue;
  if (chunk <= 0 || chunk % 128 != 0 || tokens <= 0 || tokens % chunk != 0 || kv_heads < 1) return hipErrorInvalidValue;
  if (stride_token < static_cast<int64_t>(kv_heads) * head_bytes || stride_token % 16 != 0) return hipErrorInvalidValue;
  if (reinterpret_cast<uintptr_t>(k) % 16 != 0 || reinterpret_cast<uintptr_t>(v) % 16 != 0) return hipErrorInvalidValue;
  if (15 * stride_token + head_bytes > 0xffffffffll) return hipErrorInvalidValue;  // one 16-row buffer range
  const int64_t splits = tokens / chunk;
  if (kv_heads > 65535 || splits * kv_heads > (int64_t{1} << 24)) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(splits), static_cast<unsigned>(kv_heads));
  const char* kc = static_cast<const char*>(k);
  const char* vc = static_cast<const char*>(v);
  if (head_bytes == 256)
    hipLaunchKernelGGL(read_kv_heads_kernel<256>, grid, dim3(256), 0, static_cast<hipStream_t>(hip_stream), kc, vc,
                       stride_token, chunk, sink);
  else
    hipLaunchKernelGGL(read_kv_heads_kernel<128>, grid, dim3(256), 0, static_cast<hipStream_t>(hip_stream), kc, vc,
                       stride_token, chunk, sink);
  return hipGetLastError();
}
