// Shared device code of the decode-attention kernels (gfx950).
//
// Every kernel here computes, for one (sequence b, KV head hk, split j), the
// softmax attention of the G query heads of hk over the split's token range
// (paper Sec. 2.2: the new query token attends over the whole KV cache), as
// a partial output normalised over the range plus its log-sum-exp. This file
// holds what follows the token loop: merging the per-wave partial states of a
// workgroup, writing the split's partial result, and the merge of all splits
// of a (b, hk) by whichever split finishes last (a ticket counter per (b, hk)
// in the workspace decides which). The merge visits splits in index order, so
// the result does not depend on which workgroup runs it.
//
// Scores are kept in the log2 domain: x = scale * log2(e) * q.k, so weights
// are exp2(x - m). lse values stored in the workspace are in log2 units; the
// lse written to the caller is converted to natural log.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace comem {

constexpr int kWaves = 4;           // waves per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxGroup = 16;       // largest GQA group handled in one workgroup
constexpr float kLn2 = 0.69314718055994530942f;

// Kernel arguments (passed by value). Offsets and strides are in bytes.
struct AttnParams {
  const char* q;       // [B, Hq, D] elements of the plan's dtype
  const char* k;       // K base, already offset by hk * stride_head per block
  const char* v;
  float* out;          // [B, Hq, D]
  float* lse;          // [B, Hq] or nullptr
  const int64_t* seq_start;   // contiguous layout
  const int32_t* ctx_lens;
  const int32_t* block_table; // paged layout, [B, max_pages]
  int64_t stride_token;
  int64_t stride_head;
  int64_t stride_page;
  int32_t max_pages;
  int32_t page_shift;  // log2(page_size)
  int32_t page_mask;   // page_size - 1
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;       // G = Hq / Hkv
  int32_t chunk;       // tokens per split (multiple of 32)
  int32_t num_splits;  // gridDim.x
  float scale_log2;    // scale * log2(e)
  uint32_t* tickets;   // [max_batch * Hkv], zero between calls
  float* lse_part;     // [B, Hkv, S, G]   (log2 units)
  float* o_part;       // [B, Hkv, S, G, D]
};

// Per-wave partial state handed from the token loop to the finalize step.
template <int D>
struct WaveState {
  float m[kWaves][kMaxGroup];   // running max (log2 units), -inf if no token seen
  float l[kWaves][kMaxGroup];   // sum of exp2(x - m)
  float o[kWaves][kMaxGroup][D];  // sum of exp2(x - m) * v
};

__device__ inline int64_t uniform_i64(int64_t x) {
  uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x));
  uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(static_cast<uint64_t>(x) >> 32));
  return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

__device__ inline int uniform_i32(int x) {
  return static_cast<int>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x)));
}

// Byte offset of token t of sequence b relative to the (hk-offset) K/V base.
template <bool PAGED>
__device__ inline int64_t row_offset(const AttnParams& p, int b, int64_t seq0, int t) {
  if constexpr (PAGED) {
    const int page = p.block_table[static_cast<int64_t>(b) * p.max_pages + (t >> p.page_shift)];
    return static_cast<int64_t>(page) * p.stride_page +
           static_cast<int64_t>(t & p.page_mask) * p.stride_token;
  } else {
    return (seq0 + t) * p.stride_token;
  }
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Partial results cross workgroups that may run on different XCDs, whose L2
// caches are not coherent with each other. They are written and read with
// device-scope accesses (relaxed atomics at agent scope: stores write through
// to the device coherence point, loads bypass any stale cached copy), so no
// cache-wide writeback or invalidate is needed. A writer waits until its
// stores are acknowledged before the workgroup takes its ticket.
__device__ inline void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline float load_coherent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void wait_stores_done() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Merge the workgroup's wave states, write the split's result, and if this
// split is the last of its (b, hk) to finish, merge all splits of (b, hk).
// Must be called by every thread of the workgroup after a barrier that
// follows the writes to `ws`.
template <int D>
__device__ void finalize_split(const AttnParams& p, const WaveState<D>& ws, int b, int hk, int j,
                               int nsplit_b) {
  __shared__ int sm_last;
  const int G = p.group;
  const int tid = threadIdx.x;
  const int head0 = b * p.num_q_heads + hk * G;  // first query head row of this (b, hk)
  const bool single = nsplit_b == 1;
  const int64_t part0 = (static_cast<int64_t>(b) * p.num_kv_heads + hk) * p.num_splits;

  for (int idx = tid; idx < G * D; idx += kThreads) {
    const int h = idx / D;
    const int d = idx - h * D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, ws.m[w][h]);
    float o = 0.f, lt = 0.f;
    if (M > -INFINITY) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float a = fast_exp2(ws.m[w][h] - M);  // exp2(-inf) = 0 for idle waves
        o += a * ws.o[w][h][d];
        lt += a * ws.l[w][h];
      }
    }
    const bool live = lt > 0.f;
    const float on = live ? o / lt : 0.f;
    const float lse2 = live ? M + log2f(lt) : -INFINITY;
    if (single) {
      p.out[static_cast<int64_t>(head0 + h) * D + d] = on;
      if (d == 0 && p.lse != nullptr) p.lse[head0 + h] = live ? lse2 * kLn2 : -INFINITY;
    } else {
      const int64_t slot = (part0 + j) * G + h;
      store_coherent(&p.o_part[slot * D + d], on);
      if (d == 0) store_coherent(&p.lse_part[slot], lse2);
    }
  }
  if (single) return;

  // Publish this split's partial result, then take a ticket.
  wait_stores_done();
  __syncthreads();
  if (tid == 0) {
    const uint32_t prev = atomicAdd(&p.tickets[b * p.num_kv_heads + hk], 1u);
    sm_last = prev == static_cast<uint32_t>(nsplit_b - 1);
  }
  __syncthreads();
  if (!sm_last) return;
  if (tid == 0) atomicExch(&p.tickets[b * p.num_kv_heads + hk], 0u);

  // Per-head maximum of the split lse values. G divides kThreads, so thread
  // tid only ever reads head tid % G; partial maxima meet in LDS.
  __shared__ float sm_red[kThreads];
  __shared__ float sm_max[kMaxGroup];
  const float* lp = p.lse_part + part0 * G;
  {
    float mloc = -INFINITY;
    for (int idx = tid; idx < nsplit_b * G; idx += kThreads) mloc = fmaxf(mloc, load_coherent(lp + idx));
    sm_red[tid] = mloc;
  }
  __syncthreads();
  if (tid < G) {
    float M = -INFINITY;
    for (int i = tid; i < kThreads; i += G) M = fmaxf(M, sm_red[i]);
    sm_max[tid] = M;
  }
  __syncthreads();

  // Weighted sum over splits, 4 head_dim values per slot. When there are
  // fewer slots than threads, tps threads share a slot, taking splits
  // sub, sub + tps, ...; their sums are then added in sub order.
  const int slots = G * D / 4;
  const int tps = slots >= kThreads ? 1 : kThreads / slots;
  __shared__ float4 sm_acc[kThreads];
  __shared__ float sm_wsum[kThreads];
  for (int slot = tid / tps; slot < slots; slot += kThreads / tps) {
    const int sub = tid % tps;
    const int h = (slot * 4) / D;
    const int d0 = slot * 4 - h * D;
    const float M = sm_max[h];
    const float* op = p.o_part + (part0 * G + h) * D + d0;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    float wsum = 0.f;
#pragma unroll 8
    for (int s = sub; s < nsplit_b; s += tps) {
      const float w = fast_exp2(load_coherent(lp + static_cast<int64_t>(s) * G + h) - M);
      const float* o = op + static_cast<int64_t>(s) * G * D;
      acc.x += w * load_coherent(o);
      acc.y += w * load_coherent(o + 1);
      acc.z += w * load_coherent(o + 2);
      acc.w += w * load_coherent(o + 3);
      wsum += w;
    }
    if (tps == 1) {
      const float inv = 1.f / wsum;
      *reinterpret_cast<float4*>(p.out + static_cast<int64_t>(head0 + h) * D + d0) =
          make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
      if (d0 == 0 && p.lse != nullptr) p.lse[head0 + h] = (M + log2f(wsum)) * kLn2;
    } else {
      sm_acc[tid] = acc;
      sm_wsum[tid] = wsum;
    }
  }
  if (tps == 1) return;
  __syncthreads();
  if (tid % tps == 0) {
    const int slot = tid / tps;
    const int h = (slot * 4) / D;
    const int d0 = slot * 4 - h * D;
    float4 acc = sm_acc[tid];
    float wsum = sm_wsum[tid];
    for (int i = 1; i < tps; ++i) {
      const float4 o = sm_acc[tid + i];
      acc.x += o.x;
      acc.y += o.y;
      acc.z += o.z;
      acc.w += o.w;
      wsum += sm_wsum[tid + i];
    }
    const float inv = 1.f / wsum;
    *reinterpret_cast<float4*>(p.out + static_cast<int64_t>(head0 + h) * D + d0) =
        make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
    if (d0 == 0 && p.lse != nullptr) p.lse[head0 + h] = (sm_max[h] + log2f(wsum)) * kLn2;
  }
}

}  // namespace comem
