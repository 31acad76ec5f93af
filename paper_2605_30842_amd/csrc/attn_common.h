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

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;           // waves per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxGroup = 16;       // largest GQA group handled in one workgroup
constexpr int kMergeBatch = 16;     // split partials loaded together by one thread in the merge
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
  int32_t num_splits;  // most splits of one sequence (the stride of the partial results)
  int32_t tail_chunk;  // work-queue form: tokens of each short last split, or 0 for none
  int32_t tail_splits; // work-queue form: short last splits per sequence (at most a quarter of its splits)
  float scale_log2;    // scale * log2(e)
  uint32_t* tickets;   // [max_batch * Hkv] tickets, then 2 queue counters; zero between calls
  int32_t queue_slot;  // index of the queue counters in tickets
  float* lse_part;     // [B, Hkv, S, G]   (log2 units)
  float* o_part;       // [B, Hkv, S, G, D]
  const char* new_k;   // fused append: new rows [B, Hkv, D], or nullptr for attention only
  const char* new_v;
  int64_t num_pages;   // paged layout: pool size (bounds every page access)
  float out_scale;     // multiplies every output (the V scale of an FP8 cache, else 1)
  int32_t max_ctx;     // the call's max_ctx_len: lengths are clamped to [0, max_ctx]
  uint32_t* errors;    // device error word (debug checks), or nullptr
};

// Device-side contract checks. A length outside [0, max_ctx] is clamped into
// it; a block-table entry outside [0, num_pages) becomes -1, which reads use
// as page 0 and stores skip. With an error word, each violation also sets its
// bit there (the COMEM_DEVICE_ERR_* values of the C header).
constexpr uint32_t kErrCtxLen = 1u;
constexpr uint32_t kErrBlockTable = 2u;

__device__ inline int checked_len(int L, int max_ctx, uint32_t* errors) {
  if (L < 0 || L > max_ctx) {
    if (errors != nullptr) atomicOr(errors, kErrCtxLen);
    L = L < 0 ? 0 : max_ctx;
  }
  return L;
}

__device__ inline int32_t checked_page(int32_t page, int64_t num_pages, uint32_t* errors) {
  if (page < 0 || page >= num_pages) {
    if (errors != nullptr) atomicOr(errors, kErrBlockTable);
    return -1;
  }
  return page;
}

// Per-wave partial state handed from the token loop to the finalize step.
template <int D>
struct WaveState {
  float m[kWaves][kMaxGroup];   // running max (log2 units), -inf if no token seen
  float l[kWaves][kMaxGroup];   // sum of exp2(x - m)
  alignas(16) float o[kWaves][kMaxGroup][D];  // sum of exp2(x - m) * v
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
    const int page = max(0, checked_page(p.block_table[static_cast<int64_t>(b) * p.max_pages + (t >> p.page_shift)],
                                         p.num_pages, p.errors));
    return static_cast<int64_t>(page) * p.stride_page +
           static_cast<int64_t>(t & p.page_mask) * p.stride_token;
  } else {
    return (seq0 + t) * p.stride_token;
  }
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Fused KV append (paper Sec. 2.2: the new token's key and value join the
// caches before it attends). Called by the one wave of the split holding
// token L - 1 that will also load that token's row, before any of its loads:
// `pieces` lanes store the K row of head hk, the next `pieces` lanes the V
// row (16 bytes each; 2 * pieces <= 64). Memory operations of one wave to
// one address take effect in program order, so the wave's later loads of
// the row return the new values without a wait; the wavefront-scope fence
// keeps the compiler from moving those loads above the stores. row_off < 0
// (a page outside the pool) skips the store.
__device__ inline void store_new_token(const AttnParams& p, int b, int hk, int64_t row_off, int pieces,
                                       int lane) {
  if (row_off >= 0 && lane < 2 * pieces) {
    const bool is_v = lane >= pieces;
    const int piece = is_v ? lane - pieces : lane;
    const int64_t src = (static_cast<int64_t>(b) * p.num_kv_heads + hk) * pieces * 16 + piece * 16;
    const uint4 val = *reinterpret_cast<const uint4*>((is_v ? p.new_v : p.new_k) + src);
    char* dst = const_cast<char*>(is_v ? p.v : p.k) + hk * p.stride_head + row_off + piece * 16;
    *reinterpret_cast<uint4*>(dst) = val;
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

// Paged layout: byte offset of the page slot of token t, or -1 when the
// block-table entry lies outside the pool.
__device__ inline int64_t checked_page_row(const AttnParams& p, int32_t page, int t) {
  page = checked_page(page, p.num_pages, p.errors);
  if (page < 0) return -1;
  return static_cast<int64_t>(page) * p.stride_page + static_cast<int64_t>(t & p.page_mask) * p.stride_token;
}

// Partial results cross workgroups that may run on different XCDs, whose L2
// caches are not coherent with each other. They are written and read with
// device-scope accesses (the sc1 cache policy: stores write through to the
// device coherence point, loads do not hit stale cached copies), so no
// cache-wide writeback or invalidate is needed. A writer waits until its
// stores are acknowledged before the workgroup takes its ticket.
constexpr int kDeviceScope = 16;           // buffer-instruction cache policy bits: sc1
constexpr int kBufferConfig = 0x00020000;  // buffer descriptor word 3 for raw buffers on CDNA

__device__ inline __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kBufferConfig);
}
__device__ inline void store4_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off, float4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, off, 0, kDeviceScope);
}
__device__ inline float4 load4_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kDeviceScope));
}
__device__ inline void store_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, off, 0, kDeviceScope);
}
__device__ inline float load_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kDeviceScope));
}
__device__ inline void wait_stores_done() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Online log-sum-exp merge state: running max m (log2 units), weight sum and
// weighted sum of 4 output values. Merging is order-dependent only through
// rounding; callers always merge in split order.
struct MergeState {
  float m = -INFINITY;
  float wsum = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);

  // Add a part whose values o and weight sum wt are relative to 2^m2. A part
  // with m2 = -inf adds nothing. Branch-free, so that callers' loads of
  // later parts can be issued ahead of earlier merges.
  __device__ void add(float m2, float wt, float4 o) {
    const float mn = fmaxf(m, m2);
    const float ref = mn == -INFINITY ? 0.f : mn;
    const float a = fast_exp2(m - ref);
    const float b = fast_exp2(m2 - ref);
    acc.x = acc.x * a + b * o.x;
    acc.y = acc.y * a + b * o.y;
    acc.z = acc.z * a + b * o.z;
    acc.w = acc.w * a + b * o.w;
    wsum = wsum * a + b * wt;
    m = mn;
  }
};

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
  // This (b, hk)'s partial results: lse [S][G] and outputs [S][G][D].
  const __amdgpu_buffer_rsrc_t rl = buffer_rsrc(p.lse_part + part0 * G, nsplit_b * G * 4);
  const __amdgpu_buffer_rsrc_t ro = buffer_rsrc(p.o_part + part0 * G * D, nsplit_b * G * D * 4);
  const int slots = G * D / 4;  // 4 head_dim values per slot

  for (int slot = tid; slot < slots; slot += kThreads) {
    const int h = (slot * 4) / D;
    const int d0 = slot * 4 - h * D;
    MergeState st;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float4 o = *reinterpret_cast<const float4*>(&ws.o[w][h][d0]);
      st.add(ws.m[w][h], ws.l[w][h], o);  // wave sums are unnormalised: weight 2^m, sum l
    }
    const bool live = st.wsum > 0.f;
    const float inv = live ? 1.f / st.wsum : 0.f;
    const float4 on = make_float4(st.acc.x * inv, st.acc.y * inv, st.acc.z * inv, st.acc.w * inv);
    const float lse2 = live ? st.m + log2f(st.wsum) : -INFINITY;
    if (single) {
      const float os = p.out_scale;
      *reinterpret_cast<float4*>(p.out + static_cast<int64_t>(head0 + h) * D + d0) =
          make_float4(on.x * os, on.y * os, on.z * os, on.w * os);
      if (d0 == 0 && p.lse != nullptr) p.lse[head0 + h] = live ? lse2 * kLn2 : -INFINITY;
    } else {
      store4_coherent(ro, ((j * G + h) * D + d0) * 4, on);
      if (d0 == 0) store_coherent(rl, (j * G + h) * 4, lse2);
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

  // Merge over splits. With fewer slots than threads, tps adjacent lanes
  // share a slot and take splits sub, sub + tps, ... Each lane visits its
  // splits in batches of kMergeBatch whose loads are all in flight together;
  // a batch's largest log-weight is found first, so its part weights are
  // independent exponentials and its sums plain multiply-add chains, and the
  // batch folds into the lane's running state with one rescale. The lanes of
  // a slot then combine their states by lane shuffles. Every sum has a fixed
  // order, so results do not depend on timing. Each split part has weight
  // sum 1 (it is normalised) and log-weight lse2.
  const int tps = slots >= kThreads ? 1 : kThreads / slots;
  for (int slot = tid / tps; slot < slots; slot += kThreads / tps) {
    const int sub = tid % tps;
    const int h = (slot * 4) / D;
    const int d0 = slot * 4 - h * D;
    float m = -INFINITY, wsum = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = sub; s0 < nsplit_b; s0 += kMergeBatch * tps) {
      float l2[kMergeBatch];
      float4 o[kMergeBatch];
#pragma unroll
      for (int i = 0; i < kMergeBatch; ++i) {
        const int si = min(s0 + i * tps, nsplit_b - 1);  // past the last split: re-read it, weight 0
        l2[i] = load_coherent(rl, (si * G + h) * 4);
        o[i] = load4_coherent(ro, ((si * G + h) * D + d0) * 4);
      }
      float mb = -INFINITY;
#pragma unroll
      for (int i = 0; i < kMergeBatch; ++i) {
        if (s0 + i * tps >= nsplit_b) l2[i] = -INFINITY;
        mb = fmaxf(mb, l2[i]);
      }
      const float mn = fmaxf(m, mb);
      const float ref = mn == -INFINITY ? 0.f : mn;
      const float a = fast_exp2(m - ref);
      acc = make_float4(acc.x * a, acc.y * a, acc.z * a, acc.w * a);
      wsum *= a;
#pragma unroll
      for (int i = 0; i < kMergeBatch; ++i) {
        const float w = fast_exp2(l2[i] - ref);
        wsum += w;
        acc = make_float4(fmaf(w, o[i].x, acc.x), fmaf(w, o[i].y, acc.y), fmaf(w, o[i].z, acc.z),
                          fmaf(w, o[i].w, acc.w));
      }
      m = mn;
    }
    for (int off = 1; off < tps; off <<= 1) {
      MergeState st;
      st.m = m;
      st.wsum = wsum;
      st.acc = acc;
      st.add(__shfl_xor(m, off), __shfl_xor(wsum, off),
             make_float4(__shfl_xor(acc.x, off), __shfl_xor(acc.y, off), __shfl_xor(acc.z, off),
                         __shfl_xor(acc.w, off)));
      m = st.m;
      wsum = st.wsum;
      acc = st.acc;
    }
    if (sub == 0) {
      const float inv = p.out_scale / wsum;
      *reinterpret_cast<float4*>(p.out + static_cast<int64_t>(head0 + h) * D + d0) =
          make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
      if (d0 == 0 && p.lse != nullptr) p.lse[head0 + h] = (m + log2f(wsum)) * kLn2;
    }
  }
  // Back to zero for the next call. Issued after the merge's loads, which
  // would otherwise wait for it (memory operations complete in order).
  if (tid == 0) atomicExch(&p.tickets[b * p.num_kv_heads + hk], 0u);
}

}  // namespace comem
