// Kernel arguments of the prefill-attention kernel (host and device side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace comem {

constexpr int kPrefillThreads = 512;  // 8 waves: two halves of the key tiles, 4 waves each
constexpr int kPrefillRows = 128;     // (query token, query head) rows per workgroup: 32 per wave
constexpr int kPrefillTileKeys = 64;  // keys per K/V tile staged in LDS

// Offsets and strides are in bytes.
struct PrefillParams {
  const char* q;               // [total_q, Hq, D] bf16, sequence b's new tokens from row q_start[b]
  const char* k;               // contiguous: [T, Hkv, D] rows; paged: page pool
  const char* v;
  float* out;                  // [total_q, Hq, D]
  float* lse;                  // [total_q, Hq] or nullptr
  const int64_t* q_start;
  const int32_t* q_lens;       // M_b new tokens (the last M_b of the L_b cached ones)
  const int64_t* seq_start;    // contiguous layout
  const int32_t* ctx_lens;     // L_b
  const int32_t* block_table;  // paged layout, [B, max_pages]
  int64_t stride_token;
  int64_t stride_head;
  int64_t stride_page;
  int32_t max_pages;
  int32_t page_shift;
  int32_t page_mask;
  int32_t num_q_heads;
  int32_t group;               // G = Hq / Hkv
  int32_t tokens_per_block;    // kPrefillRows / G new tokens per workgroup
  float scale_log2;            // scale * log2(e)
  int32_t max_ctx;             // ctx_lens[b] is clamped to [0, max_ctx]
  int32_t max_q;               // q_lens[b] is clamped to [0, min(L_b, max_q)]
  int64_t num_pages;           // paged layout: entries outside [0, num_pages) read page 0
};

using PrefillKernelFn = void (*)(PrefillParams);
// page_size 0 selects the contiguous-cache kernel.
PrefillKernelFn select_prefill_kernel(int head_dim, int page_size);

}  // namespace comem
