// Kernel arguments of the KV-append kernel (host and device side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace comem {

// Offsets and strides are in bytes. The new rows are dense [B, Hkv, D].
struct AppendParams {
  const char* new_k;
  const char* new_v;
  char* k;                     // contiguous: [T, Hkv, D] rows; paged: page pool
  char* v;
  const int64_t* seq_start;    // contiguous layout
  const int32_t* ctx_lens;     // L_b, counting the new token
  const int32_t* block_table;  // paged layout, [B, max_pages]
  int64_t stride_token;
  int64_t stride_head;
  int64_t stride_page;
  int64_t num_pages;
  int64_t max_ctx_len;
  int32_t max_pages;
  int32_t page_shift;
  int32_t page_mask;
  int32_t num_kv_heads;
  int32_t chunks_per_head;     // 16-byte pieces in one head's D elements
};

using AppendKernelFn = void (*)(AppendParams);
AppendKernelFn select_append_kernel(bool paged);

}  // namespace comem
