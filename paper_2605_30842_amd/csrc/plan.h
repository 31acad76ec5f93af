// Internal to the library: the plan object and the host-side argument checks
// shared by the decode, append and prefill entry points (api.cpp,
// api_prefill.cpp). Nothing here touches the HIP runtime.
#pragma once

#include <cstdint>
#include <cstddef>

#include "comem_decode_attn.h"

namespace comem {
namespace host {

constexpr uint64_t kPlanMagic = 0x434f4d454d444131ull;  // "COMEMDA1"
constexpr int64_t kMaxContext = int64_t{1} << 30;
constexpr int kGridYZLimit = 65535;
constexpr int64_t kMaxTokenStrideBytes = int64_t{1} << 26;  // lane offsets within a tile stay 32-bit

inline size_t align256(size_t x) { return (x + 255) & ~size_t{255}; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

}  // namespace host
}  // namespace comem

struct comem_decode_attn_plan {
  uint64_t magic;
  comem_decode_attn_config cfg;
  int device;
  int num_cus;
  size_t ticket_bytes;
  size_t workspace_bytes;
};

namespace comem {
namespace host {

inline int group_of(const comem_decode_attn_config& c) { return c.num_q_heads / c.num_kv_heads; }

// Bytes of one K or V element (q is bf16 for FP8 caches).
inline int elem_bytes(const comem_decode_attn_config& c) {
  return c.dtype == COMEM_F32 ? 4 : (c.dtype == COMEM_FP8_E4M3 ? 1 : 2);
}
inline bool is_fp8(const comem_decode_attn_config& c) { return c.dtype == COMEM_FP8_E4M3; }

inline const comem_decode_attn_plan* checked(const comem_decode_attn_plan* p) {
  return (p != nullptr && p->magic == kPlanMagic) ? p : nullptr;
}

// Checks of the paged-layout arguments shared by attention and append.
inline comem_status validate_paged(const comem_decode_attn_plan& p, int64_t stride_page, int32_t page_size,
                                   int64_t num_pages, const int32_t* block_table, int32_t max_pages_per_seq,
                            int64_t max_ctx_len) {
  if (block_table == nullptr) return COMEM_ERR_NULL_POINTER;
  if (page_size <= 0 || page_size > 4096 || (page_size & (page_size - 1)) != 0) return COMEM_ERR_INVALID_SHAPE;
  if (num_pages <= 0 || stride_page <= 0) return COMEM_ERR_INVALID_SHAPE;
  if (max_pages_per_seq <= 0 || max_pages_per_seq < ceil_div(max_ctx_len, page_size))
    return COMEM_ERR_INVALID_SHAPE;
  if ((stride_page * elem_bytes(p.cfg)) % 16 != 0) return COMEM_ERR_MISALIGNED;
  if (!aligned(block_table, 4)) return COMEM_ERR_MISALIGNED;
  return COMEM_OK;
}

inline int log2_of(int32_t pow2) {
  int shift = 0;
  while ((1 << shift) < pow2) ++shift;
  return shift;
}

// Checks shared by both compute calls.
inline comem_status validate_common(const comem_decode_attn_plan& p, const void* q, const void* k, const void* v,
                             int64_t stride_token, int64_t stride_head, const int32_t* ctx_lens,
                             int32_t batch, int64_t max_ctx_len, const float* out, const float* lse,
                             const void* workspace) {
  if (batch < 0 || batch > p.cfg.max_batch) return COMEM_ERR_INVALID_SHAPE;
  if (max_ctx_len < 0 || max_ctx_len > p.cfg.max_ctx_len) return COMEM_ERR_INVALID_SHAPE;
  if (batch == 0) return COMEM_OK;
  if (q == nullptr || k == nullptr || v == nullptr || ctx_lens == nullptr || out == nullptr)
    return COMEM_ERR_NULL_POINTER;
  if (stride_token <= 0 || stride_head < 0) return COMEM_ERR_INVALID_SHAPE;
  if (p.cfg.num_kv_heads > 1 && stride_head == 0) return COMEM_ERR_INVALID_SHAPE;
  const int64_t e = elem_bytes(p.cfg);
  if ((stride_token * e) % 16 != 0 || (stride_head * e) % 16 != 0) return COMEM_ERR_MISALIGNED;
  if (stride_token * e > kMaxTokenStrideBytes) return COMEM_ERR_INVALID_SHAPE;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16)) return COMEM_ERR_MISALIGNED;
  if (lse != nullptr && !aligned(lse, 4)) return COMEM_ERR_MISALIGNED;
  if (workspace != nullptr && !aligned(workspace, 256)) return COMEM_ERR_MISALIGNED;
  return COMEM_OK;
}

}  // namespace host
}  // namespace comem
