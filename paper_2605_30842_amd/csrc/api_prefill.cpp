// Host side of the prefill-attention C ABI (comem_prefill_attn.h): argument
// validation (before any HIP call) and launch of the prefill kernel.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>

#include "attn_common.h"
#include "comem_decode_attn.h"
#include "comem_prefill_attn.h"
#include "plan.h"
#include "prefill.h"

using namespace comem::host;

namespace {

// A prefill call with no sequence or no new token reads and writes nothing,
// so, as for batch = 0 in the decode calls, it needs no buffers.
bool prefill_is_empty(int32_t batch, int32_t max_q_len) { return batch == 0 || max_q_len == 0; }

// Checks of a prefill call shared by both layouts; fills the kernel arguments.
comem_status prepare_prefill(const comem_decode_attn_plan& p, const void* q, const int64_t* q_start,
                             const int32_t* q_lens, int32_t max_q_len, const void* k, const void* v,
                             int64_t stride_token, int64_t stride_head, const int32_t* ctx_lens, int32_t batch,
                             int64_t max_ctx_len, float* out, float* lse, comem::PrefillParams& a) {
  if (p.cfg.dtype != COMEM_BF16) return COMEM_ERR_UNSUPPORTED;
  if (batch < 0 || batch > p.cfg.max_batch) return COMEM_ERR_INVALID_SHAPE;
  if (max_ctx_len < 0 || max_ctx_len > p.cfg.max_ctx_len) return COMEM_ERR_INVALID_SHAPE;
  if (max_q_len < 0 || max_q_len > max_ctx_len) return COMEM_ERR_INVALID_SHAPE;
  if (prefill_is_empty(batch, max_q_len)) return COMEM_OK;
  const comem_status st = validate_common(p, q, k, v, stride_token, stride_head, ctx_lens, batch, max_ctx_len, out,
                                          lse, nullptr);
  if (st != COMEM_OK) return st;
  if (q_start == nullptr || q_lens == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!aligned(q_start, 8) || !aligned(q_lens, 4)) return COMEM_ERR_MISALIGNED;
  const int64_t e = elem_bytes(p.cfg);
  std::memset(&a, 0, sizeof(a));
  a.q = static_cast<const char*>(q);
  a.k = static_cast<const char*>(k);
  a.v = static_cast<const char*>(v);
  a.out = out;
  a.lse = lse;
  a.q_start = q_start;
  a.q_lens = q_lens;
  a.ctx_lens = ctx_lens;
  a.stride_token = stride_token * e;
  a.stride_head = stride_head * e;
  a.num_q_heads = p.cfg.num_q_heads;
  a.group = group_of(p.cfg);
  a.tokens_per_block = comem::kPrefillRows / a.group;
  a.scale_log2 = p.cfg.scale * 1.4426950408889634f;
  a.max_ctx = static_cast<int32_t>(max_ctx_len);
  a.max_q = max_q_len;
  return COMEM_OK;
}

comem_status launch_prefill(const comem_decode_attn_plan& p, const comem::PrefillParams& a, bool paged,
                            int32_t batch, int32_t max_q_len, void* stream) {
  const int64_t blocks = ceil_div(max_q_len, a.tokens_per_block);
  comem::PrefillKernelFn fn = comem::select_prefill_kernel(p.cfg.head_dim, paged ? a.page_mask + 1 : 0);
  if (fn == nullptr) return COMEM_ERR_UNSUPPORTED;
  comem::PrefillParams args = a;
  void* argv[] = {&args};
  const hipError_t err =
      hipLaunchKernel(reinterpret_cast<const void*>(fn),
                      dim3(static_cast<unsigned>(blocks), static_cast<unsigned>(p.cfg.num_kv_heads),
                           static_cast<unsigned>(batch)),
                      dim3(comem::kPrefillThreads), argv, 0, static_cast<hipStream_t>(stream));
  return err == hipSuccess ? COMEM_OK : COMEM_ERR_HIP;
}

}  // namespace

extern "C" {

comem_status comem_prefill_attn(const comem_decode_attn_plan* plan, const void* q, const int64_t* q_start,
                                const int32_t* q_lens, int32_t max_q_len, const void* k, const void* v,
                                int64_t stride_token, int64_t stride_head, const int64_t* seq_start,
                                const int32_t* ctx_lens, int32_t batch, int64_t max_ctx_len, float* out,
                                float* lse, void* hip_stream) {
  const comem_decode_attn_plan* p = checked(plan);
  if (p == nullptr) return COMEM_ERR_BAD_HANDLE;
  comem::PrefillParams a;
  comem_status st = prepare_prefill(*p, q, q_start, q_lens, max_q_len, k, v, stride_token, stride_head, ctx_lens,
                                    batch, max_ctx_len, out, lse, a);
  if (st != COMEM_OK || prefill_is_empty(batch, max_q_len)) return st;
  if (seq_start == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!aligned(seq_start, 8)) return COMEM_ERR_MISALIGNED;
  if (p->device == COMEM_NO_DEVICE) return COMEM_ERR_NO_DEVICE;
  a.seq_start = seq_start;
  return launch_prefill(*p, a, false, batch, max_q_len, hip_stream);
}

comem_status comem_prefill_attn_paged(const comem_decode_attn_plan* plan, const void* q, const int64_t* q_start,
                                      const int32_t* q_lens, int32_t max_q_len, const void* k_pages,
                                      const void* v_pages, int64_t stride_page, int64_t stride_token,
                                      int64_t stride_head, int32_t page_size, int64_t num_pages,
                                      const int32_t* block_table, int32_t max_pages_per_seq,
                                      const int32_t* ctx_lens, int32_t batch, int64_t max_ctx_len, float* out,
                                      float* lse, void* hip_stream) {
  const comem_decode_attn_plan* p = checked(plan);
  if (p == nullptr) return COMEM_ERR_BAD_HANDLE;
  comem::PrefillParams a;
  comem_status st = prepare_prefill(*p, q, q_start, q_lens, max_q_len, k_pages, v_pages, stride_token, stride_head,
                                    ctx_lens, batch, max_ctx_len, out, lse, a);
  if (st != COMEM_OK || prefill_is_empty(batch, max_q_len)) return st;
  st = validate_paged(*p, stride_page, page_size, num_pages, block_table, max_pages_per_seq, max_ctx_len);
  if (st != COMEM_OK) return st;
  if (p->device == COMEM_NO_DEVICE) return COMEM_ERR_NO_DEVICE;
  a.block_table = block_table;
  a.stride_page = stride_page * elem_bytes(p->cfg);
  a.max_pages = max_pages_per_seq;
  a.page_shift = log2_of(page_size);
  a.page_mask = page_size - 1;
  a.num_pages = num_pages;
  return launch_prefill(*p, a, true, batch, max_q_len, hip_stream);
}

}  // extern "C"
