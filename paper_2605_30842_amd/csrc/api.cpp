// Host side of the decode-attention C ABI: argument validation (always before
// any HIP call), split planning, kernel selection and launch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>

#include "attn_common.h"
#include "comem_decode_attn.h"
#include "kv_append.h"
#include "noalloc.h"
#include "plan.h"

namespace comem {
using KernelFn = void (*)(AttnParams);
using QueueKernelFn = void (*)(AttnParams, int);
KernelFn select_mfma_kernel(int head_dim, bool paged, int page_size, bool fp8);
QueueKernelFn select_mfma_queue_kernel(int head_dim, bool paged, int page_size, bool fp8);
int mfma_max_split_pages();
int mfma_max_queue_batch();
KernelFn select_valu_kernel(bool bf16, int head_dim, int group, bool paged);
}  // namespace comem

using namespace comem::host;

namespace {

constexpr int kAssumedCUs = 256;                        // gfx950 (MI355X) without a device query
constexpr int64_t kTargetWgsPerCu = 2;                  // workgroups per compute unit for one full round
constexpr int kQueueWgsPerCu = 2;                       // resident workgroups per compute unit (MFMA kernel)
constexpr int64_t kTailRounds = 4;                      // items per resident workgroup that enable short last splits
constexpr int64_t kMinChunk = 64;                       // tokens per split, lower bound
constexpr int64_t kMaxChunk = 2048;                     // tokens per split, upper bound (auto plan)

bool uses_mfma(const comem_decode_attn_plan& p);

// After the tickets [max_batch * Hkv]: the two work-queue counters and the
// device error word.
constexpr int kCounterWords = 3;
constexpr int kErrorWord = 2;  // index after the tickets

bool debug_checks(const comem_decode_attn_plan& p) { return (p.cfg.flags & COMEM_FLAG_DEBUG_CHECKS) != 0; }

// With debug checks the error word lives in the workspace, so one is needed.
comem_status check_debug_workspace(const comem_decode_attn_plan& p, const void* workspace, size_t ws_bytes) {
  if (!debug_checks(p)) return COMEM_OK;
  if (workspace == nullptr) return COMEM_ERR_NULL_POINTER;
  return ws_bytes < p.ticket_bytes ? COMEM_ERR_WORKSPACE_TOO_SMALL : COMEM_OK;
}

// Workspace bytes for `slots` (sequence, split) partial results: ticket
// counters, then per-head lse values, then per-head partial outputs.
size_t slots_workspace_bytes(const comem_decode_attn_plan& p, int64_t slots) {
  const size_t rows = static_cast<size_t>(slots) * static_cast<size_t>(p.cfg.num_q_heads);
  return p.ticket_bytes + align256(rows * 4) + rows * static_cast<size_t>(p.cfg.head_dim) * 4;
}

// Workspace bytes a call with `batch` sequences and `splits` splits needs.
// A single split writes the output directly and touches no workspace.
size_t call_workspace_bytes(const comem_decode_attn_plan& p, int64_t batch, int64_t splits) {
  return splits <= 1 ? 0 : slots_workspace_bytes(p, batch * splits);
}

// Tokens per split for the matrix-core kernel, from the host-side bounds of
// a call (the device-side lengths are never read on the host). Splits of
// 4096 tokens keep contexts of 128k and more at <= 32 splits; otherwise 2048
// if that still leaves >= 16 work items per resident workgroup, else 1024.
// Smaller items end the work queue more evenly (the last items handed out
// finish at nearly the same time) at the cost of one more partial result
// per item; at 8 items of 2048 tokens per workgroup the even end still wins.
int64_t mfma_chunk(const comem_decode_attn_plan& p, int64_t batch, int64_t L) {
  if (L >= 32 * 4096) return 4096;
  const int64_t resident = static_cast<int64_t>(kQueueWgsPerCu) * p.num_cus;
  if (batch * p.cfg.num_kv_heads * ceil_div(L, 2048) >= 16 * resident) return 2048;
  return 1024;
}

// Largest split, in tokens, whose block-table entries fit the matrix-core
// kernel's LDS copy (a multiple of 32), for pages of `page_size` tokens.
int64_t mfma_page_cap(int64_t page_size) {
  return std::max<int64_t>(32, (comem::mfma_max_split_pages() - 2) * page_size / 32 * 32);
}

// Choose tokens per split and the split count for one call. page_size is 0
// for a contiguous cache; for a paged one the matrix-core kernel's planned
// splits stay within the pages its LDS copy of the block table holds.
comem_status plan_call(const comem_decode_attn_plan& p, int64_t batch, int64_t max_ctx, int64_t page_size,
                       size_t ws_bytes, int64_t* chunk_out, int64_t* splits_out) {
  const int64_t L = max_ctx > 0 ? max_ctx : 1;
  const int64_t cap = page_size > 0 && uses_mfma(p) ? mfma_page_cap(page_size) : INT64_MAX;
  int64_t chunk;
  if (p.cfg.chunk_tokens > 0) {
    chunk = p.cfg.chunk_tokens;
    if (call_workspace_bytes(p, batch, ceil_div(L, chunk)) > ws_bytes) return COMEM_ERR_WORKSPACE_TOO_SMALL;
  } else {
    if (uses_mfma(p)) {
      chunk = std::min(mfma_chunk(p, batch, L), cap);
    } else {
      const int64_t target = kTargetWgsPerCu * p.num_cus;
      const int64_t per = ceil_div(batch * p.cfg.num_kv_heads * L, target);
      chunk = kMinChunk;
      while (chunk < per && chunk < kMaxChunk) chunk *= 2;
    }
    while (call_workspace_bytes(p, batch, ceil_div(L, chunk)) > ws_bytes) {
      if (chunk >= L || chunk * 2 > cap) return COMEM_ERR_WORKSPACE_TOO_SMALL;
      chunk *= 2;
    }
  }
  *chunk_out = chunk;
  *splits_out = ceil_div(L, chunk);
  return COMEM_OK;
}

comem_status validate_config(const comem_decode_attn_config& c) {
  if (c.num_q_heads <= 0 || c.num_kv_heads <= 0 || c.num_q_heads % c.num_kv_heads != 0)
    return COMEM_ERR_INVALID_SHAPE;
  if (c.num_kv_heads > kGridYZLimit) return COMEM_ERR_INVALID_SHAPE;
  const int G = group_of(c);
  if (G != 1 && G != 2 && G != 4 && G != 8 && G != 16) return COMEM_ERR_UNSUPPORTED;
  if (c.head_dim != 64 && c.head_dim != 128) return COMEM_ERR_UNSUPPORTED;
  if (c.dtype != COMEM_F32 && c.dtype != COMEM_BF16 && c.dtype != COMEM_FP8_E4M3) return COMEM_ERR_UNSUPPORTED;
  if (!std::isfinite(c.scale) || !(c.scale > 0.f)) return COMEM_ERR_INVALID_SHAPE;
  if (c.max_batch <= 0 || c.max_batch > kGridYZLimit) return COMEM_ERR_INVALID_SHAPE;
  if (c.max_ctx_len <= 0 || c.max_ctx_len > kMaxContext) return COMEM_ERR_INVALID_SHAPE;
  if (c.chunk_tokens < 0 || c.chunk_tokens % 32 != 0 || c.chunk_tokens > kMaxContext)
    return COMEM_ERR_INVALID_SHAPE;
  if (c.variant != COMEM_VARIANT_AUTO && c.variant != COMEM_VARIANT_VALU && c.variant != COMEM_VARIANT_MFMA &&
      c.variant != COMEM_VARIANT_MFMA_GRID)
    return COMEM_ERR_UNSUPPORTED;
  if ((c.flags & ~COMEM_FLAG_DEBUG_CHECKS) != 0) return COMEM_ERR_UNSUPPORTED;
  if ((c.variant == COMEM_VARIANT_MFMA || c.variant == COMEM_VARIANT_MFMA_GRID) && c.dtype == COMEM_F32)
    return COMEM_ERR_UNSUPPORTED;
  if (c.dtype == COMEM_FP8_E4M3) {
    if (c.variant == COMEM_VARIANT_VALU) return COMEM_ERR_UNSUPPORTED;
    if (!std::isfinite(c.k_scale) || !(c.k_scale > 0.f) || !std::isfinite(c.v_scale) || !(c.v_scale > 0.f))
      return COMEM_ERR_INVALID_SHAPE;
  }
  return COMEM_OK;
}





bool uses_mfma(const comem_decode_attn_plan& p) {
  return p.cfg.variant == COMEM_VARIANT_MFMA || p.cfg.variant == COMEM_VARIANT_MFMA_GRID ||
         (p.cfg.variant == COMEM_VARIANT_AUTO && p.cfg.dtype != COMEM_F32);
}

// The work-queue form of the matrix-core kernel keeps two counters after the
// tickets, so it needs a workspace (of at least the ticket region).
bool uses_queue(const comem_decode_attn_plan& p, int64_t batch, const void* workspace, size_t ws_bytes) {
  return uses_mfma(p) && p.cfg.variant != COMEM_VARIANT_MFMA_GRID && batch <= comem::mfma_max_queue_batch() &&
         workspace != nullptr && ws_bytes >= p.ticket_bytes;
}

comem_status launch(const comem_decode_attn_plan& p, bool paged, comem::AttnParams& a, int64_t batch,
                    int64_t splits, bool queue, void* stream) {
  const bool bf16 = p.cfg.dtype == COMEM_BF16;
  const int64_t items = batch * p.cfg.num_kv_heads * splits;
  const int64_t resident = static_cast<int64_t>(kQueueWgsPerCu) * p.num_cus;
  // With no more (nominal) items than resident workgroups every item gets its
  // own workgroup anyway, and the grid form saves the queue's prologue.
  if (queue && items > resident) {
    comem::QueueKernelFn qfn = comem::select_mfma_queue_kernel(p.cfg.head_dim, paged, a.page_mask + 1, is_fp8(p.cfg));
    if (qfn == nullptr) return COMEM_ERR_UNSUPPORTED;
    // With several rounds of items, each sequence ends in short splits of
    // half a chunk, about one round of them in all: the queue hands them out
    // last, so the workgroups finish closer together (quarter-chunk splits or
    // two rounds of them gained less). Only planned chunks of 1024 tokens or
    // more (and, paged, whose 1.25-chunk splits still fit the kernel's LDS
    // copy of the block table); a configured chunk_tokens keeps even splits.
    if (p.cfg.chunk_tokens == 0 && items >= kTailRounds * resident && a.chunk >= 1024 &&
        (!paged || 2 * static_cast<int64_t>(a.chunk) <= mfma_page_cap(a.page_mask + 1))) {
      a.tail_chunk = a.chunk / 2;
      a.tail_splits = static_cast<int32_t>(ceil_div(resident, batch * p.cfg.num_kv_heads));
    }
    dim3 grid(static_cast<unsigned>(items < resident ? items : resident));
    dim3 block(comem::kThreads);
    int nb = static_cast<int>(batch);
    void* args[] = {&a, &nb};
    const hipError_t err = hipLaunchKernel(reinterpret_cast<const void*>(qfn), grid, block, args, 0,
                                           static_cast<hipStream_t>(stream));
    return err == hipSuccess ? COMEM_OK : COMEM_ERR_HIP;
  }
  comem::KernelFn fn = uses_mfma(p) ? comem::select_mfma_kernel(p.cfg.head_dim, paged, a.page_mask + 1, is_fp8(p.cfg))
                                    : comem::select_valu_kernel(bf16, p.cfg.head_dim, group_of(p.cfg), paged);
  if (fn == nullptr) return COMEM_ERR_UNSUPPORTED;
  dim3 grid(static_cast<unsigned>(splits), static_cast<unsigned>(p.cfg.num_kv_heads),
            static_cast<unsigned>(batch));
  dim3 block(comem::kThreads);
  void* args[] = {&a};
  const hipError_t err = hipLaunchKernel(reinterpret_cast<const void*>(fn), grid, block, args, 0,
                                         static_cast<hipStream_t>(stream));
  return err == hipSuccess ? COMEM_OK : COMEM_ERR_HIP;
}

// Checks of an append call; fills the kernel arguments shared by both layouts.
comem_status prepare_append(const comem_decode_attn_plan& p, const void* new_k, const void* new_v, void* k,
                            void* v, int64_t stride_token, int64_t stride_head, const int32_t* ctx_lens,
                            int32_t batch, int64_t max_ctx_len, comem::AppendParams& a) {
  if (batch < 0 || batch > p.cfg.max_batch) return COMEM_ERR_INVALID_SHAPE;
  if (max_ctx_len < 0 || max_ctx_len > p.cfg.max_ctx_len) return COMEM_ERR_INVALID_SHAPE;
  if (batch == 0) return COMEM_OK;
  if (new_k == nullptr || new_v == nullptr || k == nullptr || v == nullptr || ctx_lens == nullptr)
    return COMEM_ERR_NULL_POINTER;
  if (stride_token <= 0 || stride_head < 0) return COMEM_ERR_INVALID_SHAPE;
  if (p.cfg.num_kv_heads > 1 && stride_head == 0) return COMEM_ERR_INVALID_SHAPE;
  const int64_t e = elem_bytes(p.cfg);
  if ((stride_token * e) % 16 != 0 || (stride_head * e) % 16 != 0) return COMEM_ERR_MISALIGNED;
  if (!aligned(new_k, 16) || !aligned(new_v, 16) || !aligned(k, 16) || !aligned(v, 16))
    return COMEM_ERR_MISALIGNED;
  std::memset(&a, 0, sizeof(a));
  a.new_k = static_cast<const char*>(new_k);
  a.new_v = static_cast<const char*>(new_v);
  a.k = static_cast<char*>(k);
  a.v = static_cast<char*>(v);
  a.ctx_lens = ctx_lens;
  a.stride_token = stride_token * e;
  a.stride_head = stride_head * e;
  a.max_ctx_len = max_ctx_len;
  a.num_kv_heads = p.cfg.num_kv_heads;
  a.chunks_per_head = static_cast<int32_t>(p.cfg.head_dim * e / 16);
  return COMEM_OK;
}

comem_status launch_append(const comem::AppendParams& a, bool paged, int32_t batch, void* stream) {
  comem::AppendParams args = a;
  void* argv[] = {&args};
  const hipError_t err = hipLaunchKernel(reinterpret_cast<const void*>(comem::select_append_kernel(paged)),
                                         dim3(static_cast<unsigned>(batch)), dim3(comem::kThreads), argv, 0,
                                         static_cast<hipStream_t>(stream));
  return err == hipSuccess ? COMEM_OK : COMEM_ERR_HIP;
}

void fill_common(const comem_decode_attn_plan& p, comem::AttnParams& a, const void* q, const void* k,
                 const void* v, int64_t stride_token, int64_t stride_head, const int32_t* ctx_lens,
                 float* out, float* lse, void* workspace, int64_t batch, int64_t max_ctx_len, int64_t chunk,
                 int64_t splits, bool queue, size_t ticket_region) {
  const int64_t e = elem_bytes(p.cfg);
  std::memset(&a, 0, sizeof(a));
  a.max_ctx = static_cast<int32_t>(max_ctx_len);
  if (debug_checks(p)) a.errors = static_cast<uint32_t*>(workspace) + p.cfg.max_batch * p.cfg.num_kv_heads + kErrorWord;
  a.q = static_cast<const char*>(q);
  a.k = static_cast<const char*>(k);
  a.v = static_cast<const char*>(v);
  a.out = out;
  a.lse = lse;
  a.ctx_lens = ctx_lens;
  a.stride_token = stride_token * e;
  a.stride_head = stride_head * e;
  a.num_q_heads = p.cfg.num_q_heads;
  a.num_kv_heads = p.cfg.num_kv_heads;
  a.group = group_of(p.cfg);
  a.chunk = static_cast<int32_t>(chunk);
  a.num_splits = static_cast<int32_t>(splits);
  // An FP8 cache's K scale multiplies every score; its V scale every output.
  a.scale_log2 = p.cfg.scale * (is_fp8(p.cfg) ? p.cfg.k_scale : 1.f) * 1.4426950408889634f;
  a.out_scale = is_fp8(p.cfg) ? p.cfg.v_scale : 1.f;
  a.queue_slot = p.cfg.max_batch * p.cfg.num_kv_heads;
  if (splits > 1 || queue) {
    char* ws = static_cast<char*>(workspace);
    const size_t slots = static_cast<size_t>(batch) * static_cast<size_t>(splits) *
                         static_cast<size_t>(p.cfg.num_q_heads);
    a.tickets = reinterpret_cast<uint32_t*>(ws);
    a.lse_part = reinterpret_cast<float*>(ws + ticket_region);
    a.o_part = reinterpret_cast<float*>(ws + ticket_region + align256(slots * 4));
  }
}

// The attention calls, with or without the fused append of the new rows.
comem_status decode_contiguous(const comem_decode_attn_plan* plan, const void* q, const void* new_k,
                               const void* new_v, const void* k, const void* v, int64_t stride_token,
                               int64_t stride_head, const int64_t* seq_start, const int32_t* ctx_lens,
                               int32_t batch, int64_t max_ctx_len, float* out, float* lse, void* workspace,
                               size_t workspace_bytes, void* hip_stream, bool fused, size_t ticket_region = 0) {
  const comem_decode_attn_plan* p = checked(plan);
  if (p == nullptr) return COMEM_ERR_BAD_HANDLE;
  if (ticket_region == 0) ticket_region = p->ticket_bytes;
  comem_status st = validate_common(*p, q, k, v, stride_token, stride_head, ctx_lens, batch, max_ctx_len,
                                    out, lse, workspace);
  if (st != COMEM_OK || batch == 0) return st;
  if (seq_start == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!aligned(seq_start, 8)) return COMEM_ERR_MISALIGNED;
  if (fused) {
    if (new_k == nullptr || new_v == nullptr) return COMEM_ERR_NULL_POINTER;
    if (!aligned(new_k, 16) || !aligned(new_v, 16)) return COMEM_ERR_MISALIGNED;
  }
  int64_t chunk = 0, splits = 0;
  st = plan_call(*p, batch, max_ctx_len, 0, workspace == nullptr ? 0 : workspace_bytes, &chunk, &splits);
  if (st != COMEM_OK) return st;
  st = check_debug_workspace(*p, workspace, workspace_bytes);
  if (st != COMEM_OK) return st;
  if (p->device == COMEM_NO_DEVICE) return COMEM_ERR_NO_DEVICE;
  const bool queue = uses_queue(*p, batch, workspace, workspace_bytes);
  comem::AttnParams a;
  fill_common(*p, a, q, k, v, stride_token, stride_head, ctx_lens, out, lse, workspace, batch, max_ctx_len, chunk,
              splits, queue, ticket_region);
  a.seq_start = seq_start;
  if (fused) {
    a.new_k = static_cast<const char*>(new_k);
    a.new_v = static_cast<const char*>(new_v);
  }
  return launch(*p, false, a, batch, splits, queue, hip_stream);
}

comem_status decode_paged(const comem_decode_attn_plan* plan, const void* q, const void* new_k,
                          const void* new_v, const void* k_pages, const void* v_pages, int64_t stride_page,
                          int64_t stride_token, int64_t stride_head, int32_t page_size, int64_t num_pages,
                          const int32_t* block_table, int32_t max_pages_per_seq, const int32_t* ctx_lens,
                          int32_t batch, int64_t max_ctx_len, float* out, float* lse, void* workspace,
                          size_t workspace_bytes, void* hip_stream, bool fused) {
  const comem_decode_attn_plan* p = checked(plan);
  if (p == nullptr) return COMEM_ERR_BAD_HANDLE;
  comem_status st = validate_common(*p, q, k_pages, v_pages, stride_token, stride_head, ctx_lens, batch,
                                    max_ctx_len, out, lse, workspace);
  if (st != COMEM_OK || batch == 0) return st;
  st = validate_paged(*p, stride_page, page_size, num_pages, block_table, max_pages_per_seq, max_ctx_len);
  if (st != COMEM_OK) return st;
  if (fused) {
    if (new_k == nullptr || new_v == nullptr) return COMEM_ERR_NULL_POINTER;
    if (!aligned(new_k, 16) || !aligned(new_v, 16)) return COMEM_ERR_MISALIGNED;
  }
  int64_t chunk = 0, splits = 0;
  st = plan_call(*p, batch, max_ctx_len, page_size, workspace == nullptr ? 0 : workspace_bytes, &chunk, &splits);
  if (st != COMEM_OK) return st;
  // The matrix-core kernel stages one split's block-table entries in LDS (a
  // planned split always fits; a configured chunk_tokens may not).
  if (uses_mfma(*p) && (chunk - 1) / page_size + 2 > comem::mfma_max_split_pages()) return COMEM_ERR_INVALID_SHAPE;
  st = check_debug_workspace(*p, workspace, workspace_bytes);
  if (st != COMEM_OK) return st;
  if (p->device == COMEM_NO_DEVICE) return COMEM_ERR_NO_DEVICE;
  const bool queue = uses_queue(*p, batch, workspace, workspace_bytes);
  comem::AttnParams a;
  fill_common(*p, a, q, k_pages, v_pages, stride_token, stride_head, ctx_lens, out, lse, workspace, batch,
              max_ctx_len, chunk, splits, queue, p->ticket_bytes);
  a.block_table = block_table;
  a.stride_page = stride_page * elem_bytes(p->cfg);
  a.max_pages = max_pages_per_seq;
  a.num_pages = num_pages;
  a.page_shift = log2_of(page_size);
  a.page_mask = page_size - 1;
  if (fused) {
    a.new_k = static_cast<const char*>(new_k);
    a.new_v = static_cast<const char*>(new_v);
  }
  return launch(*p, true, a, batch, splits, queue, hip_stream);
}

}  // namespace

extern "C" {

const char* comem_status_string(comem_status s) {
  switch (s) {
    case COMEM_OK: return "ok";
    case COMEM_ERR_NULL_POINTER: return "a required pointer is NULL";
    case COMEM_ERR_INVALID_SHAPE: return "invalid shape, stride or bound";
    case COMEM_ERR_UNSUPPORTED: return "unsupported dtype, head_dim, GQA group, variant or device";
    case COMEM_ERR_MISALIGNED: return "pointer or byte stride not suitably aligned";
    case COMEM_ERR_WORKSPACE_TOO_SMALL: return "workspace too small for this call";
    case COMEM_ERR_BAD_HANDLE: return "NULL or invalid plan";
    case COMEM_ERR_HIP: return "HIP runtime error";
    case COMEM_ERR_NO_DEVICE: return "plan was made without a device";
    case COMEM_ERR_SCRATCH_LIMIT: return "call needs more than the library's fixed device scratch holds";
  }
  return "unknown status";
}

comem_status comem_decode_attn_init(const comem_decode_attn_config* cfg, int device,
                                    comem_decode_attn_plan** plan_out, size_t* workspace_bytes_out) {
  if (cfg == nullptr || plan_out == nullptr || workspace_bytes_out == nullptr) return COMEM_ERR_NULL_POINTER;
  *plan_out = nullptr;
  *workspace_bytes_out = 0;
  const comem_status st = validate_config(*cfg);
  if (st != COMEM_OK) return st;
  if (device < COMEM_NO_DEVICE) return COMEM_ERR_INVALID_SHAPE;
  int num_cus = kAssumedCUs;
  if (device != COMEM_NO_DEVICE) {
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess) return COMEM_ERR_HIP;
    if (device >= count) return COMEM_ERR_INVALID_SHAPE;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, device) != hipSuccess) return COMEM_ERR_HIP;
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) return COMEM_ERR_UNSUPPORTED;
    num_cus = prop.multiProcessorCount;
  }
  auto* p = new (std::nothrow) comem_decode_attn_plan;
  if (p == nullptr) return COMEM_ERR_HIP;
  p->magic = kPlanMagic;
  p->cfg = *cfg;
  p->device = device;
  p->num_cus = num_cus > 0 ? num_cus : kAssumedCUs;
  // tickets (one per sequence and KV head), then the two work-queue counters
  p->ticket_bytes = align256((static_cast<size_t>(cfg->max_batch) * cfg->num_kv_heads + kCounterWords) * 4);
  // Largest number of (sequence, split) slots any call within the limits plans
  // (bounded for the matrix-core kernel by its smallest split of 1024 tokens);
  // calls with a smaller workspace get coarser splits.
  const int64_t B = cfg->max_batch, L = cfg->max_ctx_len;
  int64_t slots;
  if (cfg->chunk_tokens > 0) {
    slots = B * ceil_div(L, cfg->chunk_tokens);
  } else if (uses_mfma(*p)) {
    slots = B * ceil_div(L, 1024);
  } else {
    const int64_t target = kTargetWgsPerCu * p->num_cus;
    const int64_t a = ceil_div(target, cfg->num_kv_heads) + B;
    const int64_t b = B * ceil_div(L, kMaxChunk);
    slots = a > b ? a : b;
    const int64_t c = B * ceil_div(L, kMinChunk);
    if (c < slots) slots = c;
  }
  p->workspace_bytes = slots_workspace_bytes(*p, slots);
  // The allocation-free entry point's scratch on this device (looked up and
  // cleared once per device); the other entry points work without it.
  if (device != COMEM_NO_DEVICE) (void)comem::scratch_setup(device);
  *plan_out = p;
  *workspace_bytes_out = p->workspace_bytes;
  return COMEM_OK;
}

comem_status comem_decode_attn_destroy(comem_decode_attn_plan* plan) {
  if (plan == nullptr) return COMEM_OK;
  if (plan->magic != kPlanMagic) return COMEM_ERR_BAD_HANDLE;
  plan->magic = 0;
  delete plan;
  return COMEM_OK;
}

comem_status comem_decode_attn_device_errors(const comem_decode_attn_plan* plan, void* workspace,
                                             size_t workspace_bytes, uint32_t* errors_out, void* hip_stream) {
  const comem_decode_attn_plan* p = checked(plan);
  if (p == nullptr) return COMEM_ERR_BAD_HANDLE;
  if (workspace == nullptr || errors_out == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!aligned(workspace, 256)) return COMEM_ERR_MISALIGNED;
  if (workspace_bytes < p->ticket_bytes) return COMEM_ERR_WORKSPACE_TOO_SMALL;
  *errors_out = 0;
  if (p->device == COMEM_NO_DEVICE) return COMEM_ERR_NO_DEVICE;
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  uint32_t* word = static_cast<uint32_t*>(workspace) + p->cfg.max_batch * p->cfg.num_kv_heads + kErrorWord;
  uint32_t host = 0;
  if (hipMemcpyAsync(&host, word, sizeof(host), hipMemcpyDeviceToHost, s) != hipSuccess) return COMEM_ERR_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return COMEM_ERR_HIP;
  if (host != 0) {
    if (hipMemsetAsync(word, 0, sizeof(host), s) != hipSuccess) return COMEM_ERR_HIP;
    if (hipStreamSynchronize(s) != hipSuccess) return COMEM_ERR_HIP;
  }
  *errors_out = host;
  return COMEM_OK;
}

comem_status comem_decode_attn_plan_splits(const comem_decode_attn_plan* plan, int32_t batch,
                                           int64_t max_ctx_len, size_t workspace_bytes,
                                           int32_t* chunk_tokens_out, int32_t* num_splits_out) {
  const comem_decode_attn_plan* p = checked(plan);
  if (p == nullptr) return COMEM_ERR_BAD_HANDLE;
  if (chunk_tokens_out == nullptr || num_splits_out == nullptr) return COMEM_ERR_NULL_POINTER;
  if (batch < 0 || batch > p->cfg.max_batch) return COMEM_ERR_INVALID_SHAPE;
  if (max_ctx_len < 0 || max_ctx_len > p->cfg.max_ctx_len) return COMEM_ERR_INVALID_SHAPE;
  int64_t chunk = 0, splits = 0;
  const comem_status st = plan_call(*p, batch, max_ctx_len, 0, workspace_bytes, &chunk, &splits);
  if (st != COMEM_OK) return st;
  *chunk_tokens_out = static_cast<int32_t>(chunk);
  *num_splits_out = static_cast<int32_t>(splits);
  return COMEM_OK;
}

comem_status comem_decode_attn(const comem_decode_attn_plan* plan, const void* q, const void* k,
                               const void* v, int64_t stride_token, int64_t stride_head,
                               const int64_t* seq_start, const int32_t* ctx_lens, int32_t batch,
                               int64_t max_ctx_len, float* out, float* lse, void* workspace,
                               size_t workspace_bytes, void* hip_stream) {
  return decode_contiguous(plan, q, nullptr, nullptr, k, v, stride_token, stride_head, seq_start, ctx_lens, batch,
                           max_ctx_len, out, lse, workspace, workspace_bytes, hip_stream, false);
}

comem_status comem_decode_attn_noalloc(const comem_decode_attn_plan* plan, const void* q, const void* k,
                                       const void* v, int64_t stride_token, int64_t stride_head,
                                       const int64_t* seq_start, const int32_t* ctx_lens, int32_t batch,
                                       int64_t max_ctx_len, float* out, float* lse, void* hip_stream) {
  const comem_decode_attn_plan* p = checked(plan);
  if (p == nullptr) return COMEM_ERR_BAD_HANDLE;
  if (debug_checks(*p)) return COMEM_ERR_UNSUPPORTED;
  comem_status st = validate_common(*p, q, k, v, stride_token, stride_head, ctx_lens, batch, max_ctx_len, out, lse,
                                    nullptr);
  if (st != COMEM_OK || batch == 0) return st;
  if (seq_start == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!aligned(seq_start, 8)) return COMEM_ERR_MISALIGNED;
  // The splits a call with the plan's own workspace would use, and what they
  // need past the scratch's fixed counter region.
  if (p->ticket_bytes > comem::kScratchTicketBytes) return COMEM_ERR_SCRATCH_LIMIT;
  int64_t chunk = 0, splits = 0;
  st = plan_call(*p, batch, max_ctx_len, 0, p->workspace_bytes, &chunk, &splits);
  if (st != COMEM_OK) return st;
  const size_t partials = call_workspace_bytes(*p, batch, splits);
  const size_t need = comem::kScratchTicketBytes + (partials > 0 ? partials - p->ticket_bytes : 0);
  if (need > comem::kScratchBytes) return COMEM_ERR_SCRATCH_LIMIT;
  if (p->device == COMEM_NO_DEVICE) return COMEM_ERR_NO_DEVICE;
  void* scratch = comem::scratch_pointer(p->device);
  if (scratch == nullptr) return COMEM_ERR_HIP;
  return decode_contiguous(plan, q, nullptr, nullptr, k, v, stride_token, stride_head, seq_start, ctx_lens, batch,
                           max_ctx_len, out, lse, scratch, comem::kScratchBytes, hip_stream, false,
                           comem::kScratchTicketBytes);
}

comem_status comem_decode_attn_paged(const comem_decode_attn_plan* plan, const void* q,
                                     const void* k_pages, const void* v_pages, int64_t stride_page,
                                     int64_t stride_token, int64_t stride_head, int32_t page_size,
                                     int64_t num_pages, const int32_t* block_table,
                                     int32_t max_pages_per_seq, const int32_t* ctx_lens,
                                     int32_t batch, int64_t max_ctx_len, float* out, float* lse,
                                     void* workspace, size_t workspace_bytes, void* hip_stream) {
  return decode_paged(plan, q, nullptr, nullptr, k_pages, v_pages, stride_page, stride_token, stride_head,
                      page_size, num_pages, block_table, max_pages_per_seq, ctx_lens, batch, max_ctx_len, out, lse,
                      workspace, workspace_bytes, hip_stream, false);
}

comem_status comem_append_decode_attn(const comem_decode_attn_plan* plan, const void* q, const void* new_k,
                                      const void* new_v, void* k, void* v, int64_t stride_token,
                                      int64_t stride_head, const int64_t* seq_start, const int32_t* ctx_lens,
                                      int32_t batch, int64_t max_ctx_len, float* out, float* lse,
                                      void* workspace, size_t workspace_bytes, void* hip_stream) {
  return decode_contiguous(plan, q, new_k, new_v, k, v, stride_token, stride_head, seq_start, ctx_lens, batch,
                           max_ctx_len, out, lse, workspace, workspace_bytes, hip_stream, true);
}

comem_status comem_append_decode_attn_paged(const comem_decode_attn_plan* plan, const void* q,
                                            const void* new_k, const void* new_v, void* k_pages,
                                            void* v_pages, int64_t stride_page, int64_t stride_token,
                                            int64_t stride_head, int32_t page_size, int64_t num_pages,
                                            const int32_t* block_table, int32_t max_pages_per_seq,
                                            const int32_t* ctx_lens, int32_t batch, int64_t max_ctx_len,
                                            float* out, float* lse, void* workspace, size_t workspace_bytes,
                                            void* hip_stream) {
  return decode_paged(plan, q, new_k, new_v, k_pages, v_pages, stride_page, stride_token, stride_head, page_size,
                      num_pages, block_table, max_pages_per_seq, ctx_lens, batch, max_ctx_len, out, lse, workspace,
                      workspace_bytes, hip_stream, true);
}

comem_status comem_kv_append(const comem_decode_attn_plan* plan, const void* new_k, const void* new_v,
                             void* k, void* v, int64_t stride_token, int64_t stride_head,
                             const int64_t* seq_start, const int32_t* ctx_lens, int32_t batch,
                             int64_t max_ctx_len, void* hip_stream) {
  const comem_decode_attn_plan* p = checked(plan);
  if (p == nullptr) return COMEM_ERR_BAD_HANDLE;
  comem::AppendParams a;
  comem_status st = prepare_append(*p, new_k, new_v, k, v, stride_token, stride_head, ctx_lens, batch,
                                   max_ctx_len, a);
  if (st != COMEM_OK || batch == 0) return st;
  if (seq_start == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!aligned(seq_start, 8)) return COMEM_ERR_MISALIGNED;
  if (p->device == COMEM_NO_DEVICE) return COMEM_ERR_NO_DEVICE;
  a.seq_start = seq_start;
  return launch_append(a, false, batch, hip_stream);
}

comem_status comem_kv_append_paged(const comem_decode_attn_plan* plan, const void* new_k,
                                   const void* new_v, void* k_pages, void* v_pages, int64_t stride_page,
                                   int64_t stride_token, int64_t stride_head, int32_t page_size,
                                   int64_t num_pages, const int32_t* block_table,
                                   int32_t max_pages_per_seq, const int32_t* ctx_lens, int32_t batch,
                                   int64_t max_ctx_len, void* hip_stream) {
  const comem_decode_attn_plan* p = checked(plan);
  if (p == nullptr) return COMEM_ERR_BAD_HANDLE;
  comem::AppendParams a;
  comem_status st = prepare_append(*p, new_k, new_v, k_pages, v_pages, stride_token, stride_head, ctx_lens,
                                   batch, max_ctx_len, a);
  if (st != COMEM_OK || batch == 0) return st;
  st = validate_paged(*p, stride_page, page_size, num_pages, block_table, max_pages_per_seq, max_ctx_len);
  if (st != COMEM_OK) return st;
  if (p->device == COMEM_NO_DEVICE) return COMEM_ERR_NO_DEVICE;
  a.block_table = block_table;
  a.stride_page = stride_page * elem_bytes(p->cfg);
  a.num_pages = num_pages;
  a.max_pages = max_pages_per_seq;
  a.page_shift = log2_of(page_size);
  a.page_mask = page_size - 1;
  return launch_append(a, true, batch, hip_stream);
}

}  // extern "C"
