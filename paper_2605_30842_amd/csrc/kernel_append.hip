// KV append (paper Sec. 2.2): before the new query token attends, its key and
// value rows are concatenated to the caches. With L_b counting the new token,
// its row is token L_b - 1 of sequence b: row seq_start[b] + L_b - 1 of a
// packed cache, or slot (L_b - 1) % page_size of page
// block_table[b][(L_b - 1) / page_size] of a paged one.
//
// One workgroup per sequence; each thread moves 16-byte pieces of the K and V
// rows (the data are only copied, so the result is bit-exact for any dtype).
// A length outside [1, max_ctx_len] or a block-table entry outside the pool
// makes the sequence a no-op instead of a stray write.
#include "kv_append.h"

namespace comem {
namespace {

template <bool PAGED>
__global__ __launch_bounds__(256) void kv_append_kernel(AppendParams p) {
  const int b = blockIdx.x;
  const int64_t L = p.ctx_lens[b];
  if (L <= 0 || L > p.max_ctx_len) return;
  const int64_t t = L - 1;
  int64_t row;
  if constexpr (PAGED) {
    const int64_t entry = t >> p.page_shift;
    if (entry >= p.max_pages) return;
    const int64_t page = p.block_table[static_cast<int64_t>(b) * p.max_pages + entry];
    if (page < 0 || page >= p.num_pages) return;
    row = page * p.stride_page + (t & p.page_mask) * p.stride_token;
  } else {
    const int64_t start = p.seq_start[b];
    if (start < 0) return;
    row = (start + t) * p.stride_token;
  }
  const int per_tensor = p.num_kv_heads * p.chunks_per_head;
  const int64_t src = static_cast<int64_t>(b) * per_tensor * 16;
  for (int i = threadIdx.x; i < 2 * per_tensor; i += blockDim.x) {
    const bool is_v = i >= per_tensor;
    const int c = is_v ? i - per_tensor : i;
    const int hk = c / p.chunks_per_head;
    const int piece = c - hk * p.chunks_per_head;
    const uint4 val = *reinterpret_cast<const uint4*>((is_v ? p.new_v : p.new_k) + src + c * 16);
    *reinterpret_cast<uint4*>((is_v ? p.v : p.k) + row + hk * p.stride_head + piece * 16) = val;
  }
}

}  // namespace

AppendKernelFn select_append_kernel(bool paged) {
  return paged ? kv_append_kernel<true> : kv_append_kernel<false>;
}

}  // namespace comem
