/*
 * comem_prefill_attn.h -- prefill attention over a cached prefix on AMD
 * Instinct MI355X (gfx950), for bf16 caches.
 *
 * The operation (paper Algorithm 1, "cached" and "uncached" prefill of the
 * k-step-off pipeline, Sec. 3.2): while the agent's KV cache stays valid, a
 * step prefills only the new tokens of its latest observation over the
 * cached prefix; after the memory model's summary replaces the history, the
 * whole context (summary plus recent buffer) is prefilled from scratch.
 * Both are one operation. Sequence b holds L_b cached tokens of which the
 * last M_b are the new ones (their keys and values already in the cache, as
 * for decode in Sec. 2.2). New token i (0 <= i < M_b) sits at cache position
 * L_b - M_b + i and, for query head h (KV head h / G, G = h_q / h_kv):
 *
 *     s_t = scale * dot(q[i, h, :], K_b[t, h / G, :])     t = 0 .. L_b - M_b + i
 *     out = sum_t softmax(s)_t * V_b[t, h / G, :]
 *     lse = ln sum_t exp(s_t)
 *
 * An uncached prefill is M_b = L_b (plain causal attention); M_b = 1 is a
 * decode step. Scores and sums are fp32; the probabilities enter the matrix
 * cores as a sum of two bf16 values, so an output differs from exact
 * arithmetic by at most about 2^-15 * sum_t softmax(s)_t * |V_b[t, h / G, d]|
 * plus fp32 rounding.
 *
 * Both calls take a plan from comem_decode_attn_init (comem_decode_attn.h)
 * whose dtype is COMEM_BF16; its heads, head_dim (64 or 128), scale,
 * max_batch and max_ctx_len apply, its chunk_tokens and variant do not. They
 * need no workspace, enqueue one kernel on the given stream and return; they
 * never allocate, synchronise, or read device memory from the host.
 *
 * Ownership: the caller owns every device buffer. Errors: as for the decode
 * calls, every argument is checked on the host before any HIP call and a bad
 * argument returns its status with nothing enqueued. Device-side contract:
 * 0 <= q_lens[b] <= ctx_lens[b] <= max_ctx_len, q_lens[b] <= max_q_len,
 * contexts and query rows lie inside the given buffers, and for the paged
 * call 0 <= block_table[b][i] < num_pages for i < ceil(ctx_lens[b] /
 * page_size). The kernel clamps ctx_lens[b] into [0, max_ctx_len] and
 * q_lens[b] into [0, min(ctx_lens[b], max_q_len)], and reads an entry outside
 * [0, num_pages) as page 0, so a violation gives wrong rows for its sequence
 * but no read outside the page pool; these calls have no workspace and record
 * no error word (COMEM_FLAG_DEBUG_CHECKS does not apply). A sequence with
 * q_lens[b] == 0 writes nothing; rows of other sequences are never touched.
 */
#ifndef COMEM_PREFILL_ATTN_H
#define COMEM_PREFILL_ATTN_H

#include "comem_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Contiguous / ragged cache.
 *   q          device bf16 [total_q, h_q, d_h], dense, 16-byte aligned; the
 *              new tokens of sequence b are rows q_start[b] .. q_start[b] +
 *              q_lens[b] - 1.
 *   q_start    device int64 [batch].
 *   q_lens     device int32 [batch]: M_b.
 *   max_q_len  host bound >= every q_lens[b], 0 .. max_ctx_len. A call with
 *              max_q_len = 0 or batch = 0 enqueues nothing and, once batch,
 *              max_ctx_len and max_q_len are in range, returns COMEM_OK
 *              without looking at any pointer (empty buffers may be NULL).
 *   k, v, stride_token, stride_head, seq_start, ctx_lens, batch, max_ctx_len:
 *              as in comem_decode_attn (ctx_lens[b] = L_b counts the new tokens).
 *   out        device float32 [total_q, h_q, d_h], 16-byte aligned.
 *   lse        device float32 [total_q, h_q] (natural log) or NULL. */
comem_status comem_prefill_attn(const comem_decode_attn_plan* plan, const void* q, const int64_t* q_start,
                                const int32_t* q_lens, int32_t max_q_len, const void* k, const void* v,
                                int64_t stride_token, int64_t stride_head, const int64_t* seq_start,
                                const int32_t* ctx_lens, int32_t batch, int64_t max_ctx_len, float* out,
                                float* lse, void* hip_stream);

/* Paged cache; pages, strides and block table as in comem_decode_attn_paged,
 * queries and outputs as in comem_prefill_attn. */
comem_status comem_prefill_attn_paged(const comem_decode_attn_plan* plan, const void* q, const int64_t* q_start,
                                      const int32_t* q_lens, int32_t max_q_len, const void* k_pages,
                                      const void* v_pages, int64_t stride_page, int64_t stride_token,
                                      int64_t stride_head, int32_t page_size, int64_t num_pages,
                                      const int32_t* block_table, int32_t max_pages_per_seq,
                                      const int32_t* ctx_lens, int32_t batch, int64_t max_ctx_len, float* out,
                                      float* lse, void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* COMEM_PREFILL_ATTN_H */
