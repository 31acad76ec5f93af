/*
 * comem_decode_attn.h -- single-token decode attention over a long KV cache
 * on AMD Instinct MI355X (gfx950).
 *
 * The operation (paper Sec. 2.2, "LLM Inference"): after prefill, each
 * sequence b holds a key cache and a value cache of L_b tokens, each token a
 * [h_kv, d_h] block; at every decode step the new token's key and value are
 * appended first (so L_b counts the new token) and the one new query token,
 * [h_q, d_h], attends over the whole cache. The paper states that this step
 * is bound by HBM bandwidth because every generated token re-reads the entire
 * KV cache (Sec. 2.2; latency model of Sec. 3.3). Query head h reads KV head
 * h / G with G = h_q / h_kv (grouped-query attention, consecutive grouping).
 * For query head h of sequence b:
 *
 *     s_t   = scale * dot(q[b, h, :], K_b[t, h / G, :])       t = 0 .. L_b-1
 *     out   = sum_t softmax(s)_t * V_b[t, h / G, :]
 *     lse   = ln sum_t exp(s_t)
 *
 * L_b = 0 gives out = 0 and lse = -inf. The agent's full history and the
 * memory model's compressed context (summary plus recent buffer, Sec. 3.2)
 * are both just a shorter or longer cache, so one API serves both.
 *
 * Execution: the key axis of each (sequence, KV head) is split across
 * workgroups (split-K / flash-decoding); each split produces a partial output
 * and its log-sum-exp, and the last split of each (sequence, KV head) to
 * finish merges them in a fixed order, so results are bitwise reproducible.
 * Both compute calls enqueue work on the given HIP stream and return; they
 * never allocate, synchronise, or read device memory from the host.
 *
 * Ownership: the caller owns every device buffer (q, K, V, block table,
 * lengths, outputs, workspace). The plan is owned by the library from
 * comem_decode_attn_init until comem_decode_attn_destroy.
 *
 * Errors: every argument is checked on the host before any HIP call; a bad
 * argument returns its status and enqueues nothing. Launch failures return
 * COMEM_ERR_HIP. The library never aborts, exits or throws across this ABI.
 * Device-side contract: 0 <= ctx_lens[b] <= max_ctx_len, contexts lie
 * inside the given buffers, and for the paged call 0 <= block_table[b][i] <
 * num_pages for every i < ceil(ctx_lens[b] / page_size). Block-table entries
 * past that are never read. The kernels hold the first and the last part of
 * the contract themselves: a length outside [0, max_ctx_len] is clamped into
 * it, and an entry outside [0, num_pages) is read as page 0 and never written
 * through (the fused append skips the store). A violation therefore gives
 * wrong results for its sequence but no access outside the page pool or the
 * workspace. With COMEM_FLAG_DEBUG_CHECKS in the plan's flags, every violation
 * also sets its COMEM_DEVICE_ERR_* bit in an error word in the workspace,
 * which comem_decode_attn_device_errors reads. Whether a contiguous context
 * lies inside its buffer cannot be checked (the buffer sizes are not passed).
 */
#ifndef COMEM_DECODE_ATTN_H
#define COMEM_DECODE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  COMEM_OK = 0,
  COMEM_ERR_NULL_POINTER = 1,        /* a required pointer is NULL */
  COMEM_ERR_INVALID_SHAPE = 2,       /* sizes, strides or bounds inconsistent */
  COMEM_ERR_UNSUPPORTED = 3,         /* dtype, head_dim, GQA group or variant not built */
  COMEM_ERR_MISALIGNED = 4,          /* pointer or byte stride not 16-byte aligned */
  COMEM_ERR_WORKSPACE_TOO_SMALL = 5, /* workspace_bytes below what the call needs */
  COMEM_ERR_BAD_HANDLE = 6,          /* NULL or foreign plan */
  COMEM_ERR_HIP = 7,                 /* HIP runtime error (device query or launch) */
  COMEM_ERR_NO_DEVICE = 8,           /* plan made with device = COMEM_NO_DEVICE */
  COMEM_ERR_SCRATCH_LIMIT = 9        /* call needs more than the library's fixed scratch holds */
} comem_status;

typedef enum {
  COMEM_F32 = 0,     /* q, K, V in IEEE float32 */
  COMEM_BF16 = 1,    /* q, K, V in bfloat16 */
  COMEM_FP8_E4M3 = 2 /* q in bfloat16; K and V as OCP FP8 E4M3 codes (one byte, bias 7, no
                        infinities), attended as code value * k_scale and code value * v_scale
                        (KV quantization, the prior art the paper cites beside KV eviction) */
} comem_dtype;

typedef enum {
  COMEM_VARIANT_AUTO = 0,     /* bf16, fp8 -> matrix-core kernel; f32 -> vector kernel */
  COMEM_VARIANT_VALU = 1,     /* vector-ALU kernel (f32 and bf16), one workgroup per split */
  COMEM_VARIANT_MFMA = 2,     /* matrix-core kernel (bf16, fp8); persistent workgroups take
                                 splits from a work queue when a workspace is given and
                                 batch <= 4096, else one workgroup per split */
  COMEM_VARIANT_MFMA_GRID = 3 /* matrix-core kernel, always one workgroup per split */
} comem_variant;

/* Plan flags (comem_decode_attn_config.flags). */
#define COMEM_FLAG_DEBUG_CHECKS 1u /* record device-side contract violations (needs a workspace) */

/* Bits of the device error word (COMEM_FLAG_DEBUG_CHECKS). */
#define COMEM_DEVICE_ERR_CTX_LEN 1u     /* some ctx_lens[b] outside [0, max_ctx_len] (clamped) */
#define COMEM_DEVICE_ERR_BLOCK_TABLE 2u /* some block-table entry read outside [0, num_pages) */

/* Pass as `device` to comem_decode_attn_init to make a plan without touching
 * the HIP runtime (a gfx950 with 256 compute units is assumed). Such a plan
 * sizes workspaces and validates arguments; compute calls with it return
 * COMEM_ERR_NO_DEVICE after validation. */
#define COMEM_NO_DEVICE (-1)

typedef struct {
  int32_t num_q_heads;  /* h_q > 0 */
  int32_t num_kv_heads; /* h_kv > 0, h_q % h_kv == 0, G = h_q / h_kv in {1,2,4,8,16} */
  int32_t head_dim;     /* d_h in {64, 128} */
  int32_t dtype;        /* comem_dtype of q, K and V (see COMEM_FP8_E4M3 for the FP8 cache) */
  float scale;          /* softmax scale, finite and > 0 (1/sqrt(d_h) is usual) */
  int32_t max_batch;    /* largest batch any call will pass (> 0) */
  int64_t max_ctx_len;  /* largest context any call will pass (> 0) */
  int32_t chunk_tokens; /* tokens per split: 0 = planned per call; else a multiple of 32 */
  int32_t variant;      /* comem_variant (fp8 caches: not COMEM_VARIANT_VALU) */
  float k_scale;        /* COMEM_FP8_E4M3 only: finite and > 0, the per-tensor K scale */
  float v_scale;        /* COMEM_FP8_E4M3 only: finite and > 0, the per-tensor V scale */
  uint32_t flags;       /* 0 or COMEM_FLAG_DEBUG_CHECKS */
} comem_decode_attn_config;

typedef struct comem_decode_attn_plan comem_decode_attn_plan;

/* Validate `cfg`, query `device` (a HIP device ordinal, or COMEM_NO_DEVICE)
 * for its compute-unit count, and create a plan. *workspace_bytes_out gets
 * the workspace size that every call within the plan's limits fits in.
 * The caller allocates the workspace (device memory, 256-byte aligned) and
 * must zero-fill it once before its first use; the library keeps the
 * counters it holds at zero between calls. A workspace must not be used by
 * two calls that can run at the same time. */
comem_status comem_decode_attn_init(const comem_decode_attn_config* cfg, int device,
                                    comem_decode_attn_plan** plan_out,
                                    size_t* workspace_bytes_out);

/* Free a plan (NULL is a no-op returning COMEM_OK). */
comem_status comem_decode_attn_destroy(comem_decode_attn_plan* plan);

/* Static, human-readable text for a status code. */
const char* comem_status_string(comem_status status);

/* Tokens per split and number of splits a call would use (for tests and
 * reports): same planning as the contiguous compute call. A paged call with
 * pages of 1 or 2 tokens may plan shorter splits, so that the block-table
 * entries of one split fit the matrix-core kernel's on-chip copy (2048
 * entries); a configured chunk_tokens that does not fit is refused with
 * COMEM_ERR_INVALID_SHAPE. A sequence of L tokens has ceil(L / chunk)
 * splits. When the matrix-core kernel's work queue has several rounds of
 * work items and the chunk was planned (chunk_tokens = 0), a sequence's last
 * splits are half a chunk each and the others up to 1.25 chunk; the split
 * boundaries depend only on L and the plan, so results stay reproducible. */
comem_status comem_decode_attn_plan_splits(const comem_decode_attn_plan* plan, int32_t batch,
                                           int64_t max_ctx_len, size_t workspace_bytes,
                                           int32_t* chunk_tokens_out, int32_t* num_splits_out);

/* Device-side contract violations (plan made with COMEM_FLAG_DEBUG_CHECKS):
 * waits for hip_stream, stores in *errors_out the COMEM_DEVICE_ERR_* bits
 * that calls using this workspace have set since the last read, and clears
 * them. It synchronises the stream and copies four bytes to the host, so it
 * is for tests and debugging, not for the decode loop, and must not be
 * captured in a graph. workspace and workspace_bytes are those of the calls.
 * The standalone append calls take no workspace and record nothing; their
 * kernel skips a sequence that violates the contract. */
comem_status comem_decode_attn_device_errors(const comem_decode_attn_plan* plan, void* workspace,
                                             size_t workspace_bytes, uint32_t* errors_out, void* hip_stream);

/* Placement of V relative to K: a recommendation, not a requirement (every
 * placement gives the same bits). Each wave requests the K and the V rows of
 * the same tokens and KV head together, and those rows sit at the same
 * offset within their caches. Measured on MI355X, the step is faster when the
 * V base lies COMEM_V_BASE_OFFSET_BYTES past the K base modulo
 * COMEM_V_BASE_OFFSET_MODULUS than when the two bases are congruent modulo
 * 512 (any two separate allocations of 4 KB granularity are): the batch-1
 * 32768-token bf16 step takes 27.7-28.0 instead of 29.0-29.2 us (depending
 * on the device), its FP8 form 18.9 instead of 20.7 us, and multi-GB batches
 * are 0.7-1.4% faster. Differences
 * of 256, 768, 1280, 1792 and 2304 bytes all give the faster time; 0, 1024,
 * 2048 and 3072 the slower one. For paged caches the same applies to the V
 * pool's base against the K pool's. One way to get it: allocate K and V as
 * one buffer with V starting at the first address past K's end that is 256
 * bytes past K's base modulo 512. What counts is the address difference
 * between the V and the K row of the same token and head: for K and V
 * interleaved in one buffer (for example [T, 2, h_kv, d_h]) it is the offset
 * of the V part within a token, which should then be 256 modulo 512 too
 * (the batch-1 32768-token step over [T, 2, 8, 128]: 31.9 us single calls
 * with V at +2048 bytes, 29.1 us with each token row padded by 256 bytes and
 * V at +2304). A head-major cache ([h_kv, T, d_h] per tensor, passed through
 * stride_token = d_h and stride_head = T * d_h) needs no such care: the same
 * step ran in 27.1 us for either placement, as fast as the token-major cache
 * placed as recommended. */
#define COMEM_V_BASE_OFFSET_BYTES 256
#define COMEM_V_BASE_OFFSET_MODULUS 512

/* Contiguous / ragged cache (paper Sec. 2.2: K_cache, V_cache of l tokens,
 * each token an [h_kv, d_h] block). Strides count elements of the cache's
 * dtype (bytes for FP8 caches).
 *   q          [batch, h_q, d_h] dense, dtype of the plan (bf16 for FP8
 *              caches), 16-byte aligned.
 *   k, v       element (b, t, hk, d) at k[(seq_start[b] + t) * stride_token
 *              + hk * stride_head + d]; d contiguous. 16-byte aligned; the
 *              byte sizes of both strides must be multiples of 16.
 *   seq_start  device int64 [batch]: first row of each sequence.
 *   ctx_lens   device int32 [batch]: L_b, including the appended token.
 *   batch      0 <= batch <= plan max_batch (0 enqueues nothing).
 *   max_ctx_len host bound >= every ctx_lens[b], <= plan max_ctx_len.
 *   out        device float32 [batch, h_q, d_h], 16-byte aligned.
 *   lse        device float32 [batch, h_q] (natural log) or NULL.
 *   workspace  device buffer of workspace_bytes (see init).
 *   hip_stream hipStream_t to enqueue on (NULL = default stream). */
comem_status comem_decode_attn(const comem_decode_attn_plan* plan, const void* q, const void* k,
                               const void* v, int64_t stride_token, int64_t stride_head,
                               const int64_t* seq_start, const int32_t* ctx_lens, int32_t batch,
                               int64_t max_ctx_len, float* out, float* lse, void* workspace,
                               size_t workspace_bytes, void* hip_stream);

/* Allocation-free form of comem_decode_attn, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc. Instead of a caller workspace it uses a
 * scratch array that the library holds in device memory, one copy of
 * COMEM_NOALLOC_SCRATCH_BYTES per GPU, from the first comem_decode_attn_init
 * on that device until the process ends. It calls no allocating routine.
 * Arguments, results and planning are those of comem_decode_attn with a
 * workspace of the plan's workspace_bytes (same kernels, same splits, same
 * bits). The scratch starts with a fixed 64 KiB of counters, then the split
 * partial results:
 *   COMEM_ERR_SCRATCH_LIMIT  the call's partial results would not fit in the
 *                            rest of the scratch (for example batch 16 of
 *                            64K-token contexts with 32 query heads of 128 fits;
 *                            a call past that does not), or the plan's
 *                            max_batch * h_kv exceeds 16381 counters;
 *   COMEM_ERR_UNSUPPORTED    plan made with COMEM_FLAG_DEBUG_CHECKS (its error
 *                            word needs a caller workspace);
 *   COMEM_ERR_HIP            the scratch of the plan's device could not be set up.
 * Every call on one GPU shares that GPU's scratch, which keeps the last call's
 * contents: the counters return to zero at the end of each call, and partial
 * results are written before they are read. Calls that can overlap on one
 * GPU (different streams, or different host threads) race on it and give
 * wrong results: serialise them. */
#define COMEM_NOALLOC_SCRATCH_BYTES (32u << 20)
comem_status comem_decode_attn_noalloc(const comem_decode_attn_plan* plan, const void* q, const void* k,
                                       const void* v, int64_t stride_token, int64_t stride_head,
                                       const int64_t* seq_start, const int32_t* ctx_lens, int32_t batch,
                                       int64_t max_ctx_len, float* out, float* lse, void* hip_stream);

/* Paged cache driven by a block table (the paging scheme that the paper's
 * serving engine uses, cited in Sec. 1 and configured in Sec. 4.2).
 *   k_pages, v_pages element (b, t, hk, d) at
 *              k_pages[block_table[b * max_pages_per_seq + t / page_size] * stride_page
 *                      + (t % page_size) * stride_token + hk * stride_head + d].
 *              16-byte aligned; the byte sizes of all three strides must be
 *              multiples of 16.
 *   page_size  a power of two, 1 .. 4096.
 *   num_pages  number of pages in the pool (> 0 when batch > 0).
 *   block_table device int32 [batch, max_pages_per_seq], with
 *              max_pages_per_seq >= ceil(max_ctx_len / page_size).
 *   Other arguments as in comem_decode_attn. */
comem_status comem_decode_attn_paged(const comem_decode_attn_plan* plan, const void* q,
                                     const void* k_pages, const void* v_pages, int64_t stride_page,
                                     int64_t stride_token, int64_t stride_head, int32_t page_size,
                                     int64_t num_pages, const int32_t* block_table,
                                     int32_t max_pages_per_seq, const int32_t* ctx_lens,
                                     int32_t batch, int64_t max_ctx_len, float* out, float* lse,
                                     void* workspace, size_t workspace_bytes, void* hip_stream);

/* KV append (paper Sec. 2.2): before the new query token attends, its key
 * and value are concatenated to the caches. With ctx_lens[b] = L_b counting
 * the new token, these calls store new_k[b] and new_v[b] as token L_b - 1 of
 * sequence b, in the layout the matching attention call reads; every other
 * cache element is left as it was. Run on the same stream before the
 * attention call, it gives the append-then-attend order of a decode step.
 * The rows are copied, so the stored bits equal the given ones.
 *   new_k, new_v device [batch, h_kv, d_h] dense, the cache's dtype (FP8 caches: codes), 16-byte aligned.
 *   k, v          the cache (written), addressed as in comem_decode_attn.
 *   max_ctx_len   host bound, <= plan max_ctx_len.
 * A sequence whose ctx_lens[b] is outside [1, max_ctx_len] (or, paged,
 * whose block-table entry for token L_b - 1 lies outside [0, num_pages)) is
 * skipped on the device; no error is reported for it. Other errors as for
 * the attention calls; the plan's variant and workspace play no part. */
comem_status comem_kv_append(const comem_decode_attn_plan* plan, const void* new_k, const void* new_v,
                             void* k, void* v, int64_t stride_token, int64_t stride_head,
                             const int64_t* seq_start, const int32_t* ctx_lens, int32_t batch,
                             int64_t max_ctx_len, void* hip_stream);

/* Paged form: token L_b - 1 goes to slot (L_b - 1) % page_size of page
 * block_table[b * max_pages_per_seq + (L_b - 1) / page_size]; pages, strides
 * and block table as in comem_decode_attn_paged. */
comem_status comem_kv_append_paged(const comem_decode_attn_plan* plan, const void* new_k,
                                   const void* new_v, void* k_pages, void* v_pages, int64_t stride_page,
                                   int64_t stride_token, int64_t stride_head, int32_t page_size,
                                   int64_t num_pages, const int32_t* block_table,
                                   int32_t max_pages_per_seq, const int32_t* ctx_lens, int32_t batch,
                                   int64_t max_ctx_len, void* hip_stream);

/* One decode step in one launch (paper Sec. 2.2: append, then attend): the
 * same result as comem_kv_append followed by comem_decode_attn on one
 * stream. The split that holds token L_b - 1 of each KV head stores that
 * head's new K and V rows before it reads them; no other cache element is
 * written. new_k, new_v: device [batch, h_kv, d_h] dense, dtype of the plan,
 * 16-byte aligned. A sequence with ctx_lens[b] == 0 stores nothing. Unlike
 * comem_kv_append, the device-side contract of the attention call applies
 * (0 <= ctx_lens[b] <= max_ctx_len); only a block-table entry outside
 * [0, num_pages) for token L_b - 1 skips the store. Other arguments as in
 * comem_decode_attn. */
comem_status comem_append_decode_attn(const comem_decode_attn_plan* plan, const void* q, const void* new_k,
                                      const void* new_v, void* k, void* v, int64_t stride_token,
                                      int64_t stride_head, const int64_t* seq_start, const int32_t* ctx_lens,
                                      int32_t batch, int64_t max_ctx_len, float* out, float* lse,
                                      void* workspace, size_t workspace_bytes, void* hip_stream);

/* Paged form of comem_append_decode_attn; other arguments as in
 * comem_decode_attn_paged. */
comem_status comem_append_decode_attn_paged(const comem_decode_attn_plan* plan, const void* q,
                                            const void* new_k, const void* new_v, void* k_pages,
                                            void* v_pages, int64_t stride_page, int64_t stride_token,
                                            int64_t stride_head, int32_t page_size, int64_t num_pages,
                                            const int32_t* block_table, int32_t max_pages_per_seq,
                                            const int32_t* ctx_lens, int32_t batch, int64_t max_ctx_len,
                                            float* out, float* lse, void* workspace, size_t workspace_bytes,
                                            void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* COMEM_DECODE_ATTN_H */
