/*
 * comem_probe.h -- measurement kernels used beside the decode-attention
 * library: a streaming read (the practical HBM read ceiling of the device)
 * and a plain copy of known size (to calibrate byte counters of a profiler).
 * Neither is part of the attention computation.
 *
 * Both enqueue one kernel on `hip_stream` and return a HIP error code
 * (0 = success). Buffers are device memory owned by the caller, 16-byte
 * aligned, with `bytes` a multiple of 16; `sink` must hold 256 * blocks
 * 32-bit words (the read kernel writes there only in a case that does not
 * occur for finite inputs, so that the loads cannot be removed).
 */
#ifndef COMEM_PROBE_H
#define COMEM_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Read `bytes` starting at `src` with `blocks` workgroups of 256 threads,
 * each streaming one contiguous slice with 16-byte loads. */
int comem_probe_read(const void* src, size_t bytes, uint32_t* sink, int blocks, void* hip_stream);

/* Copy `bytes` from `src` to `dst` (non-overlapping) with `blocks` workgroups. */
int comem_probe_copy(const void* src, void* dst, size_t bytes, int blocks, void* hip_stream);

/* Read a token-major K and V cache pair the way the decode kernel's grid form
 * does, with no arithmetic: the ceiling of that access pattern. `k` and `v`
 * hold `tokens` rows of `stride_token` bytes; KV head h's slice of a row is
 * bytes [h * head_bytes, (h + 1) * head_bytes). One workgroup of 4 waves per
 * (split of `chunk` tokens, KV head), the KV head fastest in the linear
 * workgroup id; wave w takes the 32-token tiles w, w + 4, ... of its split
 * with two tiles in flight, each lane loading what the kernel's lane loads:
 * head_bytes 256 (bf16, head_dim 128) or 128 (FP8 codes, head_dim 128).
 * Requires tokens a positive multiple of chunk, chunk a multiple of 128,
 * 1 <= kv_heads, stride_token >= kv_heads * head_bytes, stride_token, k and v
 * 16-byte aligned, and at most 2^24 workgroups; otherwise returns
 * hipErrorInvalidValue and launches nothing. `sink` must hold 256 words. */
int comem_probe_read_kv_heads(const void* k, const void* v, int64_t tokens, int kv_heads, int head_bytes,
                              int64_t stride_token, int chunk, uint32_t* sink, void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* COMEM_PROBE_H */
