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

#ifdef __cplusplus
}
#endif

#endif /* COMEM_PROBE_H */
