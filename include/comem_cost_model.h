/*
 * comem_cost_model.h -- the decode-latency trade-off of the paper's Sec. 3.3
 * ("Determination of Summary Length"), evaluated on the host.
 *
 * Decode is memory-bound, so generating one token over a context of L tokens
 * takes L * S / W seconds (S: KV-cache bytes per token, W: the bandwidth the
 * decode attention sustains). Attending over a summary of L_sum tokens
 * instead of the full L_full saves (L_full - L_sum) * S / W per generated
 * token, and costs one prefill of the summary, L_sum / P seconds (P: prefill
 * throughput in tokens/s). Over Y generated tokens the summary pays off when
 * Y * (L_full - L_sum) * S / W > L_sum / P, i.e. when
 *
 *     L_sum / L_full < Y S P / (Y S P + W)        ( = 1 / (1 + W / (Y S P)) ).
 *
 * W is meant to be the bandwidth measured for comem_decode_attn on the
 * target GPU (the value bench.py reports), S the model's per-token KV bytes
 * over all layers (comem_cost_kv_bytes_per_token).
 *
 * Units: bytes, seconds, tokens. Every function checks its arguments and
 * writes its result only on COMEM_OK: a NULL pointer gives
 * COMEM_ERR_NULL_POINTER; a non-finite value, a non-positive S, W or P, a
 * negative Y or context length, or L_sum > L_full gives
 * COMEM_ERR_INVALID_SHAPE. No function touches the GPU.
 */
#ifndef COMEM_COST_MODEL_H
#define COMEM_COST_MODEL_H

#include <stdint.h>

#include "comem_decode_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  double kv_bytes_per_token;   /* S > 0 */
  double hbm_bytes_per_s;      /* W > 0 */
  double prefill_tokens_per_s; /* P > 0 */
  double generated_tokens;     /* Y >= 0 */
} comem_cost_inputs;

/* S = 2 (K and V) * num_layers * num_kv_heads * head_dim * elem_bytes
 * (Sec. 2.2: a cache holds one [h_kv, d_h] key and value block per token per
 * layer). All four arguments must be > 0. */
comem_status comem_cost_kv_bytes_per_token(int32_t num_layers, int32_t num_kv_heads, int32_t head_dim,
                                           int32_t elem_bytes, double* bytes_out);

/* Time of one memory-bound decode step over ctx_tokens tokens: ctx_tokens * S / W. */
comem_status comem_cost_decode_time(const comem_cost_inputs* in, double ctx_tokens, double* seconds_out);

/* Per-token decode saving of a summary: (l_full - l_sum) * S / W. */
comem_status comem_cost_decode_saving(const comem_cost_inputs* in, double l_full, double l_sum,
                                      double* seconds_out);

/* One-time prefill of the summary: l_sum / P. */
comem_status comem_cost_prefill_time(const comem_cost_inputs* in, double l_sum, double* seconds_out);

/* Y * decode saving - prefill time (> 0 means the summary is a net speedup). */
comem_status comem_cost_net_saving(const comem_cost_inputs* in, double l_full, double l_sum,
                                   double* seconds_out);

/* Largest L_sum / L_full with a net speedup: Y S P / (Y S P + W). */
comem_status comem_cost_max_compression_ratio(const comem_cost_inputs* in, double* ratio_out);

#ifdef __cplusplus
}
#endif

#endif /* COMEM_COST_MODEL_H */
