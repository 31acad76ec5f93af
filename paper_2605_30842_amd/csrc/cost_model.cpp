// Host-side evaluation of the decode-latency trade-off (paper Sec. 3.3).
#include "comem_cost_model.h"

#include <cmath>

namespace {

bool valid(const comem_cost_inputs& c) {
  return std::isfinite(c.kv_bytes_per_token) && c.kv_bytes_per_token > 0 && std::isfinite(c.hbm_bytes_per_s) &&
         c.hbm_bytes_per_s > 0 && std::isfinite(c.prefill_tokens_per_s) && c.prefill_tokens_per_s > 0 &&
         std::isfinite(c.generated_tokens) && c.generated_tokens >= 0;
}

bool length_ok(double l) { return std::isfinite(l) && l >= 0; }

// Seconds to stream `tokens` tokens' KV bytes at the decode bandwidth.
double stream_seconds(const comem_cost_inputs& c, double tokens) {
  return tokens * c.kv_bytes_per_token / c.hbm_bytes_per_s;
}

}  // namespace

extern "C" {

comem_status comem_cost_kv_bytes_per_token(int32_t num_layers, int32_t num_kv_heads, int32_t head_dim,
                                           int32_t elem_bytes, double* bytes_out) {
  if (bytes_out == nullptr) return COMEM_ERR_NULL_POINTER;
  if (num_layers <= 0 || num_kv_heads <= 0 || head_dim <= 0 || elem_bytes <= 0) return COMEM_ERR_INVALID_SHAPE;
  *bytes_out = 2.0 * num_layers * num_kv_heads * head_dim * elem_bytes;
  return COMEM_OK;
}

comem_status comem_cost_decode_time(const comem_cost_inputs* in, double ctx_tokens, double* seconds_out) {
  if (in == nullptr || seconds_out == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!valid(*in) || !length_ok(ctx_tokens)) return COMEM_ERR_INVALID_SHAPE;
  *seconds_out = stream_seconds(*in, ctx_tokens);
  return COMEM_OK;
}

comem_status comem_cost_decode_saving(const comem_cost_inputs* in, double l_full, double l_sum,
                                      double* seconds_out) {
  if (in == nullptr || seconds_out == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!valid(*in) || !length_ok(l_full) || !length_ok(l_sum) || l_sum > l_full) return COMEM_ERR_INVALID_SHAPE;
  *seconds_out = stream_seconds(*in, l_full - l_sum);
  return COMEM_OK;
}

comem_status comem_cost_prefill_time(const comem_cost_inputs* in, double l_sum, double* seconds_out) {
  if (in == nullptr || seconds_out == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!valid(*in) || !length_ok(l_sum)) return COMEM_ERR_INVALID_SHAPE;
  *seconds_out = l_sum / in->prefill_tokens_per_s;
  return COMEM_OK;
}

comem_status comem_cost_net_saving(const comem_cost_inputs* in, double l_full, double l_sum,
                                   double* seconds_out) {
  if (in == nullptr || seconds_out == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!valid(*in) || !length_ok(l_full) || !length_ok(l_sum) || l_sum > l_full) return COMEM_ERR_INVALID_SHAPE;
  *seconds_out = in->generated_tokens * stream_seconds(*in, l_full - l_sum) - l_sum / in->prefill_tokens_per_s;
  return COMEM_OK;
}

comem_status comem_cost_max_compression_ratio(const comem_cost_inputs* in, double* ratio_out) {
  if (in == nullptr || ratio_out == nullptr) return COMEM_ERR_NULL_POINTER;
  if (!valid(*in)) return COMEM_ERR_INVALID_SHAPE;
  // Y * (1 - r) * S / W = r / P  <=>  r = Y S P / (Y S P + W)
  const double ysp = in->generated_tokens * in->kv_bytes_per_token * in->prefill_tokens_per_s;
  *ratio_out = ysp / (ysp + in->hbm_bytes_per_s);
  return COMEM_OK;
}

}  // extern "C"
