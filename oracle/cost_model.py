"""Memory-bound decode latency model and the summary-length bound (paper Sec. 3.3).

TEST INFRASTRUCTURE ONLY (see the package docstring): the product-side helper
that evaluates the same model with a measured bandwidth is written separately.

With S the KV-cache bytes per token (GB), W the HBM bandwidth (GB/s), P the
prefill throughput (tokens/s) and Y the number of generated tokens:

  * decoding over a context of L_sum instead of L_full tokens saves, per
    generated token, (L_full - L_sum) * S / W seconds (decode is taken to be
    memory-bound: its time is the KV bytes read over the bandwidth);
  * a summary pays once for prefilling L_sum tokens, L_sum / P seconds;
  * the saving wins when Y * (L_full - L_sum) * S / W > L_sum / P, which
    rearranges to L_sum / L_full < 1 / (1 + W / (Y * S * P)).
"""

from __future__ import annotations


def decode_time(context_len, kv_bytes_per_token, bandwidth):
    """Per-token decode time of a memory-bound step: context_len * S / W."""
    return context_len * kv_bytes_per_token / bandwidth


def decode_saving(l_full, l_sum, kv_bytes_per_token, bandwidth):
    """Per-token decode saving of attending over l_sum instead of l_full tokens."""
    return (l_full - l_sum) * kv_bytes_per_token / bandwidth


def prefill_cost(l_sum, prefill_throughput):
    """One-time cost of prefilling the summary context."""
    return l_sum / prefill_throughput


def net_saving(y_tokens, l_full, l_sum, kv_bytes_per_token, bandwidth, prefill_throughput):
    """Decode savings over y_tokens minus the summary prefill cost (positive = net speedup)."""
    return (y_tokens * decode_saving(l_full, l_sum, kv_bytes_per_token, bandwidth)
            - prefill_cost(l_sum, prefill_throughput))


def max_compression_ratio(bandwidth, y_tokens, kv_bytes_per_token, prefill_throughput):
    """Upper bound on L_sum / L_full for a net speedup: 1 / (1 + W / (Y * S * P))."""
    return 1 / (1 + bandwidth / (y_tokens * kv_bytes_per_token * prefill_throughput))
