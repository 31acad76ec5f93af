"""CPU fp64 oracle for single-token decode attention over a KV cache.

TEST INFRASTRUCTURE ONLY. Nothing on the product path imports this module:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may use it. It shares no code, table or helper with the HIP path.

What it computes (paper, Sec. 2.2 "LLM Inference"): at decode step t the new
token's key and value are appended to the per-KV-head caches, so the cache
holds ``l`` rows of shape ``[h_kv, d_h]`` including the new token, and the one
new query token (``[h_q, d_h]``) attends over all of them. The paper gives the
shapes and the append-then-attend order but not the attention formula; this
oracle writes out the textbook scaled dot-product softmax attention, with
grouped-query attention (GQA, the paper's footnote on KV heads vs attention
heads) mapping query head ``h`` to KV head ``h // (h_q / h_kv)``:

    s_t   = scale * sum_d q[h, d] * K[t, h_kv(h), d]
    m     = max_t s_t
    Z     = sum_t exp(s_t - m)
    out_h = sum_t exp(s_t - m) / Z * V[t, h_kv(h), :]
    lse_h = m + ln Z

A context of length zero gives ``out = 0`` and ``lse = -inf`` (the paper is
silent; an idle batch slot is the reading taken).

Split-K ("flash-decoding") reaches the same result by attending over disjoint
token ranges and merging the partial results with their log-sum-exps; the
merge is also written out here (``lse_combine``) so it can be checked against
unsplit attention. Every value is float64, computed on the exact values the
GPU sees (bf16 bit patterns are widened exactly).

FP8 KV caches (KV quantization, the prior art the paper cites next to KV
eviction) store OCP FP8 E4M3 codes with a per-tensor scale; the attended
keys and values are the decoded codes times that scale (``dequantize``),
and the attention itself is unchanged.
"""

from __future__ import annotations

import math
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np


def fp8_e4m3_value(codes: np.ndarray) -> np.ndarray:
    """Float64 values of OCP FP8 E4M3 codes (uint8), from the format's definition.

    Sign bit 7, exponent bits 6..3 (bias 7), mantissa bits 2..0. Exponent 0
    is subnormal: m/8 * 2^-6. Otherwise (1 + m/8) * 2^(e - 7). Exponent 15
    with mantissa 7 is NaN; the format has no infinities (max 448).
    """
    return _e4m3_values_of_all_codes()[np.asarray(codes, dtype=np.uint8)]


def _e4m3_values_of_all_codes() -> np.ndarray:
    """The definition above evaluated once for each of the 256 codes (indexed by code)."""
    global _E4M3_ALL
    if _E4M3_ALL is None:
        c = np.arange(256, dtype=np.int64)
        sign = np.where(c >> 7, -1.0, 1.0)
        e = (c >> 3) & 15
        m = (c & 7).astype(np.float64)
        mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * np.exp2(e - 7.0))
        _E4M3_ALL = np.where((e == 15) & (m == 7), np.nan, sign * mag)
        _E4M3_ALL.setflags(write=False)
    return _E4M3_ALL


_E4M3_ALL = None


def widen(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of the stored data ("bf16": uint16 bit patterns; "fp8": E4M3 codes, unscaled)."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        bits = np.asarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    if dtype == "fp8":
        return fp8_e4m3_value(x)
    raise ValueError(f"unknown dtype {dtype!r}")


def dequantize(x: np.ndarray, dtype: str, scale: float = 1.0) -> np.ndarray:
    """Float64 K or V values as attended: the stored values, times the tensor's scale for fp8."""
    v = widen(x, dtype)
    return v * float(scale) if dtype == "fp8" else v


def attend(q_rows: np.ndarray, keys: np.ndarray, values: np.ndarray,
           scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Softmax attention of G query rows over L key/value rows of one KV head.

    q_rows [G, D], keys [L, D], values [L, D] (float64) -> out [G, D], lse [G].
    This is the definition written out: scores, their maximum, the exponentials
    relative to it, their sum, the weighted sum of values, and m + ln Z.
    """
    G, D = q_rows.shape
    L = keys.shape[0]
    if L == 0:
        return np.zeros((G, D)), np.full(G, -np.inf)
    s = scale * (keys @ q_rows.T)  # [L, G]
    m = s.max(axis=0)  # [G]
    w = np.exp(s - m)  # [L, G]
    z = w.sum(axis=0)  # [G]
    out = (w.T @ values) / z[:, None]  # [G, D]
    lse = m + np.log(z)
    return out, lse


def lse_combine(parts: Sequence[Tuple[np.ndarray, np.ndarray]]) -> Tuple[np.ndarray, np.ndarray]:
    """Merge attention results over disjoint token ranges.

    Each part is (out_j [G, D], lse_j [G]) for one range. With M = max_j lse_j,
    w_j = exp(lse_j - M): lse = M + ln sum_j w_j and out = sum_j w_j out_j / sum_j w_j.
    Ranges with lse_j = -inf (empty) get weight 0; if every range is empty the
    result is out = 0, lse = -inf.
    """
    outs = np.stack([np.asarray(o, dtype=np.float64) for o, _ in parts])  # [S, G, D]
    lses = np.stack([np.asarray(l, dtype=np.float64) for _, l in parts])  # [S, G]
    M = lses.max(axis=0)  # [G]
    live = np.isfinite(M)
    Msafe = np.where(live, M, 0.0)
    w = np.where(np.isfinite(lses), np.exp(lses - Msafe), 0.0)  # [S, G]
    wsum = w.sum(axis=0)
    out = np.zeros(outs.shape[1:])
    out[live] = (np.einsum("sg,sgd->gd", w, outs)[live]) / wsum[live, None]
    lse = np.where(live, Msafe + np.log(np.where(live, wsum, 1.0)), -np.inf)
    return out, lse


def attend_split(q_rows: np.ndarray, keys: np.ndarray, values: np.ndarray, scale: float,
                 bounds: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
    """Attention computed as partial results over [bounds[i], bounds[i+1]) merged by lse_combine."""
    parts = [attend(q_rows, keys[a:b], values[a:b], scale) for a, b in zip(bounds[:-1], bounds[1:])]
    return lse_combine(parts)


# ---------------------------------------------------------------- KV layouts


def contiguous_context(kv: np.ndarray, seq_start: np.ndarray, ctx_lens: np.ndarray,
                       b: int) -> np.ndarray:
    """Rows of sequence b in a packed [T, Hkv, D] cache: kv[seq_start[b] : seq_start[b] + L_b]."""
    a = int(seq_start[b])
    return kv[a: a + int(ctx_lens[b])]


def paged_context(kv_pages: np.ndarray, block_table: np.ndarray, ctx_lens: np.ndarray,
                  b: int) -> np.ndarray:
    """Logical [L_b, Hkv, D] context of sequence b in a paged cache.

    Token t of sequence b sits in page block_table[b, t // page_size] at slot
    t % page_size; only the first ceil(L_b / page_size) entries are read.
    """
    page_size = kv_pages.shape[1]
    L = int(ctx_lens[b])
    rows = []
    for t in range(0, L, page_size):
        page = int(block_table[b, t // page_size])
        if not 0 <= page < kv_pages.shape[0]:
            raise IndexError(f"block_table[{b}, {t // page_size}] = {page} outside the pool")
        rows.append(kv_pages[page, : min(page_size, L - t)])
    if not rows:
        return kv_pages[:0, 0]
    return np.concatenate(rows, axis=0)


# ---------------------------------------------------------------- KV append


def append_contiguous(kv: np.ndarray, seq_start: np.ndarray, ctx_lens: np.ndarray,
                      new_rows: np.ndarray) -> np.ndarray:
    """Copy of a packed [T, Hkv, D] cache with each sequence's new token stored.

    The decode step of Sec. 2.2 concatenates the new token's key (value) to
    the cache before attending: with ctx_lens counting that token, its row is
    seq_start[b] + ctx_lens[b] - 1. new_rows is [B, Hkv, D]; sequences with
    ctx_lens[b] == 0 have no token to store.
    """
    out = np.array(kv, copy=True)
    for b in range(len(ctx_lens)):
        if int(ctx_lens[b]) > 0:
            out[int(seq_start[b]) + int(ctx_lens[b]) - 1] = new_rows[b]
    return out


def append_paged(kv_pages: np.ndarray, block_table: np.ndarray, ctx_lens: np.ndarray,
                 new_rows: np.ndarray) -> np.ndarray:
    """Copy of a paged [P, page, Hkv, D] cache with each sequence's new token stored.

    Token t = ctx_lens[b] - 1 of sequence b goes to page block_table[b, t // page] at slot t % page.
    """
    page_size = kv_pages.shape[1]
    out = np.array(kv_pages, copy=True)
    for b in range(len(ctx_lens)):
        t = int(ctx_lens[b]) - 1
        if t >= 0:
            page = int(block_table[b, t // page_size])
            if not 0 <= page < kv_pages.shape[0]:
                raise IndexError(f"block_table[{b}, {t // page_size}] = {page} outside the pool")
            out[page, t % page_size] = new_rows[b]
    return out


# ---------------------------------------------------------------- whole batch


def _attend_sequence(q_b: np.ndarray, keys: np.ndarray, values: np.ndarray, dtype: str,
                     scale: float, heads: Optional[Iterable[int]] = None, kv_scales=(1.0, 1.0)):
    """All (or selected) query heads of one sequence; keys/values are [L, Hkv, D] stored values.

    dtype "fp8": q is bf16, K and V are E4M3 codes scaled by kv_scales = (k_scale, v_scale).
    """
    Hq, D = q_b.shape
    Hkv = keys.shape[1]
    G = Hq // Hkv
    qf = widen(q_b, "bf16" if dtype == "fp8" else dtype)
    want = set(range(Hq)) if heads is None else set(heads)
    out = np.zeros((Hq, D))
    lse = np.full(Hq, -np.inf)
    for hk in range(Hkv):
        hs = [h for h in range(hk * G, (hk + 1) * G) if h in want]
        if not hs:
            continue
        kf = dequantize(keys[:, hk], dtype, kv_scales[0])
        vf = dequantize(values[:, hk], dtype, kv_scales[1])
        o, l = attend(qf[hs], kf, vf, scale)
        out[hs] = o
        lse[hs] = l
    return out, lse


def decode_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, seq_start: np.ndarray,
                     ctx_lens: np.ndarray, scale: float, dtype: str, kv_scales=(1.0, 1.0)):
    """Contiguous/ragged layout: q [B, Hq, D]; k, v [T, Hkv, D]. Returns out [B,Hq,D], lse [B,Hq]."""
    B, Hq, D = q.shape
    if Hq % k.shape[1] != 0:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    out = np.zeros((B, Hq, D))
    lse = np.full((B, Hq), -np.inf)
    for b in range(B):
        out[b], lse[b] = _attend_sequence(q[b], contiguous_context(k, seq_start, ctx_lens, b),
                                          contiguous_context(v, seq_start, ctx_lens, b), dtype, scale,
                                          kv_scales=kv_scales)
    return out, lse


def decode_attention_paged(q: np.ndarray, k_pages: np.ndarray, v_pages: np.ndarray,
                           block_table: np.ndarray, ctx_lens: np.ndarray, scale: float, dtype: str,
                           kv_scales=(1.0, 1.0)):
    """Paged layout: k_pages, v_pages [P, page_size, Hkv, D]; block_table [B, max_pages]."""
    B, Hq, D = q.shape
    if Hq % k_pages.shape[2] != 0:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    out = np.zeros((B, Hq, D))
    lse = np.full((B, Hq), -np.inf)
    for b in range(B):
        out[b], lse[b] = _attend_sequence(q[b], paged_context(k_pages, block_table, ctx_lens, b),
                                          paged_context(v_pages, block_table, ctx_lens, b), dtype, scale,
                                          kv_scales=kv_scales)
    return out, lse


def decode_attention_rows(workload, rows: Sequence[Tuple[int, int]]) -> List[Tuple[np.ndarray, float]]:
    """Selected (b, h) outputs of a drawn workload, one by one (for full-size sampled checks)."""
    spec = workload.spec
    results = []
    by_seq = {}
    for b, h in rows:
        by_seq.setdefault(b, []).append(h)
    cache = {}
    for b, hs in by_seq.items():
        if spec.layout == "paged":
            keys = paged_context(workload.k_pages, workload.block_table, workload.ctx_lens, b)
            values = paged_context(workload.v_pages, workload.block_table, workload.ctx_lens, b)
        else:
            keys = contiguous_context(workload.k, workload.seq_start, workload.ctx_lens, b)
            values = contiguous_context(workload.v, workload.seq_start, workload.ctx_lens, b)
        o, l = _attend_sequence(workload.q[b], keys, values, spec.dtype, float(spec.scale), heads=hs,
                                kv_scales=kv_scales_of(spec))
        for h in hs:
            cache[(b, h)] = (o[h], float(l[h]))
    for b, h in rows:
        results.append(cache[(b, h)])
    return results


def kv_scales_of(spec):
    """(k_scale, v_scale) of a workload spec: its FP8 scales, else (1, 1)."""
    return (float(spec.k_scale), float(spec.v_scale)) if spec.dtype == "fp8" else (1.0, 1.0)


def reference(workload):
    """Full oracle result (out [B,Hq,D] float64, lse [B,Hq] float64) for a drawn workload."""
    spec = workload.spec
    if spec.layout == "paged":
        return decode_attention_paged(workload.q, workload.k_pages, workload.v_pages,
                                      workload.block_table, workload.ctx_lens, float(spec.scale), spec.dtype,
                                      kv_scales=kv_scales_of(spec))
    return decode_attention(workload.q, workload.k, workload.v, workload.seq_start, workload.ctx_lens,
                            float(spec.scale), spec.dtype, kv_scales=kv_scales_of(spec))
