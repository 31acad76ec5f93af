"""CPU fp64 oracle for cached-prefix prefill attention.

TEST INFRASTRUCTURE ONLY: nothing on the product path imports this module
(only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may). It shares no code with the HIP path.

What it computes (paper Algorithm 1 and the k-step-off pipeline of Sec. 3.2):
while the agent's KV cache stays valid, a step prefills only the new
observation's tokens over the cached prefix ("cached" prefill); after a
summary update the whole context (summary plus recent buffer) is prefilled
from scratch ("uncached" prefill). Both are the same operation: sequence b
holds L_b cached tokens whose last M_b are the new ones (their keys and
values already appended, as in Sec. 2.2), and new token i (0 <= i < M_b),
which sits at cache position p = L_b - M_b + i, attends over cache tokens
0 .. p (a causal mask among the new tokens; every earlier token is visible).
The uncached case is M_b = L_b. For query head h of new token i:

    s_t   = scale * sum_d q[i, h, d] * K[t, h_kv(h), d]     t = 0 .. p
    out   = sum_t softmax(s)_t * V[t, h_kv(h), :]
    lse   = ln sum_t exp(s_t)

with h_kv(h) = h // (h_q / h_kv) as in the decode oracle. The paper gives
the cached/uncached structure but no formula; this is textbook causal
softmax attention written out (scores, masked maximum, exponentials, sum,
weighted values) in float64 on the exact stored values.
"""

from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

from oracle.decode_attention import contiguous_context, paged_context, widen

_ROW_CHUNK = 256  # new tokens per block of the score matrix (memory bound of the oracle only)


def attend_causal(q_rows: np.ndarray, keys: np.ndarray, values: np.ndarray, scale: float,
                  positions: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Row r (float64 [R, D]) attends over keys[0 .. positions[r]] (inclusive).

    keys, values: float64 [L, D]. Returns out [R, D], lse [R]. A row whose
    position is negative sees no key: out 0, lse -inf.
    """
    R, D = q_rows.shape
    L = keys.shape[0]
    s = scale * (q_rows @ keys.T)  # [R, L]
    visible = np.arange(L)[None, :] <= positions[:, None]
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, initial=-np.inf)
    live = np.isfinite(m)
    w = np.where(visible, np.exp(s - np.where(live, m, 0.0)[:, None]), 0.0)
    z = w.sum(axis=1)
    out = np.zeros((R, D))
    out[live] = (w[live] @ values) / z[live, None]
    lse = np.where(live, np.where(live, m, 0.0) + np.log(np.where(live, z, 1.0)), -np.inf)
    return out, lse


def _sequence(q_b: np.ndarray, keys: np.ndarray, values: np.ndarray, dtype: str, scale: float,
              tokens: Sequence[int] = None, heads: Sequence[int] = None):
    """New tokens of one sequence: q_b [M, Hq, D] stored values; keys/values [L, Hkv, D] stored values.

    Returns out [M, Hq, D], lse [M, Hq] (rows not asked for stay 0 / -inf).
    """
    M, Hq, D = q_b.shape
    L, Hkv, _ = keys.shape
    G = Hq // Hkv
    if M > L:
        raise ValueError("more new tokens than cached tokens")
    out = np.zeros((M, Hq, D))
    lse = np.full((M, Hq), -np.inf)
    tok = np.arange(M) if tokens is None else np.asarray(sorted(set(tokens)), dtype=np.int64)
    want = set(range(Hq)) if heads is None else set(heads)
    for hk in range(Hkv):
        hs = [h for h in range(hk * G, (hk + 1) * G) if h in want]
        if not hs or len(tok) == 0:
            continue
        kf = widen(keys[:, hk], dtype)
        vf = widen(values[:, hk], dtype)
        for c0 in range(0, len(tok), _ROW_CHUNK):
            ti = tok[c0: c0 + _ROW_CHUNK]
            for h in hs:
                qf = widen(q_b[ti, h], dtype)
                o, l = attend_causal(qf, kf, vf, scale, (L - M) + ti)
                out[ti, h] = o
                lse[ti, h] = l
    return out, lse


def prefill_attention(q, k, v, seq_start, ctx_lens, q_start, q_lens, scale: float, dtype: str):
    """Contiguous cache: q [sum M_b, Hq, D] packed at q_start; k, v [T, Hkv, D] at seq_start.

    Returns out [sum M_b, Hq, D] and lse [sum M_b, Hq] (float64).
    """
    total, Hq, D = q.shape
    out = np.zeros((total, Hq, D))
    lse = np.full((total, Hq), -np.inf)
    for b in range(len(ctx_lens)):
        a, M = int(q_start[b]), int(q_lens[b])
        o, l = _sequence(q[a: a + M], contiguous_context(k, seq_start, ctx_lens, b),
                         contiguous_context(v, seq_start, ctx_lens, b), dtype, scale)
        out[a: a + M], lse[a: a + M] = o, l
    return out, lse


def prefill_attention_paged(q, k_pages, v_pages, block_table, ctx_lens, q_start, q_lens, scale: float,
                            dtype: str):
    """Paged cache [P, page, Hkv, D] with a block table; queries as in prefill_attention."""
    total, Hq, D = q.shape
    out = np.zeros((total, Hq, D))
    lse = np.full((total, Hq), -np.inf)
    for b in range(len(ctx_lens)):
        a, M = int(q_start[b]), int(q_lens[b])
        o, l = _sequence(q[a: a + M], paged_context(k_pages, block_table, ctx_lens, b),
                         paged_context(v_pages, block_table, ctx_lens, b), dtype, scale)
        out[a: a + M], lse[a: a + M] = o, l
    return out, lse


def reference(pw):
    """Full result for a drawn prefill workload (see workloads.synth.generate_prefill)."""
    w, s = pw.kv, pw.kv.spec
    if s.layout == "paged":
        return prefill_attention_paged(pw.q, w.k_pages, w.v_pages, w.block_table, w.ctx_lens, pw.q_start,
                                       pw.q_lens, float(s.scale), s.dtype)
    return prefill_attention(pw.q, w.k, w.v, w.seq_start, w.ctx_lens, pw.q_start, pw.q_lens, float(s.scale),
                             s.dtype)


def prefill_attention_rows(pw, rows: Sequence[Tuple[int, int, int]]) -> List[Tuple[np.ndarray, float]]:
    """Selected (sequence b, new token i, query head h) results, for sampled full-size checks."""
    w, s = pw.kv, pw.kv.spec
    by_seq = {}
    for b, i, h in rows:
        by_seq.setdefault(b, []).append((i, h))
    got = {}
    for b, items in by_seq.items():
        if s.layout == "paged":
            keys = paged_context(w.k_pages, w.block_table, w.ctx_lens, b)
            values = paged_context(w.v_pages, w.block_table, w.ctx_lens, b)
        else:
            keys = contiguous_context(w.k, w.seq_start, w.ctx_lens, b)
            values = contiguous_context(w.v, w.seq_start, w.ctx_lens, b)
        a, M = int(pw.q_start[b]), int(pw.q_lens[b])
        toks = [i for i, _ in items]
        hs = sorted({h for _, h in items})
        o, l = _sequence(pw.q[a: a + M], keys, values, s.dtype, float(s.scale), tokens=toks, heads=hs)
        for i, h in items:
            got[(b, i, h)] = (o[i, h], float(l[i, h]))
    return [got[r] for r in rows]
