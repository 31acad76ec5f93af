"""Pins of the prefill-attention oracle (cached and uncached prefill).

Each ``pin_*`` checks the oracle (looked up at call time through ``pa``)
against a library routine, pure-Python brute force, the decode oracle, or an
invariant of causal attention; the ``test_mutant_*`` tests plant plausible
mistakes on the CPU and check that a pin catches each.
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle.decode_attention as da
import oracle.prefill_attention as pa
from workloads.synth import PREFILL_WORKLOADS, generate_prefill, small_prefill_spec

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _close(a, b, tol, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    same_inf = np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))
    err = np.where(same_inf, 0.0, np.abs(a - b))
    assert np.all(np.isfinite(err)), f"{what}: non-finite mismatch"
    assert float(err.max(initial=0.0)) <= tol, f"{what}: max |err| {float(err.max()):.3e} > {tol:.1e}"


def _ragged_case(seed=3, layout_base=1):
    spec = small_prefill_spec(PREFILL_WORKLOADS[layout_base], [40, 7, 1, 64], [5, 7, 1, 16], seed=seed)
    return generate_prefill(spec)


def _seq_tensors(pw, b):
    w, s = pw.kv, pw.kv.spec
    if s.layout == "paged":
        keys = da.paged_context(w.k_pages, w.block_table, w.ctx_lens, b)
        values = da.paged_context(w.v_pages, w.block_table, w.ctx_lens, b)
    else:
        keys = da.contiguous_context(w.k, w.seq_start, w.ctx_lens, b)
        values = da.contiguous_context(w.v, w.seq_start, w.ctx_lens, b)
    a, M = int(pw.q_start[b]), int(pw.q_lens[b])
    return (da.widen(pw.q[a: a + M], s.dtype), da.widen(keys, s.dtype), da.widen(values, s.dtype))


# ------------------------------------------------------------------ pins


def pin_torch_sdpa_with_offset_mask():
    """torch SDPA (CPU, float64) with the mask t <= L - M + i and GQA by repeat_interleave."""
    pw = _ragged_case()
    s = pw.kv.spec
    out, _ = pa.reference(pw)
    for b in range(s.batch):
        q, k, v = _seq_tensors(pw, b)
        M, L = q.shape[0], k.shape[0]
        G = s.num_q_heads // s.num_kv_heads
        qt = torch.from_numpy(q).permute(1, 0, 2)[None]                       # [1, Hq, M, D]
        kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, 0)[None]
        vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, 0)[None]
        mask = torch.arange(L)[None, :] <= (L - M + torch.arange(M))[:, None]
        ref = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=float(s.scale))[0].permute(1, 0, 2)
        a = int(pw.q_start[b])
        _close(out[a: a + M], ref.numpy(), 1e-12, f"SDPA sequence {b}")


def pin_brute_force():
    """Pure-Python math.exp / math.fsum on tiny shapes, every (token, head), out and lse."""
    r = np.random.default_rng(11)
    for L, M, D, Hq, Hkv in [(5, 5, 3, 2, 1), (8, 3, 4, 4, 2), (6, 1, 2, 2, 2), (7, 4, 3, 3, 1)]:
        q = r.standard_normal((M, Hq, D)).astype(np.float32)
        k = r.standard_normal((L, Hkv, D)).astype(np.float32)
        v = r.standard_normal((L, Hkv, D)).astype(np.float32)
        scale = 0.7
        out, lse = pa.prefill_attention(q, k, v, np.array([0]), np.array([L]), np.array([0]), np.array([M]),
                                        scale, "f32")
        G = Hq // Hkv
        for i in range(M):
            p = L - M + i
            for h in range(Hq):
                hk = h // G
                sc = [scale * math.fsum(float(q[i, h, d]) * float(k[t, hk, d]) for d in range(D))
                      for t in range(p + 1)]
                mx = max(sc)
                w = [math.exp(x - mx) for x in sc]
                z = math.fsum(w)
                o = [math.fsum(w[t] * float(v[t, hk, d]) for t in range(p + 1)) / z for d in range(D)]
                _close(out[i, h], o, 1e-13, f"brute out L={L} M={M} i={i} h={h}")
                _close(lse[i, h], mx + math.log(z), 1e-13, f"brute lse L={L} M={M} i={i} h={h}")


def pin_one_new_token_is_decode():
    """M_b = 1: the new token sees the whole cache, so prefill equals the decode oracle."""
    spec = small_prefill_spec(PREFILL_WORKLOADS[3], [33, 100, 16], [1, 1, 1], seed=12)
    pw = generate_prefill(spec)
    out, lse = pa.reference(pw)
    w = pw.kv
    d_out, d_lse = da.decode_attention_paged(pw.q, w.k_pages, w.v_pages, w.block_table, w.ctx_lens,
                                             float(w.spec.scale), w.spec.dtype)
    _close(out, d_out, 1e-12, "M=1 out")
    _close(lse, d_lse, 1e-12, "M=1 lse")


def pin_last_new_token_sees_everything():
    """The last new token of a sequence (position L - 1) attends like a decode step over all L tokens."""
    pw = _ragged_case(seed=13)
    out, lse = pa.reference(pw)
    s = pw.kv.spec
    for b in range(s.batch):
        q, k, v = _seq_tensors(pw, b)
        G = s.num_q_heads // s.num_kv_heads
        a, M = int(pw.q_start[b]), int(pw.q_lens[b])
        for h in range(s.num_q_heads):
            o, l = da.attend(q[M - 1, h][None], k[:, h // G], v[:, h // G], float(s.scale))
            _close(out[a + M - 1, h], o[0], 1e-12, f"last token b={b} h={h}")
            _close(lse[a + M - 1, h], l[0], 1e-12, f"last token lse b={b} h={h}")


def pin_uncached_first_token():
    """Uncached prefill (M = L): token 0 sees only itself, so out = V_0 exactly and lse = its own score."""
    spec = small_prefill_spec(PREFILL_WORKLOADS[2], [9, 30], [9, 30], seed=14)
    pw = generate_prefill(spec)
    out, lse = pa.reference(pw)
    s = pw.kv.spec
    G = s.num_q_heads // s.num_kv_heads
    for b in range(2):
        q, k, v = _seq_tensors(pw, b)
        a = int(pw.q_start[b])
        for h in range(s.num_q_heads):
            assert np.array_equal(out[a, h], v[0, h // G]), "uncached token 0: out != V_0"
            _close(lse[a, h], float(s.scale) * float(q[0, h] @ k[0, h // G]), 1e-12, "uncached token 0 lse")


def pin_causality():
    """Changing K/V after position p leaves new token i (p = L - M + i) unchanged; changing row p does not."""
    pw = _ragged_case(seed=15)
    s = pw.kv.spec
    out0, _ = pa.reference(pw)
    b = 0
    L, M = int(pw.kv.ctx_lens[b]), int(pw.q_lens[b])
    i = 1
    p = L - M + i
    w = pw.kv
    st = int(w.seq_start[b])
    for rows, changed in (((st + p + 1, st + L), False), ((st + p, st + p + 1), True)):
        k0, v0 = w.k.copy(), w.v.copy()
        w.k[rows[0]: rows[1]] ^= np.uint16(0x0001)  # a finite change of the last mantissa bit
        w.v[rows[0]: rows[1]] ^= np.uint16(0x0001)
        out1, _ = pa.reference(pw)
        w.k, w.v = k0, v0
        a = int(pw.q_start[b])
        same = np.array_equal(out1[a + i], out0[a + i])
        assert same != changed, f"causality: rows {rows} changed={changed} but output same={same}"


def pin_paged_equals_contiguous():
    """The same logical contexts through a block table and packed give identical results."""
    spec = small_prefill_spec(PREFILL_WORKLOADS[3], [40, 17], [6, 17], seed=16)
    pw = generate_prefill(spec, spare_pages=2)
    out_p, lse_p = pa.reference(pw)
    w = pw.kv
    ks = [da.paged_context(w.k_pages, w.block_table, w.ctx_lens, b) for b in range(2)]
    vs = [da.paged_context(w.v_pages, w.block_table, w.ctx_lens, b) for b in range(2)]
    starts = np.array([0, ks[0].shape[0]])
    out_c, lse_c = pa.prefill_attention(pw.q, np.concatenate(ks), np.concatenate(vs), starts, w.ctx_lens,
                                        pw.q_start, pw.q_lens, float(w.spec.scale), w.spec.dtype)
    assert np.array_equal(out_p, out_c) and np.array_equal(lse_p, lse_c)


def pin_sampled_rows_match_full():
    pw = _ragged_case(seed=17)
    out, lse = pa.reference(pw)
    rows = [(0, 0, 0), (0, 4, 31), (3, 15, 7), (2, 0, 8), (1, 6, 1)]
    for (b, i, h), (o, l) in zip(rows, pa.prefill_attention_rows(pw, rows)):
        a = int(pw.q_start[b])
        _close(o, out[a + i, h], 1e-13, f"sampled row {(b, i, h)}")  # BLAS blocking may differ by shape
        _close(l, lse[a + i, h], 1e-13, f"sampled lse {(b, i, h)}")


def pin_score_count():
    """Visible pairs per head: sum over new tokens of (L - M + i + 1)."""
    pw = _ragged_case(seed=18)
    want = sum(int(L) - int(M) + i + 1 for L, M in zip(pw.kv.ctx_lens, pw.q_lens) for i in range(int(M)))
    assert pw.score_count == want


PINS = [pin_torch_sdpa_with_offset_mask, pin_brute_force, pin_one_new_token_is_decode,
        pin_last_new_token_sees_everything, pin_uncached_first_token, pin_causality,
        pin_paged_equals_contiguous, pin_sampled_rows_match_full, pin_score_count]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin()


# ------------------------------------------------------------------ planted mistakes


def _failing_pins():
    failed = []
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin()
        except Exception:  # noqa: BLE001 - any failure counts as "caught"
            failed.append(pin.__name__)
    return failed


def _with_positions(shift):
    real = pa.attend_causal

    def mutant(q_rows, keys, values, scale, positions):
        return real(q_rows, keys, values, scale, shift(positions, keys.shape[0], q_rows.shape[0]))
    return mutant


MUTANTS = {
    "mask_strict": _with_positions(lambda p, L, R: p - 1),              # t < p instead of t <= p
    "mask_one_past": _with_positions(lambda p, L, R: p + 1),
    "mask_no_prefix_offset": _with_positions(lambda p, L, R: p - (p.min() if len(p) else 0)),
    "mask_reversed_rows": _with_positions(lambda p, L, R: p[::-1].copy()),
    "no_mask": _with_positions(lambda p, L, R: np.full_like(p, L)),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_mask_is_caught(name, monkeypatch):
    monkeypatch.setattr(pa, "attend_causal", MUTANTS[name])
    assert _failing_pins(), f"no pin catches mutant {name}"


def test_mutant_no_max_subtraction_is_caught(monkeypatch):
    def mutant(q_rows, keys, values, scale, positions):
        s = scale * (q_rows @ keys.T)
        vis = np.arange(keys.shape[0])[None, :] <= positions[:, None]
        w = np.where(vis, np.exp(s), 0.0)
        z = w.sum(axis=1)
        return (w @ values) / z[:, None], np.log(z) + 1e-9
    monkeypatch.setattr(pa, "attend_causal", mutant)
    assert _failing_pins()


def test_mutant_gqa_mapping_is_caught(monkeypatch):
    real = pa._sequence

    def modulo(q_b, keys, values, dtype, scale, tokens=None, heads=None):
        Hq, Hkv = q_b.shape[1], keys.shape[1]
        G = Hq // Hkv
        perm = np.array([(h % Hkv) * G + h // Hkv for h in range(Hq)])
        inv = np.argsort(perm)
        out, lse = real(q_b[:, inv], keys, values, dtype, scale, tokens, None)
        return out[:, perm], lse[:, perm]

    monkeypatch.setattr(pa, "_sequence", modulo)
    assert _failing_pins()


def test_mutant_query_offset_is_caught(monkeypatch):
    """Queries read from the wrong packed rows (q_start ignored)."""
    real = pa._sequence

    def shifted(q_b, keys, values, dtype, scale, tokens=None, heads=None):
        return real(np.roll(q_b, 1, axis=0), keys, values, dtype, scale, tokens, heads)

    monkeypatch.setattr(pa, "_sequence", shifted)
    assert _failing_pins()
