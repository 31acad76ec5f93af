"""Pins of the CPU oracle against what mathematics and the paper fix.

Each ``pin_*`` function raises AssertionError when the oracle (looked up at
call time through the module ``da``) disagrees with a closed form, an
invariant, a brute-force evaluation, a library routine or a worked example.
The ``test_mutant_*`` tests plant plausible mistakes in the oracle (on the
CPU) and check that at least one pin catches each of them.
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle.cost_model as cm
import oracle.decode_attention as da
from workloads.synth import WORKLOADS, f32_to_bf16_bits, generate, small_spec

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _rng(seed):
    return np.random.default_rng(seed)


def _close(a, b, tol, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    same_inf = np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))
    err = np.where(same_inf, 0.0, np.abs(a - b))
    assert np.all(np.isfinite(err)), f"{what}: non-finite mismatch"
    m = float(err.max(initial=0.0))
    assert m <= tol, f"{what}: max |err| {m:.3e} > {tol:.1e}"


# ------------------------------------------------------------------ pins


def pin_one_key():
    """A one-token context returns its value row exactly and lse = its score."""
    r = _rng(1)
    for G, D in [(1, 4), (4, 64), (8, 128)]:
        q = r.standard_normal((G, D))
        k = r.standard_normal((1, D))
        v = r.standard_normal((1, D))
        out, lse = da.attend(q, k, v, 0.3)
        assert np.array_equal(out, np.repeat(v, G, axis=0)), "one key: out != V_0"
        _close(lse, 0.3 * (q @ k[0]), 1e-13, "one key: lse")


def pin_uniform_scores():
    """q = 0 makes every score equal: out = mean of V, lse = ln L."""
    r = _rng(2)
    for L in [1, 2, 7, 300]:
        v = r.standard_normal((L, 16))
        out, lse = da.attend(np.zeros((3, 16)), r.standard_normal((L, 16)), v, 0.7)
        _close(out, np.repeat(v.mean(axis=0, keepdims=True), 3, axis=0), 1e-14, "q=0: mean(V)")
        _close(lse, np.full(3, math.log(L)), 1e-14, "q=0: lse")
    # structured values: row t holds (t mod 97) / 32, exactly representable
    L = 5000
    v = ((np.arange(L) % 97) / 32.0)[:, None] * np.ones((1, 8))
    out, _ = da.attend(np.zeros((1, 8)), r.standard_normal((L, 8)), v, 1.0)
    expect = math.fsum(((np.arange(L) % 97) / 32.0).tolist()) / L
    _close(out, np.full((1, 8), expect), 1e-13, "q=0 structured V")


def pin_weights_sum_to_one():
    """Softmax weights sum to 1: a constant value row c is returned as c."""
    r = _rng(3)
    for L in [1, 5, 1000]:
        q = 3 * r.standard_normal((4, 32))
        k = r.standard_normal((L, 32))
        out, _ = da.attend(q, k, np.full((L, 32), -2.5), 0.5)
        _close(out, np.full((4, 32), -2.5), 1e-13, "sum of weights")


def pin_golden_closed_forms():
    with open(os.path.join(GOLDEN, "softmax_closed_form.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        q = np.asarray(c["q"], dtype=np.float32)[None]  # [1, Hq, D]
        k = np.asarray(c["k"], dtype=np.float32)  # [L, Hkv, D]
        v = np.asarray(c["v"], dtype=np.float32)
        L = k.shape[0]
        out, lse = da.decode_attention(q, k, v, np.array([0]), np.array([L], dtype=np.int32),
                                       c["scale"], "f32")
        _close(out[0], c["out"], c["tol"], c["name"] + " out")
        _close(lse[0], c["lse"], max(c["tol"], 1e-15), c["name"] + " lse")


def pin_split_combine():
    """Split-K partial results merged by log-sum-exp equal unsplit attention."""
    r = _rng(4)
    for L, n in [(1, 1), (10, 3), (513, 8), (2000, 40)]:
        q = 2 * r.standard_normal((4, 32))
        k = r.standard_normal((L, 32))
        v = r.standard_normal((L, 32))
        full = da.attend(q, k, v, 0.25)
        cuts = np.sort(r.integers(0, L + 1, size=n))
        bounds = [0, *cuts.tolist(), L]  # repeated cuts give empty ranges
        split = da.attend_split(q, k, v, 0.25, bounds)
        _close(split[0], full[0], 1e-12, "split-K out")
        _close(split[1], full[1], 1e-12, "split-K lse")
    # large scores: the merge must not overflow
    q = np.full((2, 8), 40.0)
    k = np.full((64, 8), 40.0) + r.standard_normal((64, 8))
    v = r.standard_normal((64, 8))
    full = da.attend(q, k, v, 1.0)
    split = da.attend_split(q, k, v, 1.0, [0, 10, 10, 50, 64])
    assert np.all(np.isfinite(full[0])) and np.all(np.isfinite(split[0])), "overflow"
    _close(split[0], full[0], 1e-11, "split-K large scores")
    _close(split[1] / full[1], np.ones(2), 1e-14, "split-K large lse")
    # all ranges empty
    o, l = da.lse_combine([da.attend(q, k[:0], v[:0], 1.0)] * 3)
    assert np.array_equal(o, np.zeros((2, 8))) and np.all(l == -np.inf), "all-empty merge"


def pin_permutation_invariance():
    """Reordering (key, value) pairs jointly leaves attention unchanged."""
    r = _rng(5)
    q = r.standard_normal((8, 64))
    k = r.standard_normal((777, 64))
    v = r.standard_normal((777, 64))
    p = r.permutation(777)
    a = da.attend(q, k, v, 0.125)
    b = da.attend(q, k[p], v[p], 0.125)
    _close(a[0], b[0], 1e-13, "permutation out")
    _close(a[1], b[1], 1e-13, "permutation lse")


def pin_key_shift():
    """Adding one vector u to every key adds scale*q.u to all scores of a head."""
    r = _rng(6)
    q = r.standard_normal((4, 32))
    k = r.standard_normal((300, 32))
    v = r.standard_normal((300, 32))
    u = 5 * r.standard_normal(32)
    a = da.attend(q, k, v, 0.2)
    b = da.attend(q, k + u, v, 0.2)
    _close(b[0], a[0], 1e-12, "key shift out")
    _close(b[1], a[1] + 0.2 * (q @ u), 1e-12, "key shift lse")


def pin_brute_force():
    """Tiny shapes against a pure-Python evaluation with math.exp and math.fsum."""
    r = _rng(7)
    for L, G, D in [(1, 1, 1), (2, 2, 3), (5, 3, 4), (8, 4, 2)]:
        q = r.standard_normal((G, D))
        k = r.standard_normal((L, D))
        v = r.standard_normal((L, D))
        sc = 0.9
        out, lse = da.attend(q, k, v, sc)
        for g in range(G):
            s = [sc * math.fsum(q[g, d] * k[t, d] for d in range(D)) for t in range(L)]
            m = max(s)
            w = [math.exp(x - m) for x in s]
            z = math.fsum(w)
            for d in range(D):
                ref = math.fsum(w[t] * v[t, d] for t in range(L)) / z
                assert abs(out[g, d] - ref) <= 1e-14 * max(1.0, abs(ref)), "brute force out"
            assert abs(lse[g] - (m + math.log(z))) <= 1e-14 * max(1.0, abs(lse[g])), "brute force lse"


def _sdpa(q, k, v, scale):
    """torch SDPA (CPU, float64, enable_gqa): q [Hq, D], k/v [L, Hkv, D] -> [Hq, D]."""
    qt = torch.from_numpy(q)[None, :, None, :]
    kt = torch.from_numpy(np.ascontiguousarray(k.transpose(1, 0, 2)))[None]
    vt = torch.from_numpy(np.ascontiguousarray(v.transpose(1, 0, 2)))[None]
    o = F.scaled_dot_product_attention(qt, kt, vt, scale=scale, enable_gqa=True)
    return o[0, :, 0, :].numpy()


def pin_torch_sdpa():
    """Whole-batch oracle against torch's scaled_dot_product_attention (library routine)."""
    spec = small_spec(WORKLOADS[2], [1, 37, 500], seed=11).replace(num_q_heads=16, num_kv_heads=4,
                                                                   head_dim=64)
    w = generate(spec)
    out, lse = da.reference(w)
    for b in range(spec.batch):
        L = int(w.ctx_lens[b])
        a = int(w.seq_start[b])
        q = da.widen(w.q[b], "bf16")
        k = da.widen(w.k[a:a + L], "bf16")
        v = da.widen(w.v[a:a + L], "bf16")
        _close(out[b], _sdpa(q, k, v, float(spec.scale)), 1e-13, "vs torch SDPA")
    # fp32 workload with G = 4 at a non-default scale
    spec = small_spec(WORKLOADS[1], [64], seed=12)
    w = generate(spec)
    out, _ = da.decode_attention(w.q, w.k, w.v, w.seq_start, w.ctx_lens, 0.37, "f32")
    ref = _sdpa(da.widen(w.q[0], "f32"), da.widen(w.k, "f32"), da.widen(w.v, "f32"), 0.37)
    _close(out[0], ref, 1e-13, "vs torch SDPA f32")


def pin_gqa_expansion():
    """GQA equals plain multi-head attention with each KV head repeated G times in a row."""
    spec = small_spec(WORKLOADS[2], [40, 3], seed=13).replace(num_q_heads=8, num_kv_heads=2, head_dim=16)
    w = generate(spec)
    out, lse = da.reference(w)
    k_rep = np.repeat(w.k, 4, axis=1)
    v_rep = np.repeat(w.v, 4, axis=1)
    out2, lse2 = da.decode_attention(w.q, k_rep, v_rep, w.seq_start, w.ctx_lens, float(spec.scale), "bf16")
    _close(out, out2, 1e-14, "GQA expansion out")
    _close(lse, lse2, 1e-14, "GQA expansion lse")


def pin_paged_equals_contiguous():
    """A paged cache and a packed cache holding the same logical rows give the same result."""
    for ps in (1, 16, 64):
        spec = small_spec(WORKLOADS[4], [0, 1, 15, 16, 17, 130], seed=14 + ps, max_ctx_len=256).replace(
            page_size=ps, key_scale_frac=0.05)
        w = generate(spec, spare_pages=3)
        lens = w.ctx_lens
        starts = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
        rows_k, rows_v = [], []
        for b in range(spec.batch):
            for t in range(int(lens[b])):
                page = w.block_table[b, t // ps]
                rows_k.append(w.k_pages[page, t % ps])
                rows_v.append(w.v_pages[page, t % ps])
        k = np.stack(rows_k)
        v = np.stack(rows_v)
        a = da.reference(w)
        b = da.decode_attention(w.q, k, v, starts, lens, float(spec.scale), "bf16")
        _close(a[0], b[0], 0.0, f"paged vs packed out (page {ps})")
        _close(a[1], b[1], 0.0, f"paged vs packed lse (page {ps})")


def pin_empty_context():
    spec = small_spec(WORKLOADS[2], [0, 5, 0], seed=15).replace(num_q_heads=4, num_kv_heads=2, head_dim=8)
    w = generate(spec)
    out, lse = da.reference(w)
    assert np.array_equal(out[0], np.zeros((4, 8))) and np.all(lse[0] == -np.inf), "L=0 convention"
    assert np.array_equal(out[2], np.zeros((4, 8))) and np.all(lse[2] == -np.inf), "L=0 convention"
    assert np.all(np.isfinite(out[1])) and np.all(np.isfinite(lse[1]))


def pin_widen_bf16():
    """bf16 bit patterns widen to the values torch assigns them."""
    r = _rng(16)
    x = r.standard_normal(4096).astype(np.float32) * np.float32(100)
    bits = f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(da.widen(bits, "bf16"), ref), "bf16 widening"
    assert np.array_equal(da.widen(x, "f32"), x.astype(np.float64)), "f32 widening"


def pin_large_scores():
    """Scores in the thousands: the maximum subtraction keeps everything finite."""
    q = np.full((2, 4), 30.0)
    k = np.array([[30.0, 30, 30, 30], [29.0, 30, 30, 30], [-30.0, 0, 0, 0]])
    v = np.array([[1.0, 0, 0, 0], [0, 1.0, 0, 0], [0, 0, 1.0, 0]])
    out, lse = da.attend(q, k, v, 1.0)
    w = np.array([1.0, math.exp(-30.0), 0.0])
    w = w / w.sum()
    _close(out, np.repeat(w[None], 2, axis=0) @ v, 1e-15, "large scores out")
    _close(lse, np.full(2, 3600.0 + math.log1p(math.exp(-30.0))), 1e-12, "large scores lse")


def _rows_cases():
    """Small workloads of every layout the full-size checks use: packed ragged, paged with pages of 16
    and 64 tokens, a GQA group of 8, and an FP8 cache with its per-tensor scales."""
    yield generate(small_spec(WORKLOADS[3], [70, 0, 33, 129], seed=17).replace(head_dim=16), gap_rows=3)
    yield generate(small_spec(WORKLOADS[4], [40, 1, 17, 96], seed=18, max_ctx_len=128).replace(head_dim=16),
                   spare_pages=2)
    yield generate(small_spec(WORKLOADS[5], [150, 64, 65], seed=19, max_ctx_len=192).replace(head_dim=16),
                   spare_pages=1)
    yield generate(small_spec(WORKLOADS[6], [90, 7], seed=20).replace(head_dim=16, k_scale=2.0 ** -5,
                                                                     v_scale=2.0 ** -3))
    yield generate(small_spec(WORKLOADS[7], [130, 64], seed=21, max_ctx_len=192).replace(head_dim=16,
                                                                                     k_scale=2.0 ** -4))


def pin_rows_equal_reference():
    """Rows computed one by one (the full-size sampled checks and the CPU baseline use them) equal the
    same rows of the whole-batch result, for every layout, a GQA group of 8 and FP8 scales; asking for
    a subset of a sequence's heads, in any order and with repeats, changes nothing."""
    for w in _rows_cases():
        s = w.spec
        ref_out, ref_lse = da.reference(w)
        every = [(b, h) for b in range(s.batch) for h in range(s.num_q_heads)]
        r = _rng(22)
        subset = [every[i] for i in r.permutation(len(every))[: max(3, len(every) // 5)]]
        for rows in (every, subset + subset[:2]):
            got = da.decode_attention_rows(w, rows)
            assert len(got) == len(rows), f"{s.name}: row count"
            for (b, h), (o, l) in zip(rows, got):
                _close(o, ref_out[b, h], 1e-12, f"{s.name} rows out ({b}, {h})")
                _close([l], [ref_lse[b, h]], 1e-12, f"{s.name} rows lse ({b}, {h})")


def pin_cost_model_case_study():
    with open(os.path.join(GOLDEN, "cost_model_case_study.json")) as f:
        g = json.load(f)
    W = Fraction(g["bandwidth_GBps"])
    P = Fraction(g["prefill_tokens_per_s"])
    S = Fraction(g["kv_GB_per_token"])
    Y = Fraction(g["generated_tokens"])
    bound = cm.max_compression_ratio(W, Y, S, P)
    assert bound == Fraction(*g["bound_exact"]), f"bound {bound}"
    assert round(float(bound), 2) == g["bound_paper_rounded"]
    assert math.isclose(g["bound_paper_rounded"] * g["prefix_K_tokens"], g["summary_bound_K_tokens_paper"])
    # at the bound the savings exactly pay for the prefill; below it they win
    L_full = Fraction(32000)
    assert cm.net_saving(Y, L_full, bound * L_full, S, W, P) == 0
    assert cm.net_saving(Y, L_full, bound * L_full * Fraction(99, 100), S, W, P) > 0
    assert cm.net_saving(Y, L_full, bound * L_full * Fraction(101, 100), S, W, P) < 0
    # per-token decode time is linear in context: t(L_full) - t(L_sum) is the saving
    assert (cm.decode_time(L_full, S, W) - cm.decode_time(Fraction(7000), S, W)
            == cm.decode_saving(L_full, Fraction(7000), S, W))
    assert cm.prefill_cost(Fraction(3000), P) == 1


PINS = [
    pin_one_key, pin_uniform_scores, pin_weights_sum_to_one, pin_golden_closed_forms,
    pin_split_combine, pin_permutation_invariance, pin_key_shift, pin_brute_force, pin_torch_sdpa,
    pin_gqa_expansion, pin_paged_equals_contiguous, pin_empty_context, pin_widen_bf16,
    pin_large_scores, pin_cost_model_case_study, pin_rows_equal_reference,
]


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


def _attend_variant(*, scale_on=True, log2=False, sign=1.0, submax=True, drop_last=False, norm="z",
                    transpose=False):
    def attend(q_rows, keys, values, scale):
        G, D = q_rows.shape
        if drop_last and keys.shape[0] > 1:
            keys, values = keys[:-1], values[:-1]
        L = keys.shape[0]
        if L == 0:
            return np.zeros((G, D)), np.full(G, -np.inf)
        s = (scale if scale_on else 1.0) * (keys @ (q_rows[:, ::-1] if transpose else q_rows).T)
        m = s.max(axis=0)
        w = np.exp(s - sign * m) if submax else np.exp(s)
        z = w.sum(axis=0)
        out = (w.T @ values) / (z[:, None] if norm == "z" else L)
        lse = (m if submax else 0) + (np.log2(z) if log2 else np.log(z))
        return out, lse
    return attend


MUTANTS = {
    "no_scale": ("attend", _attend_variant(scale_on=False)),
    "lse_log2": ("attend", _attend_variant(log2=True)),
    "max_sign": ("attend", _attend_variant(sign=-1.0)),
    "no_max_subtraction": ("attend", _attend_variant(submax=False)),
    "dropped_last_key": ("attend", _attend_variant(drop_last=True)),
    "normalise_by_L": ("attend", _attend_variant(norm="L")),
    "reversed_query": ("attend", _attend_variant(transpose=True)),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_attend_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(da, attr, fn)
    assert _failing_pins(), f"no pin catches mutant {name}"


def test_mutant_gqa_modulo_mapping_is_caught(monkeypatch):
    real = da._attend_sequence

    def modulo(q_b, keys, values, dtype, scale, heads=None):
        Hq, Hkv = q_b.shape[0], keys.shape[1]
        G = Hq // Hkv
        perm = np.array([(h % Hkv) * G + h // Hkv for h in range(Hq)])  # head h reads KV head h % Hkv
        inv = np.argsort(perm)
        out, lse = real(q_b[inv], keys, values, dtype, scale, heads)
        return out[perm], lse[perm]

    monkeypatch.setattr(da, "_attend_sequence", modulo)
    assert _failing_pins()


def test_mutant_paged_index_is_caught(monkeypatch):
    def swapped(kv_pages, block_table, ctx_lens, b):
        ps = kv_pages.shape[1]
        L = int(ctx_lens[b])
        rows = [kv_pages[block_table[b, t // ps], (t + 1) % ps if ps > 1 else 0] for t in range(L)]
        return np.stack(rows) if rows else kv_pages[:0, 0]

    monkeypatch.setattr(da, "paged_context", swapped)
    assert _failing_pins()


def test_mutant_combine_is_caught(monkeypatch):
    real = da.lse_combine

    def no_division(parts):
        out, lse = real(parts)
        lses = np.stack([l for _, l in parts])
        wsum = np.where(np.isfinite(lses), np.exp(lses - lse), 0.0).sum(axis=0)
        return out * (wsum[:, None] + 0.5), lse

    def plain_exp(parts):
        outs = np.stack([o for o, _ in parts])
        lses = np.stack([l for _, l in parts])
        w = np.exp(lses)
        return np.einsum("sg,sgd->gd", w, outs) / w.sum(axis=0)[:, None], np.log(w.sum(axis=0))

    for fn in (no_division, plain_exp):
        monkeypatch.setattr(da, "lse_combine", fn)
        assert _failing_pins(), fn.__name__


def test_mutant_widen_is_caught(monkeypatch):
    def bad(x, dtype):
        if dtype == "bf16":
            bits = (np.asarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(15))
            return bits.view(np.float32).astype(np.float64)
        return np.asarray(x, dtype=np.float64)

    monkeypatch.setattr(da, "widen", bad)
    assert _failing_pins()


def test_mutant_rows_are_caught(monkeypatch):
    """Plausible mistakes in the one-by-one rows are each caught by a pin."""
    real = da.decode_attention_rows

    def neighbour_head(w, rows):  # the head next to the one asked for
        return real(w, [(b, (h + 1) % w.spec.num_q_heads) for b, h in rows])

    def no_fp8_scales(w, rows):  # FP8 codes attended without their per-tensor scales
        import dataclasses
        return real(dataclasses.replace(w, spec=w.spec.replace(k_scale=1.0, v_scale=1.0)), rows)

    def pages_as_packed(w, rows):  # the page pool read as if it were one packed cache
        import dataclasses
        if w.spec.layout != "paged":
            return real(w, rows)
        P, ps, Hkv, D = w.k_pages.shape
        starts = np.concatenate([[0], np.cumsum(w.ctx_lens)[:-1]]).astype(np.int64)
        flat = dataclasses.replace(w, spec=w.spec.replace(layout="contiguous", page_size=0),
                                   k=w.k_pages.reshape(P * ps, Hkv, D), v=w.v_pages.reshape(P * ps, Hkv, D),
                                   seq_start=np.minimum(starts, P * ps - np.maximum(w.ctx_lens, 1)))
        return real(flat, rows)

    def first_sequence(w, rows):  # every row attends over sequence 0
        return real(w, [(0, h) for _, h in rows])

    for fn in (neighbour_head, no_fp8_scales, pages_as_packed, first_sequence):
        monkeypatch.setattr(da, "decode_attention_rows", fn)
        assert "pin_rows_equal_reference" in _failing_pins(), fn.__name__


def test_mutant_cost_model_is_caught(monkeypatch):
    monkeypatch.setattr(cm, "max_compression_ratio", lambda W, Y, S, P: 1 / (1 + Y * S * P / W))
    assert _failing_pins()


def test_append_then_context_is_concatenation():
    """After appending, each sequence's logical context is the old one with the new row last (Sec. 2.2)."""
    spec = small_spec(WORKLOADS[4], [1, 16, 17, 40], seed=50, max_ctx_len=64)
    w = generate(spec, spare_pages=1)
    r = np.random.default_rng(50)
    new = f32_to_bf16_bits(r.standard_normal((4, spec.num_kv_heads, spec.head_dim)).astype(np.float32))
    grown = w.ctx_lens  # lengths count the new token: its row is the last one of each context
    after = da.append_paged(w.k_pages, w.block_table, grown, new)
    for b in range(4):
        before = da.paged_context(w.k_pages, w.block_table, grown, b)
        ctx = da.paged_context(after, w.block_table, grown, b)
        assert np.array_equal(ctx[:-1], before[:-1]) and np.array_equal(ctx[-1], new[b])
    # every other pool row is untouched
    changed = np.argwhere((after != w.k_pages).any(axis=(2, 3)))
    assert len(changed) <= 4
    spec_c = small_spec(WORKLOADS[2], [3, 0, 5], seed=51)
    wc = generate(spec_c, gap_rows=2)
    newc = f32_to_bf16_bits(r.standard_normal((3, 8, 128)).astype(np.float32))
    afterc = da.append_contiguous(wc.k, wc.seq_start, wc.ctx_lens, newc)
    assert np.array_equal(afterc[2], newc[0]) and np.array_equal(afterc[wc.seq_start[2] + 4], newc[2])
    mask = np.ones(len(afterc), bool)
    mask[[2, wc.seq_start[2] + 4]] = False
    assert np.array_equal(afterc[mask], wc.k[mask])
