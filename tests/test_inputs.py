"""Checks of the seeded workload generator (no attention arithmetic involved)."""

import numpy as np
import pytest
import torch

from workloads import synth
from workloads.synth import WORKLOADS, f32_to_bf16_bits, generate, small_spec


def test_bf16_rne_matches_torch_bitwise():
    r = np.random.default_rng(0)
    x = np.concatenate([
        r.standard_normal(1 << 16).astype(np.float32),
        (r.standard_normal(4096) * 1e30).astype(np.float32),
        (r.standard_normal(4096) * 1e-38).astype(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 3.3895314e38], np.float32),
    ])
    # ties: mantissa low half exactly 0x8000
    ties = (r.integers(0, 1 << 15, 2048, dtype=np.uint32) << 16 | 0x8000).view(np.float32)
    x = np.concatenate([x, ties[np.isfinite(ties)]])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(f32_to_bf16_bits(x), ref)
    nan = f32_to_bf16_bits(np.array([np.nan], np.float32))
    assert (nan[0] & 0x7F80) == 0x7F80 and (nan[0] & 0x7F) != 0


def test_scale_by_8_commutes_with_cast():
    r = np.random.default_rng(1)
    x = r.standard_normal(1 << 16).astype(np.float32)
    a = f32_to_bf16_bits(x * np.float32(8))
    b = (f32_to_bf16_bits(x).astype(np.uint32) << 16).view(np.float32) * np.float32(8)
    assert np.array_equal(a, f32_to_bf16_bits(b))


def test_deterministic_and_thread_independent(monkeypatch):
    spec = small_spec(WORKLOADS[3], [3000, 70, 2100], seed=5)
    a = generate(spec)
    monkeypatch.setattr(synth, "_THREADS", 1)
    b = generate(spec)
    for name in ("q", "k", "v", "ctx_lens", "seq_start"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
    c = generate(spec, seed=6)
    assert not np.array_equal(a.k, c.k)


def test_named_workload_shapes():
    w = generate(WORKLOADS[1])
    assert w.q.shape == (1, 8, 64) and w.q.dtype == np.float32
    assert w.k.shape == (2048, 2, 64) and w.ctx_lens.tolist() == [2048]
    s = WORKLOADS[3]
    lens = synth.draw_lengths(s, np.random.default_rng(np.random.SeedSequence(s.seed).spawn(6)[0]))
    assert lens.shape == (16,) and lens.min() >= 4096 and lens.max() <= 65536
    assert WORKLOADS[5].group == 8 and WORKLOADS[2].group == 4
    assert WORKLOADS[2].scale == np.float32(1 / np.sqrt(128))


def test_paged_block_table_is_a_permutation_of_the_pool():
    spec = small_spec(WORKLOADS[4], [2048, 17, 1, 4000], seed=9, max_ctx_len=16384)
    w = generate(spec, spare_pages=5)
    ps = spec.page_size
    need = [(-(-int(L) // ps)) for L in w.ctx_lens]
    used = np.concatenate([w.block_table[b, :n] for b, n in enumerate(need)])
    assert sorted(used.tolist()) == sorted(set(used.tolist()))
    assert used.min() >= 0 and used.max() < w.k_pages.shape[0]
    assert w.k_pages.shape[0] == sum(need) + 5
    for b, n in enumerate(need):
        assert np.all(w.block_table[b, n:] == -1)
    assert w.block_table.shape == (4, 1024)


def test_key_scale_fraction():
    spec = WORKLOADS[4]
    small = small_spec(spec, [16384] * 4, seed=3)
    w = generate(small)
    seqs = np.random.SeedSequence(small.seed).spawn(6)
    pool_rows = w.k_pages.shape[0] * spec.page_size * spec.num_kv_heads
    frac = (np.random.default_rng(seqs[5]).random(pool_rows) < 0.05).mean()
    assert abs(frac - 0.05) < 0.005
    # the scaled rows are exactly 8x an N(0,1) draw: their spread is 8x larger
    kf = (w.k_pages.astype(np.uint32) << 16).view(np.float32).reshape(-1, 128)
    big = np.abs(kf).max(axis=1) > 6
    assert 0.03 < big.mean() < 0.06


def test_poison_marks_exactly_the_uncovered_rows():
    spec = small_spec(WORKLOADS[4], [5, 16, 33], seed=4, max_ctx_len=64)
    w = generate(spec, spare_pages=2, poison=True)
    nan_rows = np.isnan((w.k_pages.astype(np.uint32) << 16).view(np.float32)).all(axis=-1)
    # covered rows: 5 + 16 + 33 tokens x 8 heads are finite; the rest is NaN
    assert (~nan_rows).sum() == (5 + 16 + 33) * spec.num_kv_heads
    spec_c = small_spec(WORKLOADS[2], [3, 4], seed=4)
    wc = generate(spec_c, gap_rows=2, poison=True)
    assert wc.k.shape[0] == 3 + 4 + 4 and wc.seq_start.tolist() == [0, 5]
    assert np.isnan((wc.k.astype(np.uint32) << 16).view(np.float32)[[3, 4, 9, 10]]).all()


@pytest.mark.parametrize("i", [2, 3])
def test_kv_bytes_formula(i):
    spec = WORKLOADS[i]
    lens = synth.draw_lengths(spec, np.random.default_rng(np.random.SeedSequence(spec.seed).spawn(6)[0]))
    assert int(lens.sum()) * 8 * 128 * 2 * 2 == (134217728 if i == 2 else int(lens.sum()) * 4096)


def test_prefill_workloads_recipe():
    """New-token counts stay within the context, queries are packed, and the K/V side equals the decode draw."""
    from workloads.synth import PREFILL_WORKLOADS, generate, generate_prefill, small_prefill_spec

    spec = small_prefill_spec(PREFILL_WORKLOADS[3], [40, 7, 300], [50, 7, 128], seed=9)
    pw = generate_prefill(spec)
    assert pw.q_lens.tolist() == [40, 7, 128]  # capped at L_b
    assert pw.q_start.tolist() == [0, 40, 47]
    assert pw.q.shape == (175, 32, 128) and pw.q.dtype == np.uint16
    again = generate_prefill(spec)
    assert np.array_equal(again.q, pw.q)
    kv = generate(spec.kv, seed=9)
    assert np.array_equal(kv.k_pages, pw.kv.k_pages) and np.array_equal(kv.block_table, pw.kv.block_table)
    full = generate_prefill(PREFILL_WORKLOADS[2].__class__(
        "x", PREFILL_WORKLOADS[2].kv.replace(lengths=("fixed", 64), max_ctx_len=64), ("all",), seed=4))
    assert full.q_lens.tolist() == [64]
    assert full.score_count == 64 * 65 // 2
