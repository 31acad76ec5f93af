"""Prefill attention over a cached prefix: HIP path vs the fp64 oracle, through the C ABI.

Small cases cover ragged batches of cached and uncached prefills with partial
key tiles and partial query blocks, every GQA group and head size, page sizes
below and above a tile, and NaN-poisoned memory outside the contexts; the
three named prefill workloads are checked on sampled rows at full size.
Every element must meet the official bf16 gate and the bound that splitting
the probabilities into two bf16 implies (see tests/gpu_util.check_prefill).
"""

import numpy as np
import pytest

import oracle.decode_attention as da
import oracle.prefill_attention as pa
from tests.gpu_util import (DevicePrefill, DeviceWorkload, abs_values, check_prefill, make_op, run, run_prefill,
                            say)
from workloads.synth import PREFILL_WORKLOADS, WORKLOADS, generate, generate_prefill, small_prefill_spec

pytestmark = pytest.mark.gpu

# (cached tokens L_b, new tokens M_b): long prefix + few new, uncached (M = L), single tokens, partial tiles
RAGGED_L = [40, 7, 1, 64, 300, 1000, 129, 2100]
RAGGED_M = [5, 7, 1, 16, 129, 1000, 33, 70]


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2605_30842_amd import binding

    binding.load_library()
    yield


def _prefill_case(spec, **gen):
    pw = generate_prefill(spec, **gen)
    s = pw.kv.spec
    say(f"prefill case {spec.name} B={s.batch} L={pw.kv.ctx_lens.tolist()[:8]} M={pw.q_lens.tolist()[:8]} "
        f"G={s.group} D={s.head_dim} {s.layout} ps={s.page_size}")
    dp = DevicePrefill(pw)
    op = make_op(s)
    out, lse = run_prefill(dp, op)
    ref_out, ref_lse = pa.reference(pw)
    ref_abs, _ = pa.reference(abs_values(pw))
    return pw, dp, op, out, lse, ref_out, ref_lse, ref_abs


def test_ragged_contiguous():
    spec = small_prefill_spec(PREFILL_WORKLOADS[1], RAGGED_L, RAGGED_M, seed=51)
    *_, out, lse, ro, rl, ra = _prefill_case(spec)
    err = check_prefill(out, lse, ro, rl, ra, "ragged contiguous")
    say(f"max |err| {err:.2e}")


@pytest.mark.parametrize("G", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("D", [64, 128])
def test_groups_and_head_dims(G, D):
    spec = small_prefill_spec(PREFILL_WORKLOADS[1], [200, 77, 500], [200, 3, 150], seed=52 + G + D)
    spec = spec.__class__(spec.name, spec.kv.replace(num_q_heads=2 * G, num_kv_heads=2, head_dim=D),
                          spec.new_tokens, spec.seed)
    *_, out, lse, ro, rl, ra = _prefill_case(spec)
    check_prefill(out, lse, ro, rl, ra, f"G={G} D={D}")


@pytest.mark.parametrize("ps", [1, 2, 4, 8, 16, 64, 128])
def test_paged_with_poison(ps):
    spec = small_prefill_spec(PREFILL_WORKLOADS[3], RAGGED_L, RAGGED_M, seed=53 + ps, max_ctx_len=2176)
    spec = spec.__class__(spec.name, spec.kv.replace(page_size=ps), spec.new_tokens, spec.seed)
    *_, out, lse, ro, rl, ra = _prefill_case(spec, spare_pages=3, poison=True)
    check_prefill(out, lse, ro, rl, ra, f"paged ps={ps} poisoned")


@pytest.mark.parametrize("ps", [0, 16, 8, 1])
def test_grid_sizes(ps):
    """The same sequences (uncached, long-prefix, one-tile and odd tile counts) in a grid that fits the
    compute units at once (6 sequences, 240 workgroups) and inside a batch of 48 (one workgroup per
    sequence and KV head, over 256 workgroups, which the GPU runs in turns) match the oracle. Both halves
    of each workgroup's key tiles see every kind of tile: the first, a masked last one, one past the
    keys. ps: 0 for the contiguous cache, else the page size (pages of 8 and 1 tokens take per-lane
    addresses)."""
    paged = ps > 0
    lens = [1, 64, 65, 700, 300, 129]
    news = [1, 64, 33, 31, 150, 2]
    base = PREFILL_WORKLOADS[3 if paged else 1]
    def with_pages(spec):
        return spec.__class__(spec.name, spec.kv.replace(page_size=ps), spec.new_tokens, spec.seed) if paged else spec
    small = with_pages(small_prefill_spec(base, lens, news, seed=58, **({"max_ctx_len": 704} if paged else {})))
    r = np.random.default_rng(59)
    big_l = lens + [int(x) for x in r.integers(1, 400, size=42)]
    big_m = news + [int(min(L, m)) for L, m in zip(big_l[len(lens):], r.integers(1, 33, size=42))]
    big = with_pages(small_prefill_spec(base, big_l, big_m, seed=58, **({"max_ctx_len": 704} if paged else {})))
    def workgroups(spec):  # grid: blocks of 128 / G new tokens x KV heads x sequences
        return -(-max(spec.new_tokens[1]) // (128 // spec.kv.group)) * spec.kv.num_kv_heads * spec.kv.batch

    assert workgroups(small) <= 256 < workgroups(big)
    for spec in (small, big):
        # Paged: spare pages poisoned with NaN, so a read outside the block table's pages would show.
        _, _, _, out, lse, ro, rl, ra = _prefill_case(spec, **({"spare_pages": 3, "poison": True} if paged else {}))
        check_prefill(out, lse, ro, rl, ra, f"{f'paged ps={ps}' if paged else 'contiguous'} B={spec.kv.batch}")


def test_contiguous_gaps_poisoned():
    spec = small_prefill_spec(PREFILL_WORKLOADS[1], [65, 130, 1], [65, 2, 1], seed=54)
    *_, out, lse, ro, rl, ra = _prefill_case(spec, gap_rows=50, poison=True)
    check_prefill(out, lse, ro, rl, ra, "contiguous gaps poisoned")


def test_zero_query_gives_mean_over_visible_prefix():
    """q = 0: every visible key has weight exactly 1, so new token i gets the mean of V[0 .. L - M + i].
    V[t] = (t mod 97) / 32 makes every partial sum exact in fp32: an off-by-one in the causal limit moves
    the mean by far more than the rounding of the final division."""
    from workloads.synth import f32_to_bf16_bits

    L, M = 1500, 300
    spec = small_prefill_spec(PREFILL_WORKLOADS[1], [L], [M], seed=55)
    pw = generate_prefill(spec)
    pw.q[:] = 0
    vals = ((np.arange(L) % 97) / 32.0).astype(np.float32)
    pw.kv.v[:] = f32_to_bf16_bits(np.broadcast_to(vals[:, None, None], pw.kv.v.shape).copy())
    say("prefill case q=0 structured V")
    out, lse = run_prefill(DevicePrefill(pw), make_op(pw.kv.spec))
    csum = np.cumsum(vals.astype(np.float64))
    for i in range(M):
        n = L - M + i + 1
        want = csum[n - 1] / n
        assert np.abs(out[i] - want).max() <= 2e-6 * max(want, 1e-3), (i, out[i, 0, 0], want)
        assert np.abs(lse[i] - np.log(n)).max() <= 1e-5


@pytest.mark.parametrize("D", [64, 128])
def test_tile_probability_sums_around_the_lazy_bound(D):
    """Scores built so that the vector stage takes each of its paths: a tile whose probabilities against
    the running maximum all stay below 1 (kept at the first try), a tile whose probabilities are about 8
    each, so a lane's sum passes 2^8 while no probability does (taken again, no rescale), and a tile whose
    scores jump by more than 8 in log2 units (taken again, rescaled). q is zero except head_dim 0, so a
    key's score is q0 * K[t, hk, 0]: the value of K[., ., 0] per 64-key tile sets the pattern, in both
    halves of the key tiles (16 tiles, the last one partial and masked)."""
    from workloads.synth import f32_to_bf16_bits

    L, M = 1000, 40
    spec = small_prefill_spec(PREFILL_WORKLOADS[1], [L], [M], seed=60)
    spec = spec.__class__(spec.name, spec.kv.replace(head_dim=D), spec.new_tokens, spec.seed)
    pw = generate_prefill(spec)
    c = float(pw.kv.spec.scale) * np.log2(np.e)  # log2 units per unit of score
    # Tile levels in log2 units, relative to the start: 0, +3.1 (kept after a second try), +12.5 (rescale),
    # equal (kept), back to 0 (kept), +3.1 above the new maximum twice (second try), +14.5 (rescale).
    levels = np.array([0.0, 3.1, 12.5, 12.5, 0.0, 15.6, 15.6, 27.0] * 2)
    k0 = f32_to_bf16_bits((levels / c).astype(np.float32)).astype(np.uint16)
    k0f = (k0.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert 32 * 2.0 ** ((k0f[1] - k0f[0]) * c) > 256 > 2.0 ** ((k0f[1] - k0f[0]) * c)
    assert 32 * 2.0 ** ((k0f[5] - k0f[2]) * c) > 256 > 2.0 ** ((k0f[5] - k0f[2]) * c)
    assert (k0f[2] - k0f[1]) * c > 8 and (k0f[7] - k0f[5]) * c > 8
    pw.q[:] = 0
    pw.q[:, :, 0] = f32_to_bf16_bits(np.ones(1, np.float32))[0]
    pw.kv.k[:L, :, 0] = k0[np.arange(L) // 64][:, None]
    say(f"prefill case lazy-bound tiles D={D}")
    dp = DevicePrefill(pw)
    out, lse = run_prefill(dp, make_op(pw.kv.spec))
    ro, rl = pa.reference(pw)
    ra, _ = pa.reference(abs_values(pw))
    check_prefill(out, lse, ro, rl, ra, f"lazy-bound tiles D={D}")


def test_single_new_token_matches_decode():
    """M_b = 1 is a decode step: the prefill kernel agrees with the oracle and with the decode kernel."""
    lens = [1, 33, 700, 4097]
    spec = small_prefill_spec(PREFILL_WORKLOADS[1], lens, [1] * len(lens), seed=56)
    pw, dp, op, out, lse, ro, rl, ra = _prefill_case(spec)
    check_prefill(out, lse, ro, rl, ra, "M=1")
    w = pw.kv
    w.q[:] = pw.q  # one new token per sequence: the decode query rows
    dout, dlse = run(DeviceWorkload(w), make_op(w.spec))
    dref, _ = da.reference(w)
    assert np.abs(dout - dref).max() <= 1e-4 * max(1.0, np.abs(dref).max())
    bound = 2 * 2.0 ** -15 * np.asarray(ra) + 1e-5 * np.abs(ro) + 1e-6
    assert np.all(np.abs(out - dout) <= 2 * bound)
    assert np.abs(lse - dlse).max() <= 2e-5 * max(1.0, np.abs(dlse).max())


def test_rows_outside_the_call_untouched_and_reproducible():
    """Sequences with no new tokens write nothing; rows past the packed queries keep their contents;
    two runs agree bit for bit."""
    import torch

    spec = small_prefill_spec(PREFILL_WORKLOADS[1], [100, 50, 300], [0, 50, 7], seed=57)
    pw = generate_prefill(spec)
    say("prefill case untouched rows")
    dp = DevicePrefill(pw)
    op = make_op(pw.kv.spec)
    total = dp.q.shape[0]
    out = torch.full((total + 5, pw.kv.spec.num_q_heads, pw.kv.spec.head_dim), 7.0, dtype=torch.float32,
                     device=dp.q.device)
    a, _ = run_prefill(dp, op, out=out[:total])
    b, _ = run_prefill(dp, op, out=out[:total])
    assert np.array_equal(a, b)
    tail = out[total:].cpu().numpy()
    assert np.all(tail == 7.0)
    ro, rl = pa.reference(pw)
    ra, _ = pa.reference(abs_values(pw))
    check_prefill(a, None, ro, rl, ra, "untouched rows")


@pytest.mark.parametrize("n", [1, 2, 3])
def test_named_workload_sampled_rows(n):
    """Full-size workload, checked on sampled rows (first, last and random new tokens and heads)."""
    pw = generate_prefill(PREFILL_WORKLOADS[n])
    s = pw.kv.spec
    say(f"prefill workload {PREFILL_WORKLOADS[n].name}: B={s.batch} total new {int(pw.q_lens.sum())}")
    dp = DevicePrefill(pw)
    out, lse = run_prefill(dp, make_op(s))
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse))
    rng = np.random.default_rng(58 + n)
    rows = []
    for b in range(s.batch):
        M = int(pw.q_lens[b])
        for i in sorted({0, M - 1, *rng.integers(0, M, 2).tolist()}):
            rows.append((b, int(i), int(rng.integers(0, s.num_q_heads))))
    got = pa.prefill_attention_rows(pw, rows)
    got_abs = pa.prefill_attention_rows(abs_values(pw), rows)
    for (b, i, h), (ro, rl), (ra, _) in zip(rows, got, got_abs):
        r = int(pw.q_start[b]) + i
        check_prefill(out[r, h][None], lse[r, h][None], ro[None], np.array([rl]), ra[None], f"row {(b, i, h)}")


@pytest.mark.parametrize("base", [1, 3])
def test_kv_placement_gives_the_same_bits(base):
    """K and V carved from one allocation with V's base 256 bytes past K's
    modulo 512 (how the bench places them) give the same bits as two separate
    allocations, contiguous and paged."""
    import torch

    from paper_2605_30842_amd import binding

    spec = small_prefill_spec(PREFILL_WORKLOADS[base], RAGGED_L, RAGGED_M, seed=57 + base)
    pw, dp, op, out, lse, ro, rl, ra = _prefill_case(spec)
    k, v = binding.kv_cache_pair(tuple(dp.kv.k.shape), dp.kv.k.dtype, dp.kv.k.device)
    k.copy_(dp.kv.k)
    v.copy_(dp.kv.v)
    assert (v.data_ptr() - k.data_ptr()) % 512 == 256
    dp.kv.k, dp.kv.v = k, v
    out2, lse2 = run_prefill(dp, op)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)
    check_prefill(out2, lse2, ro, rl, ra, f"placement prefill {base}")
    torch.cuda.synchronize()
