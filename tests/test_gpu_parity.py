"""HIP path vs the fp64 oracle, element by element, through the C ABI.

Small cases span several 32-token tiles, several splits and ragged tails;
edge cases cover empty and one-token contexts, every supported GQA group and
head size, page sizes below and above a tile, NaN-poisoned memory outside the
contexts, strided (fused) K/V buffers and bitwise reproducibility.
"""

import numpy as np
import pytest

import oracle.decode_attention as da
from tests.gpu_util import DeviceWorkload, check, make_op, run, say
from workloads.synth import WORKLOADS, generate, small_spec

pytestmark = pytest.mark.gpu

RAGGED = [1, 31, 32, 33, 100, 1000, 4097]


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2605_30842_amd import binding

    binding.load_library()
    yield


def _case(spec, variant="auto", chunk=0, seed=None, **gen):
    w = generate(spec, seed=seed, **gen)
    say(f"case {spec.name} B={spec.batch} lens={w.ctx_lens.tolist()[:8]} G={spec.group} D={spec.head_dim} "
        f"{spec.dtype} {spec.layout} ps={spec.page_size} variant={variant} chunk={chunk}")
    dw = DeviceWorkload(w)
    op = make_op(spec, chunk=chunk, variant=variant)
    out, lse = run(dw, op)
    ref_out, ref_lse = da.reference(w)
    return w, dw, op, out, lse, ref_out, ref_lse


def test_fp32_tiny_workload():
    w, dw, op, out, lse, ro, rl = _case(WORKLOADS[1])
    check(out, lse, ro, rl, "f32", "fp32 L=2048")


@pytest.mark.parametrize("chunk", [0, 32, 64, 256])
def test_fp32_ragged(chunk):
    spec = small_spec(WORKLOADS[1], RAGGED, seed=21)
    _, _, _, out, lse, ro, rl = _case(spec, chunk=chunk)
    check(out, lse, ro, rl, "f32", f"fp32 ragged chunk={chunk}")


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
@pytest.mark.parametrize("chunk", [0, 32, 96, 256, 2048])
def test_bf16_ragged_contiguous(variant, chunk):
    spec = small_spec(WORKLOADS[2], RAGGED, seed=22)
    _, _, _, out, lse, ro, rl = _case(spec, variant=variant, chunk=chunk)
    check(out, lse, ro, rl, "bf16", f"bf16 ragged {variant} chunk={chunk}")


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
@pytest.mark.parametrize("G", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("D", [64, 128])
def test_groups_and_head_dims(variant, G, D):
    spec = small_spec(WORKLOADS[2], [5, 77, 700], seed=23 + G + D).replace(
        num_q_heads=2 * G, num_kv_heads=2, head_dim=D)
    _, _, _, out, lse, ro, rl = _case(spec, variant=variant, chunk=128)
    check(out, lse, ro, rl, "bf16", f"G={G} D={D} {variant}")


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid"])
@pytest.mark.parametrize("hkv", [1, 3, 5, 8, 12])
def test_kv_head_counts(variant, hkv):
    """KV head counts that do and do not divide the 8 XCDs: the grid form orders its workgroups
    head-major within a sequence, so every (split, head) pair must still be run exactly once."""
    spec = small_spec(WORKLOADS[2], [1, 700, 3000], seed=40 + hkv).replace(num_q_heads=2 * hkv, num_kv_heads=hkv)
    _, _, _, out, lse, ro, rl = _case(spec, variant=variant, chunk=128)
    check(out, lse, ro, rl, "bf16", f"Hkv={hkv} {variant}")


@pytest.mark.parametrize("G,D", [(4, 64), (8, 128), (16, 64)])
def test_fp32_groups(G, D):
    spec = small_spec(WORKLOADS[1], [3, 200], seed=24).replace(num_q_heads=2 * G, num_kv_heads=2, head_dim=D)
    _, _, _, out, lse, ro, rl = _case(spec, chunk=64)
    check(out, lse, ro, rl, "f32", f"fp32 G={G} D={D}")


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
@pytest.mark.parametrize("ps", [1, 8, 16, 64, 128])
def test_paged_small(variant, ps):
    spec = small_spec(WORKLOADS[4], RAGGED, seed=25 + ps, max_ctx_len=4224).replace(page_size=ps)
    _, _, _, out, lse, ro, rl = _case(spec, variant=variant, chunk=256, spare_pages=3)
    check(out, lse, ro, rl, "bf16", f"paged ps={ps} {variant}")


@pytest.mark.parametrize("ps", [1, 2])
def test_long_context_tiny_pages_planned(ps):
    """140000 tokens in 1- or 2-token pages: the planner shortens its 4096-token
    splits (to 2016 / 4064) so that a split's block-table entries fit the
    kernel's LDS copy; the result still matches the oracle."""
    spec = small_spec(WORKLOADS[4], [140000], seed=60 + ps).replace(page_size=ps)
    _, _, _, out, lse, ro, rl = _case(spec)
    check(out, lse, ro, rl, "bf16", f"long context, page size {ps}")


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
def test_empty_and_one_token(variant):
    spec = small_spec(WORKLOADS[2], [0, 1, 0, 1, 2], seed=26)
    w, _, _, out, lse, ro, rl = _case(spec, variant=variant)
    for b in (0, 2):
        assert np.array_equal(out[b], np.zeros_like(out[b])) and np.all(lse[b] == -np.inf)
    for b in (1, 3):
        v0 = da.widen(w.v[w.seq_start[b]], "bf16")  # [Hkv, D]
        assert np.array_equal(out[b].astype(np.float64), np.repeat(v0, spec.group, axis=0)), "L=1 must be exact"
    check(out, lse, ro, rl, "bf16", f"empty/one {variant}")


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
def test_zero_query_gives_mean_of_structured_values(variant):
    """q = 0: every weight equal, out = mean of V. V[t] = (t mod 97) / 32 is exact in bf16."""
    from workloads.synth import f32_to_bf16_bits

    L = 5000
    spec = small_spec(WORKLOADS[2], [L], seed=27)
    w = generate(spec)
    w.q[:] = 0
    vals = ((np.arange(L) % 97) / 32.0).astype(np.float32)
    w.v[:] = f32_to_bf16_bits(np.broadcast_to(vals[:, None, None], w.v.shape).copy())
    say(f"case q=0 structured V {variant}")
    op = make_op(spec, variant=variant, chunk=256)
    out, lse = run(DeviceWorkload(w), op)
    mean = float(np.sum(vals.astype(np.float64)) / L)
    assert np.abs(out - mean).max() <= 2e-6 * mean, np.abs(out - mean).max()
    assert np.abs(lse - np.log(L)).max() <= 1e-5


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
def test_nan_poison_outside_contexts(variant):
    spec = small_spec(WORKLOADS[2], [5, 33, 0, 300], seed=28)
    _, _, _, out, lse, ro, rl = _case(spec, variant=variant, chunk=64, gap_rows=40, poison=True)
    check(out, lse, ro, rl, "bf16", f"poison contiguous {variant}")
    spec = small_spec(WORKLOADS[4], [5, 33, 0, 300], seed=29, max_ctx_len=320).replace(page_size=16)
    _, _, _, out, lse, ro, rl = _case(spec, variant=variant, chunk=64, spare_pages=4, poison=True)
    check(out, lse, ro, rl, "bf16", f"poison paged {variant}")


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
@pytest.mark.parametrize("ps", [16, 64])
def test_paged_equals_contiguous_bitwise(variant, ps):
    """Same logical rows, same split plan: the paged and packed calls agree bit for bit."""
    import torch

    spec = small_spec(WORKLOADS[4], [17, 2048, 999, 64], seed=30, max_ctx_len=2048).replace(page_size=ps)
    w = generate(spec, spare_pages=2)
    say(f"case paged==contiguous ps={ps} {variant}")
    dwp = DeviceWorkload(w)
    op = make_op(spec, variant=variant, chunk=256)
    out_p, lse_p = run(dwp, op)
    lens = w.ctx_lens.astype(np.int64)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    kp = da.paged_context  # logical gather on the host
    k = np.concatenate([kp(w.k_pages, w.block_table, w.ctx_lens, b) for b in range(spec.batch)])
    v = np.concatenate([kp(w.v_pages, w.block_table, w.ctx_lens, b) for b in range(spec.batch)])
    wc = generate(spec.replace(layout="contiguous", page_size=0))
    wc.q[:] = w.q
    wc.k, wc.v, wc.seq_start, wc.ctx_lens = k, v, starts, w.ctx_lens
    out_c, lse_c = run(DeviceWorkload(wc), op)
    assert np.array_equal(out_p, out_c) and np.array_equal(lse_p, lse_c)
    torch.cuda.synchronize()


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
def test_bitwise_reproducible(variant):
    spec = small_spec(WORKLOADS[2], [4096, 3000, 77], seed=31)
    w = generate(spec)
    dw = DeviceWorkload(w)
    op = make_op(spec, variant=variant, chunk=128)
    say(f"case reproducible {variant}")
    first = run(dw, op)
    for _ in range(3):
        again = run(dw, op)
        assert np.array_equal(first[0], again[0]) and np.array_equal(first[1], again[1])


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
def test_fused_kv_buffer_strides(variant):
    """K and V interleaved in one [T, 2, Hkv, D] buffer: stride_token = 2 * Hkv * D."""
    import torch

    spec = small_spec(WORKLOADS[2], [300, 1, 129], seed=32)
    w = generate(spec)
    dw = DeviceWorkload(w)
    T = dw.k.shape[0]
    fused = torch.empty((T, 2, spec.num_kv_heads, spec.head_dim), dtype=dw.k.dtype, device=dw.k.device)
    fused[:, 0] = dw.k
    fused[:, 1] = dw.v
    dw.k, dw.v = fused[:, 0], fused[:, 1]
    op = make_op(spec, variant=variant, chunk=64)
    say(f"case fused kv {variant}")
    out, lse = run(dw, op)
    ro, rl = da.reference(w)
    check(out, lse, ro, rl, "bf16", f"fused kv {variant}")


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
def test_head_major_cache_strides(variant):
    """K and V stored head-major ([Hkv, T, D] per tensor) and passed as [T, Hkv, D] views
    (stride_token = D, stride_head = T * D): the same bits as the token-major cache."""
    spec = small_spec(WORKLOADS[2], [300, 1, 2100, 0, 129], seed=35)
    w = generate(spec)
    dw = DeviceWorkload(w)
    op = make_op(spec, variant=variant, chunk=128)
    say(f"case head-major cache {variant}")
    want = run(dw, op)
    dw.k = dw.k.permute(1, 0, 2).contiguous().permute(1, 0, 2)
    dw.v = dw.v.permute(1, 0, 2).contiguous().permute(1, 0, 2)
    assert dw.k.stride() == (spec.head_dim, dw.k.shape[0] * spec.head_dim, 1)
    got = run(dw, op)
    assert np.array_equal(want[0], got[0]) and np.array_equal(want[1], got[1])
    check(got[0], got[1], *da.reference(w), "bf16", f"head-major {variant}")


def test_workspace_reused_across_changing_calls():
    """Ticket counters return to zero: calls with different split counts share one workspace."""
    base = small_spec(WORKLOADS[2], [2000], seed=33, max_ctx_len=8192)
    op = make_op(base.replace(batch=3), chunk=64, max_batch=3, max_ctx_len=8192)
    for i, lens in enumerate([[2000, 5, 8192], [64, 65, 63], [8192, 8192, 8192], [1, 0, 4000], [2000]]):
        spec = small_spec(base, lens, seed=40 + i, max_ctx_len=8192)
        w = generate(spec)
        say(f"case workspace reuse call {i} lens={lens}")
        out, lse = run(DeviceWorkload(w), op, max_ctx_len=max(lens))
        ro, rl = da.reference(w)
        check(out, lse, ro, rl, "bf16", f"reuse call {i}")


def test_lse_optional():
    spec = small_spec(WORKLOADS[2], [100, 3000], seed=34)
    w = generate(spec)
    say("case lse=None")
    out, lse = run(DeviceWorkload(w), make_op(spec, chunk=256), want_lse=False)
    assert lse is None
    check(out, None, *da.reference(w), "bf16", "no lse")


def _tail_lengths(B, max_len, seed):
    """Ragged lengths with the cases of the short last splits: empty, one token,
    fewer than 4 splits (none short), exact multiples of the split, a ragged last tile."""
    r = np.random.default_rng(seed)
    lens = r.integers(1, max_len + 1, size=B)
    lens[:10] = [0, 1, 31, 1025, 3072, 3073, 4096, 4097, max_len, max_len - 1]
    return lens.tolist()


@pytest.mark.parametrize("base,ps", [(2, 0), (4, 16), (4, 64), (4, 2), (6, 0)])
def test_short_last_splits(base, ps):
    """Planned splits of 1024 tokens with 32 sequences x 8 KV heads x up to 8
    splits: at least 4 work items per resident workgroup, so each sequence of 4
    or more splits ends in short splits of 512 tokens that the queue hands out
    last (two per sequence on 256 compute units). Parity, then three more calls
    bit for bit equal."""
    import torch

    spec = small_spec(WORKLOADS[base], _tail_lengths(32, 8192, 36 + ps), seed=37 + base + ps, max_ctx_len=8192)
    if ps:
        spec = spec.replace(page_size=ps)
    op = make_op(spec)
    chunk, splits = op.splits(spec.batch, spec.max_ctx_len)
    resident = 2 * torch.cuda.get_device_properties(0).multi_processor_count
    assert chunk == 1024 and spec.batch * spec.num_kv_heads * splits >= 4 * resident
    w = generate(spec, spare_pages=2) if ps else generate(spec)
    dw = DeviceWorkload(w)
    say(f"case short last splits {spec.dtype} {spec.layout} ps={ps} lens={w.ctx_lens.tolist()[:10]}")
    first = run(dw, op)
    ro, rl = da.reference(w)
    check(*first, ro, rl, spec.dtype, f"short last splits {spec.layout} ps={ps}")
    for _ in range(3):
        again = run(dw, op)
        assert np.array_equal(first[0], again[0]) and np.array_equal(first[1], again[1])


@pytest.mark.parametrize("base,ps", [(2, 0), (4, 16), (4, 2)])
def test_short_last_splits_fused_append(base, ps):
    """The fused append under short last splits: the split that ends at L is a
    short one. One launch (store, then attend) leaves the same cache bits and
    output bits as the append call followed by the attention call."""
    import torch
    from workloads.synth import draw_new_rows
    from tests.gpu_util import to_torch

    spec = small_spec(WORKLOADS[base], _tail_lengths(32, 8191, 46 + ps), seed=47 + ps, max_ctx_len=8192)
    if ps:
        spec = spec.replace(page_size=ps)
    w = generate(spec, spare_pages=2) if ps else generate(spec)
    nk, nv = draw_new_rows(spec, seed=48 + ps)
    tk, tv = to_torch(nk, spec.dtype, "cuda:0"), to_torch(nv, spec.dtype, "cuda:0")
    a, b = DeviceWorkload(w), DeviceWorkload(w)
    op = make_op(spec)
    assert op.splits(spec.batch, spec.max_ctx_len)[0] == 1024
    say(f"case short last splits, fused append {spec.layout} ps={ps}")
    lse_a, lse_b = (torch.empty((spec.batch, spec.num_q_heads), dtype=torch.float32, device="cuda:0")
                    for _ in range(2))
    if ps:
        op.append_paged(tk, tv, a.k, a.v, a.block_table, a.ctx_lens, spec.max_ctx_len)
        out_a, _ = op.forward_paged(a.q, a.k, a.v, a.block_table, a.ctx_lens, spec.max_ctx_len, lse=lse_a)
        out_b, _ = op.append_forward_paged(b.q, tk, tv, b.k, b.v, b.block_table, b.ctx_lens, spec.max_ctx_len,
                                           lse=lse_b)
    else:
        op.append(tk, tv, a.k, a.v, a.seq_start, a.ctx_lens, spec.max_ctx_len)
        out_a, _ = op.forward(a.q, a.k, a.v, a.seq_start, a.ctx_lens, spec.max_ctx_len, lse=lse_a)
        out_b, _ = op.append_forward(b.q, tk, tv, b.k, b.v, b.seq_start, b.ctx_lens, spec.max_ctx_len, lse=lse_b)
    torch.cuda.synchronize()
    assert torch.equal(a.k, b.k) and torch.equal(a.v, b.v)
    assert torch.equal(out_a, out_b) and torch.equal(lse_a, lse_b)
    if ps:
        w.k_pages = da.append_paged(w.k_pages, w.block_table, w.ctx_lens, nk)
        w.v_pages = da.append_paged(w.v_pages, w.block_table, w.ctx_lens, nv)
        got_k = b.k.view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(got_k, w.k_pages)
    else:
        w.k = da.append_contiguous(w.k, w.seq_start, w.ctx_lens, nk)
        w.v = da.append_contiguous(w.v, w.seq_start, w.ctx_lens, nv)
        assert np.array_equal(b.k.view(torch.int16).cpu().numpy().view(np.uint16), w.k)
    ro, rl = da.reference(w)
    check(out_b.cpu().numpy(), lse_b.cpu().numpy(), ro, rl, spec.dtype, f"fused append, short splits ps={ps}")


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid", "valu"])
def test_split_merge_stress(variant):
    """Up to 256 splits per (sequence, KV head) and 16k workgroups: every split's
    partial result must reach the merging workgroup, call after call."""
    spec = small_spec(WORKLOADS[2], [8192, 4096, 8191, 33, 6000, 8192, 1, 7777], seed=35)
    w = generate(spec)
    dw = DeviceWorkload(w)
    op = make_op(spec, variant=variant, chunk=32)
    say(f"case split-merge stress {variant} splits={op.splits(spec.batch, spec.max_ctx_len)}")
    ro, rl = da.reference(w)
    first = run(dw, op)
    check(*first, ro, rl, "bf16", f"stress {variant}")
    for _ in range(4):
        again = run(dw, op)
        assert np.array_equal(first[0], again[0]) and np.array_equal(first[1], again[1])


@pytest.mark.parametrize("base,lens", [(2, [4100, 777, 1, 0]), (5, [3000, 65, 1]), (6, [4100, 777, 1]),
                                       (7, [3000, 65, 1])])
def test_kv_placement_gives_the_same_bits(base, lens):
    """The recommended placement (K and V in one buffer, V's base 256 bytes past
    K's modulo 512) changes only where the rows sit: the outputs equal those of
    two separate allocations bit for bit, and pass the gate."""
    import torch

    from paper_2605_30842_amd import binding

    spec = small_spec(WORKLOADS[base], lens, seed=41 + base)
    w = generate(spec)
    dw = DeviceWorkload(w)
    op = make_op(spec)
    say(f"case kv placement workload {base} {spec.dtype} {spec.layout} lens={lens}")
    separate = run(dw, op)
    k, v = binding.kv_cache_pair(tuple(dw.k.shape), dw.k.dtype, dw.k.device)
    k.copy_(dw.k)
    v.copy_(dw.v)
    assert (v.data_ptr() - k.data_ptr()) % 512 == 256
    dw.k, dw.v = k, v
    placed = run(dw, op)
    assert np.array_equal(separate[0], placed[0]) and np.array_equal(separate[1], placed[1])
    ro, rl = da.reference(w)
    check(*placed, ro, rl, spec.dtype, f"placement workload {base}")
    torch.cuda.synchronize()
