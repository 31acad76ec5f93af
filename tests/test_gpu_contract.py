"""Device-side contract violations, through the C ABI: no access outside the
pool or the workspace, the documented result, and the debug error word.

A length outside [0, max_ctx_len] is clamped into it; a block-table entry
outside [0, num_pages) is read as page 0 and never written through. The
expected values are the oracle's on the same inputs with those two rules
applied (the clamped length, page 0 in place of the bad entry), so every
check below is exact against the oracle. With debug checks the plan's error
word reports each kind of violation; without them it stays zero.
"""

import copy

import numpy as np
import pytest

import oracle.decode_attention as da
import oracle.prefill_attention as pa
from paper_2605_30842_amd import binding as B
from tests.gpu_util import (DevicePrefill, DeviceWorkload, abs_values, check, check_prefill, make_op, run,
                            run_prefill, say, to_torch)
from workloads.synth import PREFILL_WORKLOADS, WORKLOADS, generate, generate_prefill, small_prefill_spec, small_spec

pytestmark = pytest.mark.gpu

VARIANTS = ["mfma", "mfma_grid", "valu"]


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.load_library()
    yield


@pytest.mark.parametrize("debug", [False, True])
@pytest.mark.parametrize("variant", VARIANTS)
def test_length_above_max_ctx_len_is_clamped(variant, debug):
    """ctx_lens[1] = 5000 with max_ctx_len = 4096: that sequence attends over its first 4096 tokens."""
    spec = small_spec(WORKLOADS[2], [300, 5000, 100], seed=71)
    w = generate(spec)
    say(f"contract: length 5000 > max 4096, {variant}, debug={debug}")
    dw = DeviceWorkload(w)
    op = make_op(spec, variant=variant, max_ctx_len=4096, debug_checks=debug)
    out, lse = run(dw, op, max_ctx_len=4096)
    want = copy.copy(w)
    want.ctx_lens = np.minimum(w.ctx_lens, 4096)
    ro, rl = da.reference(want)
    check(out, lse, ro, rl, "bf16", f"clamped length {variant}")
    assert op.device_errors() == (B.DEVICE_ERR_CTX_LEN if debug else 0)
    assert op.device_errors() == 0  # read and cleared


@pytest.mark.parametrize("variant", VARIANTS)
def test_negative_length_is_an_empty_context(variant):
    import torch

    spec = small_spec(WORKLOADS[2], [0, 200, 33], seed=72)
    w = generate(spec)
    say(f"contract: negative length, {variant}")
    dw = DeviceWorkload(w)
    dw.ctx_lens[0] = -5
    op = make_op(spec, variant=variant, debug_checks=True)
    out, lse = run(dw, op)
    assert np.all(out[0] == 0) and np.all(lse[0] == -np.inf)
    ro, rl = da.reference(w)
    check(out, lse, ro, rl, "bf16", f"negative length {variant}")
    assert op.device_errors() == B.DEVICE_ERR_CTX_LEN
    torch.cuda.synchronize()


@pytest.mark.parametrize("debug", [False, True])
@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("ps", [1, 16, 64])
def test_block_table_entry_outside_the_pool_reads_page_zero(ps, variant, debug):
    spec = small_spec(WORKLOADS[4], [300, 700, 50], seed=73 + ps, max_ctx_len=768).replace(page_size=ps)
    w = generate(spec)
    say(f"contract: bad block-table entries, ps={ps} {variant} debug={debug}")
    dw = DeviceWorkload(w)
    num_pages = w.k_pages.shape[0]
    bad = {(1, 3 * 16 // ps): num_pages + 7, (2, 0): -2}  # entries the two sequences do read
    want = copy.copy(w)
    want.block_table = w.block_table.copy()
    for (b, i), page in bad.items():
        dw.block_table[b, i] = page
        want.block_table[b, i] = 0
    op = make_op(spec, variant=variant, debug_checks=debug)
    out, lse = run(dw, op)
    ro, rl = da.reference(want)
    check(out, lse, ro, rl, "bf16", f"bad entries ps={ps} {variant}")
    assert op.device_errors() == (B.DEVICE_ERR_BLOCK_TABLE if debug else 0)


@pytest.mark.parametrize("layout_base", [2, 4])
def test_fused_append_never_writes_through_a_violation(layout_base):
    """The fused append skips the store of a sequence whose length was clamped
    or whose last token's entry lies outside the pool; other sequences store."""
    import torch

    kw = {"max_ctx_len": 320} if layout_base == 4 else {}
    spec = small_spec(WORKLOADS[layout_base], [100, 300, 64], seed=74, **kw)
    w = generate(spec)
    say(f"contract: fused append with violations, {spec.layout}")
    from workloads.synth import draw_new_rows

    nk, nv = draw_new_rows(spec, seed=75)
    dw = DeviceWorkload(w)
    tk, tv = to_torch(nk, "bf16", "cuda:0"), to_torch(nv, "bf16", "cuda:0")
    op = make_op(spec, chunk=64, debug_checks=True)
    k0, v0 = dw.k.clone(), dw.v.clone()
    if spec.layout == "paged":
        last = (int(w.ctx_lens[1]) - 1) // spec.page_size
        dw.block_table[1, last] = 10**6
        op.append_forward_paged(dw.q, tk, tv, dw.k, dw.v, dw.block_table, dw.ctx_lens, spec.max_ctx_len)
        lens = w.ctx_lens.copy()
        lens[1] = 0  # no append for sequence 1
        want_k = da.append_paged(w.k_pages, w.block_table, lens, nk)
        want_v = da.append_paged(w.v_pages, w.block_table, lens, nv)
        err = B.DEVICE_ERR_BLOCK_TABLE
    else:
        dw.ctx_lens[1] = 301  # one past max_ctx_len = 300: clamped, so no store for sequence 1
        op.append_forward(dw.q, tk, tv, dw.k, dw.v, dw.seq_start, dw.ctx_lens, spec.max_ctx_len)
        lens = w.ctx_lens.copy()
        lens[1] = 0  # no append for sequence 1
        want_k = da.append_contiguous(w.k, w.seq_start, lens, nk)
        want_v = da.append_contiguous(w.v, w.seq_start, lens, nv)
        err = B.DEVICE_ERR_CTX_LEN
    torch.cuda.synchronize()
    assert np.array_equal(dw.k.view(torch.int16).cpu().numpy(), want_k.view(np.int16))
    assert np.array_equal(dw.v.view(torch.int16).cpu().numpy(), want_v.view(np.int16))
    assert not torch.equal(dw.k, k0) and not torch.equal(dw.v, v0)  # the other sequences did store
    assert op.device_errors() == err


def test_debug_checks_need_a_workspace():
    import torch

    spec = small_spec(WORKLOADS[2], [10], seed=76)
    op = make_op(spec, debug_checks=True)
    dw = DeviceWorkload(generate(spec))
    out = torch.empty((1, 32, 128), dtype=torch.float32, device="cuda:0")
    st = B.load_library().comem_decode_attn(op.plan, dw.q.data_ptr(), dw.k.data_ptr(), dw.v.data_ptr(), 8 * 128,
                                            128, dw.seq_start.data_ptr(), dw.ctx_lens.data_ptr(), 1, 10,
                                            out.data_ptr(), None, None, 0, None)
    assert st == B.ERR_NULL_POINTER  # rejected on the host: nothing is launched


@pytest.mark.parametrize("ps", [1, 16])
def test_prefill_block_table_entry_outside_the_pool_reads_page_zero(ps):
    spec = small_prefill_spec(PREFILL_WORKLOADS[3], [200, 500], [50, 120], seed=77 + ps, max_ctx_len=512)
    spec = spec.__class__(spec.name, spec.kv.replace(page_size=ps), spec.new_tokens, spec.seed)
    pw = generate_prefill(spec)
    say(f"contract: prefill, bad block-table entries, ps={ps}")
    dp = DevicePrefill(pw)
    num_pages = pw.kv.k_pages.shape[0]
    want = copy.deepcopy(pw)
    for (b, i), page in {(0, 0): -9, (1, 100 // ps): num_pages}.items():
        dp.kv.block_table[b, i] = page
        want.kv.block_table[b, i] = 0
    out, lse = run_prefill(dp, make_op(pw.kv.spec))
    ro, rl = pa.reference(want)
    ra, _ = pa.reference(abs_values(want))
    check_prefill(out, lse, ro, rl, ra, f"prefill bad entries ps={ps}")
