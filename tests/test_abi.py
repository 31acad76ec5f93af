"""C-ABI checks that need no GPU: exported symbols and host-side validation.

Every call here uses a plan made with COMEM_NO_DEVICE, so nothing reaches the
HIP runtime: argument errors come back before any HIP call, and a call whose
arguments are all valid stops with COMEM_ERR_NO_DEVICE.
"""

import ctypes
import os
import re

import pytest

from paper_2605_30842_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("comem_decode_attn.h", "comem_prefill_attn.h")]

A = 1 << 20  # a 256-byte aligned fake device address (never dereferenced)


def _declared_functions():
    names = set()
    for header in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(header).read(), flags=re.S)
        names |= set(re.findall(r"\b(comem_[a-z_]+)\s*\(", text))
    return sorted(names)


def test_header_declares_what_the_binding_expects():
    assert _declared_functions() == sorted(B.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = B.load_library()
    for name in _declared_functions():
        assert hasattr(lib, name), name


def test_probe_library_exports_its_header():
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "comem_probe.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(comem_[a-z_]+)\s*\(", text)))
    assert names == sorted(B.PROBE_EXPORTED)
    lib = B.load_probe_library()
    for name in names:
        assert hasattr(lib, name), name


def test_probe_read_kv_heads_rejects_bad_arguments():
    """Every argument rule of the pattern-read probe is checked on the host, before any launch
    (hipErrorInvalidValue = 1); the pointers are never dereferenced on the host."""
    lib = B.load_probe_library()
    k, v, sink = 1 << 20, 2 << 20, 3 << 20
    good = dict(k=k, v=v, tokens=32768, kv_heads=8, head_bytes=256, stride_token=2048, chunk=1024, sink=sink)
    bad = [dict(k=0), dict(v=0), dict(sink=0), dict(head_bytes=64), dict(head_bytes=512), dict(chunk=0),
           dict(chunk=96), dict(tokens=0), dict(tokens=1000), dict(kv_heads=0), dict(stride_token=1024),
           dict(stride_token=2056), dict(k=k + 8), dict(v=v + 4), dict(kv_heads=70000, stride_token=70000 * 256),
           dict(tokens=1 << 31, chunk=128, kv_heads=2, stride_token=512)]
    for change in bad:
        a = dict(good, **change)
        st = lib.comem_probe_read_kv_heads(a["k"], a["v"], a["tokens"], a["kv_heads"], a["head_bytes"],
                                           a["stride_token"], a["chunk"], a["sink"], None)
        assert st == 1, change


def _cfg(**kw):
    base = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype=B.BF16, scale=0.088, max_batch=4,
                max_ctx_len=4096, chunk_tokens=0, variant=B.VARIANT_AUTO, k_scale=1.0, v_scale=1.0)
    base.update(kw)
    return B.Config(**base)


def _status_init(cfg, device=B.NO_DEVICE):
    plan = ctypes.c_void_p()
    ws = ctypes.c_size_t()
    st = B.load_library().comem_decode_attn_init(ctypes.byref(cfg), device, ctypes.byref(plan), ctypes.byref(ws))
    if st == B.OK:
        B.comem_decode_attn_destroy(plan.value)
    return st


@pytest.mark.parametrize("kw,status", [
    (dict(num_q_heads=0), B.ERR_INVALID_SHAPE),
    (dict(num_kv_heads=0), B.ERR_INVALID_SHAPE),
    (dict(num_q_heads=30), B.ERR_INVALID_SHAPE),
    (dict(num_q_heads=24, num_kv_heads=8), B.ERR_UNSUPPORTED),  # G = 3
    (dict(num_q_heads=256, num_kv_heads=8), B.ERR_UNSUPPORTED),  # G = 32
    (dict(head_dim=96), B.ERR_UNSUPPORTED),
    (dict(dtype=7), B.ERR_UNSUPPORTED),
    (dict(scale=0.0), B.ERR_INVALID_SHAPE),
    (dict(scale=float("nan")), B.ERR_INVALID_SHAPE),
    (dict(max_batch=0), B.ERR_INVALID_SHAPE),
    (dict(max_batch=70000), B.ERR_INVALID_SHAPE),
    (dict(max_ctx_len=0), B.ERR_INVALID_SHAPE),
    (dict(max_ctx_len=(1 << 30) + 1), B.ERR_INVALID_SHAPE),
    (dict(chunk_tokens=48), B.ERR_INVALID_SHAPE),
    (dict(chunk_tokens=-32), B.ERR_INVALID_SHAPE),
    (dict(variant=9), B.ERR_UNSUPPORTED),
    (dict(variant=B.VARIANT_MFMA, dtype=B.F32), B.ERR_UNSUPPORTED),
    (dict(), B.OK),
    (dict(dtype=B.F32, head_dim=64, num_q_heads=8, num_kv_heads=2), B.OK),
])
def test_init_validation(kw, status):
    assert _status_init(_cfg(**kw)) == status


def test_init_null_arguments():
    lib = B.load_library()
    plan = ctypes.c_void_p()
    ws = ctypes.c_size_t()
    assert lib.comem_decode_attn_init(None, -1, ctypes.byref(plan), ctypes.byref(ws)) == B.ERR_NULL_POINTER
    cfg = _cfg()
    assert lib.comem_decode_attn_init(ctypes.byref(cfg), -1, None, ctypes.byref(ws)) == B.ERR_NULL_POINTER
    assert lib.comem_decode_attn_init(ctypes.byref(cfg), -2, ctypes.byref(plan), ctypes.byref(ws)) == \
        B.ERR_INVALID_SHAPE


def test_status_strings_and_null_destroy():
    for s in range(10):
        assert B.status_string(s) and B.status_string(s) != "unknown status"
    assert B.status_string(99) == "unknown status"
    assert B.load_library().comem_decode_attn_destroy(None) == B.OK


@pytest.fixture
def plan():
    p, ws = B.comem_decode_attn_init(_cfg(), B.NO_DEVICE)
    yield p, ws
    B.comem_decode_attn_destroy(p)


def _contig_args(plan, ws, **kw):
    args = dict(plan=plan, q=A, k=A, v=A, stride_token=8 * 128, stride_head=128, seq_start=A, ctx_lens=A,
                batch=2, max_ctx_len=4096, out=A, lse=A, workspace=A, workspace_bytes=ws, stream=None)
    args.update(kw)
    return args


def _call(args):
    lib = B.load_library()
    return lib.comem_decode_attn(*args.values())


@pytest.mark.parametrize("kw,status", [
    (dict(), B.ERR_NO_DEVICE),
    (dict(batch=0, q=None), B.OK),
    (dict(batch=-1), B.ERR_INVALID_SHAPE),
    (dict(batch=5), B.ERR_INVALID_SHAPE),
    (dict(max_ctx_len=4097), B.ERR_INVALID_SHAPE),
    (dict(max_ctx_len=-1), B.ERR_INVALID_SHAPE),
    (dict(q=None), B.ERR_NULL_POINTER),
    (dict(k=None), B.ERR_NULL_POINTER),
    (dict(v=None), B.ERR_NULL_POINTER),
    (dict(ctx_lens=None), B.ERR_NULL_POINTER),
    (dict(out=None), B.ERR_NULL_POINTER),
    (dict(seq_start=None), B.ERR_NULL_POINTER),
    (dict(lse=None), B.ERR_NO_DEVICE),
    (dict(stride_token=0), B.ERR_INVALID_SHAPE),
    (dict(stride_head=0), B.ERR_INVALID_SHAPE),
    (dict(stride_token=8 * 128 + 4), B.ERR_MISALIGNED),
    (dict(stride_head=132), B.ERR_MISALIGNED),
    (dict(q=A + 8), B.ERR_MISALIGNED),
    (dict(k=A + 2), B.ERR_MISALIGNED),
    (dict(v=A + 4), B.ERR_MISALIGNED),
    (dict(out=A + 4), B.ERR_MISALIGNED),
    (dict(lse=A + 2), B.ERR_MISALIGNED),
    (dict(workspace=A + 16), B.ERR_MISALIGNED),
    (dict(seq_start=A + 4), B.ERR_MISALIGNED),
    (dict(workspace_bytes=64), B.ERR_NO_DEVICE),  # planner falls back to fewer, longer splits
    (dict(workspace=None, workspace_bytes=0), B.ERR_NO_DEVICE),
])
def test_contiguous_validation(plan, kw, status):
    p, ws = plan
    assert _call(_contig_args(p, ws, **kw)) == status


def test_bad_handle():
    args = _contig_args(None, 0)
    assert _call(args) == B.ERR_BAD_HANDLE
    junk = ctypes.create_string_buffer(256)
    args = _contig_args(ctypes.addressof(junk), 0)
    assert _call(args) == B.ERR_BAD_HANDLE


def _noalloc_args(plan, **kw):
    args = dict(plan=plan, q=A, k=A, v=A, stride_token=8 * 128, stride_head=128, seq_start=A, ctx_lens=A,
                batch=2, max_ctx_len=4096, out=A, lse=A, stream=None)
    args.update(kw)
    return args


@pytest.mark.parametrize("kw,status", [
    (dict(), B.ERR_NO_DEVICE),
    (dict(batch=0, q=None), B.OK),
    (dict(batch=5), B.ERR_INVALID_SHAPE),
    (dict(max_ctx_len=4097), B.ERR_INVALID_SHAPE),
    (dict(q=None), B.ERR_NULL_POINTER),
    (dict(seq_start=None), B.ERR_NULL_POINTER),
    (dict(seq_start=A + 4), B.ERR_MISALIGNED),
    (dict(out=A + 4), B.ERR_MISALIGNED),
    (dict(stride_token=8 * 128 + 4), B.ERR_MISALIGNED),
    (dict(plan=None), B.ERR_BAD_HANDLE),
])
def test_noalloc_validation(plan, kw, status):
    p, _ = plan
    args = _noalloc_args(p)
    args.update(kw)
    assert B.load_library().comem_decode_attn_noalloc(*args.values()) == status


def _scratch_need(batch, splits, hq, d):
    rows = batch * splits * hq
    return 64 * 1024 + ((rows * 4 + 255) // 256) * 256 + rows * d * 4


def test_noalloc_rejects_calls_past_the_scratch():
    """Planned as the workspace form would plan them; a call whose partial results do not fit the fixed
    scratch is refused (before any HIP call), one that fits passes validation."""
    lib = B.load_library()
    fits, too_big = None, None
    p, ws = B.comem_decode_attn_init(_cfg(max_batch=64, max_ctx_len=65536), B.NO_DEVICE)
    try:
        for batch in (1, 2, 4, 8, 16, 32, 64):
            for L in (4096, 16384, 65536):
                chunk, splits = B.comem_decode_attn_plan_splits(p, batch, L, ws)
                need = _scratch_need(batch, splits, 32, 128) if splits > 1 else 64 * 1024
                st = lib.comem_decode_attn_noalloc(*_noalloc_args(p, batch=batch, max_ctx_len=L).values())
                if need <= B.NOALLOC_SCRATCH_BYTES:
                    assert st == B.ERR_NO_DEVICE, (batch, L)
                    fits = (batch, L)
                else:
                    assert st == B.ERR_SCRATCH_LIMIT, (batch, L)
                    too_big = (batch, L)
    finally:
        B.comem_decode_attn_destroy(p)
    assert fits and too_big
    # batch 16 of 64K-token contexts (the header's example) fits
    p, ws = B.comem_decode_attn_init(_cfg(max_batch=16, max_ctx_len=65536), B.NO_DEVICE)
    try:
        assert lib.comem_decode_attn_noalloc(*_noalloc_args(p, batch=16, max_ctx_len=65536).values()) == \
            B.ERR_NO_DEVICE
    finally:
        B.comem_decode_attn_destroy(p)


def test_noalloc_refuses_debug_plans_and_huge_ticket_regions():
    lib = B.load_library()
    p, _ = B.comem_decode_attn_init(_cfg(flags=B.FLAG_DEBUG_CHECKS), B.NO_DEVICE)
    try:
        assert lib.comem_decode_attn_noalloc(*_noalloc_args(p).values()) == B.ERR_UNSUPPORTED
    finally:
        B.comem_decode_attn_destroy(p)
    # 4096 sequences x 8 KV heads = 32768 tickets: more than the 64 KiB counter region holds
    p, _ = B.comem_decode_attn_init(_cfg(max_batch=4096, max_ctx_len=64), B.NO_DEVICE)
    try:
        assert lib.comem_decode_attn_noalloc(*_noalloc_args(p, max_ctx_len=64).values()) == B.ERR_SCRATCH_LIMIT
    finally:
        B.comem_decode_attn_destroy(p)


def _paged_args(plan, ws, **kw):
    args = dict(plan=plan, q=A, k=A, v=A, stride_page=16 * 8 * 128, stride_token=8 * 128, stride_head=128,
                page_size=16, num_pages=100, block_table=A, max_pages=256, ctx_lens=A, batch=2,
                max_ctx_len=4096, out=A, lse=A, workspace=A, workspace_bytes=ws, stream=None)
    args.update(kw)
    return args


@pytest.mark.parametrize("kw,status", [
    (dict(), B.ERR_NO_DEVICE),
    (dict(block_table=None), B.ERR_NULL_POINTER),
    (dict(page_size=0), B.ERR_INVALID_SHAPE),
    (dict(page_size=24), B.ERR_INVALID_SHAPE),
    (dict(page_size=8192), B.ERR_INVALID_SHAPE),
    (dict(num_pages=0), B.ERR_INVALID_SHAPE),
    (dict(stride_page=0), B.ERR_INVALID_SHAPE),
    (dict(max_pages=255), B.ERR_INVALID_SHAPE),
    (dict(stride_page=16 * 8 * 128 + 4), B.ERR_MISALIGNED),
    (dict(block_table=A + 2), B.ERR_MISALIGNED),
    (dict(page_size=1, max_pages=4096), B.ERR_NO_DEVICE),
    (dict(batch=0, block_table=None), B.OK),
])
def test_paged_validation(plan, kw, status):
    p, ws = plan
    assert B.load_library().comem_decode_attn_paged(*_paged_args(p, ws, **kw).values()) == status


@pytest.mark.parametrize("page_size", [1, 2, 16])
def test_planned_splits_fit_the_page_table_copy(page_size):
    """A planned split of a long paged context never needs more block-table
    entries than the matrix-core kernel copies to LDS: with 1- and 2-token
    pages the planner shortens its 4096-token splits instead of refusing the
    call (the call then stops only for want of a device)."""
    L = 262144
    p, ws = B.comem_decode_attn_init(_cfg(max_batch=1, max_ctx_len=L), B.NO_DEVICE)
    try:
        args = _paged_args(p, ws, page_size=page_size, num_pages=L, max_pages=L // page_size, batch=1,
                           max_ctx_len=L, stride_page=page_size * 8 * 128)
        assert B.load_library().comem_decode_attn_paged(*args.values()) == B.ERR_NO_DEVICE
    finally:
        B.comem_decode_attn_destroy(p)


def test_configured_split_too_long_for_the_page_table_copy():
    """A chunk_tokens the caller fixed is not shortened: 4096 one-token pages per split are refused."""
    L = 262144
    p, ws = B.comem_decode_attn_init(_cfg(max_batch=1, max_ctx_len=L, chunk_tokens=4096), B.NO_DEVICE)
    try:
        args = _paged_args(p, ws, page_size=1, num_pages=L, max_pages=L, batch=1, max_ctx_len=L,
                           stride_page=8 * 128)
        assert B.load_library().comem_decode_attn_paged(*args.values()) == B.ERR_INVALID_SHAPE
    finally:
        B.comem_decode_attn_destroy(p)


def test_flags_validation():
    assert _status_init(_cfg(flags=2)) == B.ERR_UNSUPPORTED
    assert _status_init(_cfg(flags=B.FLAG_DEBUG_CHECKS)) == B.OK


def test_debug_checks_need_a_workspace_on_the_host():
    """With COMEM_FLAG_DEBUG_CHECKS the error word lives in the workspace: a call without one is refused
    before anything is launched (a plan without a device then stops at the device)."""
    p, ws = B.comem_decode_attn_init(_cfg(flags=B.FLAG_DEBUG_CHECKS), B.NO_DEVICE)
    try:
        assert _call(_contig_args(p, ws, max_ctx_len=64)) == B.ERR_NO_DEVICE
        assert _call(_contig_args(p, ws, max_ctx_len=64, workspace=None, workspace_bytes=0)) == B.ERR_NULL_POINTER
        assert _call(_contig_args(p, ws, max_ctx_len=64, workspace_bytes=64)) == B.ERR_WORKSPACE_TOO_SMALL
        args = _paged_args(p, ws, workspace=None, workspace_bytes=0, max_ctx_len=64)
        assert B.load_library().comem_decode_attn_paged(*args.values()) == B.ERR_NULL_POINTER
    finally:
        B.comem_decode_attn_destroy(p)
    p, ws = B.comem_decode_attn_init(_cfg(), B.NO_DEVICE)
    try:  # without the flag a short call needs no workspace at all
        assert _call(_contig_args(p, ws, max_ctx_len=64, workspace=None, workspace_bytes=0)) == B.ERR_NO_DEVICE
    finally:
        B.comem_decode_attn_destroy(p)


def test_device_errors_validation(plan):
    p, ws = plan
    lib = B.load_library()
    word = ctypes.c_uint32(7)
    assert lib.comem_decode_attn_device_errors(None, A, ws, ctypes.byref(word), None) == B.ERR_BAD_HANDLE
    assert lib.comem_decode_attn_device_errors(p, None, ws, ctypes.byref(word), None) == B.ERR_NULL_POINTER
    assert lib.comem_decode_attn_device_errors(p, A, ws, None, None) == B.ERR_NULL_POINTER
    assert lib.comem_decode_attn_device_errors(p, A + 16, ws, ctypes.byref(word), None) == B.ERR_MISALIGNED
    assert lib.comem_decode_attn_device_errors(p, A, 16, ctypes.byref(word), None) == B.ERR_WORKSPACE_TOO_SMALL
    assert lib.comem_decode_attn_device_errors(p, A, ws, ctypes.byref(word), None) == B.ERR_NO_DEVICE
    assert word.value == 0


def _append_args(plan, **kw):
    args = dict(plan=plan, new_k=A, new_v=A, k=A, v=A, stride_token=8 * 128, stride_head=128, seq_start=A,
                ctx_lens=A, batch=2, max_ctx_len=4096, stream=None)
    args.update(kw)
    return args


@pytest.mark.parametrize("kw,status", [
    (dict(), B.ERR_NO_DEVICE),
    (dict(batch=0, new_k=None), B.OK),
    (dict(batch=-1), B.ERR_INVALID_SHAPE),
    (dict(batch=5), B.ERR_INVALID_SHAPE),
    (dict(max_ctx_len=4097), B.ERR_INVALID_SHAPE),
    (dict(new_k=None), B.ERR_NULL_POINTER),
    (dict(new_v=None), B.ERR_NULL_POINTER),
    (dict(k=None), B.ERR_NULL_POINTER),
    (dict(v=None), B.ERR_NULL_POINTER),
    (dict(ctx_lens=None), B.ERR_NULL_POINTER),
    (dict(seq_start=None), B.ERR_NULL_POINTER),
    (dict(stride_token=0), B.ERR_INVALID_SHAPE),
    (dict(stride_head=0), B.ERR_INVALID_SHAPE),
    (dict(stride_token=8 * 128 + 4), B.ERR_MISALIGNED),
    (dict(new_k=A + 8), B.ERR_MISALIGNED),
    (dict(new_v=A + 2), B.ERR_MISALIGNED),
    (dict(k=A + 4), B.ERR_MISALIGNED),
    (dict(seq_start=A + 4), B.ERR_MISALIGNED),
])
def test_append_validation(plan, kw, status):
    p, _ = plan
    assert B.load_library().comem_kv_append(*_append_args(p, **kw).values()) == status


@pytest.mark.parametrize("kw,status", [
    (dict(), B.ERR_NO_DEVICE),
    (dict(block_table=None), B.ERR_NULL_POINTER),
    (dict(page_size=24), B.ERR_INVALID_SHAPE),
    (dict(num_pages=0), B.ERR_INVALID_SHAPE),
    (dict(max_pages=255), B.ERR_INVALID_SHAPE),
    (dict(stride_page=16 * 8 * 128 + 4), B.ERR_MISALIGNED),
    (dict(block_table=A + 2), B.ERR_MISALIGNED),
    (dict(new_v=None), B.ERR_NULL_POINTER),
    (dict(batch=0, block_table=None), B.OK),
])
def test_append_paged_validation(plan, kw, status):
    p, _ = plan
    args = dict(plan=p, new_k=A, new_v=A, k=A, v=A, stride_page=16 * 8 * 128, stride_token=8 * 128,
                stride_head=128, page_size=16, num_pages=100, block_table=A, max_pages=256, ctx_lens=A, batch=2,
                max_ctx_len=4096, stream=None)
    args.update(kw)
    assert B.load_library().comem_kv_append_paged(*args.values()) == status
    assert B.load_library().comem_kv_append_paged(*dict(args, plan=None).values()) == B.ERR_BAD_HANDLE


@pytest.mark.parametrize("kw,status", [
    (dict(), B.ERR_NO_DEVICE),
    (dict(new_k=None), B.ERR_NULL_POINTER),
    (dict(new_v=None), B.ERR_NULL_POINTER),
    (dict(new_k=A + 8), B.ERR_MISALIGNED),
    (dict(q=None), B.ERR_NULL_POINTER),
    (dict(batch=0, new_k=None), B.OK),
    (dict(batch=5), B.ERR_INVALID_SHAPE),
])
def test_fused_append_validation(plan, kw, status):
    p, ws = plan
    c = _contig_args(p, ws)
    args = dict(plan=p, q=A, new_k=A, new_v=A)
    args.update({k: c[k] for k in c if k not in ("plan", "q")})
    args.update(kw)
    assert B.load_library().comem_append_decode_attn(*args.values()) == status
    g = _paged_args(p, ws)
    pargs = dict(plan=p, q=A, new_k=A, new_v=A)
    pargs.update({k: g[k] for k in g if k not in ("plan", "q")})
    pargs.update(kw)
    assert B.load_library().comem_append_decode_attn_paged(*pargs.values()) == status


def test_forced_chunk_needs_room():
    p, ws = B.comem_decode_attn_init(_cfg(chunk_tokens=32), B.NO_DEVICE)
    try:
        assert B.comem_decode_attn_plan_splits(p, 4, 4096, ws) == (32, 128)
        st = B.load_library().comem_decode_attn(*_contig_args(p, ws, batch=4, workspace_bytes=ws - 1).values())
        assert st == B.ERR_WORKSPACE_TOO_SMALL
    finally:
        B.comem_decode_attn_destroy(p)


@pytest.mark.parametrize("batch,L", [(1, 32768), (16, 65536), (64, 16384), (8, 131072), (1, 1), (3, 300)])
def test_auto_plan_fits_init_workspace(batch, L):
    """Every call within the plan's limits fits the workspace size init reports."""
    cfg = _cfg(max_batch=max(batch, 1), max_ctx_len=L)
    p, ws = B.comem_decode_attn_init(cfg, B.NO_DEVICE)
    try:
        for b in sorted({1, max(1, batch // 2), batch}):
            for l in sorted(x for x in {1, 33, L // 3 + 1, L} if x <= L):
                chunk, splits = B.comem_decode_attn_plan_splits(p, b, l, ws)
                assert chunk % 32 == 0 and splits == -(-l // chunk)
                chunk2, _ = B.comem_decode_attn_plan_splits(p, b, l, 1 << 40)
                assert chunk2 == chunk, "init workspace forced a coarser plan"
    finally:
        B.comem_decode_attn_destroy(p)


@pytest.mark.parametrize("batch,L,chunk", [
    (1, 32768, 1024),    # batch 1, 32k: 256 items of 1024 tokens, one per workgroup
    (16, 65536, 1024),   # ragged batch up to 64k: 4096 items of 2048 would be 8 per workgroup
    (64, 16384, 1024),   # paged batch up to 16k: likewise
    (64, 65536, 2048),   # 16 items of 2048 tokens per workgroup
    (8, 131072, 4096),   # 128k and longer: 4096-token splits
])
def test_auto_plan_split_sizes(batch, L, chunk):
    """The matrix-core planner's split sizes on a 256-CU part (2 queue workgroups per CU)."""
    p, ws = B.comem_decode_attn_init(_cfg(max_batch=batch, max_ctx_len=L), B.NO_DEVICE)
    try:
        assert B.comem_decode_attn_plan_splits(p, batch, L, ws) == (chunk, -(-L // chunk))
    finally:
        B.comem_decode_attn_destroy(p)


def _prefill_args(plan, **kw):
    args = dict(plan=plan, q=A, q_start=A, q_lens=A, max_q_len=512, k=A, v=A, stride_token=8 * 128, stride_head=128,
                seq_start=A, ctx_lens=A, batch=2, max_ctx_len=4096, out=A, lse=A, stream=None)
    args.update(kw)
    return args


@pytest.mark.parametrize("kw,status", [
    (dict(), B.ERR_NO_DEVICE),
    (dict(batch=0, q=None), B.OK),
    (dict(max_q_len=0), B.OK),
    # no new token anywhere: nothing to read or write, so empty buffers may be NULL
    (dict(max_q_len=0, q=None, q_start=None, q_lens=None, k=None, v=None, seq_start=None, ctx_lens=None,
          out=None, lse=None), B.OK),
    (dict(max_q_len=0, batch=5), B.ERR_INVALID_SHAPE),
    (dict(max_q_len=0, max_ctx_len=4097), B.ERR_INVALID_SHAPE),
    (dict(batch=-1), B.ERR_INVALID_SHAPE),
    (dict(batch=5), B.ERR_INVALID_SHAPE),
    (dict(max_ctx_len=4097), B.ERR_INVALID_SHAPE),
    (dict(max_q_len=-1), B.ERR_INVALID_SHAPE),
    (dict(max_q_len=4097), B.ERR_INVALID_SHAPE),
    (dict(q=None), B.ERR_NULL_POINTER),
    (dict(q_start=None), B.ERR_NULL_POINTER),
    (dict(q_lens=None), B.ERR_NULL_POINTER),
    (dict(k=None), B.ERR_NULL_POINTER),
    (dict(seq_start=None), B.ERR_NULL_POINTER),
    (dict(ctx_lens=None), B.ERR_NULL_POINTER),
    (dict(out=None), B.ERR_NULL_POINTER),
    (dict(lse=None), B.ERR_NO_DEVICE),
    (dict(stride_token=0), B.ERR_INVALID_SHAPE),
    (dict(stride_token=8 * 128 + 4), B.ERR_MISALIGNED),
    (dict(q=A + 8), B.ERR_MISALIGNED),
    (dict(out=A + 4), B.ERR_MISALIGNED),
    (dict(q_start=A + 4), B.ERR_MISALIGNED),
    (dict(q_lens=A + 2), B.ERR_MISALIGNED),
    (dict(seq_start=A + 4), B.ERR_MISALIGNED),
])
def test_prefill_validation(plan, kw, status):
    p, _ = plan
    assert B.load_library().comem_prefill_attn(*_prefill_args(p, **kw).values()) == status


@pytest.mark.parametrize("kw,status", [
    (dict(), B.ERR_NO_DEVICE),
    (dict(block_table=None), B.ERR_NULL_POINTER),
    (dict(page_size=24), B.ERR_INVALID_SHAPE),
    (dict(num_pages=0), B.ERR_INVALID_SHAPE),
    (dict(max_pages=255), B.ERR_INVALID_SHAPE),
    (dict(block_table=A + 2), B.ERR_MISALIGNED),
    (dict(q_lens=None), B.ERR_NULL_POINTER),
    (dict(batch=0, block_table=None), B.OK),
    (dict(max_q_len=0, q=None, out=None, block_table=None, page_size=0), B.OK),
])
def test_prefill_paged_validation(plan, kw, status):
    p, _ = plan
    args = dict(plan=p, q=A, q_start=A, q_lens=A, max_q_len=512, k=A, v=A, stride_page=16 * 8 * 128,
                stride_token=8 * 128, stride_head=128, page_size=16, num_pages=100, block_table=A, max_pages=256,
                ctx_lens=A, batch=2, max_ctx_len=4096, out=A, lse=A, stream=None)
    args.update(kw)
    assert B.load_library().comem_prefill_attn_paged(*args.values()) == status
    assert B.load_library().comem_prefill_attn_paged(*dict(args, plan=None).values()) == B.ERR_BAD_HANDLE


def test_prefill_needs_bf16():
    p, _ = B.comem_decode_attn_init(_cfg(dtype=B.F32), B.NO_DEVICE)
    try:
        assert B.load_library().comem_prefill_attn(*_prefill_args(p).values()) == B.ERR_UNSUPPORTED
    finally:
        B.comem_decode_attn_destroy(p)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=B.FP8_E4M3), B.OK),
    (dict(dtype=B.FP8_E4M3, variant=B.VARIANT_MFMA), B.OK),
    (dict(dtype=B.FP8_E4M3, variant=B.VARIANT_MFMA_GRID), B.OK),
    (dict(dtype=B.FP8_E4M3, variant=B.VARIANT_VALU), B.ERR_UNSUPPORTED),
    (dict(dtype=B.FP8_E4M3, k_scale=0.0), B.ERR_INVALID_SHAPE),
    (dict(dtype=B.FP8_E4M3, v_scale=-1.0), B.ERR_INVALID_SHAPE),
    (dict(dtype=B.FP8_E4M3, k_scale=float("inf")), B.ERR_INVALID_SHAPE),
    (dict(dtype=B.FP8_E4M3, v_scale=float("nan")), B.ERR_INVALID_SHAPE),
    (dict(dtype=B.BF16, k_scale=0.0, v_scale=0.0), B.OK),  # scales are only read for FP8 caches
    (dict(dtype=3), B.ERR_UNSUPPORTED),
])
def test_fp8_config_validation(kw, status):
    assert _status_init(_cfg(**kw)) == status


def test_fp8_strides_are_bytes():
    """An FP8 cache row of 8 heads x 128 codes is 1024 bytes: strides are counted in elements = bytes."""
    p, ws = B.comem_decode_attn_init(_cfg(dtype=B.FP8_E4M3), B.NO_DEVICE)
    try:
        lib = B.load_library()
        assert lib.comem_decode_attn(*_contig_args(p, ws).values()) == B.ERR_NO_DEVICE
        assert lib.comem_decode_attn(*_contig_args(p, ws, stride_token=8 * 128 + 8).values()) == B.ERR_MISALIGNED
        assert lib.comem_decode_attn(*_contig_args(p, ws, stride_token=8 * 128 + 16).values()) == B.ERR_NO_DEVICE
        assert lib.comem_prefill_attn(*_prefill_args(p).values()) == B.ERR_UNSUPPORTED
    finally:
        B.comem_decode_attn_destroy(p)


@pytest.mark.parametrize("shape", [(1,), (3, 5, 7), (33, 8, 128), (2, 16, 8, 64)])
@pytest.mark.parametrize("dtype", ["uint8", "bfloat16", "float32"])
def test_kv_cache_pair_places_v_256_bytes_past_k_modulo_512(shape, dtype):
    """The helper's V base is K's plus 256 modulo 512 for any size and element
    type (on CPU tensors; the arithmetic does not depend on the device), and
    the two caches do not overlap."""
    import torch

    from paper_2605_30842_amd.binding import kv_cache_pair

    dt = getattr(torch, dtype)
    k, v = kv_cache_pair(shape, dt, "cpu")
    assert k.shape == v.shape == shape and k.dtype == v.dtype == dt
    assert k.is_contiguous() and v.is_contiguous()
    assert (v.data_ptr() - k.data_ptr()) % 512 == 256
    assert v.data_ptr() >= k.data_ptr() + k.numel() * k.element_size()
    k.fill_(1)
    v.fill_(2)
    assert int(k.min()) == 1 and int(v.max()) == 2
