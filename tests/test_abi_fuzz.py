"""Property-based checks of the C ABI's host-side validation (no GPU).

The ABI validates every argument on the host before any HIP call and returns
a documented status; it never aborts or reads a device pointer on the host.
These tests draw arbitrary configs and call arguments (absurd sizes,
negative and NaN values, misaligned and null pointers) and check that every
call returns a known status, that a plan which init accepts reports a usable
split plan, and that the workspace size init reports always admits a call at
the plan's limits. Plans are made with COMEM_NO_DEVICE, so a call whose
arguments are all valid stops with COMEM_ERR_NO_DEVICE and nothing is
launched. Fake device addresses are never dereferenced.
"""

import ctypes
import math

from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from paper_2605_30842_amd import binding as B

STATUSES = {B.OK, B.ERR_NULL_POINTER, B.ERR_INVALID_SHAPE, B.ERR_UNSUPPORTED, B.ERR_MISALIGNED,
            B.ERR_WORKSPACE_TOO_SMALL, B.ERR_BAD_HANDLE, B.ERR_HIP, B.ERR_NO_DEVICE}
FUZZ = settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.too_slow])

A = 1 << 20  # 256-byte aligned fake device address
pointers = st.sampled_from([None, A, A + 2, A + 4, A + 8, A + 16, A + 256])
floats = st.floats(allow_nan=True, allow_infinity=True, width=32)


def _init(cfg):
    plan, ws = ctypes.c_void_p(), ctypes.c_size_t()
    st_ = B.load_library().comem_decode_attn_init(ctypes.byref(cfg), B.NO_DEVICE, ctypes.byref(plan),
                                                   ctypes.byref(ws))
    return st_, plan.value, ws.value


configs = st.builds(
    B.Config,
    num_q_heads=st.integers(-2, 130), num_kv_heads=st.integers(-2, 40),
    head_dim=st.sampled_from([-64, 0, 16, 32, 64, 96, 128, 256]),
    dtype=st.integers(-1, 4), scale=floats,
    max_batch=st.integers(-1, 70000), max_ctx_len=st.integers(-1, 1 << 31),
    chunk_tokens=st.integers(-64, 1 << 16), variant=st.integers(-1, 4),
    k_scale=floats, v_scale=floats, flags=st.integers(0, 7))


@FUZZ
@given(configs)
def test_init_returns_a_status_and_accepted_plans_plan(cfg):
    status, plan, ws = _init(cfg)
    assert status in STATUSES
    if status != B.OK:
        assert plan is None
        return
    try:
        assert cfg.num_q_heads > 0 and cfg.num_kv_heads > 0 and cfg.num_q_heads % cfg.num_kv_heads == 0
        assert cfg.max_batch > 0 and cfg.max_ctx_len > 0 and math.isfinite(cfg.scale) and cfg.scale > 0
        # A call at the plan's own limits fits the workspace init reported.
        chunk, splits = ctypes.c_int32(), ctypes.c_int32()
        st2 = B.load_library().comem_decode_attn_plan_splits(plan, cfg.max_batch, cfg.max_ctx_len, ws,
                                                              ctypes.byref(chunk), ctypes.byref(splits))
        assert st2 == B.OK, B.load_library().comem_status_string(st2)
        assert chunk.value > 0 and chunk.value % 32 == 0
        assert splits.value == -(-cfg.max_ctx_len // chunk.value)
    finally:
        assert B.load_library().comem_decode_attn_destroy(plan) == B.OK


@st.composite
def valid_configs(draw):
    """Configs inside the documented limits: init must accept every one."""
    hkv, g = draw(st.integers(1, 64)), draw(st.sampled_from([1, 2, 4, 8, 16]))
    dtype = draw(st.sampled_from([B.F32, B.BF16, B.FP8_E4M3]))
    variants = {B.F32: [B.VARIANT_AUTO, B.VARIANT_VALU],
                B.BF16: [B.VARIANT_AUTO, B.VARIANT_VALU, B.VARIANT_MFMA, B.VARIANT_MFMA_GRID],
                B.FP8_E4M3: [B.VARIANT_AUTO, B.VARIANT_MFMA, B.VARIANT_MFMA_GRID]}[dtype]
    positive = st.floats(2.0 ** -20, 1024.0, allow_nan=False, allow_infinity=False, width=32)
    return B.Config(num_q_heads=hkv * g, num_kv_heads=hkv, head_dim=draw(st.sampled_from([64, 128])), dtype=dtype,
                    scale=draw(positive), max_batch=draw(st.integers(1, 65535)),
                    max_ctx_len=draw(st.integers(1, 1 << 30)),
                    chunk_tokens=draw(st.one_of(st.just(0), st.integers(1, 1 << 15).map(lambda c: 32 * c))),
                    variant=draw(st.sampled_from(variants)), k_scale=draw(positive), v_scale=draw(positive),
                    flags=draw(st.sampled_from([0, B.FLAG_DEBUG_CHECKS])))


@FUZZ
@given(valid_configs())
def test_valid_configs_are_accepted_and_plan_within_their_workspace(cfg):
    status, plan, ws = _init(cfg)
    assert status == B.OK, B.load_library().comem_status_string(status)
    try:
        for batch, ctx in ((cfg.max_batch, cfg.max_ctx_len), (1, cfg.max_ctx_len), (cfg.max_batch, 1),
                           (max(1, cfg.max_batch // 3), max(1, cfg.max_ctx_len // 7))):
            chunk, splits = ctypes.c_int32(), ctypes.c_int32()
            st2 = B.load_library().comem_decode_attn_plan_splits(plan, batch, ctx, ws, ctypes.byref(chunk),
                                                                  ctypes.byref(splits))
            assert st2 == B.OK, (batch, ctx, B.load_library().comem_status_string(st2))
            assert chunk.value > 0 and chunk.value % 32 == 0
            assert splits.value == -(-ctx // chunk.value)
            if cfg.chunk_tokens:
                assert chunk.value == cfg.chunk_tokens
    finally:
        assert B.load_library().comem_decode_attn_destroy(plan) == B.OK


@FUZZ
@given(valid_configs(), st.integers(0, 12))
def test_valid_calls_at_the_plan_limits_pass_validation(cfg, log_ps):
    """Planned splits (chunk_tokens = 0) and well-formed buffers: the contiguous and the paged
    call at the plan's largest batch and context pass every host check (a device-less plan then
    stops with COMEM_ERR_NO_DEVICE), whatever the page size."""
    cfg.chunk_tokens = 0
    status, plan, ws = _init(cfg)
    assert status == B.OK
    lib = B.load_library()
    try:
        D, hkv = cfg.head_dim, cfg.num_kv_heads
        batch, ctx = cfg.max_batch, cfg.max_ctx_len
        st_c = lib.comem_decode_attn(plan, A, A, A, hkv * D, D, A, A, batch, ctx, A, A, A, ws, None)
        assert st_c == B.ERR_NO_DEVICE, lib.comem_status_string(st_c)
        ps = 1 << log_ps
        st_p = lib.comem_decode_attn_paged(plan, A, A, A, ps * hkv * D, hkv * D, D, ps, 1 << 20, A,
                                           -(-ctx // ps), A, batch, ctx, A, A, A, ws, None)
        assert st_p == B.ERR_NO_DEVICE, (ps, lib.comem_status_string(st_p))
    finally:
        assert lib.comem_decode_attn_destroy(plan) == B.OK


_PLAN = []


def _plan():
    """One device-less plan shared by the call tests, made on first use (not when pytest collects)."""
    if not _PLAN:
        cfg = B.Config(num_q_heads=32, num_kv_heads=8, head_dim=128, dtype=B.BF16, scale=0.088, max_batch=8,
                       max_ctx_len=8192, chunk_tokens=0, variant=B.VARIANT_AUTO, k_scale=1.0, v_scale=1.0)
        status, plan, _ = _init(cfg)
        assert status == B.OK
        _PLAN.append(plan)
    return _PLAN[0]


sizes = st.integers(-3, 1 << 40)


@FUZZ
@given(q=pointers, k=pointers, v=pointers, out=pointers, lse=pointers, ws_ptr=pointers, seq=pointers,
       lens=pointers, stride_token=st.integers(-8, 1 << 28), stride_head=st.integers(-8, 1 << 12),
       batch=st.integers(-2, 12), max_ctx=st.integers(-2, 20000), ws_bytes=sizes)
def test_contiguous_call_returns_a_status(q, k, v, out, lse, ws_ptr, seq, lens, stride_token, stride_head,
                                          batch, max_ctx, ws_bytes):
    status = B.load_library().comem_decode_attn(_plan(), q, k, v, stride_token, stride_head, seq, lens, batch,
                                                max_ctx, out, lse, ws_ptr, ws_bytes, None)
    assert status in STATUSES
    assert status != B.OK or batch == 0  # a device-less plan launches nothing
    assert status != B.ERR_HIP  # nothing reaches the runtime


@FUZZ
@given(q=pointers, k=pointers, bt=pointers, lens=pointers, ws_ptr=pointers,
       stride_page=st.integers(-8, 1 << 30), stride_token=st.integers(-8, 1 << 28),
       page_size=st.integers(-2, 9000), num_pages=st.integers(-2, 1 << 33), max_pages=st.integers(-2, 70000),
       batch=st.integers(-2, 12), max_ctx=st.integers(-2, 20000), ws_bytes=sizes)
def test_paged_call_returns_a_status(q, k, bt, lens, ws_ptr, stride_page, stride_token, page_size, num_pages,
                                     max_pages, batch, max_ctx, ws_bytes):
    status = B.load_library().comem_decode_attn_paged(_plan(), q, k, k, stride_page, stride_token, 128, page_size,
                                                      num_pages, bt, max_pages, lens, batch, max_ctx, A, A, ws_ptr,
                                                      ws_bytes, None)
    assert status in STATUSES
    assert status != B.OK or batch == 0
    assert status != B.ERR_HIP


@FUZZ
@given(q=pointers, qs=pointers, ql=pointers, seq=pointers, lens=pointers, max_q=st.integers(-2, 1 << 20),
       stride_token=st.integers(-8, 1 << 28), batch=st.integers(-2, 12), max_ctx=st.integers(-2, 20000))
def test_prefill_call_returns_a_status(q, qs, ql, seq, lens, max_q, stride_token, batch, max_ctx):
    status = B.load_library().comem_prefill_attn(_plan(), q, qs, ql, max_q, A, A, stride_token, 128, seq, lens, batch,
                                                 max_ctx, A, A, None)
    assert status in STATUSES
    assert status != B.OK or batch == 0 or max_q == 0
    assert status != B.ERR_HIP
