"""KV append through the C ABI vs the oracle's append, bit for bit.

Each case stores seeded new rows as token L_b - 1 of every sequence, copies
the whole cache back and compares it bitwise with the oracle's appended copy
(so both the written rows and every row that must stay untouched are
checked); then attention over the appended cache is compared with the
oracle's attention over its own appended copy (append-then-attend).
Guarded sequences (length outside [1, max_ctx_len], block-table entry outside
the pool) must leave the cache unchanged.
"""

import numpy as np
import pytest

import oracle.decode_attention as da
from tests.gpu_util import DeviceWorkload, check, make_op, run, say, to_torch
from workloads.synth import WORKLOADS, draw_new_rows, generate, small_spec

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2605_30842_amd import binding

    binding.load_library()
    yield


def _host(t, dtype):
    a = t.cpu()
    if dtype == "bf16":
        import torch

        return a.view(torch.int16).numpy().view(np.uint16)
    return a.numpy()


def _append(dw, op, new_k, new_v, max_ctx_len=None):
    import torch

    s = dw.spec
    mcl = s.max_ctx_len if max_ctx_len is None else max_ctx_len
    nk, nv = to_torch(new_k, s.dtype, "cuda:0"), to_torch(new_v, s.dtype, "cuda:0")
    if s.layout == "paged":
        op.append_paged(nk, nv, dw.k, dw.v, dw.block_table, dw.ctx_lens, mcl)
    else:
        op.append(nk, nv, dw.k, dw.v, dw.seq_start, dw.ctx_lens, mcl)
    torch.cuda.synchronize()


def _oracle_append(w, new_k, new_v):
    if w.spec.layout == "paged":
        return (da.append_paged(w.k_pages, w.block_table, w.ctx_lens, new_k),
                da.append_paged(w.v_pages, w.block_table, w.ctx_lens, new_v))
    return (da.append_contiguous(w.k, w.seq_start, w.ctx_lens, new_k),
            da.append_contiguous(w.v, w.seq_start, w.ctx_lens, new_v))


def _bitwise(got, want, what):
    assert got.shape == want.shape, what
    g = got.view(np.uint32 if got.dtype == np.float32 else got.dtype)
    h = want.view(np.uint32 if want.dtype == np.float32 else want.dtype)
    bad = np.argwhere(g != h)
    assert len(bad) == 0, f"{what}: {len(bad)} elements differ, first at {bad[:3].tolist()}"


CASES = [
    ("contig_f32", 1, [1, 31, 32, 33, 0, 1000], {}),
    ("contig_bf16", 2, [1, 0, 32, 33, 100, 4097], {"gap_rows": 3}),
    ("paged16", 4, [1, 15, 16, 17, 0, 300], {"spare_pages": 5}),
    ("paged1", 4, [1, 2, 3, 64], {"page_size": 1}),
    ("paged64_g8", 5, [63, 64, 65, 1000], {}),
]


@pytest.mark.parametrize("name,base,lens,kw", CASES, ids=[c[0] for c in CASES])
def test_append_bitwise_then_attend(name, base, lens, kw):
    gen = {k: kw[k] for k in ("gap_rows", "spare_pages") if k in kw}
    spec_kw = {k: v for k, v in kw.items() if k not in gen}
    spec = small_spec(WORKLOADS[base], lens, seed=300 + base, **spec_kw)
    w = generate(spec, **gen)
    new_k, new_v = draw_new_rows(spec, seed=400 + base)
    say(f"case append {name} lens={lens} {spec.dtype} {spec.layout} ps={spec.page_size}")
    dw = DeviceWorkload(w)
    op = make_op(spec)
    _append(dw, op, new_k, new_v)
    want_k, want_v = _oracle_append(w, new_k, new_v)
    _bitwise(_host(dw.k, spec.dtype), want_k, f"{name} K cache")
    _bitwise(_host(dw.v, spec.dtype), want_v, f"{name} V cache")
    # append-then-attend: the oracle attends over its own appended copy
    if spec.layout == "paged":
        w.k_pages, w.v_pages = want_k, want_v
    else:
        w.k, w.v = want_k, want_v
    out, lse = run(dw, op)
    ro, rl = da.reference(w)
    check(out, lse, ro, rl, spec.dtype, f"{name} attention after append")


FUSED = [
    ("contig_f32", 1, [1, 31, 32, 33, 0, 1000], {}, "auto", 0),
    ("contig_bf16_mfma", 2, [1, 0, 32, 33, 100, 4097], {"gap_rows": 3}, "mfma", 0),
    ("contig_bf16_grid_c32", 2, [1, 0, 32, 33, 100, 4097], {}, "mfma_grid", 32),
    ("contig_bf16_valu", 2, [1, 0, 32, 33, 100, 4097], {}, "valu", 0),
    ("paged16_mfma", 4, [1, 15, 16, 17, 0, 300], {"spare_pages": 5}, "mfma", 0),
    ("paged16_valu", 4, [1, 15, 16, 17, 0, 300], {}, "valu", 64),
    ("paged1", 4, [1, 2, 3, 64], {"page_size": 1}, "mfma", 0),
    ("paged64_g8", 5, [63, 64, 65, 1000], {}, "mfma", 0),
    ("paged16_queue", 4, [1000 + 37 * i for i in range(16)], {}, "mfma", 32),
]


@pytest.mark.parametrize("name,base,lens,kw,variant,chunk", FUSED, ids=[c[0] for c in FUSED])
def test_fused_append_attend(name, base, lens, kw, variant, chunk):
    """One launch appends and attends: same cache bits as the oracle's append, and the same output bits
    as the separate append call followed by the attention call."""
    import torch

    gen = {k: kw[k] for k in ("gap_rows", "spare_pages") if k in kw}
    spec_kw = {k: v for k, v in kw.items() if k not in gen}
    spec = small_spec(WORKLOADS[base], lens, seed=330 + base, **spec_kw)
    w = generate(spec, **gen)
    new_k, new_v = draw_new_rows(spec, seed=430 + base)
    say(f"case fused {name} lens={lens[:6]} {spec.dtype} {spec.layout} ps={spec.page_size} {variant} chunk={chunk}")
    op = make_op(spec, chunk=chunk, variant=variant)
    nk, nv = to_torch(new_k, spec.dtype, "cuda:0"), to_torch(new_v, spec.dtype, "cuda:0")
    fused = DeviceWorkload(w)
    lse = torch.empty((spec.batch, spec.num_q_heads), dtype=torch.float32, device="cuda:0")
    if spec.layout == "paged":
        out, lse = op.append_forward_paged(fused.q, nk, nv, fused.k, fused.v, fused.block_table, fused.ctx_lens,
                                           spec.max_ctx_len, lse=lse)
    else:
        out, lse = op.append_forward(fused.q, nk, nv, fused.k, fused.v, fused.seq_start, fused.ctx_lens,
                                     spec.max_ctx_len, lse=lse)
    torch.cuda.synchronize()
    want_k, want_v = _oracle_append(w, new_k, new_v)
    _bitwise(_host(fused.k, spec.dtype), want_k, f"{name} K cache")
    _bitwise(_host(fused.v, spec.dtype), want_v, f"{name} V cache")
    sep = DeviceWorkload(w)
    _append(sep, op, new_k, new_v)
    out2, lse2 = run(sep, op)
    _bitwise(out.cpu().numpy(), out2, f"{name} out fused vs separate")
    _bitwise(lse.cpu().numpy(), lse2, f"{name} lse fused vs separate")
    if spec.layout == "paged":
        w.k_pages, w.v_pages = want_k, want_v
    else:
        w.k, w.v = want_k, want_v
    ro, rl = da.reference(w)
    check(out.cpu().numpy(), lse.cpu().numpy(), ro, rl, spec.dtype, f"{name} fused vs oracle")


def test_append_twice_grows_context():
    """Two decode steps: append at L, attend; append at L + 1, attend (lengths grow by one)."""
    import torch

    spec = small_spec(WORKLOADS[4], [17, 30, 100], seed=310, max_ctx_len=128)  # both steps stay in allocated pages
    w = generate(spec, spare_pages=2)
    w.ctx_lens = w.ctx_lens - 1  # the first step's token is appended below
    dw = DeviceWorkload(w)
    op = make_op(spec)
    for step in range(2):
        w.ctx_lens = w.ctx_lens + 1
        dw.ctx_lens = torch.from_numpy(w.ctx_lens.astype(np.int32)).to("cuda:0")
        new_k, new_v = draw_new_rows(spec, seed=500 + step)
        _append(dw, op, new_k, new_v, max_ctx_len=int(w.ctx_lens.max()) + 1)
        w.k_pages, w.v_pages = _oracle_append(w, new_k, new_v)
        _bitwise(_host(dw.k, spec.dtype), w.k_pages, f"step {step} K")
        out, lse = run(dw, op, max_ctx_len=int(w.ctx_lens.max()))
        ro, rl = da.reference(w)
        check(out, lse, ro, rl, "bf16", f"step {step}")


def test_guarded_sequences_are_skipped():
    """Lengths above max_ctx_len and table entries outside the pool write nothing."""
    import torch

    spec = small_spec(WORKLOADS[4], [20, 40, 60, 80], seed=320, max_ctx_len=128)
    w = generate(spec, spare_pages=1)
    dw = DeviceWorkload(w)
    bt = w.block_table.copy()
    bt[1, (40 - 1) // 16] = -1                  # sequence 1: entry below the pool
    bt[2, (60 - 1) // 16] = w.k_pages.shape[0]  # sequence 2: entry past the pool
    dw.block_table = torch.from_numpy(bt.astype(np.int32)).to("cuda:0")
    new_k, new_v = draw_new_rows(spec, seed=321)
    op = make_op(spec)
    _append(dw, op, new_k, new_v, max_ctx_len=70)  # sequence 3 (L = 80) is above the bound
    want_k = w.k_pages.copy()
    want_k[bt[0, 19 // 16], 19 % 16] = new_k[0]   # only sequence 0 is stored
    _bitwise(_host(dw.k, spec.dtype), want_k, "guarded K")


@pytest.mark.parametrize("i", [3, 4, 5])
def test_append_full_workload(i):
    """Full-size caches: exactly the B target rows change, to the given bits."""
    import torch

    w = generate(WORKLOADS[i])
    spec = w.spec
    say(f"case append full workload {i} {spec.name}")
    dw = DeviceWorkload(w)
    new_k, new_v = draw_new_rows(spec, seed=600 + i)
    before_k = dw.k.clone()
    op = make_op(spec)
    _append(dw, op, new_k, new_v)
    rows = tuple(range(dw.k.dim() - 2))  # leading (row) dims
    changed = (dw.k.view(torch.int16) != before_k.view(torch.int16)).any(dim=-1).any(dim=-1)
    got = torch.nonzero(changed).cpu().numpy()
    del before_k
    L = w.ctx_lens.astype(np.int64)
    if spec.layout == "paged":
        ps = spec.page_size
        want = np.array([[w.block_table[b, (L[b] - 1) // ps], (L[b] - 1) % ps] for b in range(spec.batch)])
    else:
        want = (w.seq_start + L - 1)[:, None]
    idx = tuple(torch.from_numpy(np.ascontiguousarray(want[:, c])).to("cuda:0") for c in range(want.shape[1]))
    tgt_k, tgt_v = dw.k[idx], dw.v[idx]
    assert len(rows) == want.shape[1]
    # every changed row is a target row (a target row may keep its bits only if they were equal already)
    want_set = {tuple(r) for r in want.tolist()}
    assert {tuple(r) for r in got.tolist()} <= want_set
    _bitwise(_host(tgt_k, spec.dtype), new_k, f"workload {i} K rows")
    _bitwise(_host(tgt_v, spec.dtype), new_v, f"workload {i} V rows")
