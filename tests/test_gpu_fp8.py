"""FP8 (OCP E4M3) KV caches: HIP path vs the fp64 oracle over the dequantized caches, through the C ABI.

The kernels read one-byte codes and widen them to bf16 exactly, so the
bf16 gates apply unchanged (official gate plus the internal 1e-4 gate).
Cases cover ragged contiguous and paged caches, both head sizes and every
GQA group, non-power-of-two scales, NaN codes outside the contexts, a
one-token context (exact), the append of code rows (bitwise) and the two
FP8 workloads at full size on sampled rows.
"""

import numpy as np
import pytest

import oracle.decode_attention as da
from tests.gpu_util import DeviceWorkload, check, make_op, run, say, to_torch
from workloads.synth import WORKLOADS, draw_new_rows, generate, small_spec

pytestmark = pytest.mark.gpu

RAGGED = [1, 31, 32, 33, 100, 1000, 4097]


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2605_30842_amd import binding

    binding.load_library()
    yield


def _case(spec, variant="auto", chunk=0, **gen):
    w = generate(spec, **gen)
    say(f"fp8 case {spec.name} B={spec.batch} lens={w.ctx_lens.tolist()[:8]} G={spec.group} D={spec.head_dim} "
        f"{spec.layout} ps={spec.page_size} scales=({spec.k_scale}, {spec.v_scale}) variant={variant} chunk={chunk}")
    out, lse = run(DeviceWorkload(w), make_op(spec, chunk=chunk, variant=variant))
    ro, rl = da.reference(w)
    return w, out, lse, ro, rl


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid"])
@pytest.mark.parametrize("chunk", [0, 32, 96, 2048])
def test_ragged_contiguous(variant, chunk):
    spec = small_spec(WORKLOADS[6], RAGGED, seed=61)
    _, out, lse, ro, rl = _case(spec, variant=variant, chunk=chunk)
    check(out, lse, ro, rl, "fp8", f"fp8 ragged {variant} chunk={chunk}")


@pytest.mark.parametrize("G", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("D", [64, 128])
def test_groups_and_head_dims(G, D):
    spec = small_spec(WORKLOADS[6], [5, 77, 700], seed=62 + G + D).replace(
        num_q_heads=2 * G, num_kv_heads=2, head_dim=D, k_scale=0.0137, v_scale=0.0229)
    _, out, lse, ro, rl = _case(spec, chunk=128)
    check(out, lse, ro, rl, "fp8", f"fp8 G={G} D={D}")


@pytest.mark.parametrize("variant", ["mfma", "mfma_grid"])
@pytest.mark.parametrize("ps", [1, 8, 16, 64, 128])
def test_paged_with_poison(variant, ps):
    spec = small_spec(WORKLOADS[7], RAGGED, seed=63 + ps, max_ctx_len=4224).replace(page_size=ps)
    _, out, lse, ro, rl = _case(spec, variant=variant, chunk=256, spare_pages=3, poison=True)
    check(out, lse, ro, rl, "fp8", f"fp8 paged ps={ps} {variant}")


def test_contiguous_gaps_poisoned():
    spec = small_spec(WORKLOADS[6], [5, 33, 0, 300], seed=64)
    _, out, lse, ro, rl = _case(spec, chunk=64, gap_rows=40, poison=True)
    check(out, lse, ro, rl, "fp8", "fp8 poison contiguous")


def test_one_token_is_exact():
    """L = 1 with power-of-two scales: out = decoded V row * v_scale exactly; L = 0: zeros and -inf."""
    spec = small_spec(WORKLOADS[6], [1, 0, 1], seed=65).replace(k_scale=0.5, v_scale=2.0 ** -5)
    w, out, lse, ro, rl = _case(spec)
    for b in (0, 2):
        v0 = da.fp8_e4m3_value(w.v[w.seq_start[b]]) * spec.v_scale
        assert np.array_equal(out[b].astype(np.float64), np.repeat(v0, spec.group, axis=0))
    assert np.all(out[1] == 0) and np.all(lse[1] == -np.inf)
    check(out, lse, ro, rl, "fp8", "fp8 one token")


@pytest.mark.parametrize("layout_base", [6, 7])
def test_append_codes_bitwise_then_attend(layout_base):
    """The append calls copy code rows: the cache afterwards equals the oracle's append bit for bit."""
    import torch

    kw = {"max_ctx_len": 320} if layout_base == 7 else {}
    spec = small_spec(WORKLOADS[layout_base], [1, 15, 64, 65, 300], seed=66, **kw)
    w = generate(spec)
    nk, nv = draw_new_rows(spec, seed=67)
    say(f"fp8 append {spec.layout}")
    dw = DeviceWorkload(w)
    op = make_op(spec)
    tk, tv = to_torch(nk, "fp8", "cuda:0"), to_torch(nv, "fp8", "cuda:0")
    if spec.layout == "paged":
        op.append_paged(tk, tv, dw.k, dw.v, dw.block_table, dw.ctx_lens, spec.max_ctx_len)
        want_k = da.append_paged(w.k_pages, w.block_table, w.ctx_lens, nk)
        want_v = da.append_paged(w.v_pages, w.block_table, w.ctx_lens, nv)
    else:
        op.append(tk, tv, dw.k, dw.v, dw.seq_start, dw.ctx_lens, spec.max_ctx_len)
        want_k = da.append_contiguous(w.k, w.seq_start, w.ctx_lens, nk)
        want_v = da.append_contiguous(w.v, w.seq_start, w.ctx_lens, nv)
    torch.cuda.synchronize()
    assert np.array_equal(dw.k.cpu().numpy(), want_k) and np.array_equal(dw.v.cpu().numpy(), want_v)
    out, lse = run(dw, op)
    if spec.layout == "paged":
        w.k_pages, w.v_pages = want_k, want_v
    else:
        w.k, w.v = want_k, want_v
    ro, rl = da.reference(w)
    check(out, lse, ro, rl, "fp8", f"fp8 append-then-attend {spec.layout}")


@pytest.mark.parametrize("layout_base", [6, 7])
def test_fused_append_matches_two_calls(layout_base):
    """One launch (store then attend) gives the same cache and output bits as the two calls."""
    import torch

    kw = {"max_ctx_len": 320} if layout_base == 7 else {}
    spec = small_spec(WORKLOADS[layout_base], [1, 33, 200, 300], seed=68, **kw)
    w = generate(spec)
    nk, nv = draw_new_rows(spec, seed=69)
    say(f"fp8 fused append {spec.layout}")
    tk, tv = to_torch(nk, "fp8", "cuda:0"), to_torch(nv, "fp8", "cuda:0")
    a, b = DeviceWorkload(w), DeviceWorkload(w)
    op = make_op(spec, chunk=64)
    if spec.layout == "paged":
        op.append_paged(tk, tv, a.k, a.v, a.block_table, a.ctx_lens, spec.max_ctx_len)
        out_a, lse_a = op.forward_paged(a.q, a.k, a.v, a.block_table, a.ctx_lens, spec.max_ctx_len)
        out_b, lse_b = op.append_forward_paged(b.q, tk, tv, b.k, b.v, b.block_table, b.ctx_lens, spec.max_ctx_len)
    else:
        op.append(tk, tv, a.k, a.v, a.seq_start, a.ctx_lens, spec.max_ctx_len)
        out_a, lse_a = op.forward(a.q, a.k, a.v, a.seq_start, a.ctx_lens, spec.max_ctx_len)
        out_b, lse_b = op.append_forward(b.q, tk, tv, b.k, b.v, b.seq_start, b.ctx_lens, spec.max_ctx_len)
    torch.cuda.synchronize()
    assert torch.equal(a.k, b.k) and torch.equal(a.v, b.v)
    assert torch.equal(out_a, out_b)


@pytest.mark.parametrize("i", [6, 7])
def test_full_workload_every_output(i):
    import torch

    w = generate(WORKLOADS[i])
    say(f"fp8 full workload {i} {w.spec.name} kv_bytes={w.kv_bytes}")
    dw = DeviceWorkload(w)
    out, lse = run(dw, make_op(w.spec))
    del dw
    torch.cuda.empty_cache()
    ro, rl = da.reference(w)
    err = check(out, lse, ro, rl, "fp8", w.spec.name)
    say(f"  max |err| over every output {err:.3e}")
