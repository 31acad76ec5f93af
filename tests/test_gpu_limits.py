"""The largest shapes the C ABI accepts, against the oracle.

- Contexts whose byte offsets pass 4 GiB (one KV head in a buffer 16 or 32
  heads wide): every offset on the path must be 64-bit. Decode over 1.1M
  tokens is checked in full, prefill over 600K tokens on sampled rows.
- Batches at the work queue's limit (4096 sequences), one past it (the
  one-workgroup-per-split grid takes over) and at the grid's limit (65535).
"""

import numpy as np
import pytest

import oracle.decode_attention as da
import oracle.prefill_attention as pa
from tests.gpu_util import DeviceWorkload, abs_values, check, check_prefill, make_op, run, say, to_torch
from workloads.synth import PREFILL_WORKLOADS, WORKLOADS, generate, generate_prefill, small_prefill_spec, small_spec

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2605_30842_amd import binding

    binding.load_library()
    yield


@pytest.fixture(scope="module")
def long_case():
    spec = small_spec(WORKLOADS[2], [1_100_000], seed=90).replace(num_q_heads=8, num_kv_heads=1)
    w = generate(spec)
    return spec, w, *da.reference(w)


@pytest.mark.parametrize("variant", ["mfma", "valu"])
def test_byte_offsets_beyond_4_gib(long_case, variant):
    import torch

    spec, w, ro, rl = long_case
    T = w.k.shape[0]
    say(f"limits: {T} tokens at a 4 KB token stride, {variant}")
    k_big = torch.zeros((T, 16, 128), dtype=torch.bfloat16, device="cuda:0")
    v_big = torch.zeros_like(k_big)
    k, v = k_big[:, :1, :], v_big[:, :1, :]
    k.copy_(to_torch(w.k, "bf16", "cuda:0"))
    v.copy_(to_torch(w.v, "bf16", "cuda:0"))
    assert k.stride(0) * 2 * (T - 1) > 2 ** 32
    q = to_torch(w.q, "bf16", "cuda:0")
    ss = torch.zeros(1, dtype=torch.int64, device="cuda:0")
    cl = torch.full((1,), T, dtype=torch.int32, device="cuda:0")
    op = make_op(spec, variant=variant)
    lse = torch.empty((1, spec.num_q_heads), dtype=torch.float32, device="cuda:0")
    out, lse = op.forward(q, k, v, ss, cl, spec.max_ctx_len, lse=lse)
    torch.cuda.synchronize()
    check(out.cpu().numpy(), lse.cpu().numpy(), ro, rl, "bf16", f"4 GiB offsets {variant}")
    del k_big, v_big, k, v
    torch.cuda.empty_cache()


@pytest.mark.parametrize("variant", ["mfma", "valu"])
def test_page_pool_beyond_4_gib(variant):
    """8200 pages of 64 tokens, one KV head in a 32-head-wide pool (512 KB per page): pages past the
    8192nd start beyond 4 GiB; a random block table reaches them."""
    import torch

    spec = small_spec(WORKLOADS[5], [8200 * 64], seed=99).replace(num_q_heads=8, num_kv_heads=1)
    w = generate(spec)
    P, ps = w.k_pages.shape[:2]
    say(f"limits: paged pool of {P} pages x {ps} tokens at an 8 KB token stride, {variant}")
    k_big = torch.zeros((P, ps, 32, 128), dtype=torch.bfloat16, device="cuda:0")
    v_big = torch.zeros_like(k_big)
    k, v = k_big[:, :, :1, :], v_big[:, :, :1, :]
    k.copy_(to_torch(w.k_pages, "bf16", "cuda:0"))
    v.copy_(to_torch(w.v_pages, "bf16", "cuda:0"))
    assert k.stride(0) * 2 * (P - 1) > 2 ** 32
    q = to_torch(w.q, "bf16", "cuda:0")
    bt = torch.from_numpy(w.block_table.astype(np.int32)).to("cuda:0")
    cl = torch.from_numpy(w.ctx_lens.astype(np.int32)).to("cuda:0")
    lse = torch.empty((1, spec.num_q_heads), dtype=torch.float32, device="cuda:0")
    out, lse = make_op(spec, variant=variant).forward_paged(q, k, v, bt, cl, spec.max_ctx_len, lse=lse)
    torch.cuda.synchronize()
    out, lse = out.cpu().numpy(), lse.cpu().numpy()
    del k_big, v_big, k, v
    torch.cuda.empty_cache()
    ro, rl = da.reference(w)
    check(out, lse, ro, rl, "bf16", f"paged pool past 4 GiB {variant}")


@pytest.mark.parametrize("variant", ["mfma", "valu"])
@pytest.mark.parametrize("B", [4096, 4097])
def test_batches_at_the_work_queue_limit(B, variant):
    lens = np.random.default_rng(92 + B).integers(0, 65, size=B).tolist()
    spec = small_spec(WORKLOADS[2], lens, seed=93)
    w = generate(spec)
    say(f"limits: batch {B}, {variant}")
    out, lse = run(DeviceWorkload(w), make_op(spec, variant=variant))
    ro, rl = da.reference(w)
    check(out, lse, ro, rl, "bf16", f"batch {B} {variant}")


def test_batch_at_the_grid_limit():
    B = 65535
    lens = np.random.default_rng(94).integers(0, 4, size=B)
    spec = small_spec(WORKLOADS[2], lens.tolist(), seed=95)
    w = generate(spec)
    say(f"limits: batch {B}")
    out, lse = run(DeviceWorkload(w), make_op(spec))
    empty = lens == 0
    assert np.all(out[empty] == 0) and np.all(lse[empty] == -np.inf)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse[~empty]))
    r = np.random.default_rng(96)
    rows = sorted({(0, 0), (B - 1, spec.num_q_heads - 1),
                   *[(int(r.integers(B)), int(r.integers(spec.num_q_heads))) for _ in range(60)]})
    ref = da.decode_attention_rows(w, rows)
    check(np.stack([out[b, h] for b, h in rows]), np.array([lse[b, h] for b, h in rows]),
          np.stack([o for o, _ in ref]), np.array([l for _, l in ref]), "bf16", f"batch {B} sampled rows")


def test_prefill_byte_offsets_beyond_4_gib():
    import torch

    spec = small_prefill_spec(PREFILL_WORKLOADS[1], [600_000], [256], seed=97)
    spec = spec.__class__(spec.name, spec.kv.replace(num_q_heads=8, num_kv_heads=1), spec.new_tokens, spec.seed)
    pw = generate_prefill(spec)
    w, s = pw.kv, pw.kv.spec
    T = w.k.shape[0]
    say(f"limits: prefill of 256 new tokens over {T} at an 8 KB token stride")
    k_big = torch.zeros((T, 32, 128), dtype=torch.bfloat16, device="cuda:0")
    v_big = torch.zeros_like(k_big)
    k, v = k_big[:, :1, :], v_big[:, :1, :]
    k.copy_(to_torch(w.k, "bf16", "cuda:0"))
    v.copy_(to_torch(w.v, "bf16", "cuda:0"))
    q = to_torch(pw.q, "bf16", "cuda:0")
    q_start = torch.from_numpy(pw.q_start.astype(np.int64)).to("cuda:0")
    q_lens = torch.from_numpy(pw.q_lens.astype(np.int32)).to("cuda:0")
    ss = torch.zeros(1, dtype=torch.int64, device="cuda:0")
    cl = torch.full((1,), T, dtype=torch.int32, device="cuda:0")
    assert k.stride(0) * 2 * (T - 1) > 2 ** 32
    lse = torch.empty((256, s.num_q_heads), dtype=torch.float32, device="cuda:0")
    out, lse = make_op(s).prefill(q, q_start, q_lens, 256, k, v, ss, cl, s.max_ctx_len, lse=lse)
    torch.cuda.synchronize()
    out, lse = out.cpu().numpy(), lse.cpu().numpy()
    del k_big, v_big, k, v
    torch.cuda.empty_cache()
    r = np.random.default_rng(98)
    rows = sorted({(0, 0, 0), (0, 255, 7), *[(0, int(r.integers(256)), int(r.integers(8))) for _ in range(10)]})
    ref = pa.prefill_attention_rows(pw, rows)
    ref_abs = pa.prefill_attention_rows(abs_values(pw), rows)
    check_prefill(np.stack([out[i, h] for _, i, h in rows]), np.array([lse[i, h] for _, i, h in rows]),
                  np.stack([o for o, _ in ref]), np.array([l for _, l in ref]), np.stack([o for o, _ in ref_abs]),
                  "prefill 4 GiB offsets")
