"""Randomised parity sweep: HIP path vs the fp64 oracle through the C ABI.

Seeded draws cover combinations that the hand-written cases do not
enumerate: cache dtype x kernel variant x layout and page size x GQA group x
head size x split size x ragged lengths with empty sequences, spare pool
pages and NaN poison outside the contexts. Each draw is one test case,
checked element by element against the oracle with the same gates as the
other parity tests: decode attention, decode with the fused append (cache
bits against the oracle's append, output bits against the separate calls)
and prefill over a cached prefix. The sizes keep the whole sweep under a
minute on one GPU; the environment variables COMEM_RANDOM_DECODE_CASES,
COMEM_RANDOM_PREFILL_CASES, COMEM_RANDOM_APPEND_CASES and
COMEM_RANDOM_QUEUE_CASES set larger counts for longer sweeps.
"""

import os

import numpy as np
import pytest

import oracle.decode_attention as da
from tests.gpu_util import DeviceWorkload, check, make_op, run, say
from workloads.synth import WORKLOADS, generate, small_spec

pytestmark = pytest.mark.gpu

VARIANTS = {"f32": ["auto", "valu"], "bf16": ["auto", "mfma", "mfma_grid", "valu"], "fp8": ["auto", "mfma", "mfma_grid"]}
BASE = {("f32", False): 1, ("bf16", False): 2, ("bf16", True): 4, ("fp8", False): 6, ("fp8", True): 7}
NUM_CASES = int(os.environ.get("COMEM_RANDOM_DECODE_CASES", 160))


def draw_case(i: int) -> dict:
    r = np.random.default_rng([2026, i])
    dtype = ["f32", "bf16", "bf16", "fp8"][i % 4]
    paged = dtype != "f32" and bool(r.integers(2))
    variant = str(r.choice(VARIANTS[dtype]))
    nseq = int(r.integers(1, 7))
    long = r.random(nseq) < 0.6
    lens = np.where(long, r.integers(0, 4097, nseq), r.integers(0, 41, nseq))
    lens[r.random(nseq) < 0.15] = 0
    max_ctx = int(max(lens.max(), 1) + r.integers(0, 200))
    ps = int(1 << r.integers(0, 8)) if paged else 0
    chunk = int(32 * r.integers(1, 80)) if r.random() < 0.5 else 0
    if paged and chunk and variant != "valu" and (chunk - 1) // ps + 2 > 2048:
        chunk = 0  # a configured split must fit the matrix-core kernel's block-table copy
    return dict(dtype=dtype, paged=paged, variant=variant, hkv=int(r.integers(1, 4)),
                g=int(r.choice([1, 2, 4, 8, 16])), d=int(r.choice([64, 128])), lens=lens.tolist(),
                max_ctx=max_ctx, ps=ps, chunk=chunk, seed=int(r.integers(1 << 20)), poison=bool(r.integers(2)))


def make_workload(c: dict):
    base = WORKLOADS[BASE[(c["dtype"], c["paged"])]]
    spec = small_spec(base, c["lens"], seed=c["seed"], max_ctx_len=c["max_ctx"]).replace(
        num_q_heads=c["hkv"] * c["g"], num_kv_heads=c["hkv"], head_dim=c["d"])
    if c["paged"]:
        return spec.replace(page_size=c["ps"]), generate(spec.replace(page_size=c["ps"]), spare_pages=2,
                                                        poison=c["poison"])
    return spec, generate(spec, gap_rows=3 if c["poison"] else 0, poison=c["poison"])


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2605_30842_amd import binding

    binding.load_library()
    yield


@pytest.mark.parametrize("i", range(NUM_CASES))
def test_random_case_matches_the_oracle(i):
    c = draw_case(i)
    spec, w = make_workload(c)
    say(f"random case {i}: {c}")
    out, lse = run(DeviceWorkload(w), make_op(spec, chunk=c["chunk"], variant=c["variant"]))
    ro, rl = da.reference(w)
    empty = w.ctx_lens == 0
    assert np.all(out[empty] == 0) and np.all(lse[empty] == -np.inf)
    check(out, lse, ro, rl, c["dtype"], f"random case {i}")


NUM_PREFILL_CASES = int(os.environ.get("COMEM_RANDOM_PREFILL_CASES", 64))


def draw_prefill_case(i: int) -> dict:
    r = np.random.default_rng([2027, i])
    paged = bool(i % 2)
    nseq = int(r.integers(1, 5))
    lens = r.integers(1, 1201, nseq)
    lens[r.random(nseq) < 0.2] = r.integers(1, 40)
    new = np.minimum(lens, r.integers(1, 161, nseq))
    uncached = (r.random(nseq) < 0.3) & (lens <= 160)
    new[uncached] = lens[uncached]
    new[r.random(nseq) < 0.1] = 0
    return dict(paged=paged, hkv=int(r.integers(1, 4)), g=int(r.choice([1, 2, 4, 8, 16])),
                d=int(r.choice([64, 128])), lens=lens.tolist(), new=new.tolist(),
                max_ctx=int(lens.max() + r.integers(0, 100)), ps=int(1 << r.integers(0, 8)) if paged else 0,
                seed=int(r.integers(1 << 20)), poison=bool(r.integers(2)))


@pytest.mark.parametrize("i", range(NUM_PREFILL_CASES))
def test_random_prefill_case_matches_the_oracle(i):
    import oracle.prefill_attention as pa
    from tests.gpu_util import DevicePrefill, abs_values, check_prefill, run_prefill
    from workloads.synth import PREFILL_WORKLOADS, generate_prefill, small_prefill_spec

    c = draw_prefill_case(i)
    spec = small_prefill_spec(PREFILL_WORKLOADS[3 if c["paged"] else 1], c["lens"], c["new"], seed=c["seed"],
                              max_ctx_len=c["max_ctx"])
    kv = spec.kv.replace(num_q_heads=c["hkv"] * c["g"], num_kv_heads=c["hkv"], head_dim=c["d"])
    if c["paged"]:
        kv = kv.replace(page_size=c["ps"])
    spec = spec.__class__(spec.name, kv, spec.new_tokens, spec.seed)
    gen = dict(spare_pages=2, poison=c["poison"]) if c["paged"] else dict(gap_rows=3 if c["poison"] else 0,
                                                                          poison=c["poison"])
    pw = generate_prefill(spec, **gen)
    say(f"random prefill case {i}: {c}")
    out, lse = run_prefill(DevicePrefill(pw), make_op(pw.kv.spec))
    ro, rl = pa.reference(pw)
    ra, _ = pa.reference(abs_values(pw))
    check_prefill(out, lse, ro, rl, ra, f"random prefill case {i}")


NUM_APPEND_CASES = int(os.environ.get("COMEM_RANDOM_APPEND_CASES", 48))


@pytest.mark.parametrize("i", range(NUM_APPEND_CASES))
def test_random_fused_append_case(i):
    """A decode step with its new token: the fused call leaves the oracle's appended cache bit for bit and
    gives the same output bits as the append call followed by the attention call."""
    import torch

    from tests.test_gpu_append import _append, _bitwise, _host, _oracle_append
    from tests.gpu_util import to_torch
    from workloads.synth import draw_new_rows

    c = draw_case(10_000 + i)
    spec, w = make_workload(c)
    new_k, new_v = draw_new_rows(spec, seed=c["seed"] + 1)
    say(f"random fused append case {i}: {c}")
    op = make_op(spec, chunk=c["chunk"], variant=c["variant"])
    nk, nv = to_torch(new_k, spec.dtype, "cuda:0"), to_torch(new_v, spec.dtype, "cuda:0")
    fused = DeviceWorkload(w)
    lse = torch.empty((spec.batch, spec.num_q_heads), dtype=torch.float32, device="cuda:0")
    if c["paged"]:
        out, lse = op.append_forward_paged(fused.q, nk, nv, fused.k, fused.v, fused.block_table, fused.ctx_lens,
                                           spec.max_ctx_len, lse=lse)
    else:
        out, lse = op.append_forward(fused.q, nk, nv, fused.k, fused.v, fused.seq_start, fused.ctx_lens,
                                     spec.max_ctx_len, lse=lse)
    torch.cuda.synchronize()
    want_k, want_v = _oracle_append(w, new_k, new_v)
    _bitwise(_host(fused.k, spec.dtype), want_k, f"case {i} K cache")
    _bitwise(_host(fused.v, spec.dtype), want_v, f"case {i} V cache")
    sep = DeviceWorkload(w)
    _append(sep, op, new_k, new_v)
    out2, lse2 = run(sep, op)
    _bitwise(out.cpu().numpy(), out2, f"case {i} out fused vs separate")
    _bitwise(lse.cpu().numpy(), lse2, f"case {i} lse fused vs separate")
    if c["paged"]:
        w.k_pages, w.v_pages = want_k, want_v
    else:
        w.k, w.v = want_k, want_v
    ro, rl = da.reference(w)
    check(out.cpu().numpy(), lse.cpu().numpy(), ro, rl, spec.dtype, f"random fused append case {i}")


NUM_QUEUE_CASES = int(os.environ.get("COMEM_RANDOM_QUEUE_CASES", 12))


def draw_queue_case(i: int) -> dict:
    """Batches large enough for the work queue's short last splits: 8 KV heads, up to 16K tokens, planned
    splits (at least 4 items per resident workgroup on 256 compute units)."""
    r = np.random.default_rng([2028, i])
    dtype = ["bf16", "fp8"][i % 2]
    paged = bool((i // 2) % 2)
    nseq = int(r.integers(16, 41))
    lens = r.integers(0, 16385, nseq)
    lens[r.random(nseq) < 0.1] = 0
    lens[0] = 16384
    return dict(dtype=dtype, paged=paged, variant=str(r.choice(["auto", "mfma"])), hkv=8,
                g=int(r.choice([4, 8])), d=128, lens=lens.tolist(), max_ctx=16384,
                ps=int(r.choice([2, 16, 64, 128])) if paged else 0, chunk=0, seed=int(r.integers(1 << 20)),
                poison=bool(r.integers(2)))


@pytest.mark.parametrize("i", range(NUM_QUEUE_CASES))
def test_random_queue_case_matches_the_oracle(i):
    import torch

    c = draw_queue_case(i)
    spec, w = make_workload(c)
    op = make_op(spec, chunk=0, variant=c["variant"])
    chunk, splits = op.splits(spec.batch, spec.max_ctx_len)
    resident = 2 * torch.cuda.get_device_properties(0).multi_processor_count
    assert chunk == 1024 and spec.batch * spec.num_kv_heads * splits >= 4 * resident
    say(f"random queue case {i}: {dict(c, lens=c['lens'][:6])}")
    out, lse = run(DeviceWorkload(w), op)
    if c["dtype"] == "bf16":
        ro, rl = da.reference(w)
        check(out, lse, ro, rl, c["dtype"], f"random queue case {i}")
        return
    # FP8: sampled rows of six sequences, the longest among them (the oracle widens a sequence's every code)
    r = np.random.default_rng([2029, i])
    hq = spec.num_q_heads
    seqs = {0, *(int(b) for b in r.choice(spec.batch, size=5, replace=False))}
    rows = sorted({*((b, 0) for b in seqs), *((b, hq - 1) for b in seqs),
                   *((b, int(r.integers(hq))) for b in seqs for _ in range(3))})
    ref = da.decode_attention_rows(w, rows)
    check(np.stack([out[b, h] for b, h in rows]), np.array([lse[b, h] for b, h in rows]),
          np.stack([o for o, _ in ref]), np.array([l for _, l in ref]), c["dtype"], f"random queue case {i}")
    empty = w.ctx_lens == 0
    assert np.all(out[empty] == 0) and np.all(lse[empty] == -np.inf)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(lse[~empty]))
