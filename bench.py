"""Decode-attention bandwidth benchmark (one MI355X).

One step = one call of the whole hot path (split-K partial attention and the
log-sum-exp merge, one kernel launch) over one batch of synthetic input that
is already resident in HBM. The default workload is batch 1, 32 query / 8 KV
heads, head_dim 128, bf16, 32768-token context (128 MiB of K+V per step).
Because that fits the 256 MB last-level cache, the timed steps cycle over
enough identical copies of the cache that each step reads memory no recent
step touched.

Prints one JSON line: effective GB/s = algorithmic K+V bytes / step time,
the roofline object for the kernel (HBM bound, 8 TB/s peak), and the CPU
oracle timed on a bounded sample as a reported baseline.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
METRIC = "decode-attention effective HBM GB/s (% of peak) and µs/step at 32k-128k ctx"
MALL_BYTES = 256 << 20


def _args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=2, help="named workload 1..5 (2 = the headline one)")
    ap.add_argument("--variant", default="auto", choices=["auto", "mfma", "valu"])
    ap.add_argument("--chunk", type=int, default=0, help="tokens per split (0 = planned)")
    ap.add_argument("--copies", type=int, default=0, help="KV copies to cycle over (0 = enough to exceed the LLC)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="budget of the CPU oracle baseline (0 = skip)")
    ap.add_argument("--timing", default="graph", choices=["graph", "eager"],
                    help="graph: replay captured launches (no host launch cost in the timed region)")
    return ap.parse_args()


def _cpu_baseline(w, budget_s):
    """Time the fp64 oracle on whole steps of the same workload (a bounded number of them)."""
    import oracle.decode_attention as da

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # noqa: BLE001
        threads = 1
    spec = w.spec
    # A bounded sample: the first sequences of the batch, enough for about budget_s of work.
    t0 = time.perf_counter()
    da.reference(w) if spec.batch == 1 else da.decode_attention_rows(w, [(0, h) for h in range(spec.num_q_heads)])
    one = time.perf_counter() - t0
    per_bytes = (int(w.ctx_lens[0]) * spec.num_kv_heads * spec.head_dim * 2 * spec.elem_bytes)
    reps = max(1, int(budget_s / max(one, 1e-3)))
    t0 = time.perf_counter()
    for _ in range(reps):
        if spec.batch == 1:
            da.reference(w)
        else:
            da.decode_attention_rows(w, [(0, h) for h in range(spec.num_q_heads)])
    dt = (time.perf_counter() - t0) / reps
    sample = (f"{reps} oracle calls over sequence 0 ({int(w.ctx_lens[0])} tokens, all {spec.num_q_heads} "
              f"query heads) of the same workload, float64 numpy")
    return {"value": round(per_bytes / dt / 1e9, 3), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": sample, "seconds_per_call": round(dt, 4),
            "host_cpus": len(os.sched_getaffinity(0))}


def main():
    a = _args()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {a.gpus}); this build has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2605_30842_amd import binding
    from paper_2605_30842_amd.binding import DecodeAttention
    from workloads.synth import WORKLOADS, generate

    binding.load_library()
    spec = WORKLOADS[a.workload]
    w = generate(spec)
    kv_bytes = w.kv_bytes
    dev = torch.device("cuda:0")

    def dev_t(x):
        if spec.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

    q = dev_t(w.q)
    ctx = torch.from_numpy(w.ctx_lens.astype(np.int32)).to(dev)
    copies = a.copies or max(1, math.ceil(4 * MALL_BYTES / kv_bytes))
    paged = spec.layout == "paged"
    k0 = dev_t(w.k_pages if paged else w.k)
    v0 = dev_t(w.v_pages if paged else w.v)
    kv = [(k0, v0)] + [(k0.clone(), v0.clone()) for _ in range(copies - 1)]
    if paged:
        bt = torch.from_numpy(w.block_table.astype(np.int32)).to(dev)
    else:
        ss = torch.from_numpy(w.seq_start.astype(np.int64)).to(dev)
    op = DecodeAttention(spec.num_q_heads, spec.num_kv_heads, spec.head_dim, spec.dtype, float(spec.scale),
                         spec.batch, spec.max_ctx_len, chunk_tokens=a.chunk, variant=a.variant)
    chunk, splits = op.splits(spec.batch, spec.max_ctx_len)
    out = torch.empty((spec.batch, spec.num_q_heads, spec.head_dim), dtype=torch.float32, device=dev)
    lse = torch.empty((spec.batch, spec.num_q_heads), dtype=torch.float32, device=dev)
    def step(i, stream):
        k, v = kv[i % copies]
        if paged:
            op.forward_paged(q, k, v, bt, ctx, spec.max_ctx_len, out=out, lse=lse, stream=stream)
        else:
            op.forward(q, k, v, ss, ctx, spec.max_ctx_len, out=out, lse=lse, stream=stream)

    stream = torch.cuda.current_stream()
    for i in range(a.warmup):
        step(i, stream)
    torch.cuda.synchronize()
    eager_out = out.clone()

    def timed(run_steps, n):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        run_steps()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    eager_ms = timed(lambda: [step(i, stream) for i in range(a.steps)], a.steps)
    steps = a.steps
    ms = eager_ms
    if a.timing == "graph":
        # One graph holds one launch per KV copy; the timed region replays it.
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.graph(graph, stream=side):
            for i in range(copies):
                step(i, torch.cuda.current_stream())
        torch.cuda.synchronize()
        for _ in range(3):  # every replay must reproduce the eager result bit for bit
            out.zero_()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(out, eager_out), "graph replay differs from eager result"
        replays = max(1, -(-a.steps // copies))
        steps = replays * copies
        ms = timed(lambda: [graph.replay() for _ in range(replays)], steps)
    gbps = kv_bytes / (ms * 1e-3) / 1e9
    assert torch.isfinite(out).all().item()

    cpu = _cpu_baseline(w, a.cpu_seconds) if a.cpu_seconds > 0 else None
    kind = "mfma" if (a.variant == "mfma" or (a.variant == "auto" and spec.dtype == "bf16")) else "valu"
    line = {
        "metric": METRIC,
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms, 6),
        "us_per_step": round(ms * 1e3, 3),
        "pct_of_peak": round(100 * gbps / PEAK_HBM_GBPS, 2),
        "decode_tok_per_s": round(spec.batch / (ms * 1e-3), 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic",
        "config": {
            "workload": spec.name, "batch": spec.batch, "num_q_heads": spec.num_q_heads,
            "num_kv_heads": spec.num_kv_heads, "head_dim": spec.head_dim, "ctx_len_total": int(w.ctx_lens.sum()),
            "layout": spec.layout, "page_size": spec.page_size, "kv_bytes_per_step": kv_bytes,
            "kv_copies_cycled": copies, "chunk_tokens": chunk, "splits": splits, "kernel": kind,
            "timing": a.timing, "eager_us_per_step": round(eager_ms * 1e3, 3),
        },
        "roofline": {
            "bound": "hbm", "achieved": round(gbps, 2), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(gbps / PEAK_HBM_GBPS, 4), "traffic": None,
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
