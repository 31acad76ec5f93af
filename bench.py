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
oracle timed on a bounded sample as a reported baseline. The same run also
times, with the same rules, the headline workload with its K and V caches in
the other placement, the other workloads of the 32k-128k range (batch 16
ragged up to 64K, batch 64 paged, batch 8 at 128K), and a streaming read of
4 GiB and of the headline's byte count (the practical read ceiling), and a
bare read of the headline's cache with the kernel's grid and per-lane loads
(the ceiling of its access pattern); those go under config.also and
roofline.read_ceiling (--no-also skips them).
"""

from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 matrix-core peak
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = ["paper_2605_30842_amd/csrc/api.cpp", "paper_2605_30842_amd/csrc/plan.h",
                  "paper_2605_30842_amd/csrc/attn_common.h",
                  "paper_2605_30842_amd/csrc/kernel_mfma.hip", "paper_2605_30842_amd/csrc/kernel_valu.hip"]
PREFILL_SOURCES = ["paper_2605_30842_amd/csrc/api_prefill.cpp", "paper_2605_30842_amd/csrc/attn_common.h",
                   "paper_2605_30842_amd/csrc/prefill.h", "paper_2605_30842_amd/csrc/kernel_prefill.hip"]
APPEND_SOURCES = ["paper_2605_30842_amd/csrc/api.cpp", "paper_2605_30842_amd/csrc/kv_append.h",
                  "paper_2605_30842_amd/csrc/kernel_append.hip"]
APPEND_PROFILED = (2, 5)  # decode workloads whose standalone append is traced (contiguous, paged)
COPY_CAL_BYTES = 256 << 20  # size of the copy used to calibrate FETCH_SIZE / WRITE_SIZE
METRIC = "decode-attention effective HBM GB/s (% of peak) and µs/step at 32k-128k ctx"
MALL_BYTES = 256 << 20


def _args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=2,
                    help="named workload 1..7 (2 = the headline one; 6, 7 = FP8 KV variants of 2 and 5)")
    ap.add_argument("--op", default="attention", choices=["attention", "append", "step", "fused"],
                    help="attention: the decode-attention call; append: the KV-append call alone; "
                         "step: the append call then the attention call; fused: both in one launch")
    ap.add_argument("--variant", default="auto", choices=["auto", "mfma", "mfma_grid", "valu"])
    ap.add_argument("--chunk", type=int, default=0, help="tokens per split (0 = planned)")
    ap.add_argument("--kv-placement", default="offset", choices=["offset", "separate"],
                    help="offset: K and V of each copy in one allocation, V's base 256 bytes past K's modulo 512 "
                         "(the placement the C header recommends); separate: two allocations (bases equal modulo 4096)")
    ap.add_argument("--copies", type=int, default=0, help="KV copies to cycle over (0 = enough to exceed the LLC)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="budget of the CPU oracle baseline (0 = skip)")
    ap.add_argument("--timing", default="graph", choices=["graph", "eager"],
                    help="graph: replay captured launches (no host launch cost in the timed region)")
    ap.add_argument("--probe", choices=["read", "copy"], default=None,
                    help="instead of attention, time the streaming-read or copy probe kernel")
    ap.add_argument("--probe-bytes", type=int, default=4 << 30)
    ap.add_argument("--probe-blocks", type=int, default=4096)
    ap.add_argument("--prefill", type=int, default=0,
                    help="instead of decode, time the prefill-attention call on named prefill workload N (1..3)")
    ap.add_argument("--no-also", dest="also", action="store_false",
                    help="time only the named workload (by default the run also times the other placement of its "
                         "K/V caches, the other long-context workloads and the streaming-read ceiling)")
    ap.add_argument("--also-workloads", type=lambda s: [int(x) for x in s.split(",") if x], default=[3, 4, 5],
                    help="comma-separated workloads timed beside the headline (default 3,4,5)")
    ap.add_argument("--also-steps", type=int, default=200, help="timed steps of each of those workloads")
    ap.add_argument("--summarize", metavar="DIR", default=None,
                    help="write profiles/ summaries from rocprofv3 outputs under DIR (layout in summarize())")
    return ap.parse_args()


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def kernel_source_hash(sources=KERNEL_SOURCES) -> str:
    """Hash of the sources' code: comments and whitespace do not count, so a
    recorded profile stays valid across edits that change no code."""
    import re

    h = hashlib.sha256()
    for rel in sources:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def _counter_medians(path):
    """Median per counter over dispatches of the attention kernel (or of the copy probe)."""
    vals = {}
    for f in glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            k = r["Kernel_Name"]
            kind = "attn" if ("decode_" in k or "prefill_" in k) else ("copy" if "copy_kernel" in k else None)
            if kind:
                vals.setdefault((kind, r["Counter_Name"]), []).append(float(r["Counter_Value"]))
    return {k: sorted(v)[len(v) // 2] for k, v in vals.items()}


# Counter passes of each workload (one rocprofv3 --pmc run each, within the
# per-block limits: at most 8 SQ, 4 TCC and 2 GRBM counters per run).
COUNTER_PASSES = {
    "sq": "SQ_WAVES SQ_WAVE_CYCLES SQ_BUSY_CU_CYCLES SQ_ACTIVE_INST_VALU SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_LDS "
          "SQ_LDS_IDX_ACTIVE SQ_LDS_BANK_CONFLICT GRBM_GUI_ACTIVE GRBM_COUNT",
    "tcc": "TCC_HIT_sum TCC_MISS_sum TCC_EA0_RDREQ_sum TCC_BUBBLE_sum",
    "tcc2": "TCC_EA0_RDREQ_32B_sum TCC_EA0_RDREQ_DRAM_sum",
}


def _gpu_agent(path):
    for f in glob.glob(os.path.join(path, "**", "*agent_info.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r.get("Agent_Type") == "GPU":
                return r
    return None


def _derived_counters(d, tag, kv_bytes):
    """Occupancy, VALU / MFMA busy, LDS bank conflicts, L2 hits and EA read bytes of the attention kernel.

    Medians over its dispatches of the passes in COUNTER_PASSES; None if the
    runs are absent. The busy and conflict percentages use rocprofv3's own
    definitions (VALUBusy, MfmaUtil, LDSBankConflict) with the GPU-active
    cycles of one XCD (a dispatch row sums GRBM_GUI_ACTIVE over the XCDs).
    SQ_WAVE_CYCLES / SQ_BUSY_CU_CYCLES (both in quad-cycles, summed over
    SIMDs) is the mean number of resident waves per SIMD while busy: it reads
    1.0 for a grid of one 4-wave workgroup per CU. Read bytes come from
    FETCH_SIZE with the copy calibration, not from the request counts, whose
    size classes (TCC_BUBBLE reads 0) do not add up on this GPU.
    """
    m = {}
    for sub in COUNTER_PASSES:
        for (kind, name), v in _counter_medians(os.path.join(d, "pmc", f"{tag}_{sub}")).items():
            if kind == "attn":
                m[name] = v
    ag = _gpu_agent(os.path.join(d, "pmc", f"{tag}_sq"))
    if "SQ_WAVES" not in m or "TCC_HIT_sum" not in m or ag is None:
        return None
    cu, simd, xcc = int(ag["Cu_Count"]), int(ag["Simd_Count"]), int(ag["Num_Xcc"])
    gui = m["GRBM_GUI_ACTIVE"] / xcc
    out = {"raw": {k: m[k] for k in sorted(m)},
           "waves": int(m["SQ_WAVES"]),
           "mean_waves_per_simd_while_busy": round(m["SQ_WAVE_CYCLES"] / m["SQ_BUSY_CU_CYCLES"], 2),
           "simds_per_cu": int(ag["Simd_Per_Cu"]),
           "valu_busy_pct": round(100 * m["SQ_ACTIVE_INST_VALU"] / cu / gui, 2),
           "mfma_util_pct": round(100 * m["SQ_VALU_MFMA_BUSY_CYCLES"] / (gui * simd), 2),
           "lds_bank_conflict_pct": round(100 * m["SQ_LDS_BANK_CONFLICT"] / gui / cu, 3),
           "lds_conflict_cycles_per_active_cycle": round(m["SQ_LDS_BANK_CONFLICT"] / max(m["SQ_LDS_IDX_ACTIVE"], 1), 4),
           "l2_hit_pct": round(100 * m["TCC_HIT_sum"] / max(m["TCC_HIT_sum"] + m["TCC_MISS_sum"], 1), 2)}
    if "TCC_EA0_RDREQ_DRAM_sum" in m:
        out["ea_read_requests_to_dram_pct"] = round(100 * m["TCC_EA0_RDREQ_DRAM_sum"] / max(m["TCC_EA0_RDREQ_sum"], 1), 2)
    return out


def _short_kernel_name(full):
    """decode_mfma_queue_kernel<128, Layout 1, true> -> decode_mfma_queue_D128_paged_fp8 (and similar).

    A bool template argument is the FP8 switch of the MFMA decode kernels
    and the paged switch of the others.
    """
    import re

    m = re.search(r"((?:decode|prefill)_\w+?|kv_append)(?:_kernel)?<([^>]*)>", full)
    if not m:
        return re.sub(r"\W+", "_", full.split("<")[0]).strip("_")[:60]
    base, args = m.group(1), m.group(2)
    parts = [x.strip() for x in re.split(r",\s*(?![^()]*\))", args)]
    name = base
    for a in parts:
        lay = re.search(r"Layout\)(\d)", a)
        if lay:
            name += "_" + ["contig", "paged", "pagedfine"][int(lay.group(1))]
        elif a.isdigit():
            name += f"_D{a}" if a in ("64", "128") else f"_{a}"
        elif "Bf16" in a:
            name += "_bf16"
        elif a == "float":
            name += "_f32"
        elif a in ("true", "false") and base.startswith("decode_mfma"):
            name += "_fp8" if a == "true" else ""
        elif a in ("true", "false"):
            name += "_paged" if a == "true" else "_contig"
    return name


def _kernel_stats(path):
    rows = []
    for f in glob.glob(os.path.join(path, "**", "*kernel_stats.csv"), recursive=True):
        rows += list(csv.DictReader(open(f)))
    return rows


def summarize(a):
    """profiles/<kernel>_<workload>.md from the rocprofv3 runs under DIR.

    Expected layout (each made by the command shown in the summary):
      DIR/prof/w<N>/, DIR/prof/p<N>/   --kernel-trace --stats of the default bench run of decode workload N,
                                       or of `--prefill N`
      DIR/pmc/w<N>_fetch, DIR/pmc/w<N>_write (and p<N>_...)   FETCH_SIZE / WRITE_SIZE runs of the same
      DIR/pmc/copy_fetch, DIR/pmc/copy_write   the same counters on a 256 MiB copy
    """
    from workloads.synth import PREFILL_WORKLOADS, WORKLOADS, generate, generate_prefill

    d = a.summarize
    cal_f = _counter_medians(os.path.join(d, "pmc", "copy_fetch")).get(("copy", "FETCH_SIZE"))
    cal_w = _counter_medians(os.path.join(d, "pmc", "copy_write")).get(("copy", "WRITE_SIZE"))
    fetch_scale = COPY_CAL_BYTES / 1024 / cal_f if cal_f else None
    write_scale = COPY_CAL_BYTES / 1024 / cal_w if cal_w else None
    os.makedirs(PROFILES, exist_ok=True)
    jobs = ([("w", i, spec) for i, spec in WORKLOADS.items()] +
            [("p", i, spec) for i, spec in PREFILL_WORKLOADS.items()] +
            [("a", i, WORKLOADS[i]) for i in APPEND_PROFILED])
    for tag, i, spec in jobs:
        stats = _kernel_stats(os.path.join(d, "prof", f"{tag}{i}"))
        if not stats:
            continue
        key = {"w": "decode_", "p": "prefill_", "a": "kv_append"}[tag]
        attn = [r for r in stats if key in r["Name"]]
        if tag == "a":
            # K and V rows of every (sequence, KV head): read from the inputs, written to the cache
            units = {"moved_bytes": 2 * 2 * spec.batch * spec.num_kv_heads * spec.head_dim * spec.elem_bytes}
            sources = APPEND_SOURCES
            bench_args = f"--workload {i} --op append --cpu-seconds 0"
            pmc_args = None
        elif tag == "w":
            w = generate(spec)
            units = {"algorithmic_bytes": w.kv_bytes}
            sources = KERNEL_SOURCES
            bench_args = f"--workload {i} --cpu-seconds 0 --no-also"
            pmc_args = f"--workload {i} --timing eager --steps 4 --warmup 1 --cpu-seconds 0 --no-also"
        else:
            pw = generate_prefill(spec)
            units = {"algorithmic_flops": pw.flops, "kv_bytes": pw.kv.kv_bytes}
            sources = PREFILL_SOURCES
            bench_args = f"--prefill {i} --steps 20 --warmup 3 --cpu-seconds 0"
            pmc_args = f"--prefill {i} --steps 3 --warmup 1 --cpu-seconds 0"
        fm = _counter_medians(os.path.join(d, "pmc", f"{tag}{i}_fetch")).get(("attn", "FETCH_SIZE"))
        wm = _counter_medians(os.path.join(d, "pmc", f"{tag}{i}_write")).get(("attn", "WRITE_SIZE"))
        traffic = None
        if fm and wm and fetch_scale and write_scale:
            traffic = round(fm * 1024 * fetch_scale + wm * 1024 * write_scale)
        kname = _short_kernel_name(attn[0]["Name"]) if attn else "none"
        avg_ns = float(attn[0]["AverageNs"]) if attn else None
        rec = {"workload": spec.name, "kernel": kname, "kernel_source_hash": kernel_source_hash(sources),
               "calls": int(attn[0]["Calls"]) if attn else 0, "avg_duration_us": avg_ns / 1e3 if avg_ns else None}
        rec.update(units)
        if tag == "a":
            kv = units["moved_bytes"]
            rec["achieved_GBps_from_trace"] = round(kv / avg_ns, 3) if avg_ns else None
        elif tag == "w":
            kv = units["algorithmic_bytes"]
            rec["achieved_GBps_from_trace"] = round(kv / avg_ns, 1) if avg_ns else None
        else:
            rec["achieved_TFLOPs_from_trace"] = round(units["algorithmic_flops"] / avg_ns / 1e3, 1) if avg_ns else None
            kv = units["kv_bytes"]
        rec.update({"fetch_KiB_per_dispatch": fm, "write_KiB_per_dispatch": wm, "fetch_scale": fetch_scale,
                    "write_scale": write_scale, "traffic_bytes": traffic,
                    "traffic_over_kv_bytes": round(traffic / kv, 4) if traffic else None})
        counters = _derived_counters(d, f"{tag}{i}", kv)
        name = f"{kname}_{spec.name}.md"
        with open(os.path.join(PROFILES, name), "w") as f:
            f.write(f"# {kname} on {spec.name}\n\n")
            f.write("Commands (run from the repository root on the MI355X box, after `cd /tmp && export TMPDIR=/tmp`"
                    " and returning to the root):\n\n```\n")
            f.write(f"rocprofv3 --kernel-trace --stats --output-format csv -d {d}/prof/{tag}{i} -o {tag}{i} -- "
                    f"python3 bench.py {bench_args}\n")
            for c in ("FETCH_SIZE", "WRITE_SIZE") if pmc_args else ():
                sub = "fetch" if c == "FETCH_SIZE" else "write"
                f.write(f"rocprofv3 --pmc {c} --output-format csv -d {d}/pmc/{tag}{i}_{sub} -o {tag}{i}_{sub} -- "
                        f"python3 bench.py {pmc_args}\n")
                f.write(f"rocprofv3 --pmc {c} --output-format csv -d {d}/pmc/copy_{sub} -o copy_{sub} -- "
                        f"python3 bench.py --probe copy --probe-bytes {COPY_CAL_BYTES} --steps 3 --warmup 1\n")
            if counters:
                for sub, names in COUNTER_PASSES.items():
                    f.write(f"rocprofv3 --pmc {names} --output-format csv -d {d}/pmc/{tag}{i}_{sub} -o {tag}{i}_{sub}"
                            f" -- python3 bench.py {pmc_args}\n")
            f.write(f"python3 bench.py --summarize {d}\n```\n\n")
            f.write("Kernel statistics (rocprofv3 --stats, all dispatches of the bench run):\n\n")
            f.write("| kernel | calls | avg us | min us | max us |\n|---|---|---|---|---|\n")
            for r in stats:
                f.write(f"| {_short_kernel_name(r['Name'])} | {r['Calls']} | {float(r['AverageNs'])/1e3:.2f} | "
                        f"{float(r['MinNs'])/1e3:.2f} | {float(r['MaxNs'])/1e3:.2f} |\n")
            if pmc_args:
                f.write("\nHBM traffic per dispatch: FETCH_SIZE and WRITE_SIZE medians (KiB), each scaled by the "
                        f"factor that makes the same counter read {COPY_CAL_BYTES} bytes for a copy of that size.\n\n")
            else:
                f.write("\nA few KB per dispatch: the kernel is bound by launch latency, so no traffic counters were "
                        "taken.\n\n")
            f.write("```json\n" + json.dumps(rec, indent=1) + "\n```\n")
            if counters:
                f.write("\nCounters (medians over the kernel's dispatches in the --pmc runs above; percentages as "
                        "rocprofv3 defines VALUBusy, MfmaUtil and LDSBankConflict, over one XCD's GPU-active cycles; "
                        "rocprofv3 exposes no Infinity Cache (MALL) counters on this system):\n\n")
                f.write("| quantity | value |\n|---|---|\n")
                for k, v in counters.items():
                    if k != "raw":
                        f.write(f"| {k} | {v} |\n")
                f.write("\n```json\n" + json.dumps({"counters_raw": counters["raw"]}, indent=1) + "\n```\n")
        print(f"wrote profiles/{name}", flush=True)


def recorded_traffic(workload_name, sources=KERNEL_SOURCES, unit_key="algorithmic_bytes"):
    """HBM bytes per dispatch from a profiles/ summary of the current kernel sources, else None."""
    for f in glob.glob(os.path.join(PROFILES, f"*_{workload_name}.md")):
        txt = open(f).read()
        if "```json" not in txt:
            continue
        rec = json.loads(txt.split("```json", 1)[1].split("```", 1)[0])
        if rec.get("kernel_source_hash") == kernel_source_hash(sources) and rec.get("traffic_bytes") and \
                unit_key in rec:
            return rec["traffic_bytes"]
    return None


def _probe(a):
    """Streaming read (practical HBM read ceiling) or copy (profiler byte-counter calibration)."""
    import torch

    from paper_2605_30842_amd import binding

    binding.load_probe_library()
    n = a.probe_bytes
    src = torch.ones(n // 4, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src) if a.probe == "copy" else None
    sink = torch.zeros(256 * a.probe_blocks, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    def once():
        if a.probe == "read":
            binding.comem_probe_read(src.data_ptr(), n, sink.data_ptr(), a.probe_blocks, stream.cuda_stream)
        else:
            binding.comem_probe_copy(src.data_ptr(), dst.data_ptr(), n, a.probe_blocks, stream.cuda_stream)

    for _ in range(a.warmup):
        once()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(a.steps):
        once()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / a.steps
    moved = n * (2 if a.probe == "copy" else 1)
    print(json.dumps({"probe": a.probe, "bytes": n, "bytes_moved": moved, "blocks": a.probe_blocks,
                      "us_per_call": round(ms * 1e3, 3), "GB_per_s": round(moved / (ms * 1e-3) / 1e9, 1),
                      "steps": a.steps}), flush=True)


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
            "host_cpus": len(os.sched_getaffinity(0)), "cpu_model": _cpu_model()}


def _prefill_cpu_baseline(pw, budget_s):
    """Time the fp64 prefill oracle on whole rows (new token, query head) of the same workload."""
    import oracle.prefill_attention as pa

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # noqa: BLE001
        threads = 1
    s = pw.kv.spec
    b = 0
    M = int(pw.q_lens[b])
    L = int(pw.kv.ctx_lens[b])
    rows = [(b, M - 1 - i, h) for i in range(min(M, 8)) for h in range(s.num_q_heads)]
    flops = sum(4 * s.head_dim * (L - M + i + 1) for (_, i, _) in rows)
    t0 = time.perf_counter()
    pa.prefill_attention_rows(pw, rows)
    one = time.perf_counter() - t0
    reps = max(1, int(budget_s / max(one, 1e-3)))
    t0 = time.perf_counter()
    for _ in range(reps):
        pa.prefill_attention_rows(pw, rows)
    dt = (time.perf_counter() - t0) / reps
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} oracle calls over the last {min(M, 8)} new tokens x {s.num_q_heads} heads of "
                      f"sequence 0 ({L} cached tokens), float64 numpy",
            "seconds_per_call": round(dt, 4), "host_cpus": len(os.sched_getaffinity(0)), "cpu_model": _cpu_model()}


def _prefill(a):
    """Prefill attention (cached prefix + causal new tokens) on a named prefill workload."""
    import torch

    from paper_2605_30842_amd import binding
    from paper_2605_30842_amd.binding import DecodeAttention
    from workloads.synth import PREFILL_WORKLOADS, generate_prefill

    binding.load_library()
    pspec = PREFILL_WORKLOADS[a.prefill]
    pw = generate_prefill(pspec)
    s = pw.kv.spec
    dev = torch.device("cuda:0")

    def dev_t(x):
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)

    q = dev_t(pw.q)
    q_start = torch.from_numpy(pw.q_start.astype(np.int64)).to(dev)
    q_lens = torch.from_numpy(pw.q_lens.astype(np.int32)).to(dev)
    ctx = torch.from_numpy(pw.kv.ctx_lens.astype(np.int32)).to(dev)
    paged = s.layout == "paged"
    k = dev_t(pw.kv.k_pages if paged else pw.kv.k)
    v = dev_t(pw.kv.v_pages if paged else pw.kv.v)
    if a.kv_placement == "offset":  # one allocation, V's base 256 bytes past K's modulo 512
        kc, vc = binding.kv_cache_pair(tuple(k.shape), k.dtype, dev)
        kc.copy_(k)
        vc.copy_(v)
        k, v = kc, vc
    v_minus_k = (int(v.data_ptr()) - int(k.data_ptr())) % 4096
    bt = torch.from_numpy(pw.kv.block_table.astype(np.int32)).to(dev) if paged else None
    ss = None if paged else torch.from_numpy(pw.kv.seq_start.astype(np.int64)).to(dev)
    op = DecodeAttention(s.num_q_heads, s.num_kv_heads, s.head_dim, s.dtype, float(s.scale), s.batch,
                         s.max_ctx_len)
    out = torch.empty(q.shape, dtype=torch.float32, device=dev)
    lse = torch.empty(q.shape[:2], dtype=torch.float32, device=dev)
    max_q = int(pw.q_lens.max())

    def step(stream):
        if paged:
            op.prefill_paged(q, q_start, q_lens, max_q, k, v, bt, ctx, s.max_ctx_len, out=out, lse=lse, stream=stream)
        else:
            op.prefill(q, q_start, q_lens, max_q, k, v, ss, ctx, s.max_ctx_len, out=out, lse=lse, stream=stream)

    stream = torch.cuda.current_stream()
    for _ in range(a.warmup):
        step(stream)
    torch.cuda.synchronize()
    eager_out = out.clone()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(a.steps):
        step(stream)
    e1.record(stream)
    torch.cuda.synchronize()
    eager_ms = e0.elapsed_time(e1) / a.steps
    assert torch.equal(out, eager_out), "repeated prefill calls differ"
    assert torch.isfinite(out).all().item()
    flops = pw.flops
    tflops = flops / (eager_ms * 1e-3) / 1e12
    cpu = _prefill_cpu_baseline(pw, a.cpu_seconds) if a.cpu_seconds > 0 else None
    print(json.dumps({
        "metric": "prefill-attention TFLOP/s (algorithmic: 4 * head_dim * query heads * visible pairs)",
        "value": round(tflops, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(eager_ms, 6), "us_per_step": round(eager_ms * 1e3, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": pspec.name, "batch": s.batch, "num_q_heads": s.num_q_heads,
                   "num_kv_heads": s.num_kv_heads, "head_dim": s.head_dim, "layout": s.layout,
                   "page_size": s.page_size, "new_tokens": int(pw.q_lens.sum()),
                   "cached_tokens": int(pw.kv.ctx_lens.sum()), "flops_per_step": flops, "timing": "eager",
                   "kv_placement": a.kv_placement, "v_minus_k_base_mod_4096": v_minus_k},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 3), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": recorded_traffic(pspec.name, PREFILL_SOURCES, "algorithmic_flops")},
        "cpu_baseline": cpu,
    }), flush=True)


def _measure_decode(a, wl, placement, steps, warmup, op_kind="attention", single_calls=True, want_w=False):
    """Time `steps` decode steps of named workload `wl` with graph (or eager) timing; return a result dict.

    Inputs are drawn on the host, copied to HBM before the timed region, and
    (for workloads that fit the last-level cache) replicated so that every
    step reads memory no recent step touched. Graph replays are checked bit
    for bit against the eager result.
    """
    import torch

    from paper_2605_30842_amd import binding
    from paper_2605_30842_amd.binding import DecodeAttention
    from workloads.synth import WORKLOADS, draw_new_rows, generate

    binding.load_library()
    spec = WORKLOADS[wl]
    w = generate(spec)
    kv_bytes = w.kv_bytes
    dev = torch.device("cuda:0")

    def dev_t(x, dtype=spec.dtype):
        if dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)  # f32 values or fp8 codes (uint8)

    q = dev_t(w.q, spec.q_dtype)
    ctx = torch.from_numpy(w.ctx_lens.astype(np.int32)).to(dev)
    copies = a.copies or max(1, math.ceil(4 * MALL_BYTES / kv_bytes))
    paged = spec.layout == "paged"
    k0 = dev_t(w.k_pages if paged else w.k)
    v0 = dev_t(w.v_pages if paged else w.v)
    if placement == "offset":
        kv = []
        for _ in range(copies):
            kc, vc = binding.kv_cache_pair(tuple(k0.shape), k0.dtype, dev)
            kc.copy_(k0)
            vc.copy_(v0)
            kv.append((kc, vc))
        del k0, v0
    else:
        kv = [(k0, v0)] + [(k0.clone(), v0.clone()) for _ in range(copies - 1)]
    v_minus_k = sorted({(int(vc.data_ptr()) - int(kc.data_ptr())) % 4096 for kc, vc in kv})
    bt = torch.from_numpy(w.block_table.astype(np.int32)).to(dev) if paged else None
    ss = None if paged else torch.from_numpy(w.seq_start.astype(np.int64)).to(dev)
    scales = dict(k_scale=spec.k_scale, v_scale=spec.v_scale) if spec.dtype == "fp8" else {}
    op = DecodeAttention(spec.num_q_heads, spec.num_kv_heads, spec.head_dim, spec.dtype, float(spec.scale),
                         spec.batch, spec.max_ctx_len, chunk_tokens=a.chunk, variant=a.variant, **scales)
    chunk, splits = op.splits(spec.batch, spec.max_ctx_len)
    out = torch.zeros((spec.batch, spec.num_q_heads, spec.head_dim), dtype=torch.float32, device=dev)
    lse = torch.empty((spec.batch, spec.num_q_heads), dtype=torch.float32, device=dev)
    new_k, new_v = (dev_t(x) for x in draw_new_rows(spec, seed=spec.seed + 100))

    def step(i, stream):
        k, v = kv[i % copies]
        if op_kind == "fused":  # the new token's rows are stored by the attention launch itself
            if paged:
                op.append_forward_paged(q, new_k, new_v, k, v, bt, ctx, spec.max_ctx_len, out=out, lse=lse,
                                        stream=stream)
            else:
                op.append_forward(q, new_k, new_v, k, v, ss, ctx, spec.max_ctx_len, out=out, lse=lse,
                                  stream=stream)
            return
        if op_kind != "attention":  # the new token's rows are stored first (same row on every step)
            if paged:
                op.append_paged(new_k, new_v, k, v, bt, ctx, spec.max_ctx_len, stream=stream)
            else:
                op.append(new_k, new_v, k, v, ss, ctx, spec.max_ctx_len, stream=stream)
        if op_kind != "append":
            if paged:
                op.forward_paged(q, k, v, bt, ctx, spec.max_ctx_len, out=out, lse=lse, stream=stream)
            else:
                op.forward(q, k, v, ss, ctx, spec.max_ctx_len, out=out, lse=lse, stream=stream)

    stream = torch.cuda.current_stream()
    for i in range(warmup):
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

    eager_ms = timed(lambda: [step(i, stream) for i in range(steps)], steps)
    ms = eager_ms
    if a.timing == "graph":
        # One graph holds at least 16 launches, cycling over the KV copies, so
        # the gap between graph launches is spread over many steps; the timed
        # region replays it, and a second graph of the remaining launches
        # (the copies continue in order), so that exactly `steps` are timed.
        per_graph = copies * max(1, -(-16 // copies))
        full, rem = divmod(steps, per_graph)

        def capture(n):
            g = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream()
            side.wait_stream(stream)
            with torch.cuda.graph(g, stream=side):
                for i in range(n):
                    step(i, torch.cuda.current_stream())
            torch.cuda.synchronize()
            return g

        graphs = [capture(per_graph)] * full + ([capture(rem)] if rem else [])
        for g in set(graphs):
            for _ in range(3):  # every replay must reproduce the eager result bit for bit (the copies are equal)
                out.zero_()
                g.replay()
                torch.cuda.synchronize()
                assert torch.equal(out, eager_out), "graph replay differs from eager result"
        ms = timed(lambda: [g.replay() for g in graphs], steps)
    assert torch.isfinite(out).all().item()
    pct = None
    if single_calls:
        # Spread of single calls (after the timed region): each of 100 eager
        # calls bracketed by its own pair of events on the stream.
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(100)]
        for i, (b0, b1) in enumerate(ev):
            b0.record(stream)
            step(i, stream)
            b1.record(stream)
        torch.cuda.synchronize()
        per_call = sorted(b0.elapsed_time(b1) * 1e3 for b0, b1 in ev)
        pct = {f"p{q}": round(per_call[min(len(per_call) - 1, q * len(per_call) // 100)], 3) for q in (10, 50, 90)}
    res = {"spec": spec, "ms": ms, "eager_ms": eager_ms, "single_call_us": pct, "kv_bytes": kv_bytes,
           "copies": copies, "v_minus_k": v_minus_k, "chunk": chunk, "splits": splits,
           "ctx_len_total": int(w.ctx_lens.sum()), "w": w if want_w else None}
    del kv, q, out, lse, op
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def _read_ceiling(nbytes, steps, blocks=4096):
    """Streaming read of `nbytes` (the practical HBM read ceiling), timed like the decode steps: graph replays
    of back-to-back launches, cycling over enough buffers that each launch reads memory no recent one touched."""
    import torch

    from paper_2605_30842_amd import binding

    binding.load_probe_library()
    copies = max(1, math.ceil(4 * MALL_BYTES / nbytes))
    bufs = [torch.ones(nbytes // 4, dtype=torch.int32, device="cuda") for _ in range(copies)]
    sink = torch.zeros(256 * blocks, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    per_graph = copies * max(1, -(-16 // copies))
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.graph(g, stream=side):
        for i in range(per_graph):
            binding.comem_probe_read(bufs[i % copies].data_ptr(), nbytes, sink.data_ptr(), blocks,
                                     torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    reps = max(1, steps // per_graph)
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * per_graph)
    del bufs, sink, g
    torch.cuda.empty_cache()
    return {"bytes": nbytes, "blocks": blocks, "us_per_call": round(us, 3),
            "GBps": round(nbytes / (us * 1e-6) / 1e9, 1), "frac_of_peak": round(nbytes / (us * 1e-6) / 1e9 /
                                                                               PEAK_HBM_GBPS, 4),
            "buffers_cycled": copies}


def _read_kv_heads(spec, tokens, chunk, placement, steps):
    """A bare read of the headline cache with the decode kernel's grid and per-lane loads
    (comem_probe_read_kv_heads), timed like the decode steps (graph replays, cycling over KV copies placed
    as in the decode measurement): the ceiling of the kernel's access pattern. None where it does not apply
    (paged or ragged caches, head_dim other than 128, fp32, or lengths not a multiple of the split)."""
    import torch

    from paper_2605_30842_amd import binding

    head_bytes = {"bf16": 256, "fp8": 128}.get(spec.dtype)
    if (spec.layout != "contiguous" or spec.batch != 1 or spec.head_dim != 128 or head_bytes is None or
            tokens % chunk != 0 or chunk % 128 != 0):
        return None
    binding.load_probe_library()
    dev = torch.device("cuda:0")
    shape = (tokens, spec.num_kv_heads, spec.head_dim)
    dtype = torch.bfloat16 if spec.dtype == "bf16" else torch.uint8
    kv_bytes = 2 * tokens * spec.num_kv_heads * head_bytes
    copies = max(1, math.ceil(4 * MALL_BYTES / kv_bytes))
    kv = []
    for _ in range(copies):
        if placement == "offset":
            kc, vc = binding.kv_cache_pair(shape, dtype, dev)
        else:
            kc, vc = torch.empty(shape, dtype=dtype, device=dev), torch.empty(shape, dtype=dtype, device=dev)
        kc.view(torch.uint8).fill_(1)
        vc.view(torch.uint8).fill_(1)
        kv.append((kc, vc))
    sink = torch.zeros(256, dtype=torch.int32, device=dev)
    stride = spec.num_kv_heads * head_bytes
    per_graph = copies * max(1, -(-16 // copies))
    stream = torch.cuda.current_stream()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.graph(g, stream=side):
        for i in range(per_graph):
            kc, vc = kv[i % copies]
            binding.comem_probe_read_kv_heads(kc.data_ptr(), vc.data_ptr(), tokens, spec.num_kv_heads, head_bytes,
                                              stride, chunk, sink.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    reps = max(1, steps // per_graph)
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * per_graph)
    del kv, sink, g
    torch.cuda.empty_cache()
    return {"bytes": kv_bytes, "split_tokens": chunk, "kv_placement": placement, "us_per_call": round(us, 3),
            "GBps": round(kv_bytes / (us * 1e-6) / 1e9, 1),
            "frac_of_peak": round(kv_bytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4), "buffers_cycled": copies}


def _summary(r):
    gbps = r["kv_bytes"] / (r["ms"] * 1e-3) / 1e9
    d = {"us_per_step": round(r["ms"] * 1e3, 3), "GBps": round(gbps, 1), "frac_of_peak": round(gbps / PEAK_HBM_GBPS, 4),
         "decode_tok_per_s": round(r["spec"].batch / (r["ms"] * 1e-3), 1), "kv_bytes_per_step": r["kv_bytes"],
         "ctx_len_total": r["ctx_len_total"], "chunk_tokens": r["chunk"], "splits": r["splits"],
         "kv_copies_cycled": r["copies"], "v_minus_k_base_mod_4096": r["v_minus_k"],
         "eager_us_per_step": round(r["eager_ms"] * 1e3, 3)}
    if r["single_call_us"]:
        d["single_call_us"] = r["single_call_us"]
    return d


def main():
    a = _args()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {a.gpus}); this library has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    if a.steps < 1 or a.warmup < 0:
        print("--steps must be at least 1 and --warmup at least 0", file=sys.stderr)
        sys.exit(2)
    if a.probe:
        _probe(a)
        return
    if a.summarize:
        summarize(a)
        return
    if a.prefill:
        _prefill(a)
        return

    r = _measure_decode(a, a.workload, a.kv_placement, a.steps, a.warmup, a.op, single_calls=a.op != "append",
                        want_w=a.cpu_seconds > 0 and a.op == "attention")
    spec = r["spec"]
    ms, eager_ms = r["ms"], r["eager_ms"]
    if a.op == "append":
        row_bytes = spec.batch * spec.num_kv_heads * spec.head_dim * spec.elem_bytes * 2  # K and V rows
        moved = 2 * row_bytes  # each row read once and written once
        gbps = moved / (ms * 1e-3) / 1e9
        print(json.dumps({
            "metric": "kv-append µs/step", "value": round(ms * 1e3, 3), "unit": "µs", "n_gpus": 1,
            "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms, 6), "higher_is_better": False,
            "scaling": "weak", "vs_baseline": None, "dtype": spec.dtype, "data": "synthetic",
            "config": {"workload": spec.name, "op": "append", "batch": spec.batch, "layout": spec.layout,
                       "page_size": spec.page_size, "row_bytes_per_step": row_bytes, "timing": a.timing,
                       "eager_us_per_step": round(eager_ms * 1e3, 3)},
            "roofline": {"bound": "hbm", "achieved": round(gbps, 3), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                         "frac": round(gbps / PEAK_HBM_GBPS, 6), "traffic": None},
            "cpu_baseline": None,
        }), flush=True)
        return
    kv_bytes = r["kv_bytes"]
    gbps = kv_bytes / (ms * 1e-3) / 1e9
    print(f"# headline {spec.name}: {ms * 1e3:.3f} us/step, {gbps:.1f} GB/s", file=sys.stderr, flush=True)
    cpu = _cpu_baseline(r["w"], a.cpu_seconds) if r["w"] is not None else None
    r["w"] = None

    # The rest of the metric's 32k-128k range, the other K/V placement and
    # the read ceiling, measured in the same process with the same rules.
    also = {}
    ceiling = None
    if a.also and a.op == "attention" and a.chunk == 0 and a.variant == "auto":
        other = "separate" if a.kv_placement == "offset" else "offset"
        ro = _measure_decode(a, a.workload, other, a.steps, a.warmup, single_calls=False)
        also[f"{spec.name}@{other}"] = dict(_summary(ro), kv_placement=other)
        print(f"# {spec.name} @{other}: {ro['ms'] * 1e3:.3f} us/step", file=sys.stderr, flush=True)
        for wl in a.also_workloads:
            if wl == a.workload:
                continue
            rw = _measure_decode(a, wl, a.kv_placement, a.also_steps, min(a.warmup, 5), single_calls=False)
            also[rw["spec"].name] = dict(_summary(rw), kv_placement=a.kv_placement)
            print(f"# {rw['spec'].name}: {rw['ms'] * 1e3:.3f} us/step", file=sys.stderr, flush=True)
        ceiling = {"read_4GiB": _read_ceiling(4 << 30, 160), "read_same_bytes": _read_ceiling(kv_bytes, a.steps)}
        pattern = _read_kv_heads(spec, int(r["ctx_len_total"]), r["chunk"], a.kv_placement, a.steps)
        if pattern is not None:
            ceiling["read_kernel_pattern"] = pattern
        print(f"# read ceiling: {ceiling}", file=sys.stderr, flush=True)

    kind = a.variant if a.variant != "auto" else ("valu" if spec.dtype == "f32" else "mfma")
    line = {
        "metric": METRIC,
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": a.steps,
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
            "num_kv_heads": spec.num_kv_heads, "head_dim": spec.head_dim, "ctx_len_total": r["ctx_len_total"],
            "layout": spec.layout, "page_size": spec.page_size, "kv_bytes_per_step": kv_bytes,
            "kv_copies_cycled": r["copies"], "kv_placement": a.kv_placement, "v_minus_k_base_mod_4096": r["v_minus_k"],
            "chunk_tokens": r["chunk"], "splits": r["splits"], "kernel": kind,
            "timing": a.timing, "eager_us_per_step": round(eager_ms * 1e3, 3), "op": a.op,
            "single_call_us": r["single_call_us"],
            "also": also or None,
        },
        "roofline": {
            "bound": "hbm", "achieved": round(gbps, 2), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(gbps / PEAK_HBM_GBPS, 4),
            "traffic": recorded_traffic(spec.name) if a.op == "attention" else None,
            "read_ceiling": ceiling,
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)

if __name__ == "__main__":
    main()
