"""Helpers shared by the GPU tests: move a drawn workload to the device, run
the HIP path through the C ABI, and compare with the oracle."""

from __future__ import annotations

import sys

import numpy as np

TOL_BF16_ABS, TOL_BF16_REL = 2e-3, 1e-2  # official gate for bf16 inputs with fp32 accumulation
TOL_F32_ABS = 1e-5                        # official gate for fp32 inputs
TOL_DIAG = 1e-4                           # internal gate: |err| <= 1e-4 * max(1, max|ref|)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_torch(arr, dtype, device):
    """bf16 bit patterns -> a bfloat16 tensor; fp8 codes stay uint8; other arrays as they are."""
    import torch

    if dtype == "bf16" and arr.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr)).to(device)


class DeviceWorkload:
    """Device copies of a drawn workload's arrays."""

    def __init__(self, w, device="cuda:0"):
        import torch

        s = w.spec
        self.w = w
        self.spec = s
        self.q = to_torch(w.q, s.q_dtype, device)
        self.ctx_lens = torch.from_numpy(w.ctx_lens.astype(np.int32)).to(device)
        if s.layout == "paged":
            self.k = to_torch(w.k_pages, s.dtype, device)
            self.v = to_torch(w.v_pages, s.dtype, device)
            self.block_table = torch.from_numpy(w.block_table.astype(np.int32)).to(device)
        else:
            self.k = to_torch(w.k, s.dtype, device)
            self.v = to_torch(w.v, s.dtype, device)
            self.seq_start = torch.from_numpy(w.seq_start.astype(np.int64)).to(device)


def make_op(spec, chunk=0, variant="auto", max_batch=None, max_ctx_len=None, debug_checks=False):
    from paper_2605_30842_amd.binding import DecodeAttention

    scales = dict(k_scale=spec.k_scale, v_scale=spec.v_scale) if spec.dtype == "fp8" else {}
    return DecodeAttention(spec.num_q_heads, spec.num_kv_heads, spec.head_dim, spec.dtype, float(spec.scale),
                           max_batch or spec.batch, max_ctx_len or spec.max_ctx_len, chunk_tokens=chunk,
                           variant=variant, debug_checks=debug_checks, **scales)


def run(dw: DeviceWorkload, op, want_lse=True, max_ctx_len=None):
    """One call of the HIP path; returns (out, lse) as numpy float32 (lse None if not asked)."""
    import torch

    s = dw.spec
    B = s.batch
    lse = torch.empty((B, s.num_q_heads), dtype=torch.float32, device=dw.q.device) if want_lse else None
    mcl = s.max_ctx_len if max_ctx_len is None else max_ctx_len
    if s.layout == "paged":
        out, lse = op.forward_paged(dw.q, dw.k, dw.v, dw.block_table, dw.ctx_lens, mcl, lse=lse)
    else:
        out, lse = op.forward(dw.q, dw.k, dw.v, dw.seq_start, dw.ctx_lens, mcl, lse=lse)
    torch.cuda.synchronize()
    return out.cpu().numpy(), (None if lse is None else lse.cpu().numpy())


def check(out, lse, ref_out, ref_lse, dtype, what=""):
    """Assert the official gate (and, for bf16 and fp8 caches, the internal diagnostic gate); return max |err|."""
    out = np.asarray(out, dtype=np.float64)
    ref_out = np.asarray(ref_out, dtype=np.float64)
    assert out.shape == ref_out.shape, what
    assert np.all(np.isfinite(out)), f"{what}: non-finite output"
    err = np.abs(out - ref_out)
    scale = max(1.0, float(np.abs(ref_out).max(initial=0.0)))
    if dtype == "f32":
        assert err.max(initial=0) <= TOL_F32_ABS, f"{what}: max |err| {err.max():.3e}"
    else:
        bad = err > TOL_BF16_ABS + TOL_BF16_REL * np.abs(ref_out)
        assert not bad.any(), f"{what}: {bad.sum()} elements outside 2e-3 + 1e-2|ref| (max {err.max():.3e})"
        assert err.max(initial=0) <= TOL_DIAG * scale, f"{what}: diagnostic max |err| {err.max():.3e}"
    if lse is not None and ref_lse is not None:
        lse = np.asarray(lse, dtype=np.float64)
        ref_lse = np.asarray(ref_lse, dtype=np.float64)
        inf = np.isinf(ref_lse)
        assert np.array_equal(np.isinf(lse), inf), f"{what}: lse -inf pattern"
        assert np.all(lse[inf] == ref_lse[inf])
        lerr = np.abs(lse[~inf] - ref_lse[~inf])
        lim = (TOL_F32_ABS if dtype == "f32" else TOL_DIAG) * np.maximum(1.0, np.abs(ref_lse[~inf]))
        assert np.all(lerr <= lim), f"{what}: lse max err {lerr.max(initial=0):.3e}"
    return float(err.max(initial=0.0))


# ------------------------------------------------------------------ prefill

PREFILL_P_ROUNDING = 2.0 ** -15  # relative error of a probability split into two bf16 for the matrix cores


class DevicePrefill:
    """Device copies of a drawn prefill workload: the cache side plus the packed new-token queries."""

    def __init__(self, pw, device="cuda:0"):
        import torch

        self.pw = pw
        self.kv = DeviceWorkload(pw.kv, device)
        s = pw.kv.spec
        self.q = to_torch(pw.q, s.dtype, device)
        self.q_start = torch.from_numpy(pw.q_start.astype(np.int64)).to(device)
        self.q_lens = torch.from_numpy(pw.q_lens.astype(np.int32)).to(device)
        self.max_q_len = int(pw.q_lens.max(initial=0))


def run_prefill(dp: DevicePrefill, op, out=None, want_lse=True):
    """One prefill call through the C ABI; returns (out, lse) as numpy float32."""
    import torch

    s = dp.pw.kv.spec
    total = dp.q.shape[0]
    lse = torch.full((total, s.num_q_heads), float("nan"), dtype=torch.float32, device=dp.q.device) \
        if want_lse else None
    kv = dp.kv
    if s.layout == "paged":
        out, lse = op.prefill_paged(dp.q, dp.q_start, dp.q_lens, dp.max_q_len, kv.k, kv.v, kv.block_table,
                                    kv.ctx_lens, s.max_ctx_len, out=out, lse=lse)
    else:
        out, lse = op.prefill(dp.q, dp.q_start, dp.q_lens, dp.max_q_len, kv.k, kv.v, kv.seq_start, kv.ctx_lens,
                              s.max_ctx_len, out=out, lse=lse)
    torch.cuda.synchronize()
    return out.cpu().numpy(), (None if lse is None else lse.cpu().numpy())


def abs_values(pw):
    """The same prefill workload with |V| in place of V (bf16: sign bit cleared), for error bounds."""
    import dataclasses

    kv = pw.kv
    if kv.spec.dtype != "bf16":
        raise ValueError("bf16 only")
    if kv.spec.layout == "paged":
        kv2 = dataclasses.replace(kv, v_pages=kv.v_pages & np.uint16(0x7FFF))
    else:
        kv2 = dataclasses.replace(kv, v=kv.v & np.uint16(0x7FFF))
    return dataclasses.replace(pw, kv=kv2)


def check_prefill(out, lse, ref_out, ref_lse, ref_abs, what=""):
    """The official bf16 gate, plus the bound that the split probabilities imply: every element within
    2 * 2^-15 * sum_t w_t |v_t| (ref_abs, half of it for fp32 accumulation) + 1e-5 |ref| + 1e-6.
    Returns max |err|."""
    out = np.asarray(out, dtype=np.float64)
    ref_out = np.asarray(ref_out, dtype=np.float64)
    assert out.shape == ref_out.shape, what
    assert np.all(np.isfinite(out)), f"{what}: non-finite output"
    err = np.abs(out - ref_out)
    bad = err > TOL_BF16_ABS + TOL_BF16_REL * np.abs(ref_out)
    assert not bad.any(), f"{what}: {bad.sum()} elements outside 2e-3 + 1e-2|ref| (max {err.max():.3e})"
    bound = 2 * PREFILL_P_ROUNDING * np.asarray(ref_abs, dtype=np.float64) + 1e-5 * np.abs(ref_out) + 1e-6
    over = err > bound
    assert not over.any(), (f"{what}: {over.sum()} elements beyond the split-probability bound "
                            f"(worst ratio {(err / bound).max():.3f})")
    if lse is not None:
        lse = np.asarray(lse, dtype=np.float64)
        ref_lse = np.asarray(ref_lse, dtype=np.float64)
        assert np.all(np.isfinite(lse)), f"{what}: non-finite lse"
        lerr = np.abs(lse - ref_lse)
        assert np.all(lerr <= 2e-5 * np.maximum(1.0, np.abs(ref_lse))), f"{what}: lse max err {lerr.max():.3e}"
    return float(err.max(initial=0.0))
