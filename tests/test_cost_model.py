"""The library's Sec. 3.3 cost model (C, host only) against the paper's case
study, the paper's KV-size example, the oracle's independent Python version,
and the break-even property that defines the bound."""

import ctypes
import json
import math
import os
import re
from fractions import Fraction

import numpy as np
import pytest

import oracle.cost_model as cm
from paper_2605_30842_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")


def _inputs(S, W, P, Y):
    return B.CostInputs(S, W, P, Y)


def test_header_matches_exports():
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "comem_cost_model.h")).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(comem_[a-z_0-9]+)\s*\(", text)))
    assert names == sorted(B.COST_EXPORTED)
    lib = B.load_library()
    for n in names:
        assert hasattr(lib, n)


def test_case_study():
    """Sec. 3.3: W = 2 TB/s, P = 3000 tok/s, S = 2e-4 GB, Y = 1000 -> bound 3/13 (printed 0.23; 7.36K of 32K)."""
    g = json.load(open(os.path.join(GOLDEN, "cost_model_case_study.json")))
    inp = _inputs(float(g["kv_GB_per_token"]) * 1e9, g["bandwidth_GBps"] * 1e9, g["prefill_tokens_per_s"],
                  g["generated_tokens"])
    r = B.comem_cost_max_compression_ratio(inp)
    num, den = g["bound_exact"]
    assert abs(r - num / den) <= 1e-15
    assert round(r, 2) == g["bound_paper_rounded"]
    assert round(g["bound_paper_rounded"] * g["prefix_K_tokens"], 2) == g["summary_bound_K_tokens_paper"]


def test_kv_bytes_per_token_matches_sec_2_2_example():
    """Sec. 2.2: Qwen3-32B (64 layers, 8 KV heads, head size 128) in 16-bit floats holds 64K tokens in 16 GB."""
    S = B.comem_cost_kv_bytes_per_token(64, 8, 128, 2)
    assert S == 262144
    assert S * 65536 == 16 * 2**30
    # the case study's S = 2e-4 GB is this 2.62e-4 GB cut to one significant digit
    assert 2e-4 < S / 1e9 < 3e-4


def test_agrees_with_oracle_on_random_inputs():
    r = np.random.default_rng(7)
    for _ in range(200):
        S, W, P, Y = 10 ** r.uniform(3, 6), 10 ** r.uniform(11, 13), 10 ** r.uniform(2, 5), r.integers(0, 10**4)
        Lf = float(r.integers(1, 10**6))
        Ls = float(r.integers(0, Lf + 1))
        inp = _inputs(S, W, P, float(Y))
        assert B.comem_cost_decode_time(inp, Lf) == pytest.approx(cm.decode_time(Lf, S, W), rel=1e-13)
        assert B.comem_cost_decode_saving(inp, Lf, Ls) == pytest.approx(cm.decode_saving(Lf, Ls, S, W), rel=1e-13,
                                                                         abs=1e-300)
        assert B.comem_cost_prefill_time(inp, Ls) == pytest.approx(cm.prefill_cost(Ls, P), rel=1e-13, abs=1e-300)
        want = cm.net_saving(float(Y), Lf, Ls, S, W, P)
        scale = max(abs(float(Y) * cm.decode_saving(Lf, Ls, S, W)), abs(cm.prefill_cost(Ls, P)), 1e-300)
        assert abs(B.comem_cost_net_saving(inp, Lf, Ls) - want) <= 1e-12 * scale
        assert B.comem_cost_max_compression_ratio(inp) == pytest.approx(cm.max_compression_ratio(W, float(Y), S, P),
                                                                        rel=1e-13, abs=1e-300)


def test_bound_is_the_break_even_point():
    """At L_sum = r * L_full the net saving is zero; below it positive, above it negative (exact rationals)."""
    S, W, P, Y = Fraction(262144), Fraction(6 * 10**12), Fraction(5000), Fraction(1000)
    r = Y * S * P / (Y * S * P + W)
    inp = _inputs(float(S), float(W), float(P), float(Y))
    assert B.comem_cost_max_compression_ratio(inp) == pytest.approx(float(r), rel=1e-15)
    Lf = 32768.0
    for frac, sign in ((0.9, 1), (1.1, -1)):
        assert math.copysign(1, B.comem_cost_net_saving(inp, Lf, frac * float(r) * Lf)) == sign


@pytest.mark.parametrize("fn,args", [
    ("comem_cost_decode_time", (-1.0,)),
    ("comem_cost_decode_time", (float("nan"),)),
    ("comem_cost_decode_saving", (10.0, 11.0)),
    ("comem_cost_prefill_time", (float("inf"),)),
    ("comem_cost_net_saving", (1.0, -1.0)),
])
def test_invalid_lengths(fn, args):
    inp = _inputs(1.0, 1.0, 1.0, 1.0)
    out = ctypes.c_double(123.0)
    lib = B.load_library()
    assert getattr(lib, fn)(ctypes.byref(inp), *args, ctypes.byref(out)) == B.ERR_INVALID_SHAPE
    assert out.value == 123.0  # untouched on error


@pytest.mark.parametrize("bad", [dict(kv_bytes_per_token=0.0), dict(hbm_bytes_per_s=-1.0),
                                 dict(prefill_tokens_per_s=float("nan")), dict(generated_tokens=-1.0)])
def test_invalid_inputs(bad):
    vals = dict(kv_bytes_per_token=1.0, hbm_bytes_per_s=1.0, prefill_tokens_per_s=1.0, generated_tokens=1.0)
    vals.update(bad)
    inp = B.CostInputs(**vals)
    out = ctypes.c_double()
    assert B.load_library().comem_cost_max_compression_ratio(ctypes.byref(inp), ctypes.byref(out)) == \
        B.ERR_INVALID_SHAPE
    assert B.load_library().comem_cost_max_compression_ratio(None, ctypes.byref(out)) == B.ERR_NULL_POINTER
    assert B.load_library().comem_cost_kv_bytes_per_token(0, 8, 128, 2, ctypes.byref(out)) == B.ERR_INVALID_SHAPE
    assert B.load_library().comem_cost_kv_bytes_per_token(1, 8, 128, 2, None) == B.ERR_NULL_POINTER
