"""Pins of the FP8 KV part of the oracle: the E4M3 decoder and attention over dequantized caches.

The decoder is checked against torch's float8_e4m3fn (a library routine)
on every code and against values worked out by hand from the OCP format
definition; attention over an FP8 cache is checked against torch SDPA on
the dequantized tensors and against closed forms. Planted mistakes in the
decoder are each caught by a pin.
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle.decode_attention as da
from workloads.synth import WORKLOADS, f32_to_fp8_e4m3_codes, generate, small_spec

ALL = np.arange(256, dtype=np.uint8)


def pin_matches_torch_on_every_code():
    mine = da.fp8_e4m3_value(ALL)
    ref = torch.from_numpy(ALL.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(mine), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(mine[ok], ref[ok])
    assert np.array_equal(np.signbit(mine[ok]), np.signbit(ref[ok]))


def pin_hand_values():
    """Worked from the definition: sign | 4-bit exponent (bias 7) | 3-bit mantissa."""
    cases = {0x00: 0.0, 0x38: 1.0, 0x39: 1.125, 0x3F: 1.875, 0x40: 2.0, 0x30: 0.5, 0x7E: 448.0,
             0xFE: -448.0, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x08: 2.0 ** -6, 0xB8: -1.0}
    got = da.fp8_e4m3_value(np.array(list(cases), dtype=np.uint8))
    assert np.array_equal(got, np.array(list(cases.values())))
    assert math.copysign(1.0, float(da.fp8_e4m3_value(np.array([0x80], np.uint8))[0])) == -1.0
    assert np.isnan(da.fp8_e4m3_value(np.array([0x7F, 0xFF], np.uint8))).all()


def pin_order_and_symmetry():
    """Codes 0..126 increase strictly (subnormals join normals without a gap); the sign bit negates."""
    pos = da.fp8_e4m3_value(ALL[:127])
    assert np.all(np.diff(pos) > 0)
    assert pos[8] - pos[7] == pos[1] - pos[0] == 2.0 ** -9  # subnormal spacing continues into the first binade
    assert np.array_equal(da.fp8_e4m3_value(ALL[128:255]), -pos)


def pin_generator_rounds_to_nearest():
    """Codes drawn for x are the E4M3 value nearest to x (ties to the even code)."""
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(4000).astype(np.float32) * 64,
                        np.float32([0.0, 448.0, -448.0, 1.0625, 1.1875, 2.0 ** -10])])
    codes = f32_to_fp8_e4m3_codes(x)
    table = da.fp8_e4m3_value(ALL[:127])
    got = da.fp8_e4m3_value(codes)
    dist = np.abs(np.abs(x.astype(np.float64))[:, None] - table[None, :])
    best = dist.min(axis=1)
    assert np.all(np.abs(np.abs(got) - np.abs(x)) == best)
    nz = got != 0
    assert np.array_equal(np.sign(got[nz]), np.sign(x[nz]))
    # ties go to the even mantissa: 1.0625 is halfway between 1.0 (m=0) and 1.125 (m=1)
    assert got[-3] == 1.0 and got[-2] == 1.25 and got[-1] == 0.0  # 1.1875: between 1.125 (m=1) and 1.25 (m=2)


def pin_attention_over_dequantized_cache():
    """An FP8 workload's reference equals torch SDPA (fp64) on the dequantized K/V, GQA by repeat."""
    spec = small_spec(WORKLOADS[6], [40, 1, 300], seed=11).replace(k_scale=0.013, v_scale=0.021)
    w = generate(spec)
    out, lse = da.reference(w)
    for b in range(spec.batch):
        a, L = int(w.seq_start[b]), int(w.ctx_lens[b])
        q = torch.from_numpy(da.widen(w.q[b], "bf16"))[None, :, None, :]  # [1, Hq, 1, D]
        k = torch.from_numpy(da.fp8_e4m3_value(w.k[a:a + L]) * spec.k_scale).permute(1, 0, 2)[None]
        v = torch.from_numpy(da.fp8_e4m3_value(w.v[a:a + L]) * spec.v_scale).permute(1, 0, 2)[None]
        k = k.repeat_interleave(spec.group, dim=1)
        v = v.repeat_interleave(spec.group, dim=1)
        ref = F.scaled_dot_product_attention(q, k, v, scale=float(spec.scale))[0, :, 0].numpy()
        assert np.abs(out[b] - ref).max() <= 1e-12


def pin_one_key_gives_scaled_value():
    """L = 1: out = decoded V row times v_scale exactly; lse = the one score (with k_scale)."""
    spec = small_spec(WORKLOADS[6], [1], seed=12).replace(k_scale=0.5, v_scale=0.25)
    w = generate(spec)
    out, lse = da.reference(w)
    v0 = da.fp8_e4m3_value(w.v[0]) * 0.25  # [Hkv, D]
    assert np.array_equal(out[0], np.repeat(v0, spec.group, axis=0))
    k0 = da.fp8_e4m3_value(w.k[0]) * 0.5
    q = da.widen(w.q[0], "bf16")
    s = np.einsum("hd,hd->h", q, np.repeat(k0, spec.group, axis=0)) * float(spec.scale)
    assert np.abs(lse[0] - s).max() <= 1e-12


PINS = [pin_matches_torch_on_every_code, pin_hand_values, pin_order_and_symmetry, pin_generator_rounds_to_nearest,
        pin_attention_over_dequantized_cache, pin_one_key_gives_scaled_value]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()


def _failing_pins():
    failed = []
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failed.append(pin.__name__)
    return failed


def _bias8(codes):
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    e, m = (c >> 3) & 15, (c & 7).astype(np.float64)
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -7, (1.0 + m / 8.0) * np.exp2(e - 8.0))
    return np.where((e == 15) & (m == 7), np.nan, np.where(c >> 7, -1.0, 1.0) * mag)


def _subnormal_as_normal(codes):
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    e, m = (c >> 3) & 15, (c & 7).astype(np.float64)
    mag = np.where((e == 0) & (m == 0), 0.0, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    return np.where((e == 15) & (m == 7), np.nan, np.where(c >> 7, -1.0, 1.0) * mag)


def _no_sign(codes):
    return np.abs(_ORIG(codes))


def _mantissa_sixteenths(codes):
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    e, m = (c >> 3) & 15, (c & 7).astype(np.float64)
    mag = np.where(e == 0, m / 16.0 * 2.0 ** -6, (1.0 + m / 16.0) * np.exp2(e - 7.0))
    return np.where((e == 15) & (m == 7), np.nan, np.where(c >> 7, -1.0, 1.0) * mag)


def _no_nan(codes):
    v = _ORIG(codes)
    return np.where(np.isnan(v), 480.0, v)


_ORIG = da.fp8_e4m3_value
MUTANTS = {"bias8": _bias8, "subnormal_as_normal": _subnormal_as_normal, "no_sign": _no_sign,
           "mantissa_sixteenths": _mantissa_sixteenths, "no_nan": _no_nan}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_decoder_is_caught(name, monkeypatch):
    monkeypatch.setattr(da, "fp8_e4m3_value", MUTANTS[name])
    assert _failing_pins(), f"no pin catches mutant {name}"


def test_mutant_scale_dropped_is_caught(monkeypatch):
    monkeypatch.setattr(da, "dequantize", lambda x, dtype, scale=1.0: da.widen(x, dtype))
    assert _failing_pins()
