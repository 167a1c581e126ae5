"""Pins for the oracle's scalar formats: OCP E4M3FN and binary16.

E4M3 is checked against torch's independent float8_e4m3fn conversion over
every fp32 bit pattern whose magnitude lies in the representable range, and
against spot values of the format's definition.  binary16 is checked against
numpy's fp64 -> fp16 conversion (one correct rounding) and constructed ties.
"""
import numpy as np
import pytest
import torch


def test_e4m3_spot_values(orc):
    v = orc.e4m3_to_f64
    assert v(0x7E) == 448.0 and v(0xFE) == -448.0
    assert v(0x01) == 2.0 ** -9 and v(0x08) == 2.0 ** -6 and v(0x07) == 7 * 2.0 ** -9
    assert v(0x38) == 1.0 and v(0x39) == 1.125 and v(0x00) == 0.0
    assert np.isnan(v(0x7F)) and np.isnan(v(0xFF))


def test_e4m3_roundtrip_all_finite_codes(orc):
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    vals = orc.e4m3_to_f64(codes).astype(np.float32)
    back = orc.e4m3_from_f32(vals)
    # -0.0 keeps its sign bit; every other code round-trips exactly
    assert np.array_equal(back, codes)


def test_e4m3_ties_and_saturation(orc):
    x = np.array([1.0625, 1.1875, 448.0, 449.0, 463.99, 1e30, -1e30, 2.0 ** -10, 3 * 2.0 ** -10,
                  np.inf, -np.inf], np.float32)
    want = np.array([0x38, 0x3A, 0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0x00, 0x02, 0x7E, 0xFE], np.uint8)
    assert np.array_equal(orc.e4m3_from_f32(x), want)
    assert orc.e4m3_from_f32(np.array([np.nan], np.float32))[0] & 0x7F == 0x7F


def test_e4m3_matches_torch_over_range(orc):
    # every fp32 pattern with biased exponent 100..135 (2^-27 .. <2^9), both
    # signs, restricted to |x| < 464 where torch and the saturating definition agree
    chunk = 1 << 23
    for e in range(100, 136):
        for sign in (0, 1):
            bits = (np.uint32(sign << 31) | np.uint32(e << 23)) + np.arange(chunk, dtype=np.uint32)
            x = bits.view(np.float32)
            x = x[np.abs(x) < 464.0]
            if x.size == 0:
                continue
            ours = orc.e4m3_from_f32(x)
            ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
            bad = np.nonzero(ours != ref)[0]
            assert bad.size == 0, (e, sign, x[bad[:5]], ours[bad[:5]], ref[bad[:5]])


def test_f16_matches_numpy(orc):
    rng = np.random.default_rng(7)
    x = np.concatenate([
        rng.standard_normal(200000) * np.exp2(rng.integers(-30, 16, 200000)),
        rng.uniform(-65504, 65504, 10000),
        rng.uniform(-2.0 ** -14, 2.0 ** -14, 10000),  # subnormal range
    ])
    x = x[np.abs(x) < 65504.0]  # beyond the largest half numpy gives inf, we saturate
    ours = orc.f16_from_f64(x)
    ref = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(ours, ref)


def test_f16_ties_to_even_single_rounding(orc):
    # exact midpoints between neighbouring halves round to the even one
    h = np.arange(0x0001, 0x7BFF, 37, dtype=np.uint16)
    lo = orc.f16_to_f64(h)
    hi = orc.f16_to_f64(h + 1)
    mid = (lo + hi) / 2  # exact in fp64
    got = orc.f16_from_f64(mid)
    want = np.where(h % 2 == 0, h, h + 1).astype(np.uint16)
    assert np.array_equal(got, want)
    # a value just above a midpoint (in fp64 but below fp32 resolution) rounds up:
    # a double rounding through fp32 would land on the midpoint and go to even
    above = mid + mid * 2.0 ** -40
    assert np.array_equal(orc.f16_from_f64(above), (h + 1).astype(np.uint16))


def test_f16_saturates(orc):
    got = orc.f16_from_f64(np.array([65504.0, 65519.0, 1e9, -1e9]))
    assert list(got) == [0x7BFF, 0x7BFF, 0x7BFF, 0xFBFF]
