"""Pins of the oracle's number formats against independent implementations:
numpy's float16 cast and torch's bfloat16 cast (both round to nearest even),
over every fp32 bit pattern, and a brute-force nearest-grid-point check of
the single-rounding fp64 -> bf16 conversion."""
import os

import numpy as np
import pytest
import torch

import oracle

CHUNK = 1 << 25


def _patterns(start):
    return np.arange(start, start + CHUNK, dtype=np.uint64).astype(np.uint32)


def _same(a: np.ndarray, b: np.ndarray, nan_a: np.ndarray, nan_b: np.ndarray) -> bool:
    return bool(np.array_equal(nan_a, nan_b) and np.array_equal(a[~nan_a], b[~nan_b]))


FULL = os.environ.get("WUSHKV_EXHAUSTIVE") == "1"


def _check_f16(x):
    ours = oracle.f32_to_f16(x)
    with np.errstate(over="ignore", invalid="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    nan_o = (ours & 0x7C00 == 0x7C00) & (ours & 0x03FF != 0)
    nan_r = (ref & 0x7C00 == 0x7C00) & (ref & 0x03FF != 0)
    return _same(ours, ref, nan_o, nan_r)


def _check_bf16(x):
    ours = oracle.f32_to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan_o = (ours & 0x7F80 == 0x7F80) & (ours & 0x007F != 0)
    nan_r = (ref & 0x7F80 == 0x7F80) & (ref & 0x007F != 0)
    return _same(ours, ref, nan_o, nan_r)


@pytest.mark.skipif(not FULL, reason="full 2^32 sweep (about 12 min): set WUSHKV_EXHAUSTIVE=1")
def test_f32_to_f16_exhaustive():
    for start in range(0, 1 << 32, CHUNK):
        assert _check_f16(_patterns(start).view(np.float32)), "fp16 mismatch at %#x" % start


@pytest.mark.skipif(not FULL, reason="full 2^32 sweep (about 12 min): set WUSHKV_EXHAUSTIVE=1")
def test_f32_to_bf16_exhaustive():
    for start in range(0, 1 << 32, CHUNK):
        assert _check_bf16(_patterns(start).view(np.float32)), "bf16 mismatch at %#x" % start


def test_f32_to_bf16_every_rounding_class():
    # every upper half (sign, exponent, 7 kept bits) with the dropped 16 bits
    # at each decision point (below / at / above the midpoint, extremes)
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF], np.uint32)
    lows = np.concatenate([lows, np.random.default_rng(0).integers(0, 1 << 16, 20).astype(np.uint32)])
    x = (hi[:, None] | lows[None, :]).reshape(-1).view(np.float32)
    assert _check_bf16(x)


def test_f32_to_f16_every_rounding_class():
    # normal fp16 range: every kept pattern (sign, exponent, 10 bits) with the
    # dropped 13 bits at each decision point
    top = np.arange(1 << 19, dtype=np.uint32) << 13
    lows = np.array([0x0000, 0x0001, 0x0FFF, 0x1000, 0x1001, 0x1FFF], np.uint32)
    lows = np.concatenate([lows, np.random.default_rng(1).integers(0, 1 << 13, 6).astype(np.uint32)])
    assert _check_f16((top[:, None] | lows[None, :]).reshape(-1).view(np.float32))
    # subnormal and underflow range (fp32 exponents 100..113): here more bits
    # are dropped, so sweep every mantissa of those binades
    for e in range(100, 114):
        m = np.arange(1 << 23, dtype=np.uint32)
        for sign in (0, 1):
            x = ((np.uint32(sign) << 31) | (np.uint32(e) << 23) | m).view(np.float32)
            assert _check_f16(x), "fp16 mismatch in binade %d" % e


def test_f16_to_f32_all_patterns():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = oracle.f16_to_f32(h)
    ref = h.view(np.float16).astype(np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])


def _bf16_neighbours(v: np.ndarray):
    """Adjacent bf16 values below and above each positive finite bf16 v."""
    bits = (v.astype(np.float32).view(np.uint32) >> 16).astype(np.uint32)
    lo = ((bits - 1) << 16).view(np.float32).astype(np.float64)
    hi = ((bits + 1) << 16).view(np.float32).astype(np.float64)
    return lo, hi


def test_f64_to_bf16_is_nearest_even():
    rng = np.random.default_rng(1)
    # random doubles spanning normal magnitudes, plus exact midpoints (ties)
    x = rng.standard_normal(200000) * np.exp(rng.uniform(-30, 30, 200000))
    mids = []
    for v in rng.standard_normal(2000):
        b = int(oracle.f32_to_bf16(np.float32(v)))
        lo = float(oracle.bf16_to_f32(b))
        hi = float(oracle.bf16_to_f32(b + 1))
        mids.append((lo + hi) / 2.0)
    x = np.concatenate([x, np.array(mids)])
    ours = oracle.bf16_to_f32(oracle.f64_to_bf16(x)).astype(np.float64)
    a = np.abs(x)
    r = np.abs(ours)
    lo, hi = _bf16_neighbours(r)
    # nearest: no neighbour is strictly closer
    assert np.all(np.abs(r - a) <= np.abs(lo - a))
    assert np.all(np.abs(r - a) <= np.abs(hi - a))
    # ties go to the even significand
    tie = (np.abs(r - a) == np.abs(lo - a)) | (np.abs(r - a) == np.abs(hi - a))
    tie &= np.abs(r - a) > 0
    bits = (ours.astype(np.float32).view(np.uint32) >> 16)
    assert np.all((bits[tie] & 1) == 0)
    assert tie.sum() > 1000  # the midpoints were exercised
    assert np.array_equal(np.sign(ours), np.sign(x))


def test_f64_to_bf16_agrees_with_f32_path_when_exact():
    # doubles that are exactly fp32 values round the same way as the fp32 path
    rng = np.random.default_rng(2)
    x = rng.standard_normal(100000).astype(np.float32)
    assert np.array_equal(oracle.f64_to_bf16(x.astype(np.float64)), oracle.f32_to_bf16(x))
