"""Pins for the oracle's fp8 E4M3 codebook snapping."""

import numpy as np
import pytest

from oracle import codec, fp8


def test_hand_checked_codes_and_roundings():
    # (value, nearest E4M3 value, code)
    cases = [
        (1.0, 1.0, 0x38), (-2.0, -2.0, 0xC0), (448.0, 448.0, 0x7E), (-448.0, -448.0, 0xFE),
        (2.0 ** -9, 2.0 ** -9, 0x01), (2.0 ** -6, 2.0 ** -6, 0x08), (7 * 2.0 ** -9, 7 * 2.0 ** -9, 0x07),
        (1.0625, 1.0, 0x38),          # halfway between 1 and 1.125: the even mantissa
        (1.1875, 1.25, 0x3A),         # halfway between 1.125 and 1.25: the even mantissa
        (1.07, 1.125, 0x39),
        (1000.0, 448.0, 0x7E),        # saturation
        (2.0 ** -10, 0.0, 0x00),      # halfway between 0 and the smallest subnormal
        (3 * 2.0 ** -10, 2.0 ** -8, 0x02),
        (15.5, 16.0, 0x58),           # rounds up into the next binade
        (0.3, 0.3125, 0x2A),
    ]
    for x, v, code in cases:
        got = fp8.snap_e4m3(np.array([x]))[0]
        assert got == v, (x, got, v)
        assert int(fp8.e4m3_bits(np.array([v]))[0]) == code, (x, hex(code))


def test_every_finite_code_round_trips():
    codes = np.arange(256, dtype=np.uint8)
    vals = fp8.e4m3_value(codes)
    finite = ~np.isnan(vals)
    assert finite.sum() == 254                        # two NaN codes, no infinities
    assert np.array_equal(fp8.snap_e4m3(vals[finite]), vals[finite])
    nz = finite & (vals != 0)
    assert np.array_equal(fp8.e4m3_bits(vals[nz]), codes[nz])
    pos = np.sort(vals[finite & (vals > 0)])
    assert pos[0] == 2.0 ** -9 and pos[-1] == 448.0 and np.all(np.diff(pos) > 0)


def test_snapping_is_the_nearest_value():
    rng = np.random.default_rng(4)
    x = rng.standard_normal(20000) * np.exp(rng.uniform(-8, 6, 20000))
    y = fp8.snap_e4m3(x)
    grid = fp8.e4m3_value(np.arange(256, dtype=np.uint8))
    grid = np.unique(grid[~np.isnan(grid)])
    inside = np.abs(x) <= 448
    d_best = np.min(np.abs(x[inside, None] - grid[None, :]), axis=1)
    assert np.allclose(np.abs(x[inside] - y[inside]), d_best, rtol=0, atol=0)
    assert np.all(np.abs(y[~inside]) == 448) and np.all(np.signbit(y) == np.signbit(x))


def test_snapped_codebooks_are_exact_in_fp16():
    rng = np.random.default_rng(5)
    cb = (rng.standard_normal((4, 256, 4)) * 3).astype(np.float16)
    s = fp8.snap_codebooks(cb)
    assert s.dtype == np.float16
    assert np.array_equal(s.astype(np.float64), fp8.snap_e4m3(cb.astype(np.float64)))
    # the nearest-codeword search runs unchanged on snapped books
    u = rng.standard_normal((50, 16))
    codes, _ = codec.encode(u, s)
    assert codes.shape == (50, 4)
