"""Pins of the oracle's E4M3 codec against the format definition and torch."""

import os

import numpy as np
import pytest
import torch

from oracle import e4m3

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e4m3_ocp_values.txt")
ALL = np.arange(256, dtype=np.uint8)
FINITE = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)


def _golden():
    rows = []
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if line:
            code, val = line.split()[:2]
            rows.append((int(code, 16), float(val)))
    return rows


def test_golden_ocp_values():
    for code, val in _golden():
        got = e4m3.decode(np.array([code], np.uint8))[0]
        if np.isnan(val):
            assert np.isnan(got)
        else:
            assert got == val and np.signbit(got) == np.signbit(val), hex(code)
            assert e4m3.encode(np.array([val], np.float32))[0] == code


def test_decode_matches_torch_for_all_codes():
    ref = torch.from_numpy(ALL.copy()).view(torch.float8_e4m3fn).to(torch.float32).numpy()
    got = e4m3.decode(ALL)
    np.testing.assert_array_equal(np.isnan(got), np.isnan(ref))
    fin = ~np.isnan(ref)
    np.testing.assert_array_equal(got[fin], ref[fin].astype(np.float64))
    np.testing.assert_array_equal(np.signbit(got[fin]), np.signbit(ref[fin]))


def test_round_trip_all_finite_codes():
    v = e4m3.decode(FINITE).astype(np.float32)
    np.testing.assert_array_equal(e4m3.encode(v), FINITE)


def test_nan_codes():
    assert np.isnan(e4m3.decode(np.array([0x7F, 0xFF], np.uint8))).all()
    assert e4m3.encode(np.array([np.nan], np.float32))[0] == 0x7F


def test_codes_are_monotone():
    pos = e4m3.decode(np.arange(0x00, 0x7F, dtype=np.uint8))
    assert np.all(np.diff(pos) > 0)
    neg = e4m3.decode(np.arange(0x80, 0xFF, dtype=np.uint8))
    assert np.all(np.diff(neg) < 0)


@pytest.mark.parametrize("sign", [1.0, -1.0])
def test_midpoints_round_to_even_and_neighbours_to_nearest(sign):
    for c in range(0x00, 0x7E):                    # adjacent finite pairs c, c+1
        lo = e4m3.decode(np.array([c], np.uint8))[0]
        hi = e4m3.decode(np.array([c + 1], np.uint8))[0]
        mid = np.float32((lo + hi) / 2)             # exact in fp32
        assert float(mid) == (lo + hi) / 2
        even = c if c % 2 == 0 else c + 1
        sbit = 0x80 if sign < 0 else 0
        got = e4m3.encode(np.array([sign * mid], np.float32))[0]
        assert got == (even | sbit), (hex(c), mid)
        above = np.nextafter(mid, np.float32(np.inf))
        below = np.nextafter(mid, np.float32(0))
        assert e4m3.encode(np.array([sign * above], np.float32))[0] == ((c + 1) | sbit)
        assert e4m3.encode(np.array([sign * below], np.float32))[0] == (c | sbit)


def test_saturation():
    big = np.array([448.0, np.nextafter(np.float32(448), np.float32(1e9)), 464.0, 480.0,
                    1e30, np.inf], np.float32)
    assert (e4m3.encode(big) == 0x7E).all()
    assert (e4m3.encode(-big) == 0xFE).all()


def test_underflow_and_signed_zero():
    tiny = np.float32(2.0 ** -10)                   # half the smallest subnormal: tie -> 0
    assert e4m3.encode(np.array([tiny], np.float32))[0] == 0x00
    assert e4m3.encode(np.array([np.nextafter(tiny, np.float32(1))], np.float32))[0] == 0x01
    assert e4m3.encode(np.array([-2.0 ** -11], np.float32))[0] == 0x80
    assert e4m3.encode(np.array([-0.0], np.float32))[0] == 0x80
    assert e4m3.encode(np.array([1e-45], np.float32))[0] == 0x00   # fp32 subnormal input


def test_encode_matches_torch_cast_inside_range():
    rng = np.random.default_rng(123)
    n = 1 << 20
    mag = np.exp2(rng.uniform(-14, np.log2(448.0), n)).astype(np.float32)
    mag = np.minimum(mag, np.float32(448.0))
    y = np.where(rng.random(n) < 0.5, -mag, mag).astype(np.float32)
    ref = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(e4m3.encode(y), ref)


def test_encode_is_nearest():
    """Brute force: the chosen code minimises |dec(code) - y| over all codes."""
    rng = np.random.default_rng(5)
    y = (rng.standard_normal(4096) * rng.choice([1e-3, 0.05, 1.0, 30.0, 300.0], 4096)).astype(np.float32)
    y = np.clip(y, -448, 448)
    tab = e4m3.decode(FINITE)
    codes = e4m3.encode(y)
    err = np.abs(e4m3.decode(codes) - y.astype(np.float64))
    best = np.min(np.abs(tab[None, :] - y.astype(np.float64)[:, None]), axis=1)
    np.testing.assert_array_equal(err, best)
