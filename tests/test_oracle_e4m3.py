"""Pins for the oracle's E4M3 codec against things other than itself.

* hand-derived code points of the format (tests/golden/, section 2.1.1 + ref. [12]);
* torch's float8_e4m3fn cast (a library routine) on every bf16 value and on
  dense fp32 neighbourhoods of every rounding midpoint;
* a brute-force nearest-value search on random samples.
"""
import os

import numpy as np
import pytest
import torch

from oracle import e4m3

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_points(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                rows.append(line.split())
    return rows


def torch_cast_codes(v: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_matches_golden_points():
    for code_s, val_s in _read_points("e4m3_format_points.txt"):
        code = int(code_s, 16)
        got = e4m3.decode(np.array([code], np.uint8))[0]
        if val_s == "nan":
            assert np.isnan(got), hex(code)
        else:
            want = float(val_s)
            assert got == want and np.signbit(got) == np.signbit(want), (hex(code), got, want)


def test_encode_matches_golden_rounding_points():
    for row in _read_points("e4m3_rounding_points.txt"):
        v, code = float(row[0]), int(row[1], 16)
        got = int(e4m3.encode(np.array([v], np.float32))[0])
        assert got == code, (v, hex(got), hex(code))


def test_decode_table_matches_torch_for_all_256_codes():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = e4m3.decode(codes)
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(got))
    assert np.array_equal(ref[~nan], got[~nan])
    assert np.array_equal(np.signbit(ref[~nan]), np.signbit(got[~nan]))
    assert int(nan.sum()) == 2                      # only 0x7F and 0xFF
    assert np.nanmax(got) == 448.0 and np.nanmin(got) == -448.0


def test_every_finite_code_round_trips():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    vals = e4m3.decode(codes).astype(np.float32)
    assert np.array_equal(e4m3.encode(vals), codes)


def test_encode_matches_torch_on_every_bf16_value_below_464():
    bits = np.arange(65536, dtype=np.uint32) << np.uint32(16)
    v = bits.view(np.float32)
    keep = np.isfinite(v) & (np.abs(v) < 464.0)
    v = v[keep]
    assert np.array_equal(e4m3.encode(v), torch_cast_codes(v))


def _midpoints():
    vals = np.unique(np.abs(e4m3.decode(np.arange(0x7F, dtype=np.uint8))))
    return (vals[:-1] + vals[1:]) / 2.0          # 126 midpoints between finite magnitudes


def test_encode_matches_torch_around_every_midpoint():
    # every fp32 within 4096 ulps of each rounding midpoint, both signs
    mids = _midpoints().astype(np.float32)
    offs = np.arange(-4096, 4097, dtype=np.int64)
    b = (mids.view(np.uint32).astype(np.int64)[:, None] + offs[None, :]).ravel()
    b = b[(b >= 0) & (b < 0x7F800000)].astype(np.uint32)
    v = b.view(np.float32)
    v = np.concatenate([v, -v])
    v = v[np.abs(v) < 464.0]
    assert np.array_equal(e4m3.encode(v), torch_cast_codes(v))


def test_encode_matches_torch_on_random_fp32():
    rng = np.random.default_rng(7)
    b = rng.integers(0, 0x43E80000, size=2_000_000, dtype=np.uint64).astype(np.uint32)  # |v| < 464
    v = b.view(np.float32)
    v = np.where(rng.random(v.shape) < 0.5, -v, v).astype(np.float32)
    assert np.array_equal(e4m3.encode(v), torch_cast_codes(v))


def test_encode_saturates_where_torch_does_not():
    # the satfinite branch: torch returns NaN (0x7F) from 465 up, the reading here is 448
    v = np.array([465.0, 480.0, 1e6, 3.3895e38, np.inf, -465.0, -np.inf], np.float32)
    assert e4m3.encode(v).tolist() == [0x7E] * 5 + [0xFE] * 2


def test_encode_matches_bruteforce_nearest_search():
    rng = np.random.default_rng(11)
    v = np.concatenate([
        rng.standard_normal(300).astype(np.float32) * 50,
        (rng.random(100) * 2.0 ** -6).astype(np.float32),
        _midpoints().astype(np.float32)[::3],
        np.array([0.0, -0.0, 448.0, 447.9, 460.0, 464.0, 500.0], np.float32),
    ])
    got = e4m3.encode(v)
    for x, c in zip(v.tolist(), got.tolist()):
        assert c == e4m3.encode_nearest_bruteforce(x), (x, hex(c))


@pytest.mark.slow
def test_encode_matches_torch_exhaustive_fp32_below_464():
    # all 2^31 magnitudes below 464, both signs, in chunks (minutes)
    step = 1 << 24
    for start in range(0, 0x43E80000, step):
        b = np.arange(start, min(start + step, 0x43E80000), dtype=np.uint32)
        v = b.view(np.float32)
        assert np.array_equal(e4m3.encode(v), torch_cast_codes(v)), hex(start)
        assert np.array_equal(e4m3.encode(-v), torch_cast_codes(-v)), hex(start)
