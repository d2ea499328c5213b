"""Pins of the oracle's E4M3 cache codes (oracle/fp8.py): torch's own
float8_e4m3fn conversions (a library routine) for every code and for values in
range, closed forms for the saturating and non-finite cases and the ties."""
import numpy as np
import pytest
import torch

from oracle import fp8 as F


def test_decode_matches_torch_for_every_code():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = F.e4m3_decode(codes)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    fin = ~np.isnan(ref)
    assert np.array_equal(got[fin], ref[fin])
    assert np.isnan(got).sum() == 2 and F.e4m3_decode(0x7E) == 448.0


def test_encode_matches_torch_in_range():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * s for s in (1e-3, 0.05, 1.0, 30.0, 150.0)]).astype(np.float32)
    x = x[np.abs(x) <= 448.0]
    # every code's value and every midpoint between neighbouring values (ties)
    vals = F.e4m3_decode(np.arange(0, 0x7F, dtype=np.uint8))
    mids = (vals[1:] + vals[:-1]) / 2
    x = np.concatenate([x, vals, -vals, mids, -mids]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(F.e4m3_encode(x), ref)


def test_round_trip_and_order():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    assert np.array_equal(F.e4m3_encode(F.e4m3_decode(codes)), codes)
    pos = np.sort(np.abs(np.random.default_rng(1).standard_normal(5000) * 100))
    assert np.all(np.diff(F.e4m3_encode(pos).astype(np.int64)) >= 0)


@pytest.mark.parametrize("x,code", [(1e6, 0x7E), (-1e6, 0xFE), (np.inf, 0x7E), (-np.inf, 0xFE), (449.0, 0x7E),
                                    (2.0 ** -9, 0x01), (2.0 ** -10, 0x00), (3 * 2.0 ** -10, 0x02),
                                    (2.0 ** -6, 0x08), (1.0, 0x38), (1.0625, 0x38), (1.1875, 0x3A), (-0.0, 0x80)])
def test_closed_forms(x, code):
    assert int(F.e4m3_encode(np.array([x]))[0]) == code


def test_nan_keeps_sign():
    assert int(F.e4m3_encode(np.array([np.nan]))[0]) & 0x7F == 0x7F


def test_cache_value_round_trip_error():
    # values already in bf16, scale 1/8: the read-back error is at most half
    # a step of 3 mantissa bits (1/16 relative) in the normal range
    rng = np.random.default_rng(2)
    v = (rng.standard_normal(4096) * 4).astype(np.float32)
    v = np.frombuffer((v.view(np.uint32) & 0xFFFF0000).tobytes(), dtype=np.float32)
    back = F.dequantize(F.quantize_cache_value(v, 0.125), 0.125)
    big = np.abs(v) > 0.125 * 2 ** -6
    assert np.all(np.abs(back[big] - v[big]) <= np.abs(v[big]) / 16 + 1e-12)
