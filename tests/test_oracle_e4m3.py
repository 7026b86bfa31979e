"""Pins of the oracle's e4m3fn codec against torch's float8_e4m3fn cast and hand-checked values."""
import os

import numpy as np
import pytest
import torch

from oracle import e4m3

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e4m3_worked_values.txt")


def torch_encode(x32):
    return torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_all_codes_matches_torch():
    codes = np.arange(256, dtype=np.uint8)
    ours = e4m3.decode(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    fin = ~np.isnan(ref)
    assert np.array_equal(ours[fin], ref[fin])
    assert np.array_equal(np.signbit(ours[fin]), np.signbit(ref[fin]))
    assert set(np.nonzero(np.isnan(ours))[0]) == {0x7F, 0xFF}
    assert np.nanmax(ours) == 448.0


def test_worked_values():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            expr, code = line.split()[:2]
            rows.append((eval(expr, {"__builtins__": {}}), int(code, 16)))
    vals = np.array([r[0] for r in rows])
    got = e4m3.encode_rne(vals)
    assert [hex(c) for c in got] == [hex(r[1]) for r in rows]


def _tie_sensitive_patterns():
    # every fp32 bit pattern's upper 16 bits with lower halves that put the
    # discarded bits at 0, 1 ulp, just below / at / above half, and all ones.
    # This is as strong as trying all 2^32 patterns: an e4m3 result keeps at
    # most 3 mantissa bits, so the rounding bit of a fp32 input is mantissa bit
    # 19 or higher (higher still for subnormal results), inside the upper 16
    # bits; the lower 16 bits can only act as sticky bits, where all that counts
    # is whether they are zero, and every upper half is tried with both.
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    u = (hi[:, None] | lows[None, :]).ravel()
    x = u.view(np.float32)
    return x[np.isfinite(x) & (np.abs(x) <= 448.0)]


def test_encode_matches_torch_on_all_tie_sensitive_fp32_patterns():
    x = _tie_sensitive_patterns()
    assert x.size > 200_000
    assert np.array_equal(e4m3.encode_rne(x), torch_encode(x))


def test_encode_matches_torch_on_random_fp32():
    rng = np.random.default_rng(123)
    u = rng.integers(0, 1 << 32, size=2_000_000, dtype=np.uint64).astype(np.uint32)
    x = u.view(np.float32)
    x = x[np.isfinite(x) & (np.abs(x) <= 448.0)]
    y = rng.uniform(-448.0, 448.0, size=1_000_000).astype(np.float32)
    for arr in (x, y):
        assert np.array_equal(e4m3.encode_rne(arr), torch_encode(arr))


def test_round_trip_of_every_finite_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    assert np.array_equal(e4m3.encode_rne(e4m3.decode(codes)), codes)


def test_rejects_out_of_range():
    with pytest.raises(ValueError):
        e4m3.encode_rne(np.array([449.0]))
    with pytest.raises(ValueError):
        e4m3.encode_rne(np.array([np.nan]))
