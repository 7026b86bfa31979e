"""Pins of the oracle quantizer (Eq. (2), shared train-query scale) against
the absmax rule, power-of-two equivariance, IEEE division and the paper's
printed quantization error."""
import os

import numpy as np

from oracle import quantize as Q
from oracle.e4m3 import decode

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "quantization_error.txt")


def _x(shape, seed, mult=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(shape).astype(np.float32)
    if mult:
        x *= rng.uniform(0.25, 8.0, size=(1, 1, shape[2], 1)).astype(np.float32)
    return x


def test_absmax_element_maps_to_448_and_codes_stay_finite():
    x = _x((3, 257, 4, 64), 1)
    s = Q.scale_from_amax(Q.absmax_per_head(x))
    c = Q.quantize_with_scale(x, s)                       # (B,H,S,D)
    xt = x.transpose(0, 2, 1, 3)
    for b in range(3):
        for h in range(4):
            i = np.unravel_index(np.argmax(np.abs(xt[b, h])), xt[b, h].shape)
            assert c[b, h][i] == (0xFE if xt[b, h][i] < 0 else 0x7E)
    assert np.all((c & 0x7F) <= 0x7E)


def test_scale_is_amax_over_448_in_fp32_and_zero_head_uses_one():
    x = _x((2, 100, 3, 64), 2)
    x[1, :, 2, :] = 0.0
    amax = Q.absmax_per_head(x)
    assert np.array_equal(amax[0], np.abs(x[0]).max(axis=(0, 2)))
    s = Q.scale_from_amax(amax)
    assert s.dtype == np.float32
    assert s[1, 2] == 1.0
    assert s[0, 0] == np.float32(np.float64(amax[0, 0]) / 448.0)   # fl32(a/448) = fl32(fl64(a/448))
    c = Q.quantize_with_scale(x, s)
    assert np.all(c[1, 2] == 0)


def test_fp32_division_is_correctly_rounded():
    # fl32(x/s) equals the fp32 rounding of the fp64 quotient (double rounding is
    # harmless for division when 53 >= 2*24 + 2), so numpy's fp32 divide is IEEE.
    rng = np.random.default_rng(3)
    x = rng.standard_normal(1_000_000).astype(np.float32) * np.float32(50)
    s = np.float32(0.0123456)
    assert np.array_equal(np.divide(x, s, dtype=np.float32), (x.astype(np.float64) / np.float64(s)).astype(np.float32))


def test_power_of_two_equivariance():
    x = _x((1, 300, 2, 64), 4)
    a = Q.quantize_qkv_per_head(x, x, x, x[:, :50])
    for k in (-7, 3, 11):
        y = (x * np.float32(2.0 ** k)).astype(np.float32)
        b = Q.quantize_qkv_per_head(y, y, y, y[:, :50])
        for key in ("q8_train", "k8", "v8", "q8_test"):
            assert np.array_equal(a[key], b[key])
        assert np.array_equal(b["s_q"], a["s_q"] * np.float32(2.0 ** k))


def test_paper_quantization_error_on_gaussian_heads():
    with open(GOLDEN) as f:
        val, tol = [float(t) for t in next(l for l in f if not l.startswith("#")).split()]
    rng = np.random.default_rng(5)
    x = rng.standard_normal((1, 1 << 15, 2, 64)).astype(np.float32)   # 2M elements per head
    s = Q.scale_from_amax(Q.absmax_per_head(x))
    c = Q.quantize_with_scale(x, s)
    for h in range(2):
        xh = x[0, :, h, :].astype(np.float64)
        xhat = decode(c[0, h]) * float(s[0, h])
        rel = np.sqrt(np.mean((xhat - xh) ** 2)) / np.sqrt(np.mean(xh ** 2))
        assert abs(rel - val) <= tol, rel


def test_test_queries_use_train_scale_saturate_and_are_batch_invariant():
    x = _x((1, 400, 2, 64), 6)
    q_test = _x((1, 64, 2, 64), 7)
    q_test[0, 5, 1, 3] = 10.0 * np.abs(x[0, :, 1, :]).max()      # beyond the train amax
    full = Q.quantize_qkv_per_head(x, x, x, q_test)
    assert np.array_equal(full["s_q"], Q.scale_from_amax(Q.absmax_per_head(x)))
    assert full["q8_test"][0, 1, 5, 3] == 0x7E                    # clamped to +448
    sub = Q.quantize_qkv_per_head(x, x, x, q_test[:, [40, 5, 17]])
    assert np.array_equal(sub["q8_test"], full["q8_test"][:, :, [40, 5, 17]])


def test_layout_and_dequantization_error_bound():
    x = _x((2, 33, 3, 64), 8)
    s = Q.scale_from_amax(Q.absmax_per_head(x))
    c = Q.quantize_with_scale(x, s)
    assert c.shape == (2, 3, 33, 64) and c.dtype == np.uint8
    xhat = decode(c) * s[:, :, None, None]
    xt = x.transpose(0, 2, 1, 3).astype(np.float64)
    y = np.abs(xt) / s[:, :, None, None]
    # half an e4m3 ulp: 2^-4 relative in the normal range, 2^-10 absolute below 2^-6 (+ fp32 division)
    bound = s[:, :, None, None] * (np.maximum(y * 2.0 ** -4, 2.0 ** -10) * (1 + 1e-6) + 1e-6 * y)
    assert np.all(np.abs(xhat - xt) <= bound)
