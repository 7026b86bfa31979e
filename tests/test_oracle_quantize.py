"""Pins of the oracle quantizer (Eq. (2), shared train-query scale) against
the absmax rule, power-of-two equivariance, IEEE division and the paper's
printed quantization error."""
import os

import numpy as np

from oracle import quantize as Q
from oracle.e4m3 import decode, encode_rne

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


def test_quantizer_divides_where_the_reciprocal_would_move_a_tie():
    # Eq. (2) divides by s.  Inputs x = fl32(t s) for which the IEEE quotient x / s is
    # exactly an e4m3 rounding midpoint t, but x * fl32(1/s) is one fp32 ulp off it, so
    # a reciprocal multiply would round to the other neighbour where the tie goes down.
    rng = np.random.default_rng(31)
    mids = np.array([(1 + (2 * m + 1) / 16) * 2.0 ** e for e in range(-3, 8) for m in range(8)
                     if (1 + (2 * m + 1) / 16) * 2.0 ** e < 448])
    found = []
    for s in rng.uniform(1e-3, 10.0, 3000).astype(np.float32):
        x = (mids * np.float64(s)).astype(np.float32)
        exact = (x.astype(np.float64) / np.float64(s)).astype(np.float32)
        recip = x * (np.float32(1.0) / s)
        for i in np.nonzero((exact == mids) & (recip != exact))[0]:
            found.append((x[i], s))
    assert len(found) > 50
    for x, s in found:
        code = Q.quantize_with_scale(np.full((1, 1, 1, 1), x, np.float32), np.full((1, 1), s, np.float32))
        want = encode_rne(np.float32(np.float64(x) / np.float64(s)))
        assert code[0, 0, 0, 0] == want, (x, s)


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


def test_per_call_test_scale_is_the_test_batch_absmax_and_couples_test_rows():
    # Table 1, "per-call query scale": the test queries get a scale of their own.
    x = _x((1, 300, 2, 64), 11)
    q_test = _x((1, 50, 2, 64), 12) * np.float32(0.0625)           # far below the train amax
    q_test[0, 9, 0, 7] = np.float32(3.0) * np.abs(q_test[0, :, 0, :]).max()
    shared = Q.quantize_qkv_per_head(x, x, x, q_test)
    per = Q.quantize_qkv_per_head(x, x, x, q_test, q_scale_mode="per_call")
    for key in ("q8_train", "k8", "v8", "s_q", "s_k", "s_v"):
        assert np.array_equal(per[key], shared[key])
    assert np.array_equal(shared["s_q_test"], shared["s_q"])
    # the test absmax element maps to 448 under its own scale, and no code saturates beyond it
    dec = np.abs(decode(per["q8_test"]))
    assert np.array_equal(dec.max(axis=(2, 3)), np.full((1, 2), 448.0))
    assert per["q8_test"][0, 0, 9, 7] == 0x7E
    assert not np.array_equal(per["s_q_test"], per["s_q"])
    # scaling the test batch by a power of two leaves its codes unchanged
    per4 = Q.quantize_qkv_per_head(x, x, x, q_test * np.float32(4.0), q_scale_mode="per_call")
    assert np.array_equal(per4["q8_test"], per["q8_test"])
    assert np.array_equal(per4["s_q_test"], per["s_q_test"] * np.float32(4.0))
    # dropping the row that holds head 0's absmax changes the other rows' codes (Sec. 3: the
    # per-call scale couples the test rows); the shared scale does not
    keep = [r for r in range(50) if r != 9]
    sub_per = Q.quantize_qkv_per_head(x, x, x, q_test[:, keep], q_scale_mode="per_call")
    sub_sh = Q.quantize_qkv_per_head(x, x, x, q_test[:, keep])
    assert not np.array_equal(sub_per["q8_test"][:, 0], per["q8_test"][:, 0][:, keep])
    assert np.array_equal(sub_sh["q8_test"], shared["q8_test"][:, :, keep])


def test_joint_scale_is_one_scale_over_train_and_test_queries():
    # The single ICL call over all rows of the TabICLv2 experiments: one per-head scale over
    # the union of the train and test query rows.
    x = _x((2, 200, 3, 64), 13)
    q_test = _x((2, 40, 3, 64), 14)
    q_test[1, 3, 2, 5] = np.float32(6.0) * np.abs(x[1, :, 2, :]).max()   # head (1,2): test amax wins
    joint = Q.quantize_qkv_per_head(x, x, x, q_test, q_scale_mode="joint")
    assert np.array_equal(joint["s_q_test"], joint["s_q"])
    both = np.concatenate([x, q_test], axis=1)
    s = Q.scale_from_amax(Q.absmax_per_head(both))
    codes = Q.quantize_with_scale(both, s)
    assert np.array_equal(joint["s_q"], s)
    assert np.array_equal(joint["q8_train"], codes[:, :, :200])
    assert np.array_equal(joint["q8_test"], codes[:, :, 200:])
    # where the train amax is the larger, joint and shared agree bit for bit
    shared = Q.quantize_qkv_per_head(x, x, x, q_test)
    at_train = np.abs(x).max(axis=(1, 3)) >= np.abs(q_test).max(axis=(1, 3))
    assert at_train.sum() >= 3 and not at_train[1, 2]
    for b, h in zip(*np.nonzero(at_train)):
        assert np.array_equal(joint["q8_test"][b, h], shared["q8_test"][b, h])
        assert joint["s_q"][b, h] == shared["s_q"][b, h]
    # head (1,2): the shared scale saturates the large test value, the joint one does not clip it
    assert shared["q8_test"][1, 2, 3, 5] == 0x7E and joint["q8_test"][1, 2, 3, 5] == 0x7E
    assert (np.abs(decode(joint["q8_train"][1, 2])).max() < 448.0 / 4)
    assert (np.abs(decode(shared["q8_train"][1, 2])).max() == 448.0)


def test_unknown_query_scale_mode_is_rejected():
    x = _x((1, 8, 1, 64), 15)
    try:
        Q.quantize_qkv_per_head(x, x, x, x, q_scale_mode="per_head")
    except ValueError:
        return
    raise AssertionError("expected ValueError")
