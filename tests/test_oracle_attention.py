"""Pins of the oracle's attention references: brute force, a library SDPA,
closed forms, and the exact-arithmetic limit of the one-pass kernel model."""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import quantize as Q
from oracle.e4m3 import decode, encode_rne


def brute_force_attention(q, k, v, alpha):
    out = []
    for qi in q:
        logits = [alpha * sum(a * b for a, b in zip(qi, kj)) for kj in k]
        mx = max(logits)
        w = [math.exp(t - mx) for t in logits]
        z = sum(w)
        out.append([sum(wj * vj[c] for wj, vj in zip(w, v)) / z for c in range(len(v[0]))])
    return np.array(out)


@pytest.mark.parametrize("R,N,D", [(1, 1, 1), (3, 5, 2), (8, 8, 4), (2, 7, 3)])
def test_softmax_attention_matches_brute_force(R, N, D):
    rng = np.random.default_rng(R * 100 + N * 10 + D)
    q, k, v = rng.standard_normal((R, D)), rng.standard_normal((N, D)), rng.standard_normal((N, D))
    ours = A.softmax_attention(q, k, v, 0.7)
    ref = brute_force_attention(q.tolist(), k.tolist(), v.tolist(), 0.7)
    assert np.allclose(ours, ref, rtol=1e-12, atol=1e-12)


def test_softmax_attention_matches_torch_sdpa_fp64():
    rng = np.random.default_rng(11)
    q, k, v = rng.standard_normal((70, 64)) * 3, rng.standard_normal((300, 64)) * 3, rng.standard_normal((300, 64))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None], scale=0.125)[0].numpy()
    ours = A.softmax_attention(q, k, v, 0.125, chunk_rows=16)
    assert np.allclose(ours, ref, rtol=1e-11, atol=1e-12)


def test_rows_sum_to_one_constant_v_and_identical_keys():
    rng = np.random.default_rng(12)
    q, k = rng.standard_normal((20, 16)) * 5, rng.standard_normal((40, 16)) * 5
    ones = np.ones((40, 3))
    assert np.allclose(A.softmax_attention(q, k, ones, 1.0), 1.0, atol=1e-12)
    v = rng.standard_normal((40, 5))
    same_k = np.tile(k[:1], (40, 1))
    assert np.allclose(A.softmax_attention(q, same_k, v, 1.0), v.mean(axis=0), atol=1e-12)


def test_one_hot_row_returns_that_value_row():
    k = np.eye(8)[:5] * 40.0
    q = np.eye(8)[[2]]
    v = np.arange(15.0).reshape(5, 3)
    assert np.allclose(A.softmax_attention(q, k, v, 1.0), v[2], atol=1e-12)


def _small_qkv(seed, B=1, N=200, M=30, H=2, D=64, spread=3.0):
    rng = np.random.default_rng(seed)
    mk = lambda n: (rng.standard_normal((B, n, H, D)) * rng.uniform(0.5, spread, (1, 1, H, 1))).astype(np.float32)
    return mk(N), mk(N), mk(N), mk(M)


def test_icl_attention_two_calls_share_keys_and_values():
    qt, k, v, qe = _small_qkv(13)
    o_tr, o_te = A.icl_attention(qt, k, v, qe, 0.125)
    for h in range(2):
        assert np.allclose(o_te[0, :, h], A.softmax_attention(qe[0, :, h], k[0, :, h], v[0, :, h], 0.125), atol=1e-13)
        assert np.allclose(o_tr[0, :, h], A.softmax_attention(qt[0, :, h], k[0, :, h], v[0, :, h], 0.125), atol=1e-13)
    # test queries equal to train queries give identical rows
    o_tr2, o_te2 = A.icl_attention(qt, k, v, qt[:, :30], 0.125)
    assert np.allclose(o_te2, o_tr2[:, :30], rtol=0, atol=1e-13)
    # row selection (BLAS may block differently for different row counts)
    s_tr, s_te = A.icl_attention(qt, k, v, qe, 0.125, rows_train=[5, 199], rows_test=[0, 29])
    assert np.allclose(s_tr, o_tr[:, [5, 199]], rtol=0, atol=1e-13)
    assert np.allclose(s_te, o_te[:, [0, 29]], rtol=0, atol=1e-13)


@pytest.mark.parametrize("block_kv", [1, 16, 64, 77, 200, 4096])
def test_kernel_model_without_p_rounding_equals_exact_attention(block_kv):
    # With P kept exact, the one-pass online softmax must reproduce Eq. (1) on the
    # dequantized inputs for any key-tile size (ragged tails included).
    qt, k, v, qe = _small_qkv(14)
    qz = Q.quantize_qkv_per_head(qt, k, v, qe)
    ref_tr, ref_te = A.icl_attention_dequantized(qz, 0.125)
    for row_sum in ("p8", "ptilde"):
        o_tr, o_te = A.icl_attention_fp8_kernel_model(qz, 0.125, block_kv, quantize_p=False, row_sum=row_sum)
        assert np.allclose(o_tr, ref_tr, rtol=1e-11, atol=1e-11 * np.abs(ref_tr).max())
        assert np.allclose(o_te, ref_te, rtol=1e-11, atol=1e-11 * np.abs(ref_te).max())


def p_rounding_bound(q, k, v, c):
    """Elementwise bound on |O_qp - O_q| from the e4m3 rounding of P alone.

    Each exact weight p_j = 2^(c(s_j - m) + 8) (m the final row max) is
    replaced by a rounded one with |error| <= 2^-4 p_j (normal e4m3) or
    <= 2^-10 (subnormal half step; later rescales only shrink it), and
    O_qp - O_q = sum_j (w_j - p_j)(v_j - O_q) / sum_j w_j.
    """
    s = q @ k.T
    p = np.exp2(c * (s - s.max(axis=1, keepdims=True)) + 8.0)
    o = (p @ v) / p.sum(axis=1, keepdims=True)
    e = 2.0 ** -4 * p + 2.0 ** -10
    num = np.einsum("rj,rjc->rc", e, np.abs(v[None, :, :] - o[:, None, :]))
    return o, num / (p.sum(axis=1) - e.sum(axis=1))[:, None]


@pytest.mark.parametrize("block_kv,seed", [(64, 15), (32, 16), (500, 17)])
def test_kernel_model_with_p_rounding_within_e4m3_bound(block_kv, seed):
    qt, k, v, qe = _small_qkv(seed, N=300, M=20, spread=4.0)
    qz = Q.quantize_qkv_per_head(qt, k, v, qe)
    o_tr, o_te = A.icl_attention_fp8_kernel_model(qz, 0.125, block_kv)
    ref_tr, ref_te = A.icl_attention_dequantized(qz, 0.125)
    for h in range(2):
        c = 0.125 * float(qz["s_q"][0, h]) * float(qz["s_k"][0, h]) * A.LOG2E
        kq, vq = decode(qz["k8"][0, h]), decode(qz["v8"][0, h]) * float(qz["s_v"][0, h])
        for q8, got, ref in ((qz["q8_train"], o_tr, ref_tr), (qz["q8_test"], o_te, ref_te)):
            o, bnd = p_rounding_bound(decode(q8[0, h]), kq, vq, c)
            assert np.allclose(o, ref[0, :, h], atol=1e-9 * np.abs(o).max())
            err = np.abs(got[0, :, h] - ref[0, :, h])
            assert np.all(err <= bnd * (1 + 1e-9) + 1e-12)
            assert err.max() > 0                                      # P really is rounded


def test_kernel_model_identical_keys_constant_v_and_one_hot():
    rng = np.random.default_rng(18)
    D, N = 64, 150
    q8 = decode(encode_rne(np.clip(rng.standard_normal((10, D)) * 60, -448, 448)))
    k8 = np.tile(decode(encode_rne(np.clip(rng.standard_normal((1, D)) * 60, -448, 448))), (N, 1))
    v8 = decode(encode_rne(np.clip(rng.standard_normal((N, D)) * 60, -448, 448)))
    # identical keys: every lifted weight is exactly 2^8, so the output is the mean of V exactly
    o = A.one_pass_fp8_attention(q8, k8, v8, 0.01, 0.5, 64)
    assert np.allclose(o, 0.5 * v8.mean(axis=0), rtol=0, atol=1e-12)
    # constant V: the rounded weights are normalised by their own sum
    k8 = decode(encode_rne(np.clip(rng.standard_normal((N, D)) * 60, -448, 448)))
    vc = np.full((N, D), 3.5)
    assert np.allclose(A.one_pass_fp8_attention(q8, k8, vc, 0.003, 2.0, 64), 7.0, rtol=0, atol=1e-12)
    # one-hot: key 37 exceeds all others by > 20 in the base-2 logit, others round to 0
    k8 = np.zeros((N, D)); k8[37, 0] = 448.0; q8 = np.zeros((1, D)); q8[0, 0] = 448.0
    assert np.array_equal(A.one_pass_fp8_attention(q8, k8, v8, 1e-4, 1.0, 64)[0], v8[37])


def test_kernel_model_lifts_row_max_to_256_and_weights_are_e4m3_values():
    # V = identity reveals the normalised weights; with one key tile the largest weight is 2^8.
    rng = np.random.default_rng(19)
    N = D = 64
    q8 = decode(encode_rne(np.clip(rng.standard_normal((5, D)) * 60, -448, 448)))
    k8 = decode(encode_rne(np.clip(rng.standard_normal((N, D)) * 60, -448, 448)))
    w = A.one_pass_fp8_attention(q8, k8, np.eye(N), 2e-4, 1.0, N)
    p8 = 256.0 * w / w.max(axis=1, keepdims=True)
    assert np.all(np.argmax(w, axis=1) == np.argmax(q8 @ k8.T, axis=1))
    assert np.allclose(p8, decode(encode_rne(np.round(p8, 9))), rtol=0, atol=1e-9)


def test_running_max_lift_worked_example():
    # One query, two blocks of two keys, c = 0.1 and one-hot V rows, so the output is the
    # normalised weight vector.  In [128, 256) the e4m3 values are 16 apart, in [64, 128)
    # 8 apart.  Block 1 (scores 0, -3): its running max is 0, the lifted weights are
    # 2^8 = 256 and 2^7.7 = 207.9, which rounds to 208.  Block 2 (scores 15, 10): the max
    # moves to 15, block 1's state is rescaled by 2^(0.1 (0 - 15)) = 2^-1.5, and the new
    # weights are 256 and 2^7.5 = 181.0, which rounds to 176 (the midpoint to 192 is 184).
    # A lift relative to the row's final max would give block 1 the weights 2^6.5 = 90.5
    # -> 88 and 2^6.2 = 73.5 -> 72 instead of 256 r = 90.5 and 208 r = 73.5.
    r = 2.0 ** -1.5
    w = np.array([256 * r, 208 * r, 256.0, 176.0])
    o = A.one_pass_fp8_attention(np.array([[1.0]]), np.array([[0.0], [-3.0], [15.0], [10.0]]), np.eye(4), 0.1,
                                 1.0, 2)
    assert np.allclose(o[0], w / w.sum(), rtol=1e-14, atol=0)


def test_lift_keeps_subnormal_weights():
    # Base-2 logits 0 and -17.5: with the 2^8 lift the small weight is 2^-9.5, which
    # rounds to the smallest subnormal 2^-9 (a lift of 2^7 would round it to 0).
    q8 = np.zeros((1, 64)); q8[0, 0] = 1.0
    k8 = np.zeros((2, 64)); k8[0, 0] = 64.0; k8[1, 0] = 32.0
    w = A.one_pass_fp8_attention(q8, k8, np.eye(2), 17.5 / 32.0, 1.0, 64)[0]
    assert w[1] == 2.0 ** -9 / (256.0 + 2.0 ** -9)
    assert w[0] == 256.0 / (256.0 + 2.0 ** -9)


def test_tie_allowance_bounds_the_effect_of_perturbed_exponents():
    # With a single key tile the output depends on c only through the e4m3
    # rounding of P~ (the lifted weights are normalised by their own sum), so it
    # is piecewise constant in c.  Moving c by a relative amount that moves every
    # P~ by less than tie_rel can only flip the rounding of P~ values inside the
    # tie window, so the result moves by at most the returned allowance.
    rng = np.random.default_rng(25)
    N, D = 700, 64
    q8 = decode(encode_rne(np.clip(rng.standard_normal((40, D)) * 80, -448, 448)))
    k8 = decode(encode_rne(np.clip(rng.standard_normal((N, D)) * 80, -448, 448)))
    v8 = decode(encode_rne(np.clip(rng.standard_normal((N, D)) * 80, -448, 448)))
    c = 1.3e-5
    o, allow = A.one_pass_fp8_attention(q8, k8, v8, c, 0.01, N, tie_rel=1e-4)
    assert np.array_equal(o, A.one_pass_fp8_attention(q8, k8, v8, c, 0.01, N))
    assert allow.max() > 0
    # relative move of P~ = 2^(c f (s - m) + 8) is (2^((f-1) c |s - m|) - 1) <= 1e-4 here
    span = c * np.max((q8 @ k8.T).max(axis=1) - (q8 @ k8.T).min(axis=1))
    moved = 0
    for f in (1 + 0.9e-4 / span, 1 - 0.9e-4 / span, 1 + 0.3e-4 / span):
        o2 = A.one_pass_fp8_attention(q8, k8, v8, c * f, 0.01, N)
        d = np.abs(o2 - o)
        moved += np.count_nonzero(d > 1e-12 * np.abs(o).max())
        assert np.all(d <= allow * 1.001 + 1e-12 * np.abs(o).max())
    assert moved > 0
    # with a tiny window nothing is flagged in a generic row
    _, allow0 = A.one_pass_fp8_attention(q8[:3], k8, v8, c, 0.01, N, tie_rel=1e-15)
    assert allow0.max() < 1e-9 * np.abs(o).max()


def _repeat_heads(x, H, G, axis):
    """The standard grouped-query expansion: head h of the result is head h // (H // G) of x."""
    return np.repeat(np.take(x, np.arange(G), axis=axis), H // G, axis=axis)


@pytest.mark.parametrize("G", [1, 2, 4])
def test_grouped_test_heads_equal_attention_over_repeated_kv_heads(G):
    # Appendix (noise experiment): TabPFN-v3's test rows attend, grouped-query style, to the
    # first K/V head(s) of the train-train call.
    qt, k, v, qe = _small_qkv(21, B=2, N=150, M=20, H=4)
    o_tr, o_te = A.icl_attention(qt, k, v, qe, 0.125, test_kv_heads=G)
    ref_tr, _ = A.icl_attention(qt, k, v, qe, 0.125)
    _, ref_te = A.icl_attention(qt, _repeat_heads(k, 4, G, 2), _repeat_heads(v, 4, G, 2), qe, 0.125)
    assert np.allclose(o_tr, ref_tr, rtol=0, atol=1e-13)
    assert np.allclose(o_te, ref_te, rtol=0, atol=1e-13)
    # the FP8 kernel model reads that K/V head's codes and scales for the test rows
    qz = Q.quantize_qkv_per_head(qt, k, v, qe)
    rep = dict(qz)
    for key in ("k8", "v8", "s_k", "s_v"):
        rep[key] = _repeat_heads(qz[key], 4, G, 1)
    m_tr, m_te = A.icl_attention_fp8_kernel_model(qz, 0.125, 64, test_kv_heads=G)
    r_tr, _ = A.icl_attention_fp8_kernel_model(qz, 0.125, 64)
    _, r_te = A.icl_attention_fp8_kernel_model(rep, 0.125, 64)
    assert np.array_equal(m_tr, r_tr) and np.array_equal(m_te, r_te)
    d_tr, d_te = A.icl_attention_dequantized(qz, 0.125, test_kv_heads=G)
    _, e_te = A.icl_attention_dequantized(rep, 0.125)
    assert np.allclose(d_te, e_te, rtol=0, atol=1e-13)
    if G < 4:
        assert not np.allclose(o_te, A.icl_attention(qt, k, v, qe, 0.125)[1], atol=1e-3)


def test_grouped_test_heads_must_divide_h():
    qt, k, v, qe = _small_qkv(22, N=10, M=3, H=4)
    with pytest.raises(ValueError):
        A.icl_attention(qt, k, v, qe, 0.125, test_kv_heads=3)


@pytest.mark.parametrize("mode,test_mult", [("per_call", 0.0625), ("joint", 2.0)])
def test_kernel_model_uses_the_test_query_scale(mode, test_mult):
    # per_call: test queries 16x below the train amax get a scale ~16x below s_q, so a test
    # call that used s_q for them would scale its logits by ~16.  joint: test queries above the
    # train amax set the one scale of both calls.
    qt, k, v, qe = _small_qkv(23, N=300, M=24, spread=1.0)
    qe = qe * np.float32(test_mult)
    qz = Q.quantize_qkv_per_head(qt, k, v, qe, q_scale_mode=mode)
    assert np.all(np.abs(qz["s_q_test"] / qz["s_q"] - test_mult) < 0.5 * test_mult) if mode == "per_call" else \
        np.array_equal(qz["s_q_test"], qz["s_q"])
    ex_tr, ex_te = A.icl_attention(qt, k, v, qe, 0.125)
    o_tr, o_te = A.icl_attention_fp8_kernel_model(qz, 0.125, 64)
    d_tr, d_te = A.icl_attention_dequantized(qz, 0.125)
    for h in range(2):
        c = 0.125 * float(qz["s_q_test"][0, h]) * float(qz["s_k"][0, h]) * A.LOG2E
        kq, vq = decode(qz["k8"][0, h]), decode(qz["v8"][0, h]) * float(qz["s_v"][0, h])
        o, bnd = p_rounding_bound(decode(qz["q8_test"][0, h]), kq, vq, c)
        assert np.allclose(o, d_te[0, :, h], atol=1e-9 * np.abs(o).max())
        assert np.all(np.abs(o_te[0, :, h] - d_te[0, :, h]) <= bnd * (1 + 1e-9) + 1e-12)
    # and O_q and O_qp stay within the FP8 quantization error of the exact result on both calls
    for got, ex in ((d_tr, ex_tr), (d_te, ex_te), (o_tr, ex_tr), (o_te, ex_te)):
        assert np.linalg.norm(got - ex) / np.linalg.norm(ex) < 0.1      # a wrong query scale gives ~1


def test_kernel_model_with_a_vanishing_softmax_factor_returns_the_mean_of_v():
    # c = 0 (alpha s_q s_k underflowing): every logit is 0, Eq. (1) gives the plain mean of V,
    # and the replay must not rescale its empty first state by 2^(0 * -inf)
    rng = np.random.default_rng(27)
    N, D = 300, 64
    q8 = decode(encode_rne(np.clip(rng.standard_normal((7, D)) * 60, -448, 448)))
    k8 = decode(encode_rne(np.clip(rng.standard_normal((N, D)) * 60, -448, 448)))
    v8 = decode(encode_rne(np.clip(rng.standard_normal((N, D)) * 60, -448, 448)))
    for c in (0.0, 1e-300):
        o = A.one_pass_fp8_attention(q8, k8, v8, c, 0.25, 128)
        assert np.allclose(o, 0.25 * v8.mean(axis=0), rtol=0, atol=1e-12 * np.abs(v8).max())


def test_kernel_model_scores_hook_and_per_row_tie_windows():
    # scores given explicitly stand for Q_8 K_8^T: the exact products reproduce the default,
    # and scores doubled with c halved give the same logits, hence the same output
    rng = np.random.default_rng(28)
    N, D = 400, 64
    q8 = decode(encode_rne(np.clip(rng.standard_normal((6, D)) * 60, -448, 448)))
    k8 = decode(encode_rne(np.clip(rng.standard_normal((N, D)) * 60, -448, 448)))
    v8 = decode(encode_rne(np.clip(rng.standard_normal((N, D)) * 60, -448, 448)))
    c = 3e-4
    base = A.one_pass_fp8_attention(q8, k8, v8, c, 0.5, 128)
    assert np.array_equal(A.one_pass_fp8_attention(q8, k8, v8, c, 0.5, 128, scores=q8 @ k8.T), base)
    assert np.allclose(A.one_pass_fp8_attention(q8, k8, v8, c / 2, 0.5, 128, scores=2 * (q8 @ k8.T)), base,
                       rtol=1e-13, atol=1e-13 * np.abs(base).max())
    moved = A.one_pass_fp8_attention(q8, k8, v8, c, 0.5, 128, scores=q8 @ k8.T + 1500.0 * (np.arange(N) == 5))
    assert not np.allclose(moved, base)
    # a tie window given per row equals the scalar one on every row
    _, a1 = A.one_pass_fp8_attention(q8, k8, v8, c, 0.5, 128, tie_rel=1e-3)
    _, a2 = A.one_pass_fp8_attention(q8, k8, v8, c, 0.5, 128, tie_rel=np.full(6, 1e-3))
    assert np.array_equal(a1, a2)
