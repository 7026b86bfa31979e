"""Softmax attention references in fp64 (test oracle).

* ``softmax_attention`` -- Eq. (1): Attn(Q,K,V) = P V, P = softmax(alpha Q K^T)
  row-wise, alpha a scalar (Sec. 3).  Softmax is evaluated after subtracting
  the row maximum, which leaves it unchanged mathematically.
* ``icl_attention`` -- the ICL stage evaluates Eq. (1) twice per head: the N
  train queries and the M test queries both attend to the same N train keys
  and values (Sec. 3, second paragraph).  Used on the exact inputs (O_exact)
  and on the dequantized inputs s*X_8 (O_q).  With ``test_kv_heads`` G < H
  the test call is grouped-query attention over the first G heads of the
  train K/V: query head h reads K/V head h // (H / G).  TabPFN-v3's test
  rows attend to the first K/V head this way (G = 1), and the two calls then
  consume the very same K/V entries (appendix, noise experiment).
* ``icl_attention_fp8_kernel_model`` -- a replay, in fp64, of the one-pass
  fused kernel the paper describes (Sec. 3 and Fig. 2): tiles of ``block_kv``
  keys in order, a running row maximum, the Q and K scales applied together
  with the softmax scale, P lifted so that the running row maximum maps to
  2^8 and rounded to e4m3 inside the kernel, and the V scale applied in the
  epilogue (O_qp).

Readings (the paper is silent; each is also listed in the design notes):
* the 2^8 lift is relative to the running maximum after the current key
  tile, the only maximum a one-pass kernel knows;
* the row sum l accumulates the rounded P_8 values (``row_sum="p8"``), so
  the effective weights of every row sum to one; ``row_sum="ptilde"`` sums
  the unrounded P~ instead;
* alpha is an fp32 value (default 1/sqrt(d)), widened to fp64 here.
"""
import math

import numpy as np

from .e4m3 import decode, round_to_e4m3

LOG2E = math.log2(math.e)
P_LIFT_LOG2 = 8.0          # the row maximum of P is lifted to 2^8 = 256


def softmax_attention(q, k, v, alpha, chunk_rows=1024):
    """Eq. (1) in fp64: q (R,D), k (N,D), v (N,D) -> (R,D)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    out = np.empty((q.shape[0], v.shape[1]), dtype=np.float64)
    for r0 in range(0, q.shape[0], chunk_rows):
        s = float(alpha) * (q[r0:r0 + chunk_rows] @ k.T)
        s -= s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[r0:r0 + chunk_rows] = p @ v
    return out


def _pick(rows, n):
    return np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)


def grouped_kv_head(h, H, test_kv_heads):
    """The K/V head that test query head h reads (test_kv_heads None or 0 means H)."""
    G = H if not test_kv_heads else int(test_kv_heads)
    if G < 1 or G > H or H % G:
        raise ValueError("test_kv_heads must divide H")
    return h // (H // G)


def icl_attention(q_train, k, v, q_test, alpha, rows_train=None, rows_test=None, test_kv_heads=None):
    """Train-train and test-train attention on (B,S,H,D) inputs, fp64.

    Returns (o_train, o_test) with shapes (B, R_train, H, D) and
    (B, R_test, H, D) for the selected query rows (all rows by default).
    """
    q_train = np.asarray(q_train)
    B, N, H, D = q_train.shape
    rt = _pick(rows_train, N)
    M = 0 if q_test is None else np.asarray(q_test).shape[1]
    re = _pick(rows_test, M)
    o_tr = np.zeros((B, len(rt), H, D))
    o_te = np.zeros((B, len(re), H, D))
    for b in range(B):
        for h in range(H):
            kk = k[b, :, h, :]
            vv = v[b, :, h, :]
            o_tr[b, :, h] = softmax_attention(q_train[b, rt, h, :], kk, vv, alpha)
            if len(re):
                hk = grouped_kv_head(h, H, test_kv_heads)
                o_te[b, :, h] = softmax_attention(q_test[b, re, h, :], k[b, :, hk, :], v[b, :, hk, :], alpha)
    return o_tr, o_te


def dequantize(codes, scale):
    """s * X_8 as (B,S,H,D) fp64 from (B,H,S,D) codes and (B,H) scales."""
    x = decode(codes) * np.asarray(scale, dtype=np.float64)[:, :, None, None]
    return x.transpose(0, 2, 1, 3)


def icl_attention_dequantized(qz, alpha, rows_train=None, rows_test=None, test_kv_heads=None):
    """O_q: Eq. (1) in fp64 on the dequantized tensors of ``quantize_qkv_per_head``
    (test queries with their own scale s_q_test)."""
    q_te = dequantize(qz["q8_test"], qz.get("s_q_test", qz["s_q"])) if "q8_test" in qz else None
    return icl_attention(dequantize(qz["q8_train"], qz["s_q"]),
                         dequantize(qz["k8"], qz["s_k"]),
                         dequantize(qz["v8"], qz["s_v"]),
                         q_te, alpha, rows_train, rows_test, test_kv_heads)


def one_pass_fp8_attention(q8, k8, v8, c, s_v, block_kv, quantize_p=True, row_sum="p8", tie_rel=None,
                           scores=None):
    """One head of the fused FP8 kernel, replayed in fp64.

    q8 (R,D), k8 (N,D), v8 (N,D) are the e4m3 *values* (decoded codes),
    c = alpha * s_q * s_k * log2(e) is the factor that turns a raw code dot
    product into a base-2 logit, s_v the V dequantization scale.  ``scores``
    (R,N), if given, stands for the code dot products Q_8 K_8^T (by default
    they are computed exactly), so that the same replay can be run on the
    scores of a particular FP8 dot-product arithmetic.  Before the first key
    block the state is empty; its rescale factor is 0 (as 2^(c (-inf)) is for
    any c > 0, and also when c underflows to 0).

    With ``tie_rel`` set (a scalar, or one value per row), also returns the
    sensitivity of the result to
    rounding ties of P: for every P~ whose e4m3 rounding changes when P~ moves
    by a relative tie_rel, the two candidate codes differ by ``spread``; if an
    implementation picks the other one for any such keys, its output moves by
    at most sum_j spread_j r_j (|v_j| + |o|) / l (r_j the later rescales), which
    is returned elementwise as (o, allowance).
    """
    R, D = q8.shape
    N = k8.shape[0]
    m = np.full(R, -np.inf)
    l = np.zeros(R)
    acc = np.zeros((R, v8.shape[1]))
    tie_l = np.zeros(R)
    tie_acc = np.zeros((R, v8.shape[1]))
    if tie_rel is not None and np.ndim(tie_rel):
        tie_rel = np.asarray(tie_rel, dtype=np.float64).reshape(R, 1)
    for j0 in range(0, N, block_kv):
        if scores is None:
            s = q8 @ k8[j0:j0 + block_kv].T      # exact: products of e4m3 values
        else:
            s = np.asarray(scores[:, j0:j0 + block_kv], dtype=np.float64)
        m_new = np.maximum(m, s.max(axis=1))
        p = np.exp2(c * (s - m_new[:, None]) + P_LIFT_LOG2)   # <= 2^8
        p8 = round_to_e4m3(p) if quantize_p else p
        # rescale of the old state; the empty state before the first block has none
        first = np.isneginf(m)
        r = np.where(first, 0.0, np.exp2(c * (np.where(first, m_new, m) - m_new)))
        l = l * r + (p8 if row_sum == "p8" else p).sum(axis=1)
        acc = acc * r[:, None] + p8 @ v8[j0:j0 + block_kv]
        if tie_rel is not None:
            spread = round_to_e4m3(p * (1 + tie_rel)) - round_to_e4m3(p * (1 - tie_rel))
            tie_l = tie_l * r + spread.sum(axis=1)
            tie_acc = tie_acc * r[:, None] + spread @ np.abs(v8[j0:j0 + block_kv])
        m = m_new
    o = acc * float(s_v) / l[:, None]
    if tie_rel is None:
        return o
    return o, (tie_acc * float(s_v) + tie_l[:, None] * np.abs(o)) / l[:, None]


def icl_attention_fp8_kernel_model(qz, alpha, block_kv, rows_train=None, rows_test=None,
                                   quantize_p=True, row_sum="p8", tie_rel=None, test_kv_heads=None,
                                   score_fn=None):
    """O_qp: both ICL calls through ``one_pass_fp8_attention`` for every (b, h).

    ``qz`` is the output of ``quantize_qkv_per_head``.  The test call of head
    h uses the test-query scale s_q_test and the codes and scales of K/V head
    ``grouped_kv_head(h, H, test_kv_heads)``.  Returns (o_train, o_test) as
    (B, R, H, D) fp64 for the selected rows; with ``tie_rel`` set, returns
    ((o_train, allowance_train), (o_test, allowance_test)).  ``score_fn``,
    if given, maps (query codes (R,D), key codes (N,D)) to the scores the
    replay uses in place of the exact Q_8 K_8^T.
    """
    B, H, N, D = qz["k8"].shape
    rt = _pick(rows_train, N)
    M = qz["q8_test"].shape[2] if "q8_test" in qz else 0
    re = _pick(rows_test, M)
    o_tr = np.zeros((B, len(rt), H, D))
    o_te = np.zeros((B, len(re), H, D))
    a_tr = np.zeros_like(o_tr)
    a_te = np.zeros_like(o_te)
    s_q_test = qz.get("s_q_test", qz["s_q"])
    for b in range(B):
        for h in range(H):
            hk = grouped_kv_head(h, H, test_kv_heads)
            calls = ((o_tr, a_tr, "q8_train", rt, qz["s_q"][b, h], h),
                     (o_te, a_te, "q8_test", re, s_q_test[b, h], hk))
            for o, a, key, rows, s_query, hkv in calls:
                if len(rows) == 0:
                    continue
                c = float(alpha) * float(s_query) * float(qz["s_k"][b, hkv]) * LOG2E
                args = (decode(qz["k8"][b, hkv]), decode(qz["v8"][b, hkv]), c, qz["s_v"][b, hkv], block_kv,
                        quantize_p, row_sum, tie_rel)
                sc = None if score_fn is None else score_fn(qz[key][b, h, rows], qz["k8"][b, hkv])
                res = one_pass_fp8_attention(decode(qz[key][b, h, rows]), *args, scores=sc)
                if tie_rel is None:
                    o[b, :, h] = res
                else:
                    o[b, :, h], a[b, :, h] = res
    if tie_rel is None:
        return o_tr, o_te
    return (o_tr, a_tr), (o_te, a_te)
