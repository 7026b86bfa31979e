"""Parity checks of the FP8 path against the oracle (test infrastructure).

Every expected value comes from ``oracle/``; this module adds only the
tolerances and the bounds they rest on, each derived from a stated fact:

T0   codes and scales: bit-exact against ``oracle.quantize`` (the tests
     compare them directly).
T1   O_gpu against O_qp, the oracle's replay of the one-pass kernel
     (``oracle.attention.one_pass_fp8_attention``), in the regime where every
     FP8 dot product is exact (``narrow_range_inputs``):
         |dO| <= 1.01 * tie allowance + 1e-5 RMS + 1e-6 |O_qp|.
     The kernel's exponent c S + 8 - c m is computed in fp32; it moves P~ by
     less than TIE_REL relative there, so a key can round to the other e4m3
     neighbour only if P~ lies within TIE_REL of a midpoint, and the oracle's
     tie allowance bounds the effect of all such keys.
T1hw O_gpu against the same oracle replay fed the scores of the FP8 MFMA's
     measured arithmetic (``mfma_model.scores``, pinned against the hardware
     by ``test_gpu_mfma_precision.py``) instead of the exact Q_8 K_8^T, on any
     inputs, elementwise:
         |dO| <= 1.01 * tie allowance(row) + pv_term + 1e-5 RMS + 1e-6 |O|,
     with the tie window widened per row to cover the fp32 rounding of
     c * m (``hw_tie_rel``) and pv_term the bound of the P V and row-sum
     instructions (``pv_rowsum_term``).
T2'  O_gpu against O_q, Eq. (1) in fp64 on the dequantized inputs
     (``oracle.attention.icl_attention_dequantized``), elementwise within the
     bound that follows from the method's rounding of P to e4m3 and the FP8
     dot-product error bound (``fp8_bound``), with slack 1.25 and 1e-5 RMS.
"""
import concurrent.futures as cf
import math
import os
import time

import numpy as np
import torch

import mfma_model as MM
from oracle import attention as OA
from oracle.e4m3 import decode

TIE_REL = 2.0 ** -18
T1_OUTLIER = 2e-3
ACC_REL = 2.0 ** -22      # one fp32 accumulation into a running sum, per 64-key chunk (relative)
P_HALF_ULP = 2.0 ** -4    # e4m3 rounding of a normal P~
P_SUB_HALF = 2.0 ** -10   # e4m3 rounding of a subnormal P~ (half the 2^-9 step)
T2_SLACK = 1.25


def checker_device():
    """The GPU when there is one (the full-size checks need its speed), else the CPU."""
    return torch.device("cuda") if torch.cuda.is_available() else torch.device("cpu")


def workers():
    return max(1, min(16, os.cpu_count() or 1))


def t1_metrics(got, ref):
    d = np.abs(np.asarray(got, np.float64) - ref)
    rms = np.sqrt(np.mean(ref ** 2))
    return {"max_over_rms": float(d.max() / rms) if d.size else 0.0,
            "relF": float(np.linalg.norm(d) / np.linalg.norm(ref)) if d.size else 0.0,
            "outlier_frac": float(np.mean(d > T1_OUTLIER * rms)) if d.size else 0.0}


def assert_t1(got, ref, allowance, what=""):
    got = np.asarray(got, np.float64)
    rms = np.sqrt(np.mean(ref ** 2))
    err = np.abs(got - ref)
    tol = 1.01 * allowance + 1e-5 * rms + 1e-6 * np.abs(ref)
    assert np.all(err <= tol), (what, (err / tol).max(), t1_metrics(got, ref))
    return t1_metrics(got, ref)


def softmax_factor(alpha, s_query, s_k):
    """c = alpha * s_q * s_k * log2(e), as the oracle's replay computes it."""
    return float(alpha) * float(s_query) * float(s_k) * OA.LOG2E


def hw_tie_rel(c, scores):
    """Per-row tie window for the kernel's fp32 exponent.  The kernel forms
    t = fma(S, c, fl32(8 - fl32(c m))) with c itself rounded to fp32 (three
    roundings): the error of t is below (2 |c m| + 64) 2^-24 in log2 units for the
    keys whose weights count (|c (S - m)| <= 32 there), which moves P~ = 2^t by
    ln2 times that, relative.  A factor 4 of margin, and at least TIE_REL."""
    m = np.max(np.abs(scores), axis=1) if scores.shape[1] else np.zeros(scores.shape[0])
    return np.maximum(TIE_REL, 4 * math.log(2) * (2 * abs(c) * m + 64) * 2.0 ** -24)


def pv_rowsum_term(v_hat_absmax, o, N):
    """Bound on the error that the P V and row-sum instructions add to an output row.

    Per 64-key chunk each is one FP8 MFMA whose groups of 8 keys err by less than
    7 * 2^-13 * 2^(max e_P) * 2^(max e_V) (mfma_model); summed over the chunks, with
    2^(max e_P) <= max(P, 2^-6) and the row's lifted weights summing to l >= 2^8, the
    group terms are below 7 * 2^-13 * (1 + N 2^-17) of l * max|V_c| (P V) and of l (row
    sum).  The fp32 accumulation across the ceil(N/64) chunks adds ACC_REL per chunk.
    Returns the elementwise bound |dO_c| <= (e_pv_c + |O_c| e_l) / (1 - e_l)."""
    n_tiles = (N + 63) // 64
    grp = MM.GROUP_REL * (1 + N * 2.0 ** -17)
    e_l = grp + n_tiles * ACC_REL
    e_pv = grp * v_hat_absmax[None, :] + n_tiles * ACC_REL * np.abs(o)
    return (e_pv + np.abs(o) * e_l) / (1 - e_l)


def fp8_bound(q8, k8, v8, s_v, c, device, row_chunk=None):
    """T2': (O, bound) for query codes q8 (R,D) against key / value codes k8, v8 (N,D).

    With p_j = 2^(c (s_j - max s) + 8) the exact lifted weights (s = Q_8 K_8^T), the
    kernel's effective weight is, up to a factor common to the row, p_j 2^(c d_j)
    (1 + r_j) + z_j: d_j the FP8 dot-product error of that score (|d_j| <=
    delta_j = mfma_model.dot_error_bound), |r_j| <= 2^-4 (e4m3 half ulp) and |z_j| <=
    2^-10 2^(c max delta) (half the subnormal step, scaled by the row's common factor).
    Then O - O_q = sum_j e_j (v_j - O_q) / sum_j (p_j + e_j) with |e_j| <= A_j + z,
    A_j = p_j ((1 + 2^-4) 2^(c delta_j) - 1); the P V and row-sum instructions add
    ``pv_rowsum_term``.  Evaluated on ``device`` in fp64, row chunk by row chunk, with
    |v_j - O_q| bounded by |v_j - mu| + |O_q - mu| (mu the mean of V-hat over the keys)."""
    dev = device
    q = torch.from_numpy(decode(q8)).to(dev)
    k = torch.from_numpy(decode(k8)).to(dev)
    v_hat = torch.from_numpy(decode(v8) * float(s_v)).to(dev)
    gq = torch.from_numpy(MM.group_max_exp2(q8)).to(dev)
    gk = torch.from_numpy(MM.group_max_exp2(k8)).to(dev)
    R, D = q.shape
    N = k.shape[0]
    mu = v_hat.mean(dim=0) if N else torch.zeros(D, dtype=torch.float64, device=dev)
    v_dev = (v_hat - mu[None, :]).abs()
    o_all = np.empty((R, D))
    bnd_all = np.empty((R, D))
    if row_chunk is None:          # (rows, N) fp64 temporaries of at most 1 GB
        row_chunk = max(1, (1 << 27) // max(1, N))
    for r0 in range(0, R, row_chunk):
        r1 = min(R, r0 + row_chunk)
        s = q[r0:r1] @ k.T                                   # exact: e4m3 products, fp64 sums
        p = torch.exp2(c * (s - s.amax(dim=1, keepdim=True)) + 8.0)
        psum = p.sum(dim=1)
        o = (p @ v_hat) / psum[:, None]
        delta = MM.GROUP_REL * (gq[r0:r1] @ gk.T) + 2 * MM.ACC_REL * (q[r0:r1].abs() @ k.abs().T)
        A = p * ((1 + P_HALF_ULP) * torch.exp2(c * delta) - 1)
        z = P_SUB_HALF * torch.exp2(c * delta.amax(dim=1))
        e = A + z[:, None]                                   # (r, N)
        # sum_j e_j |v_j - o| <= sum_j e_j |v_j - mu| + |o - mu| sum_j e_j for any per-channel mu
        # (here the mean of V over the keys): two products instead of an (r, N, D) temporary
        esum = e.sum(dim=1)
        num = e @ v_dev + (o - mu[None, :]).abs() * esum[:, None]
        den = psum - esum
        b = torch.where(den[:, None] > 0, num / den.clamp(min=1e-300)[:, None], torch.full_like(num, float("inf")))
        o_all[r0:r1] = o.cpu().numpy()
        bnd_all[r0:r1] = b.cpu().numpy()
    vmax = np.abs(decode(v8) * float(s_v)).max(axis=0) if N else np.zeros(D)
    return o_all, bnd_all + pv_rowsum_term(vmax, o_all, N)


def _replay_hw(q8, k8, v8, c, s_v, block_kv, device, row_chunk=None):
    """The oracle's replay on the MFMA model's scores, with the per-row tie allowance,
    in row chunks spread over threads (numpy releases the GIL in the heavy parts)."""
    kd = torch.from_numpy(np.ascontiguousarray(k8)).to(device)
    kv, vv = decode(k8), decode(v8)
    R = q8.shape[0]
    if row_chunk is None:          # the replay loops over key blocks: small chunks cost interpreter time
        row_chunk = int(min(128, max(32, -(-R // workers()))))

    def one(r0):
        r1 = min(R, r0 + row_chunk)
        sc = MM.scores(torch.from_numpy(np.ascontiguousarray(q8[r0:r1])).to(device), kd).cpu().numpy()
        if device.type == "cuda":
            torch.cuda.synchronize()
        o, allow = OA.one_pass_fp8_attention(decode(q8[r0:r1]), kv, vv, c, s_v, block_kv,
                                             tie_rel=hw_tie_rel(c, sc), scores=sc)
        return r0, o, allow

    o = np.empty((R, kv.shape[1]))
    allow = np.empty_like(o)
    with cf.ThreadPoolExecutor(workers()) as ex:
        for r0, oo, aa in ex.map(one, range(0, R, row_chunk)):
            o[r0:r0 + len(oo)] = oo
            allow[r0:r0 + len(oo)] = aa
    return o, allow


def _head(qz, b, h, call, test_kv_heads):
    """(query code key, query scale, K/V head) of one call of head h."""
    if call == "train":
        return "q8_train", qz["s_q"][b, h], h
    hk = OA.grouped_kv_head(h, qz["k8"].shape[1], test_kv_heads)
    return "q8_test", qz.get("s_q_test", qz["s_q"])[b, h], hk


def oracle_o_q(qz, alpha, b, h, rows, call="train", test_kv_heads=None):
    """O_q rows of one (b, h) and call, from ``oracle.attention.icl_attention_dequantized``."""
    key, _, hk = _head(qz, b, h, call, test_kv_heads)
    sub = {"q8_train": qz["q8_train"][b:b + 1, h:h + 1], "s_q": qz["s_q"][b:b + 1, h:h + 1],
           "k8": qz["k8"][b:b + 1, hk:hk + 1], "s_k": qz["s_k"][b:b + 1, hk:hk + 1],
           "v8": qz["v8"][b:b + 1, hk:hk + 1], "s_v": qz["s_v"][b:b + 1, hk:hk + 1]}
    if call == "test":
        sub["q8_test"] = qz["q8_test"][b:b + 1, h:h + 1]
        sub["s_q_test"] = qz.get("s_q_test", qz["s_q"])[b:b + 1, h:h + 1]
        return OA.icl_attention_dequantized(sub, alpha, [], rows)[1][0, :, 0]
    return OA.icl_attention_dequantized(sub, alpha, rows, [])[0][0, :, 0]


def check_fp8_rows(got, qz, alpha, b, h, rows, call="train", test_kv_heads=None, block_kv=128, what="",
                   device=None, t2=True, t1hw_every=1):
    """T1hw and T2' on query rows ``rows`` of (b, h) for one call; got (R, D) the GPU rows.
    T1hw runs on every ``t1hw_every``-th of them (its replay is the costly part at full
    size), T2' on all.  Returns metrics against the oracle's O_q and its hardware-score
    replay."""
    device = checker_device() if device is None else device
    rows = np.asarray(rows, dtype=np.int64)
    got = np.asarray(got, np.float64)
    key, s_query, hk = _head(qz, b, h, call, test_kv_heads)
    if len(rows) == 0:
        return {}
    q8 = qz[key][b, h][rows]
    k8, v8 = qz["k8"][b, hk], qz["v8"][b, hk]
    s_v = qz["s_v"][b, hk]
    c = softmax_factor(alpha, s_query, qz["s_k"][b, hk])
    N = k8.shape[0]
    sub = np.arange(0, len(rows), max(1, int(t1hw_every)))
    t0 = time.perf_counter()
    o_hw, allow = _replay_hw(q8[sub], k8, v8, c, s_v, block_kv, device)
    t1 = time.perf_counter()
    vmax = np.abs(decode(v8) * float(s_v)).max(axis=0)
    rms = np.sqrt(np.mean(o_hw ** 2))
    err = np.abs(got[sub] - o_hw)
    tol = 1.01 * allow + pv_rowsum_term(vmax, o_hw, N) + 1e-5 * rms + 1e-6 * np.abs(o_hw)
    assert np.all(err <= tol), ("T1hw", what, call, b, h, float((err / tol).max()),
                                int(rows[sub][np.argmax((err / tol).max(axis=1))]), t1_metrics(got[sub], o_hw))
    out = {"vs_hw_replay": t1_metrics(got[sub], o_hw), "seconds": {"t1hw": round(t1 - t0, 2)}}
    if t2:
        t0 = time.perf_counter()
        o_q = oracle_o_q(qz, alpha, b, h, rows, call, test_kv_heads)
        t1 = time.perf_counter()
        o_b, bnd = fp8_bound(q8, k8, v8, s_v, c, device)
        out["seconds"].update(o_q=round(t1 - t0, 2), t2_bound=round(time.perf_counter() - t1, 2))
        assert np.allclose(o_b, o_q, rtol=1e-9, atol=1e-9 * np.abs(o_q).max()), "checker's O differs from O_q"
        rms_q = np.sqrt(np.mean(o_q ** 2))
        err2 = np.abs(got - o_q)
        lim = T2_SLACK * bnd + 1e-5 * rms_q
        assert np.all(err2 <= lim), ("T2'", what, call, b, h, float((err2 / lim).max()))
        out["vs_o_q"] = t1_metrics(got, o_q)
        out["t2_use"] = float((err2 / lim).max())
    return out


def check_fp8_call(o, qz, alpha, rows_train, rows_test, test_kv_heads=None, block_kv=128, what="", heads=None,
                   t2=True, t1hw_every=1):
    """check_fp8_rows over every (b, h) (or the heads listed) of both calls; o = (o_train, o_test)
    the full GPU outputs (B, rows, H, D); rows_train / rows_test the rows checked (None: all).
    Returns the worst metrics."""
    o_tr, o_te = (np.asarray(x) for x in o)
    B, H = qz["s_q"].shape
    N = qz["k8"].shape[2]
    M = qz["q8_test"].shape[2] if "q8_test" in qz else 0
    rt = np.arange(N) if rows_train is None else np.asarray(rows_train)
    re = np.arange(M) if rows_test is None else np.asarray(rows_test)
    worst = {"relF_vs_hw_replay": 0.0, "max_over_rms_vs_hw_replay": 0.0, "relF_vs_o_q": 0.0, "t2_use": 0.0,
             "seconds": {}}
    for b in range(B):
        for h in (range(H) if heads is None else heads):
            for call, oo, rows in (("train", o_tr, rt), ("test", o_te, re)):
                if len(rows) == 0:
                    continue
                m = check_fp8_rows(oo[b, rows, h], qz, alpha, b, h, rows, call, test_kv_heads, block_kv,
                                   what, t2=t2, t1hw_every=t1hw_every)
                if len(rows) >= 1024:   # progress on the long full-size checks
                    print("checked %s b=%d h=%d %s: %d rows" % (what, b, h, call, len(rows)), flush=True)
                worst["relF_vs_hw_replay"] = max(worst["relF_vs_hw_replay"], m["vs_hw_replay"]["relF"])
                worst["max_over_rms_vs_hw_replay"] = max(worst["max_over_rms_vs_hw_replay"],
                                                         m["vs_hw_replay"]["max_over_rms"])
                for k, v in m["seconds"].items():
                    worst["seconds"][k] = round(worst["seconds"].get(k, 0.0) + v, 2)
                if t2:
                    worst["relF_vs_o_q"] = max(worst["relF_vs_o_q"], m["vs_o_q"]["relF"])
                    worst["t2_use"] = max(worst["t2_use"], m["t2_use"])
    return worst


def narrow_range_inputs(B, N, M, H, D, seed):
    """Inputs whose e4m3 codes all have magnitudes in [224, 448] (|x| in [amax/2, amax]
    with random signs), so every FP8 MFMA dot product of the kernel is exact:
    Q and K products span two binades, and with alpha = 1/sqrt(D) the lifted
    P_8 lie in [2^6, 2^8], so the P V products span a few binades too."""
    rng = np.random.default_rng(seed)
    def draw(rows):
        mag = rng.uniform(0.5, 1.0, (B, rows, H, D)).astype(np.float32)
        return (mag * rng.choice(np.array([-1.0, 1.0], np.float32), size=mag.shape)).astype(np.float32)
    q = draw(N + M)
    return {"q_train": q[:, :N].copy(), "k": draw(N), "v": draw(N), "q_test": q[:, N:].copy()}


def sample_rows(n, k, seed, block=128):
    """First/last rows, rows on both sides of query-tile boundaries and random rows (sorted, unique)."""
    rng = np.random.default_rng(seed)
    pick = {0, n - 1}
    for t in range(block, n, block * max(1, (n // block) // 8)):
        pick.update((t - 1, t))
    pick.update(rng.integers(0, n, size=max(0, k - len(pick))).tolist())
    return np.array(sorted(x for x in pick if 0 <= x < n), dtype=np.int64)


def to_dev(x, dtype):
    return torch.from_numpy(np.ascontiguousarray(x)).to(dtype).cuda()


def gpu_inputs(x, dtype):
    return {k: to_dev(v, dtype) for k, v in x.items()}


def bf16_check(got, q, k, v, alpha, device=None, what=""):
    """The bf16 kernel's rows against Eq. (1) in fp64 (``oracle.attention.softmax_attention``),
    elementwise.  The kernel rounds P to bf16 for the P V product and normalises by the sum
    of the rounded weights w_j (a row-sum MFMA over the same operand), so O_bf16 - O =
    sum_j (w_j - p_j)(v_j - O) / sum_j w_j with |w_j - p_j| <= 2^-8 p_j; the bf16 MFMA adds
    fp32 accumulation errors (2^-21 of sum p |v| per instruction, measured) over the
    ceil(N/16) instructions of a row.  Bound: 1.25 times that, plus 1e-5 RMS."""
    device = checker_device() if device is None else device
    ref = OA.softmax_attention(q, k, v, alpha)
    qd, kd, vd = (torch.from_numpy(np.asarray(a, np.float64)).to(device) for a in (q, k, v))
    R, D = qd.shape
    N = kd.shape[0]
    o_all, b_all = np.empty((R, D)), np.empty((R, D))
    step = max(1, (1 << 26) // max(1, N * D))
    for r0 in range(0, R, step):
        s = float(alpha) * (qd[r0:r0 + step] @ kd.T)
        p = torch.exp(s - s.amax(dim=1, keepdim=True))
        ps = p.sum(dim=1)
        o = (p @ vd) / ps[:, None]
        num = torch.einsum("rn,rnd->rd", p, (vd[None] - o[:, None]).abs())
        pv = (p @ vd.abs()) / ps[:, None]
        b = 2.0 ** -8 * num / ((1 - 2.0 ** -8) * ps[:, None]) + ((N + 15) // 16) * 2.0 ** -21 * (pv + o.abs())
        o_all[r0:r0 + step] = o.cpu().numpy()
        b_all[r0:r0 + step] = b.cpu().numpy()
    assert np.allclose(o_all, ref, rtol=1e-9, atol=1e-9 * np.abs(ref).max()), "checker's O differs from Eq. (1)"
    err = np.abs(np.asarray(got, np.float64) - ref)
    lim = 1.25 * b_all + 1e-5 * np.sqrt(np.mean(ref ** 2))
    assert np.all(err <= lim), ("bf16", what, float((err / lim).max()))
    return t1_metrics(got, ref)
