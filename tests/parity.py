"""Shared helpers of the GPU parity tests: device transfer, row sampling and
the stated tolerances (T1 against the oracle's kernel model O_qp, T2 against
Eq. (1) on the dequantized inputs O_q)."""
import numpy as np
import torch

from oracle import attention as OA
from oracle.e4m3 import decode

# T1 -- FP8 path vs O_qp (the one-pass kernel replayed in fp64), elementwise:
#   |dO| <= 1.01 * tie allowance + 1e-5 * RMS(O_qp) + 1e-6 * |O_qp|.
# It applies where every FP8 MFMA dot product is exact (inputs whose codes
# span a narrow range, see ``narrow_range_inputs``): the kernel then differs
# from O_qp by fp32 arithmetic only.  Its exponent c*S + 8 - c*m is off by at
# most ~1e-6 (fp32 c: 3 roundings of |c S| <= 1; fp32 bias and fma: 2^-21
# each near 8), and v_exp_f32 adds < 1 ulp, so P~ moves by < 1e-6 relative:
# a key can round to the other e4m3 neighbour only if O_qp's P~ lies within
# TIE_REL (4x margin) of a rounding midpoint; the oracle's tie allowance
# bounds the effect of all such keys.  Everything else is fp32 noise.
TIE_REL = 2.0 ** -18
T1_MAX, T1_RELF, T1_OUTLIER, T1_OUTLIER_FRAC = 1e-2, 1e-4, 2e-3, 1e-3   # reported only

# The FP8 MFMA of gfx950 (v_mfma_f32_*_f8f6f4) does not round its dot product
# exactly: products are aligned to the largest one and truncated, so a 64-term
# dot product can be off by up to ~2.3e-4 of sum |a_k b_k| (measured with
# random full-range e4m3 operands; a narrow exponent range is exact), and each
# accumulation into C loses about one fp32 ulp (truncation).  EPS_DOT bounds
# the first with a 2x margin, EPS_ACC the second per key tile.
EPS_DOT = 2.0 ** -11
EPS_ACC = 2.0 ** -22
# T1' -- on general inputs the FP8 path stays within relF 2e-2 of O_qp (a
# dropped key tile or a missing rescale gives 0.17 and more), on heads whose
# logits the dot-product error above can move by at most T1P_MAX_LOGIT_ERR
# log2 units: delta = c * EPS_DOT * max_ij sum_k |q_ik k_jk|, from the codes.
# Typical heads of the workloads have delta ~0.1.  Over 160 seeded random
# cases (B <= 4, H <= 9, N up to 6000, multipliers up to 8, outliers up to 50x)
# the worst such head per case had median relF 1e-3, 90th percentile 4e-3 and
# maximum 1.07e-2, from rows whose two leading keys are within delta.  Where
# the outlier channels of Q and K coincide, sum |q_k k_k| reaches 1e5 and more
# and delta 1 to 7 log2 units, on rows whose logits span hundreds or
# thousands: two leading keys closer than delta may then swap which dominates,
# such a row's output moves by up to a few RMS (relF 1e-2 to 4e-2 measured),
# and only the elementwise T2', which bounds exactly that error, is a test;
# it is then required on every checked row instead.  An emulation that
# truncates the products to 15 bits of the largest moves O_qp by the same
# amounts on such heads.
# relF is a statistic of the rows checked: with few of them a single row whose
# leading keys are within delta dominates it (relF 2e-2 from one of 12 test
# rows in one case), so T1' also needs at least T1P_MIN_ROWS rows.
T1P_RELF = 2e-2
T1P_MAX_LOGIT_ERR = 0.25
T1P_MIN_ROWS = 32


def t1_metrics(got, ref):
    d = np.abs(np.asarray(got, np.float64) - ref)
    rms = np.sqrt(np.mean(ref ** 2))
    return {"max_over_rms": d.max() / rms,
            "relF": np.linalg.norm(d) / np.linalg.norm(ref),
            "outlier_frac": np.mean(d > T1_OUTLIER * rms)}


def assert_t1(got, ref, allowance, what=""):
    got = np.asarray(got, np.float64)
    rms = np.sqrt(np.mean(ref ** 2))
    err = np.abs(got - ref)
    tol = 1.01 * allowance + 1e-5 * rms + 1e-6 * np.abs(ref)
    assert np.all(err <= tol), (what, (err / tol).max(), t1_metrics(got, ref))
    return t1_metrics(got, ref)


def _abs_dev_sums(v, o):
    """out[r, c] = sum_j |v[j, c] - o[r, c]|, from each channel's sorted values and prefix sums."""
    N = v.shape[0]
    vs = np.sort(np.ascontiguousarray(v.T), axis=1)      # (D, N): each channel's values in order
    cs = np.empty((vs.shape[0], N + 1))
    cs[:, 0] = 0.0
    np.cumsum(vs, axis=1, out=cs[:, 1:])
    out = np.empty_like(o)
    for ch in range(vs.shape[0]):
        t = o[:, ch]
        k = np.searchsorted(vs[ch], t)
        out[:, ch] = t * k - cs[ch, k] + (cs[ch, N] - cs[ch, k]) - t * (N - k)
    return out


def _weighted_abs_dev(A, z, v, o):
    """An upper bound of sum_j (A_rj + z_r) |v_jc - o_rc| (A >= 0, z >= 0), equal to it
    up to 1e-9 relative.  The z part is summed over all keys with _abs_dev_sums; the A part
    only over keys with A_rj >= 1e-16 max_j A_rj, and the rest of its mass is counted
    at max_j |v_jc - o_rc|, so dropping them can only raise the result."""
    num = z[:, None] * _abs_dev_sums(v, o)
    vmax, vmin = v.max(axis=0), v.min(axis=0)
    N = v.shape[0]
    for r in range(A.shape[0]):
        keep = np.nonzero(A[r] >= 1e-16 * A[r].max())[0]
        if len(keep) > N // 4:   # most keys count: sum over all of them, in cache-sized pieces
            for j0 in range(0, N, 8192):
                num[r] += A[r, j0:j0 + 8192] @ np.abs(v[j0:j0 + 8192] - o[r])
        else:
            num[r] += A[r, keep] @ np.abs(v[keep] - o[r])
            num[r] += (A[r].sum() - A[r, keep].sum()) * np.maximum(vmax - o[r], o[r] - vmin)
    return num * (1 + 1e-9)


def p_rounding_bound(q8, k8, v_hat, c, eps_dot=0.0, n_tiles=0):
    """Elementwise bound on |O - O_q| for the one-pass FP8 kernel (rows of q8).

    With p_j = 2^(c (s_j - max s) + 8) the exact lifted weights, a weight the
    kernel uses is w_j = g * p_j * 2^(c d_j) (1 + r_j) + z_j: g a factor common
    to the row (it cancels), |d_j| <= eps_dot * sum_k |q_k k_jk| the error of
    the QK^T dot product, |r_j| <= 2^-4 (half an e4m3 ulp, normal range) and
    |z_j| <= 2^-10 (half the subnormal step; rescaling by 2^(c(m_old-m)) <= 1
    only shrinks it).  Then O - O_q = sum_j (w_j/g - p_j)(v_j - O_q) / sum_j w_j/g.
    The PV and row-sum dot products add eps_dot of sum_j p_j |v_j| / sum p
    each, and n_tiles accumulations into C add EPS_ACC per tile of the same.
    With eps_dot = 0 and n_tiles = 0 this is the bound of O_qp itself.
    """
    s = q8 @ k8.T
    p = np.exp2(c * (s - s.max(axis=1, keepdims=True)) + 8.0)
    psum = p.sum(axis=1)
    o = (p @ v_hat) / psum[:, None]
    a = np.abs(q8) @ np.abs(k8).T
    # e_rj = A_rj + z_r: the weight term and the subnormal term, the same for every key
    A = p * ((1 + 2.0 ** -4) * np.exp2(c * eps_dot * a) - 1)
    z = 2.0 ** -10 * np.exp2(c * eps_dot * a.max(axis=1))
    num = _weighted_abs_dev(A, z, v_hat, o)
    den = psum - (A.sum(axis=1) + z * k8.shape[0])
    bound = np.where(den[:, None] > 0, num / np.where(den > 0, den, 1.0)[:, None], np.inf)
    pv = (p @ np.abs(v_hat)) / psum[:, None]
    bound += (2 * eps_dot + n_tiles * EPS_ACC) * (pv + np.abs(o))
    return o, bound


def assert_t2(got, qz, alpha, b, h, q8_rows, slack=1.25, eps_dot=EPS_DOT, s_query=None, hk=None):
    """T2': |O_gpu - O_q| <= 1.25 * p_rounding_bound(eps_dot) + 1e-5 * RMS, elementwise.

    The query rows q8_rows have scale s_query (default s_q of head h) and attend to K/V
    head hk (default h)."""
    hk = h if hk is None else hk
    s_query = qz["s_q"][b, h] if s_query is None else s_query
    c = float(alpha) * float(s_query) * float(qz["s_k"][b, hk]) * OA.LOG2E
    k8 = decode(qz["k8"][b, hk])
    v_hat = decode(qz["v8"][b, hk]) * float(qz["s_v"][b, hk])
    n_tiles = (k8.shape[0] + 63) // 64
    o, bnd = p_rounding_bound(decode(q8_rows), k8, v_hat, c, eps_dot, n_tiles)
    rms = np.sqrt(np.mean(o ** 2))
    err = np.abs(np.asarray(got, np.float64) - o)
    assert np.all(err <= slack * bnd + 1e-5 * rms), (err / (bnd + 1e-30)).max()
    return err.max() / rms


def assert_t1p(got, ref, what=""):
    """T1': statistical agreement with O_qp on general inputs (relF only)."""
    m = t1_metrics(got, ref)
    assert m["relF"] <= T1P_RELF, (what, m)
    return m


def logit_error_scale(qz, alpha, b, h, q8_rows, s_query=None, hk=None, eps_dot=EPS_DOT):
    """delta = c * eps_dot * max over the rows and keys of sum_k |q_k k_k|: the most the FP8
    dot-product error can move a base-2 logit of these rows (log2 units)."""
    hk = h if hk is None else hk
    s_query = qz["s_q"][b, h] if s_query is None else s_query
    c = float(alpha) * float(s_query) * float(qz["s_k"][b, hk]) * OA.LOG2E
    a = np.abs(decode(q8_rows)) @ np.abs(decode(qz["k8"][b, hk])).T
    return c * eps_dot * float(a.max()) if a.size else 0.0


def assert_t1p_or_t2(got, ref, qz, alpha, b, h, q8_rows, s_query=None, hk=None, what="", t2_max_rows=None):
    """T1' against O_qp where the FP8 dot-product error moves logits by at most
    T1P_MAX_LOGIT_ERR and at least T1P_MIN_ROWS rows are checked; otherwise T2'
    against O_q on every row passed, or on t2_max_rows of them evenly spaced (the
    bound costs rows * N * D, too much at 262144 keys for every sampled row).
    Returns the metrics against O_qp and whether T1' applied."""
    delta = logit_error_scale(qz, alpha, b, h, q8_rows, s_query, hk)
    if delta <= T1P_MAX_LOGIT_ERR and len(q8_rows) >= T1P_MIN_ROWS:
        return assert_t1p(got, ref, what), True
    idx = np.arange(len(q8_rows))
    if t2_max_rows is not None and len(idx) > t2_max_rows:
        idx = np.unique(np.linspace(0, len(idx) - 1, t2_max_rows).astype(np.int64))
    assert_t2(np.asarray(got)[idx], qz, alpha, b, h, np.asarray(q8_rows)[idx], s_query=s_query, hk=hk)
    return t1_metrics(got, ref), False


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
