"""The arithmetic of gfx950's matrix instructions that the attention kernels use,
measured (tests/mfma_probe.hip) and compared with exact dot products and with
the model in tests/mfma_model.py.

The paper's kernel paragraph (Method) notes that FP8 tensor cores of earlier
GPU generations accumulate in reduced precision.  gfx950's FP8 MFMA does too:
it truncates products within groups of 8 (mfma_model).  Every tolerance of the
FP8 parity checks rests on the model pinned here:
* the model is bit-exact on dot products of e4m3-quantized normal data (the
  kind the attention kernel sees) and within 2^-21 (sum |a b| + |C|) on
  full-range random codes, structured cancellations and large accumulators;
* the hardware's error never exceeds the model's bound
  7 * 2^-13 * sum_g 2^(max e_a) 2^(max e_b) + 2^-21 (sum |a b| + |C|), and an
  adversarial group reaches at least 90% of its first term -- more than
  2^-11 sum |a b| -- so no bound proportional to sum |a b| with that constant
  would hold;
* operands within a narrow exponent range give exact dot products;
* the bf16 MFMA errs by at most 2^-21 (sum |a b| + |C|).
"""
import ctypes
import os

import numpy as np
import pytest
import torch

import mfma_model as MM
from oracle.e4m3 import decode

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libmfma_probe.so")
FINITE = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
KINDS = {0: (64, 32), 1: (128, 16)}     # kind: (K products, R rows of a tile)


def probe():
    if not os.path.exists(LIB):
        raise RuntimeError("%s not built: run __graft_entry__.build()" % LIB)
    lib = ctypes.CDLL(LIB)
    lib.mfma_probe_run.restype = ctypes.c_int
    lib.mfma_probe_run.argtypes = [ctypes.c_int] + [ctypes.c_void_p] * 4 + [ctypes.c_int]
    return lib


def run(kind, A, Bt, C):
    """D = A B + C for every tile on the GPU (A (T,R,K), Bt (T,R,K), C (T,R,R))."""
    a, bt, c = (torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in (A, Bt, C))
    assert a.shape == bt.shape and c.shape == a.shape[:2] + (a.shape[1],)
    d = torch.empty_like(c)
    rc = probe().mfma_probe_run(kind, a.data_ptr(), bt.data_ptr(), c.data_ptr(), d.data_ptr(), a.shape[0])
    assert rc == 0, rc
    return d.cpu().numpy().astype(np.float64)


def enc(x):
    c = torch.tensor(np.asarray(x, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(decode(c), np.asarray(x, np.float64))
    return c


def prod(e, mant=1.0, sign=1.0):
    """(a, b) e4m3 values with a b = sign mant 2^e, or None."""
    for x in range(7 if mant * 256 > 448 else 8, (-9 if mant == 1.0 else -6) - 1, -1):
        if -9 <= e - x <= 8:
            return sign * mant * 2.0 ** x, 2.0 ** (e - x)
    return None


def families(K, seed):
    """Seeded dot-product experiments (a[K], b[K], c) by family (values, not codes)."""
    rng = np.random.default_rng(seed)
    out = {}
    zero = lambda: (np.zeros(K), np.zeros(K))
    ex = []
    for e in range(0, 35):            # one product 2^16 and one more, e binades below it
        for sign in (1.0, -1.0):
            for mant in (1.0, 1.5, 1.875):
                for _ in range(4):
                    a, b = zero()
                    k0, k1 = rng.choice(K, 2, replace=False)
                    a[k0], b[k0] = 256.0, 256.0
                    pr = prod(16 - e, mant, sign)
                    if pr is not None:
                        a[k1], b[k1] = pr
                    ex.append((a, b, 0.0))
    out["pair"] = ex
    ex = []
    for e in range(4, 30):            # 2^16 and n products of +-2^(16 - e)
        for n in (1, 3, 7, 15, 31, K - 1):
            a, b = zero()
            ks = rng.permutation(K)
            a[ks[0]], b[ks[0]] = 256.0, 256.0
            x, y = prod(16 - e)
            for t in range(n):
                a[ks[1 + t]], b[ks[1 + t]] = x * rng.choice([-1.0, 1.0]), y
            ex.append((a, b, 0.0))
    out["many"] = ex
    ex = []
    for p in (-10, 0, 16):            # a product and accumulators of many magnitudes
        for cexp in range(-30, 40, 6):
            for sign in (1.0, -1.0):
                a, b = zero()
                k0 = rng.integers(K)
                a[k0], b[k0] = prod(p)
                ex.append((a, b, float(np.float32(sign * 2.0 ** cexp * (1 + 3 * 2.0 ** -22)))))
    out["accum"] = ex
    ex = []
    for e in range(8, 26):            # adversarial: 2^16 and 7 same-sign products just below 2^(16 - e) in its group
        for g0 in (0, K // 2 - 8, K - 8):
            a, b = zero()
            a[g0], b[g0] = 256.0, 256.0
            for t in range(1, 8):
                a[g0 + t], b[g0 + t] = prod(16 - e - 1, 1.875)
            ex.append((a, b, 0.0))
    out["adversarial"] = ex
    ex = []
    for i in range(1024):            # random full-range codes; every other one with a random C
        a, b = decode(rng.choice(FINITE, K)), decode(rng.choice(FINITE, K))
        c = float(np.float32(rng.choice([-1, 1]) * abs(np.dot(a, b)) * 2.0 ** rng.uniform(-30, 30))) if i % 2 else 0.0
        ex.append((a, b, c))
    out["random_full"] = ex
    ex = []
    for i in range(1024):            # e4m3 of N(0,1) rows scaled to amax 448, one outlier channel every third
        a, b = rng.standard_normal(K) * rng.uniform(0.5, 4), rng.standard_normal(K) * rng.uniform(0.5, 4)
        if i % 3 == 0:
            ch = rng.integers(K)
            a[ch] *= 20
            b[ch] *= 20
        a, b = a / np.abs(a).max() * 448, b / np.abs(b).max() * 448
        cast = lambda v: decode(torch.tensor(v.astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy())
        ex.append((cast(a), cast(b), 0.0))
    out["quantized_normal"] = ex
    ex = []
    for i in range(256):             # magnitudes in [224, 448]
        draw = lambda: rng.integers(0x70, 0x7F, K).astype(np.uint8) | (rng.integers(0, 2, K).astype(np.uint8) << 7)
        ex.append((decode(draw()), decode(draw()), 0.0))
    out["narrow"] = ex
    return out


def pack(exps, K, R):
    """Experiments on the diagonals of tiles (off-diagonal C = 0): codes A, Bt and C."""
    T = (len(exps) + R - 1) // R
    A = np.zeros((T, R, K), np.uint8)
    Bt = np.zeros((T, R, K), np.uint8)
    C = np.zeros((T, R, R), np.float32)
    for n, (a, b, c) in enumerate(exps):
        t, i = divmod(n, R)
        A[t, i], Bt[t, i], C[t, i, i] = enc(a), enc(b), c
    return A, Bt, C


@pytest.fixture(scope="module", params=[0, 1], ids=["32x32x64", "16x16x128"])
def measured(request):
    kind = request.param
    K, R = KINDS[kind]
    res = {}
    for name, exps in families(K, 70 + kind).items():
        A, Bt, C = pack(exps, K, R)
        d = run(kind, A, Bt, C)
        # every output of every tile is a dot product (the off-diagonal ones mix experiments)
        a = np.broadcast_to(A[:, :, None, :], A.shape[:2] + (R, K)).reshape(-1, K)
        b = np.broadcast_to(Bt[:, None, :, :], A.shape[:2] + (R, K)).reshape(-1, K)
        res[name] = (a, b, C.reshape(-1).astype(np.float64), d.reshape(-1))
    return kind, res


def test_model_matches_the_hardware(measured):
    kind, res = measured
    for name, (a, b, c, d) in res.items():
        model = MM.mfma_dot(torch.from_numpy(a), torch.from_numpy(b), torch.from_numpy(c)).numpy()
        p = decode(a) * decode(b)
        scale = np.abs(p).sum(axis=1) + np.abs(c)
        assert np.all(np.abs(d - model) <= MM.ACC_REL * scale), (kind, name, float((np.abs(d - model) / scale).max()))
        frac = np.mean(d == model)
        print(kind, name, "bit-exact fraction %.4f" % frac)
        if name in ("quantized_normal", "narrow"):
            assert frac == 1.0, (kind, name, frac)
        else:
            assert frac >= 0.85, (kind, name, frac)


def test_error_bound_holds_and_is_tight(measured):
    kind, res = measured
    for name, (a, b, c, d) in res.items():
        va, vb = decode(a), decode(b)
        p = va * vb
        exact = p.sum(axis=1) + c          # exact in fp64: e4m3 products, at most 2^25 apart, plus one fp32 value
        n, K = a.shape
        group = MM.GROUP_REL * (MM.group_max_exp2(a) * MM.group_max_exp2(b)).sum(axis=1)
        bound = group + MM.ACC_REL * (np.abs(p).sum(axis=1) + np.abs(c))
        err = np.abs(d - exact)
        assert np.all(err <= bound), (kind, name, float((err / bound).max()))
        if name == "narrow":
            assert np.array_equal(d, exact), (kind, "narrow range not exact")
        if name == "adversarial":
            R = KINDS[kind][1]                               # the tile diagonals: the constructed experiments
            idx = (np.arange(n // (R * R))[:, None] * R * R + np.arange(R)[None, :] * (R + 1)).ravel()
            idx = idx[np.abs(p[idx]).sum(axis=1) > 0]
            assert (err[idx] / group[idx]).max() >= 0.9, (err[idx] / group[idx]).max()
            assert (err[idx] / (2.0 ** -11 * np.abs(p[idx]).sum(axis=1))).max() > 1.5


def test_bf16_mfma_accumulates_in_fp32():
    rng = np.random.default_rng(72)
    T = 64
    a = (rng.standard_normal((T, 32, 16)) * 2.0 ** rng.uniform(-8, 8, (T, 32, 16))).astype(np.float32)
    b = (rng.standard_normal((T, 32, 16)) * 2.0 ** rng.uniform(-8, 8, (T, 32, 16))).astype(np.float32)
    A = torch.from_numpy(a).to(torch.bfloat16)
    Bt = torch.from_numpy(b).to(torch.bfloat16)
    C = np.zeros((T, 32, 32), np.float32)
    C[T // 2:] = (rng.standard_normal((T - T // 2, 32, 32)) * 2.0 ** rng.uniform(-4, 12, (T - T // 2, 32, 32)))
    d = run(2, A.view(torch.int16).numpy(), Bt.view(torch.int16).numpy(), C)
    av, bv = A.double().numpy(), Bt.double().numpy()
    exact = np.einsum("tik,tjk->tij", av, bv) + C     # bf16 products are exact in fp64; 16 terms, error ~2^-50
    scale = np.einsum("tik,tjk->tij", np.abs(av), np.abs(bv)) + np.abs(C)
    assert np.all(np.abs(d - exact) <= 2.0 ** -21 * scale), float((np.abs(d - exact) / scale).max())
