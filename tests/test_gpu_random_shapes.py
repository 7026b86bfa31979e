"""Seeded random shapes, dtypes and options through the fused FP8 path.

Each case draws B, H, D, N, M, the input dtype, the query-scale mode and the
grouped test K/V heads from a fixed generator, with inputs drawn like the
workloads (per-head multipliers, outlier channels).  The codes and scales must
equal the oracle's quantizer (Eq. (2)) bit for bit, and every output row must
be within T1hw of the oracle's one-pass replay on the FP8 MFMA's dot products
and within T2' of Eq. (1) on the dequantized inputs (tests/parity.py)."""
import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import quantize as OQ
from paper_2609_13031_amd import tfm
from paper_2609_13031_amd.workloads import Workload, generate
from parity import check_fp8_call, gpu_inputs, sample_rows

pytestmark = pytest.mark.gpu
MODES = ("shared", "per_call", "joint")


def draw_cases(n, seed):
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        H = int(rng.integers(1, 10))
        divisors = [g for g in range(1, H + 1) if H % g == 0]
        cases.append(dict(B=int(rng.integers(1, 4)), H=H, D=int(rng.choice([64, 128])),
                          N=int(rng.integers(1, 700)), M=0 if rng.random() < 0.25 else int(rng.integers(1, 300)),
                          dtype=str(rng.choice(["f32", "bf16"])), mode=str(rng.choice(MODES)),
                          G=int(rng.choice(divisors)), seed=1000 + i))
    return cases


@pytest.mark.parametrize("case", draw_cases(40, 80), ids=lambda c: "B%(B)dH%(H)dD%(D)dN%(N)dM%(M)d-%(dtype)s-%(mode)s-G%(G)d" % c)
def test_random_case(case):
    c = case
    w = Workload("random", B=c["B"], H=c["H"], D=c["D"], N=c["N"], M=c["M"], dtype=c["dtype"], seed=c["seed"])
    x = generate(w)
    tdt = torch.float32 if c["dtype"] == "f32" else torch.bfloat16
    g = gpu_inputs(x, tdt)
    q_test = g["q_test"] if c["M"] else None
    q = tfm.tfm_quantize_qkv_per_head(g["q_train"], g["k"], g["v"], q_test, q_scale_mode=c["mode"])
    o_tr, o_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], q_test, alpha=w.alpha,
                                           q_scale_mode=c["mode"], test_kv_heads=c["G"])
    torch.cuda.synchronize()
    ref = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"] if c["M"] else None,
                                   q_scale_mode=c["mode"])
    keys = ["q8_train", "k8", "v8", "s_q", "s_k", "s_v", "s_q_test"] + (["q8_test"] if c["M"] else [])
    for k in keys:
        assert np.array_equal(q[k].cpu().numpy(), ref[k]), (c, k)
    o_tr, o_te = o_tr.cpu().numpy(), o_te.cpu().numpy()
    check_fp8_call((o_tr, o_te), ref, w.alpha, None, None if c["M"] else [], test_kv_heads=c["G"],
                   block_kv=tfm.tfm_icl_attention_fp8_block_kv(w.D), what=c)


def draw_sharp_cases(n, seed):
    """Sharp heads: multipliers up to 8 on every tensor and 50x outlier channels (most key blocks
    of a row then round to e4m3 zero and are skipped), up to 3000 train rows."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        H = int(rng.integers(1, 7))
        divisors = [g for g in range(1, H + 1) if H % g == 0]
        cases.append(dict(B=int(rng.integers(1, 3)), H=H, D=int(rng.choice([64, 128])), N=int(rng.integers(100, 3000)),
                          M=0 if rng.random() < 0.25 else int(rng.integers(1, 400)),
                          dtype=str(rng.choice(["f32", "bf16"])), mode=str(rng.choice(MODES)),
                          G=int(rng.choice(divisors)), seed=3000 + i))
    return cases


@pytest.mark.parametrize("case", draw_sharp_cases(12, 82), ids=lambda c: "B%(B)dH%(H)dD%(D)dN%(N)dM%(M)d-%(dtype)s-%(mode)s-G%(G)d" % c)
def test_random_sharp_case(case):
    c = case
    w = Workload("sharp", B=c["B"], H=c["H"], D=c["D"], N=c["N"], M=c["M"], dtype=c["dtype"], seed=c["seed"],
                 mult_lo=0.25, mult_hi=8.0, outlier_frac=0.005, outlier_factor=50.0)
    x = generate(w)
    g = gpu_inputs(x, torch.float32 if c["dtype"] == "f32" else torch.bfloat16)
    q_test = g["q_test"] if c["M"] else None
    o_tr, o_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], q_test, alpha=w.alpha,
                                           q_scale_mode=c["mode"], test_kv_heads=c["G"])
    ref = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"] if c["M"] else None,
                                   q_scale_mode=c["mode"])
    check_fp8_call((o_tr.cpu().numpy(), o_te.cpu().numpy()), ref, w.alpha, None, None if c["M"] else [],
                   test_kv_heads=c["G"], block_kv=tfm.tfm_icl_attention_fp8_block_kv(w.D), what=c)


def draw_wide_cases(n, seed):
    """Head dimension 128, at least 65536 train rows and grids of at least 256 workgroups of
    256 rows (the 8-wave kernel)."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        c = dict(B=int(rng.integers(1, 3)), H=int(rng.choice([1, 2])), D=128, N=int(rng.integers(65536, 67000)),
                 M=int(rng.integers(0, 700)), dtype=str(rng.choice(["f32", "bf16"])), mode=str(rng.choice(MODES)),
                 seed=2000 + len(cases))
        if c["B"] * c["H"] * (-(-c["N"] // 256) + -(-c["M"] // 256)) >= 256:
            cases.append(c)
    return cases


@pytest.mark.parametrize("case", draw_wide_cases(6, 81), ids=lambda c: "B%(B)dH%(H)dN%(N)dM%(M)d-%(dtype)s-%(mode)s" % c)
def test_random_wide_d128_case(case):
    c = case
    w = Workload("random", B=c["B"], H=c["H"], D=c["D"], N=c["N"], M=c["M"], dtype=c["dtype"], seed=c["seed"])
    x = generate(w)
    g = gpu_inputs(x, torch.float32 if c["dtype"] == "f32" else torch.bfloat16)
    q_test = g["q_test"] if c["M"] else None
    o_tr, o_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], q_test, alpha=w.alpha, q_scale_mode=c["mode"])
    o_tr, o_te = o_tr.cpu().numpy(), o_te.cpu().numpy()
    ref = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"] if c["M"] else None,
                                   q_scale_mode=c["mode"])
    rt = sample_rows(w.N, 128, c["seed"])
    re = sample_rows(w.M, 48, c["seed"] + 1) if c["M"] else np.zeros(0, np.int64)
    check_fp8_call((o_tr, o_te), ref, w.alpha, rt, re, block_kv=tfm.tfm_icl_attention_fp8_block_kv(w.D), what=c)
