"""GPU parity of the ICL-call options with the oracle: the query-scale modes
(Sec. 3 and Table 1: shared train-query scale, per-call test scale; the
appendix's single-call joint scale) and grouped-query test rows over the
first K/V heads (appendix, TabPFN-v3's test-train call)."""
import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import quantize as OQ
from paper_2609_13031_amd import tfm
from paper_2609_13031_amd.workloads import Workload, generate
from parity import TIE_REL, assert_t1, check_fp8_call, gpu_inputs, narrow_range_inputs, sample_rows

pytestmark = pytest.mark.gpu
BKV = 128
MODES = ("shared", "per_call", "joint")
CODE_KEYS = ("q8_train", "k8", "v8", "q8_test")
SCALE_KEYS = ("s_q", "s_k", "s_v", "s_q_test")


def skewed_inputs(w, seed):
    """Workload inputs whose test queries are scaled per head by 1/16 ... 4, so the test
    absmax is below the train absmax on some heads and above it on others."""
    x = generate(w)
    mult = np.random.default_rng(seed).choice(np.array([0.0625, 0.5, 1.0, 2.0, 4.0], np.float32), size=w.H)
    x["q_test"] = (x["q_test"] * mult[None, None, :, None]).astype(np.float32)
    return x


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_quantize_modes_bit_exact(mode, dtype):
    w = Workload("modes", B=2, H=5, D=64, N=700, M=300, dtype=dtype, seed=41)
    x = skewed_inputs(w, 42)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    g = gpu_inputs(x, tdt)
    got = tfm.tfm_quantize_qkv_per_head(g["q_train"], g["k"], g["v"], g["q_test"], q_scale_mode=mode)
    xr = {k: torch.from_numpy(v).to(tdt).float().numpy() for k, v in x.items()}
    ref = OQ.quantize_qkv_per_head(xr["q_train"], xr["k"], xr["v"], xr["q_test"], q_scale_mode=mode)
    for k in CODE_KEYS + SCALE_KEYS:
        assert np.array_equal(got[k].cpu().numpy(), ref[k]), (mode, k)
    # the modes differ where they should
    if mode != "shared":
        assert not np.array_equal(ref["s_q_test"], OQ.quantize_qkv_per_head(xr["q_train"], xr["k"], xr["v"],
                                                                              xr["q_test"])["s_q_test"])


@pytest.mark.parametrize("mode", MODES)
def test_quantize_modes_without_test_rows(mode):
    w = Workload("modes0", B=1, H=3, D=128, N=333, M=0, dtype="bf16", seed=43)
    x = generate(w)
    g = gpu_inputs(x, torch.bfloat16)
    got = tfm.tfm_quantize_qkv_per_head(g["q_train"], g["k"], g["v"], None, q_scale_mode=mode)
    xr = {k: torch.from_numpy(v).to(torch.bfloat16).float().numpy() for k, v in x.items()}
    ref = OQ.quantize_qkv_per_head(xr["q_train"], xr["k"], xr["v"], None, q_scale_mode=mode)
    for k in ("q8_train", "k8", "v8") + SCALE_KEYS:
        assert np.array_equal(got[k].cpu().numpy(), ref[k]), (mode, k)
    assert got["q8_test"].shape == (1, 3, 0, 128)


def fp8_out(g, alpha, **opts):
    o = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=alpha, **opts)
    torch.cuda.synchronize()
    return o[0].cpu().numpy(), o[1].cpu().numpy()


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("G", [0, 1, 2])
def test_fp8_attention_modes_and_grouped_test_heads(mode, G):
    w = Workload("opts", B=2, H=4, D=64, N=1500, M=400, dtype="bf16", seed=44 + G)
    x = skewed_inputs(w, 45)
    g = gpu_inputs(x, torch.bfloat16)
    o_tr, o_te = fp8_out(g, w.alpha, q_scale_mode=mode, test_kv_heads=G)
    xr = {k: torch.from_numpy(v).to(torch.bfloat16).float().numpy() for k, v in x.items()}
    qz = OQ.quantize_qkv_per_head(xr["q_train"], xr["k"], xr["v"], xr["q_test"], q_scale_mode=mode)
    rt, re = sample_rows(w.N, 96, 46), sample_rows(w.M, 64, 47)
    check_fp8_call((o_tr, o_te), qz, w.alpha, rt, re, test_kv_heads=G or None, block_kv=BKV, what=(mode, G))
    # the split entry points and the prequantized one compute the same thing
    ws = tfm.tfm_icl_attention_fp8_quantize(g["q_train"], g["k"], g["v"], g["q_test"], q_scale_mode=mode)
    a_tr, a_te = tfm.tfm_icl_attention_fp8_attend(ws, w.B, w.H, w.D, w.N, w.M, alpha=w.alpha, test_kv_heads=G)
    assert np.array_equal(a_tr.cpu().numpy(), o_tr) and np.array_equal(a_te.cpu().numpy(), o_te)
    q = tfm.tfm_quantize_qkv_per_head(g["q_train"], g["k"], g["v"], g["q_test"], q_scale_mode=mode)
    p_tr, p_te = tfm.tfm_icl_attention_fp8_prequantized(q["q8_train"], q["k8"], q["v8"], q["q8_test"], q["s_q"],
                                                        q["s_k"], q["s_v"], alpha=w.alpha, s_q_test=q["s_q_test"],
                                                        test_kv_heads=G)
    assert np.array_equal(p_tr.cpu().numpy(), o_tr) and np.array_equal(p_te.cpu().numpy(), o_te)


@pytest.mark.parametrize("mode,G,test_mult", [("per_call", 0, 0.25), ("joint", 2, 1.0), ("shared", 1, 1.0)])
def test_exact_mfma_regime_with_options(mode, G, test_mult):
    # Narrow-range codes keep every FP8 MFMA dot product exact: T1 against O_qp.  Under
    # "per_call" the test queries, 4x smaller, still map to codes in [224, 448] on their own scale.
    B, H, D, N, M = 1, 4, 64, 600, 200
    x = narrow_range_inputs(B, N, M, H, D, seed=48)
    x["q_test"] *= np.float32(test_mult)
    g = gpu_inputs(x, torch.float32)
    alpha = np.float32(0.025)
    o_tr, o_te = fp8_out(g, float(alpha), q_scale_mode=mode, test_kv_heads=G)
    qz = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"], q_scale_mode=mode)
    (r_tr, a_tr), (r_te, a_te) = OA.icl_attention_fp8_kernel_model(qz, alpha, BKV, tie_rel=TIE_REL,
                                                                    test_kv_heads=G or None)
    for h in range(H):
        assert_t1(o_tr[0, :, h], r_tr[0, :, h], a_tr[0, :, h], ("train", mode, G, h))
        assert_t1(o_te[0, :, h], r_te[0, :, h], a_te[0, :, h], ("test", mode, G, h))


@pytest.mark.parametrize("G", [1, 2])
def test_grouped_test_heads_equal_physically_repeated_kv_heads(G):
    # Test rows of head h over K/V head h // (H/G) must be bit-identical to a call whose K/V
    # heads are repeated in memory (same codes, same scales, same arithmetic); the train
    # rows must be those of the ungrouped call.
    w = Workload("gqa", B=1, H=4, D=128, N=900, M=250, dtype="bf16", seed=49)
    x = generate(w)
    g = gpu_inputs(x, torch.bfloat16)
    idx = torch.tensor([h // (w.H // G) for h in range(w.H)], device="cuda")
    g_rep = dict(g, k=g["k"][:, :, idx].contiguous(), v=g["v"][:, :, idx].contiguous())
    for fn in (tfm.tfm_icl_attention_fp8, tfm.tfm_icl_attention_bf16):
        a_tr, a_te = fn(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha, test_kv_heads=G)
        b_tr, _ = fn(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
        _, c_te = fn(g_rep["q_train"], g_rep["k"], g_rep["v"], g_rep["q_test"], alpha=w.alpha)
        assert torch.equal(a_tr, b_tr), fn.__name__
        assert torch.equal(a_te, c_te), fn.__name__
        assert not torch.equal(a_te[:, :, -1], fn(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)[1][:, :, -1])


@pytest.mark.parametrize("N,expect_fp8", [(8192, False), (8193, True)])
def test_gate_passes_the_options_to_either_path(N, expect_fp8):
    w = Workload("gate_opts", B=1, H=2, D=64, N=N, M=40, dtype="bf16", seed=50)
    x = skewed_inputs(w, 51)
    g = gpu_inputs(x, torch.bfloat16)
    opts = dict(q_scale_mode="per_call", test_kv_heads=1)
    o_tr, o_te, used = tfm.tfm_icl_attention(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha, **opts)
    assert used == expect_fp8
    if expect_fp8:
        d = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha, **opts)
    else:
        d = tfm.tfm_icl_attention_bf16(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha, test_kv_heads=1)
    assert torch.equal(o_tr, d[0]) and torch.equal(o_te, d[1])


@pytest.mark.parametrize("mode", MODES)
def test_many_heads_and_row_slices(mode):
    # 34 heads: the quantize kernels take at most 32 heads per block, so every row splits
    # over two blocks; 1300 train rows: the amax pass keeps 82 slice maxima of 16 rows per
    # head, the last slice ragged.  Codes and scales bit-exact (Eq. (2)); the fused quantize
    # path (V into the kernel's tile layout, scales reduced inside the quantize launch)
    # bitwise equal to attention on the public codes; both within T1hw and T2' of the oracle.
    w = Workload("wide", B=2, H=34, D=64, N=1300, M=300, dtype="bf16", seed=52)
    x = skewed_inputs(w, 53)
    g = gpu_inputs(x, torch.bfloat16)
    xr = {k: torch.from_numpy(v).to(torch.bfloat16).float().numpy() for k, v in x.items()}
    ref = OQ.quantize_qkv_per_head(xr["q_train"], xr["k"], xr["v"], xr["q_test"], q_scale_mode=mode)
    q = tfm.tfm_quantize_qkv_per_head(g["q_train"], g["k"], g["v"], g["q_test"], q_scale_mode=mode)
    for k in CODE_KEYS + SCALE_KEYS:
        assert np.array_equal(q[k].cpu().numpy(), ref[k]), (mode, k)
    ws = tfm.tfm_icl_attention_fp8_quantize(g["q_train"], g["k"], g["v"], g["q_test"], q_scale_mode=mode)
    a_tr, a_te = tfm.tfm_icl_attention_fp8_attend(ws, w.B, w.H, w.D, w.N, w.M, alpha=w.alpha)
    p_tr, p_te = tfm.tfm_icl_attention_fp8_prequantized(q["q8_train"], q["k8"], q["v8"], q["q8_test"], q["s_q"],
                                                        q["s_k"], q["s_v"], alpha=w.alpha, s_q_test=q["s_q_test"])
    assert torch.equal(a_tr, p_tr) and torch.equal(a_te, p_te), mode
    rt, re = sample_rows(w.N, 32, 54), sample_rows(w.M, 16, 55)
    heads = [0, 31, 32, 33]     # both sides of the head-group boundary
    check_fp8_call((a_tr.cpu().numpy(), a_te.cpu().numpy()), ref, w.alpha, rt, re, block_kv=BKV, what=mode,
                   heads=heads)
