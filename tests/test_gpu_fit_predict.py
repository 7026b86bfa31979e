"""GPU tests of the fit-once / predict-many split of the ICL calls: every
output is bit-for-bit the one tfm_icl_attention_fp8 gives for the same inputs
(that entry point is checked against the oracle elsewhere), test batches are
independent of each other under the shared train-query scale (Sec. 3), and the
per-call scale follows the oracle."""
import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import quantize as OQ
from paper_2609_13031_amd import tfm
from paper_2609_13031_amd.workloads import Workload, generate
from parity import check_fp8_call, gpu_inputs, sample_rows

pytestmark = pytest.mark.gpu
BKV = 128


@pytest.fixture(scope="module")
def table():
    w = Workload("fitpredict", B=2, H=4, D=64, N=3000, M=700, dtype="bf16", seed=61)
    x = generate(w)
    return w, x, gpu_inputs(x, torch.bfloat16)


@pytest.mark.parametrize("mode,G", [("shared", 0), ("per_call", 0), ("shared", 1), ("per_call", 2)])
def test_fit_then_predict_equals_the_fused_call(table, mode, G):
    w, x, g = table
    f_tr, f_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha,
                                           q_scale_mode=mode, test_kv_heads=G)
    o_tr, ws = tfm.tfm_icl_attention_fp8_fit(g["q_train"], g["k"], g["v"], alpha=w.alpha, m_max=w.M)
    o_te = tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"], w.N, alpha=w.alpha, q_scale_mode=mode,
                                             test_kv_heads=G)
    assert torch.equal(o_tr, f_tr)
    assert torch.equal(o_te, f_te)


def test_workgroup_width_at_d128_changes_no_bit():
    # At head dimension 128 the fused call here runs workgroups of 8 waves (65836 train rows,
    # and its grid still gives every compute unit one), while a 40-row predict batch runs
    # workgroups of 4: the rows they share must agree bit for bit.
    w = Workload("wide", B=1, H=2, D=128, N=65836, M=300, dtype="bf16", seed=63)
    g = gpu_inputs(generate(w), torch.bfloat16)
    f_tr, f_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
    o_tr, ws = tfm.tfm_icl_attention_fp8_fit(g["q_train"], g["k"], g["v"], alpha=w.alpha, m_max=w.M)
    part = tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"][:, 17:57].contiguous(), w.N, alpha=w.alpha)
    assert torch.equal(o_tr, f_tr)
    assert torch.equal(part, f_te[:, 17:57])


def test_predict_batches_are_independent_under_the_shared_scale(table):
    w, x, g = table
    _, ws = tfm.tfm_icl_attention_fp8_fit(g["q_train"], g["k"], g["v"], alpha=w.alpha, m_max=w.M)
    full = tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"], w.N, alpha=w.alpha)
    perm = torch.from_numpy(np.random.default_rng(62).permutation(w.M)[:257]).cuda()
    part = tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"][:, perm].contiguous(), w.N, alpha=w.alpha)
    assert torch.equal(part, full[:, perm])
    one = tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"][:, 5:6].contiguous(), w.N, alpha=w.alpha)
    assert torch.equal(one, full[:, 5:6])
    # switching modes on one fit state: a per-call predict leaves the shared one unchanged
    tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"][:, :100].contiguous(), w.N, alpha=w.alpha,
                                      q_scale_mode="per_call")
    again = tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"], w.N, alpha=w.alpha)
    assert torch.equal(again, full)
    # bf16 output is the rounded fp32 output
    h = tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"], w.N, alpha=w.alpha, out_dtype=torch.bfloat16)
    assert torch.equal(h, full.to(torch.bfloat16))


def test_per_call_predict_follows_the_oracle(table):
    w, x, g = table
    _, ws = tfm.tfm_icl_attention_fp8_fit(g["q_train"], g["k"], g["v"], alpha=w.alpha, m_max=w.M)
    rows = np.arange(0, 300)
    qt = np.ascontiguousarray(x["q_test"][:, rows]) * np.float32(0.25)   # a batch with its own, smaller absmax
    gq = torch.from_numpy(qt).to(torch.bfloat16).cuda()
    o_te = tfm.tfm_icl_attention_fp8_predict(ws, gq, w.N, alpha=w.alpha, q_scale_mode="per_call").cpu().numpy()
    xr = {k: torch.from_numpy(v).to(torch.bfloat16).float().numpy() for k, v in x.items()}
    qz = OQ.quantize_qkv_per_head(xr["q_train"], xr["k"], xr["v"], gq.float().cpu().numpy(), q_scale_mode="per_call")
    check_fp8_call((np.zeros((w.B, 0, w.H, w.D)), o_te), qz, w.alpha, [], None, block_kv=BKV, what="per_call")


@pytest.mark.parametrize("G", [0, 1])
def test_shared_fit_and_predict_follow_the_oracle(table, G):
    # fit's train rows and a later predict batch, on the shared train-query scale, against
    # the oracle directly (the fused call they equal is checked elsewhere too)
    w, x, g = table
    o_tr, ws = tfm.tfm_icl_attention_fp8_fit(g["q_train"], g["k"], g["v"], alpha=w.alpha, m_max=w.M)
    rows = np.arange(100, 400)
    o_te = tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"][:, rows].contiguous(), w.N, alpha=w.alpha,
                                             test_kv_heads=G)
    xr = {k: torch.from_numpy(v).to(torch.bfloat16).float().numpy() for k, v in x.items()}
    qz = OQ.quantize_qkv_per_head(xr["q_train"], xr["k"], xr["v"], xr["q_test"][:, rows])
    check_fp8_call((o_tr.cpu().numpy(), o_te.cpu().numpy()), qz, w.alpha, sample_rows(w.N, 128, 64), None,
                   test_kv_heads=G or None, block_kv=BKV, what=("fit/predict", G))


def test_fit_predict_edge_cases(table):
    w, x, g = table
    o_tr, ws = tfm.tfm_icl_attention_fp8_fit(g["q_train"], g["k"], g["v"], alpha=w.alpha, m_max=64)
    empty = tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"][:, :0].contiguous(), w.N, alpha=w.alpha)
    assert empty.shape == (w.B, 0, w.H, w.D)
    with pytest.raises(tfm.TfmError) as e:                 # 260 test rows need more than the m_max=64 workspace
        tfm.tfm_icl_attention_fp8_predict(ws, g["q_test"][:, :260].contiguous(), w.N, alpha=w.alpha)
    assert e.value.status == 6
    with pytest.raises(tfm.TfmError) as e:
        tfm.tfm_icl_attention_fp8_fit(g["q_train"], g["k"], g["v"], alpha=w.alpha, q_scale_mode="joint")
    assert e.value.status == 8
    # a fit with fp32 inputs gives the fused call's train rows too
    g32 = {k: v.float() for k, v in g.items()}
    f_tr, _ = tfm.tfm_icl_attention_fp8(g32["q_train"], g32["k"], g32["v"], None, alpha=w.alpha)
    o32, _ = tfm.tfm_icl_attention_fp8_fit(g32["q_train"], g32["k"], g32["v"], alpha=w.alpha)
    assert torch.equal(o32, f_tr)
