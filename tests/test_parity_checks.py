"""CPU checks of the parity tests' own machinery (tests/parity.py): the T2'
bound's O is the oracle's O_q, the bound holds for the oracle's replay of the
kernel on the FP8 MFMA model's scores, and the checks reject plausible
mistakes in an output (a dropped key tile, a wrong block size, a wrong V
scale, rows swapped)."""
import numpy as np
import pytest
import torch

import mfma_model as MM
import parity as P
from oracle import attention as OA
from oracle import quantize as OQ
from oracle.e4m3 import decode
from paper_2609_13031_amd.workloads import Workload, generate

CPU = torch.device("cpu")


@pytest.fixture(scope="module")
def head():
    w = Workload("chk", B=1, H=3, D=64, N=700, M=90, dtype="bf16", mult_hi=8.0, outlier_factor=50.0, seed=77)
    x = generate(w)
    qz = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])
    return w, qz


def replay(qz, alpha, b, h, rows, block_kv=128, keys=None, call="train"):
    key, s_q = ("q8_train", qz["s_q"]) if call == "train" else ("q8_test", qz["s_q_test"])
    k8, v8 = qz["k8"][b, h], qz["v8"][b, h]
    if keys is not None:
        k8, v8 = k8[keys], v8[keys]
    q8 = qz[key][b, h][rows]
    c = P.softmax_factor(alpha, s_q[b, h], qz["s_k"][b, h])
    sc = MM.scores(torch.from_numpy(q8), torch.from_numpy(k8)).numpy()
    return OA.one_pass_fp8_attention(decode(q8), decode(k8), decode(v8), c, qz["s_v"][b, h], block_kv, scores=sc)


def test_bound_is_the_oracle_o_q_and_covers_the_hardware_score_replay(head):
    w, qz = head
    rows = np.arange(0, w.N, 3)
    for h in range(w.H):
        c = P.softmax_factor(w.alpha, qz["s_q"][0, h], qz["s_k"][0, h])
        o, bnd = P.fp8_bound(qz["q8_train"][0, h][rows], qz["k8"][0, h], qz["v8"][0, h], qz["s_v"][0, h], c, CPU)
        o_q = P.oracle_o_q(qz, w.alpha, 0, h, rows)
        assert np.allclose(o, o_q, rtol=1e-9, atol=1e-9 * np.abs(o_q).max())
        err = np.abs(replay(qz, w.alpha, 0, h, rows) - o_q)
        assert np.all(err <= bnd), (h, float((err / bnd).max()))


def test_the_checks_accept_the_hardware_score_replay(head):
    w, qz = head
    rows = np.arange(0, w.N, 5)
    for h in range(w.H):
        m = P.check_fp8_rows(replay(qz, w.alpha, 0, h, rows), qz, w.alpha, 0, h, rows, device=CPU)
        assert m["vs_hw_replay"]["relF"] < 1e-12
    te = np.arange(w.M)
    P.check_fp8_rows(replay(qz, w.alpha, 0, 1, te, call="test"), qz, w.alpha, 0, 1, te, call="test", device=CPU)


@pytest.mark.parametrize("mistake", ["dropped_tile", "block_64", "v_scale", "swapped_rows", "exact_scores"])
def test_the_checks_reject_a_mistake(head, mistake):
    w, qz = head
    rows = np.arange(0, w.N, 5)
    h = 2
    got = {
        "dropped_tile": lambda: replay(qz, w.alpha, 0, h, rows, keys=np.arange(w.N - 64)),
        "block_64": lambda: replay(qz, w.alpha, 0, h, rows, block_kv=64),
        "v_scale": lambda: replay(qz, w.alpha, 0, h, rows) * 1.01,
        "swapped_rows": lambda: replay(qz, w.alpha, 0, h, rows)[np.r_[1, 0, 2:len(rows)]],
        # the exact-arithmetic replay differs from the kernel's through the truncated dot
        # products alone: on this head (outliers 50x) T1hw must tell them apart
        "exact_scores": lambda: OA.icl_attention_fp8_kernel_model(
            {k: v[:, h:h + 1] for k, v in qz.items()}, w.alpha, 128, rows, [])[0][0, :, 0],
    }[mistake]()
    with pytest.raises(AssertionError):
        P.check_fp8_rows(got, qz, w.alpha, 0, h, rows, device=CPU)


def test_bf16_check_accepts_rounded_weights_and_rejects_a_scale_error():
    rng = np.random.default_rng(78)
    q, k, v = rng.standard_normal((20, 64)) * 3, rng.standard_normal((500, 64)) * 3, rng.standard_normal((500, 64))
    alpha = 0.125
    s = alpha * q @ k.T
    p = np.exp(s - s.max(axis=1, keepdims=True))
    pb = torch.from_numpy(p).to(torch.bfloat16).double().numpy()         # P rounded to bf16, normalised by its sum
    got = (pb @ v) / pb.sum(axis=1, keepdims=True)
    P.bf16_check(got, q, k, v, alpha, device=CPU)
    with pytest.raises(AssertionError):
        P.bf16_check(got * 1.01, q, k, v, alpha, device=CPU)
