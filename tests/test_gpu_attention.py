"""GPU parity of the FP8 and bf16 ICL attention entry points with the oracle.

FP8 (tests/parity.py): every checked row elementwise against the oracle's
one-pass replay fed the FP8 MFMA's measured dot products (T1hw) and against
Eq. (1) on the dequantized inputs O_q within the derived bound (T2'); in the
regime where every FP8 dot product is exact, against the oracle's exact replay
O_qp within fp32 rounding (T1).  Full-size workloads are checked on sampled
rows: each output row depends only on its own query and all keys, so a
sampled row is checked exactly.  Plus edge shapes, closed forms and
invariances.  bf16: against Eq. (1) in fp64 (``oracle.attention``)."""
import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import quantize as OQ
from paper_2609_13031_amd import tfm
from paper_2609_13031_amd.workloads import WORKLOADS, Workload, generate
from parity import (TIE_REL, assert_t1, bf16_check, check_fp8_call, check_fp8_rows, gpu_inputs, narrow_range_inputs,
                    pv_rowsum_term, sample_rows)

pytestmark = pytest.mark.gpu
BKV = 128   # keys per block of the FP8 kernel: the running-max granularity the oracle replays


def test_library_block_size_is_the_one_the_oracle_replays():
    assert tfm.tfm_icl_attention_fp8_block_kv(64) == BKV and tfm.tfm_icl_attention_fp8_block_kv(128) == BKV


def fp8(g, w, out_dtype=torch.float32):
    o = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha, out_dtype=out_dtype)
    torch.cuda.synchronize()
    return o[0].float().cpu().numpy(), o[1].float().cpu().numpy()


def run_workload(w):
    """The fused FP8 call on the workload's inputs, and the oracle's codes and scales."""
    print("workload", w, flush=True)
    x = generate(w)
    g = gpu_inputs(x, torch.float32 if w.dtype == "f32" else torch.bfloat16)
    o_tr, o_te = fp8(g, w)
    del g
    return o_tr, o_te, OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])


def check_workload(w, rows_tr=None, rows_te=None, run=None, heads=None, t1hw_every=1):
    """T2' on the selected rows (default all) of the selected heads (default all) of every
    table, T1hw on every t1hw_every-th of them."""
    o_tr, o_te, qz = run_workload(w) if run is None else run
    m = check_fp8_call((o_tr, o_te), qz, w.alpha, rows_tr, rows_te, block_kv=BKV, what=w.name, heads=heads,
                       t1hw_every=t1hw_every)
    print("worst:", m, flush=True)
    return m


@pytest.mark.parametrize("B,H,D,N,M", [(1, 2, 64, 512, 128), (2, 3, 64, 1000, 77), (1, 2, 128, 700, 64)])
def test_exact_mfma_regime_matches_kernel_model_tightly(B, H, D, N, M):
    # codes in [224, 448] and a small softmax scale keep every FP8 MFMA dot
    # product exact, so the kernel must agree with O_qp to fp32 rounding (T1)
    x = narrow_range_inputs(B, N, M, H, D, seed=N + D)
    w = Workload("narrow", B=B, H=H, D=D, N=N, M=M, dtype="f32")
    alpha = 0.025
    g = gpu_inputs(x, torch.float32)
    o = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=alpha)
    o_tr, o_te = o[0].cpu().numpy(), o[1].cpu().numpy()
    qz = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])
    (r_tr, a_tr), (r_te, a_te) = OA.icl_attention_fp8_kernel_model(qz, np.float32(alpha), BKV, tie_rel=TIE_REL)
    for b in range(B):
        for h in range(H):
            m1 = assert_t1(o_tr[b, :, h], r_tr[b, :, h], a_tr[b, :, h], ("train", b, h))
            m2 = assert_t1(o_te[b, :, h], r_te[b, :, h], a_te[b, :, h], ("test", b, h))
    check_fp8_call((o_tr, o_te), qz, np.float32(alpha), None, None, block_kv=BKV, what="narrow")
    print("T1 metrics (last head):", m1, m2)


def test_tiny_full():
    check_workload(WORKLOADS["tiny"])


def test_threshold_sampled():
    w = WORKLOADS["threshold"]
    check_workload(w, sample_rows(w.N, 1024, 1), sample_rows(w.M, 512, 2))


def test_many_tables_sampled():
    w = WORKLOADS["many_tables"]
    check_workload(w, sample_rows(w.N, 64, 3), sample_rows(w.M, 32, 4))


def mid_rows(w):
    # 2048 sampled train rows and 512 test rows per head, plus train rows 0..1023 (the rows
    # the benchmark's accuracy report uses)
    return np.union1d(sample_rows(w.N, 2048, 5), np.arange(1024)), sample_rows(w.M, 512, 6)


@pytest.mark.timeout(900)
def test_mid_full_size_sampled():
    w = WORKLOADS["mid"]
    check_workload(w, *mid_rows(w), t1hw_every=2)


@pytest.fixture(scope="module")
def large_run():
    return run_workload(WORKLOADS["large"])


@pytest.mark.timeout(900)
@pytest.mark.parametrize("heads", [(0, 2), (2, 4), (4, 6), (6, 8)])
def test_large_full_size_sampled(large_run, heads):
    w = WORKLOADS["large"]
    check_workload(w, sample_rows(w.N, 2048, 7), sample_rows(w.M, 512, 8), run=large_run, heads=range(*heads),
                   t1hw_every=16)


@pytest.mark.parametrize("name", ["mid", "large"])
def test_full_size_every_row(name):
    # Every output row at the full size, through properties that need no row of the
    # oracle's attention.  (1) A row depends only on its own query (Eq. (1); the
    # query scale comes from all of Q_train, which a permutation leaves alone), so
    # permuting the query rows permutes the outputs bit for bit: a missed, repeated
    # or misplaced query tile breaks this.  (2) A row is a mean of V-hat rows with
    # weights >= 0, so each channel lies within V-hat's range over the keys, up to
    # the FP8 MFMA error of the P V and row-sum products; NaN, garbage or a wrong
    # output scale leaves that range.
    w = WORKLOADS[name]
    print("workload", w, flush=True)
    x = generate(w)
    g = gpu_inputs(x, torch.bfloat16)
    a_tr, a_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
    rng = np.random.default_rng(25)
    p_tr = torch.from_numpy(rng.permutation(w.N)).cuda()
    p_te = torch.from_numpy(rng.permutation(w.M)).cuda()
    b_tr, b_te = tfm.tfm_icl_attention_fp8(g["q_train"][:, p_tr].contiguous(), g["k"], g["v"],
                                           g["q_test"][:, p_te].contiguous(), alpha=w.alpha)
    assert torch.equal(b_tr, a_tr[:, p_tr]) and torch.equal(b_te, a_te[:, p_te])
    del b_tr, b_te, g
    s_v = OQ.scale_from_amax(OQ.absmax_per_head(x["v"]))
    v_hat = OA.dequantize(OQ.quantize_with_scale(x["v"], s_v), s_v)          # (B, N, H, D)
    lo, hi = v_hat.min(axis=1), v_hat.max(axis=1)                            # (B, H, D)
    del v_hat
    vmax = np.maximum(np.abs(lo), np.abs(hi)).reshape(-1, w.D)
    slack = np.stack([pv_rowsum_term(vm, vm[None], w.N)[0] for vm in vmax]).reshape(lo.shape)
    lo = torch.from_numpy(lo - slack).float().cuda()[:, None]
    hi = torch.from_numpy(hi + slack).float().cuda()[:, None]
    for o in (a_tr, a_te):
        assert bool(torch.isfinite(o).all())
        assert bool(((o >= lo) & (o <= hi)).all()), float(torch.maximum(lo - o, o - hi).max())


def test_d128_wide_workgroups_ragged_rows():
    # 65836 train rows, B*H*ceil(rows/256) = 520 workgroups: the 8-wave kernel at head
    # dimension 128, with a ragged last key block and partial last query tiles of both calls
    w = Workload("wide", B=1, H=2, D=128, N=65836, M=300, dtype="bf16", seed=64)
    check_workload(w, sample_rows(w.N, 256, 11), sample_rows(w.M, 64, 12))


def test_tensors_beyond_4_gib():
    # B*H = 65408 heads of D = 128 and 640 train rows: every train-row tensor holds 5.4 G
    # elements (10.7 GB in bf16, 5.4 GB of codes), so element and byte offsets pass 2^32.
    # Inputs are drawn on the GPU; the heads at the start, the middle and the very end are
    # checked against the oracle (codes and scales bit for bit, outputs within T1hw and T2').
    B, H, D, N, M = 511, 128, 128, 640, 64
    gen = torch.Generator(device="cuda").manual_seed(65)
    def draw(rows):
        x = torch.randn((B, rows, H, D), generator=gen, device="cuda", dtype=torch.bfloat16)
        x *= (torch.rand((B, 1, H, 1), generator=gen, device="cuda") * 3.5 + 0.5).to(torch.bfloat16)
        return x
    g = {"q_train": draw(N), "k": draw(N), "v": draw(N), "q_test": draw(M)}
    alpha = np.float32(1.0 / np.sqrt(D))
    qz = tfm.tfm_quantize_qkv_per_head(g["q_train"], g["k"], g["v"], g["q_test"])
    assert qz["k8"].numel() > 2 ** 32 and qz["k8"].dtype == torch.uint8
    o_tr, o_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=float(alpha))
    assert o_tr.numel() > 2 ** 32
    torch.cuda.synchronize()
    for b, h in ((0, 0), (255, 77), (510, 126), (510, 127)):
        x = {k: t[b:b + 1, :, h:h + 1].float().cpu().numpy() for k, t in g.items()}
        ref = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])
        for key in ("q8_train", "k8", "v8", "q8_test"):
            assert np.array_equal(qz[key][b, h].cpu().numpy(), ref[key][0, 0]), (b, h, key)
        for key in ("s_q", "s_k", "s_v", "s_q_test"):
            assert qz[key][b, h].item() == ref[key][0, 0], (b, h, key)
        check_fp8_call((o_tr[b:b + 1, :, h:h + 1].cpu().numpy(), o_te[b:b + 1, :, h:h + 1].cpu().numpy()), ref,
                       alpha, None, None, block_kv=BKV, what=(b, h))
    # the prequantized entry point (public code layout, V re-laid into tiles) gives every row bit for bit
    p_tr, p_te = tfm.tfm_icl_attention_fp8_prequantized(qz["q8_train"], qz["k8"], qz["v8"], qz["q8_test"], qz["s_q"],
                                                        qz["s_k"], qz["s_v"], alpha=float(alpha))
    assert torch.equal(p_tr, o_tr) and torch.equal(p_te, o_te)
    del qz, o_tr, o_te, p_tr, p_te
    # the 16-bit kernel on the same tensors, against Eq. (1) in fp64
    b_tr, b_te = tfm.tfm_icl_attention_bf16(g["q_train"], g["k"], g["v"], g["q_test"], alpha=float(alpha))
    torch.cuda.synchronize()
    for b, h in ((0, 0), (510, 127)):
        k, v = (g[n][b, :, h].double().cpu().numpy() for n in ("k", "v"))
        for o, q in ((b_tr, g["q_train"]), (b_te, g["q_test"])):
            bf16_check(o[b, :, h].cpu().numpy(), q[b, :, h].double().cpu().numpy(), k, v, float(alpha), what=(b, h))
    del g, b_tr, b_te
    torch.cuda.empty_cache()


@pytest.mark.parametrize("B,H,D,N,M,dtype", [
    (1, 1, 64, 1, 1, "f32"), (1, 2, 64, 63, 0, "bf16"), (2, 1, 64, 64, 5, "f32"), (1, 3, 64, 65, 130, "bf16"),
    (1, 1, 128, 1, 0, "bf16"), (1, 2, 128, 129, 17, "f32"), (3, 2, 128, 200, 255, "bf16"), (1, 1, 64, 1000, 1, "bf16"),
    # around the first key block staged as a full block (two whole 128-key blocks) and a whole last block
    (1, 2, 64, 256, 7, "bf16"), (2, 1, 64, 257, 0, "f32"), (1, 1, 64, 384, 129, "bf16"),
])
def test_edge_shapes(B, H, D, N, M, dtype):
    check_workload(Workload("edge", B=B, H=H, D=D, N=N, M=M, dtype=dtype, seed=B * 1000 + N + M))


def test_identical_keys_give_mean_of_v_and_constant_v_is_returned():
    rng = np.random.default_rng(20)
    B, N, H, D, M = 1, 300, 2, 64, 40
    q = rng.standard_normal((B, N + M, H, D)).astype(np.float32) * 3
    k = np.repeat(rng.standard_normal((B, 1, H, D)).astype(np.float32), N, axis=1)
    v = rng.standard_normal((B, N, H, D)).astype(np.float32)
    x = {"q_train": q[:, :N], "k": k, "v": v, "q_test": q[:, N:]}
    w = Workload("closed", B=B, H=H, D=D, N=N, M=M, dtype="f32")
    o_tr, o_te = fp8(gpu_inputs(x, torch.float32), w)
    qz = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])
    v_hat = OA.dequantize(qz["v8"], qz["s_v"])
    mean_v = v_hat.mean(axis=1)                                          # (B, H, D)
    # every lifted weight is exactly 2^8; only the FP8 MFMA arithmetic of P V and of l errs
    for h in range(H):
        tol = pv_rowsum_term(np.abs(v_hat[0, :, h]).max(axis=0), mean_v[:, h], N)
        for o in (o_tr, o_te):
            assert np.all(np.abs(o[0, :, h] - mean_v[0, h]) <= tol), h
    x["v"] = np.full_like(v, 1.75)
    x["k"] = rng.standard_normal((B, N, H, D)).astype(np.float32) * 4
    o_tr, o_te = fp8(gpu_inputs(x, torch.float32), w)
    tol = pv_rowsum_term(np.full(D, 1.75), np.full((1, D), 1.75), N)
    for o in (o_tr, o_te):
        assert np.all(np.abs(o - 1.75) <= tol)


def test_vanishing_softmax_factor_gives_the_mean_of_v():
    # |Q|, |K| ~ 1e-21: s_q s_k underflows, so the kernel's factor c = alpha s_q s_k log2(e)
    # is 0 in fp32 and every lifted weight is 2^8: the output is the mean of V-hat (Eq. (1)
    # with logits that are all 0).  The empty state before the first key block is not
    # rescaled by 2^(0 * -inf).
    rng = np.random.default_rng(26)
    B, N, H, D, M = 1, 300, 2, 64, 20
    q = (rng.standard_normal((B, N + M, H, D)) * 1e-21).astype(np.float32)
    k = (rng.standard_normal((B, N, H, D)) * 1e-21).astype(np.float32)
    v = rng.standard_normal((B, N, H, D)).astype(np.float32)
    x = {"q_train": q[:, :N].copy(), "k": k, "v": v, "q_test": q[:, N:].copy()}
    o_tr, o_te = fp8(gpu_inputs(x, torch.float32), Workload("tiny_c", B=B, H=H, D=D, N=N, M=M, dtype="f32"))
    qz = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])
    assert np.float32(np.float32(1 / 8) * qz["s_q"][0, 0] * qz["s_k"][0, 0]) == 0
    mean_v = OA.dequantize(qz["v8"], qz["s_v"]).mean(axis=1)
    for h in range(H):
        tol = pv_rowsum_term(np.abs(OA.dequantize(qz["v8"], qz["s_v"])[0, :, h]).max(axis=0), mean_v[:, h], N)
        for o in (o_tr, o_te):
            assert np.all(np.isfinite(o))
            assert np.all(np.abs(o[0, :, h] - mean_v[0, h]) <= tol), h


def test_one_hot_rows():
    # key 11 matches every query far better than the rest: the output is its V row
    B, N, H, D, M = 1, 256, 1, 64, 8
    rng = np.random.default_rng(21)
    k = rng.standard_normal((B, N, H, D)).astype(np.float32) * 0.01
    k[0, 11, 0, :] = 1.0
    q = np.ones((B, N + M, H, D), np.float32) * 4.0
    v = rng.standard_normal((B, N, H, D)).astype(np.float32)
    x = {"q_train": q[:, :N], "k": k, "v": v, "q_test": q[:, N:]}
    o_tr, o_te = fp8(gpu_inputs(x, torch.float32), Workload("onehot", B=B, H=H, D=D, N=N, M=M, dtype="f32"))
    qz = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])
    v11 = OA.dequantize(qz["v8"], qz["s_v"])[0, 11, 0]
    assert np.allclose(o_tr[0, :, 0], v11, rtol=1e-6, atol=1e-6)
    assert np.allclose(o_te[0, :, 0], v11, rtol=1e-6, atol=1e-6)


@pytest.fixture(scope="module")
def thr():
    w = WORKLOADS["threshold"].with_(N=4000, M=700)
    x = generate(w)
    return w, x, gpu_inputs(x, torch.bfloat16)


def test_batch_invariance_of_test_rows(thr):
    # the train-query scale makes a test row's output independent of the other test rows
    w, x, g = thr
    _, full = fp8(g, w)
    perm = np.random.default_rng(22).permutation(w.M)[:123]
    g2 = dict(g)
    g2["q_test"] = g["q_test"][:, torch.from_numpy(perm).cuda()].contiguous()
    _, part = fp8(g2, w.with_(M=123))
    assert np.array_equal(part, full[:, perm])


def test_train_outputs_do_not_depend_on_test_rows(thr):
    w, x, g = thr
    tr_full, _ = fp8(g, w)
    g0 = dict(g)
    g0["q_test"] = None
    tr_only, te_only = fp8(g0, w.with_(M=0))
    assert te_only.shape[1] == 0
    assert np.array_equal(tr_full, tr_only)


def test_test_rows_equal_to_train_rows_give_identical_outputs(thr):
    w, x, g = thr
    g2 = dict(g)
    g2["q_test"] = g["q_train"][:, 100:300].contiguous()
    tr, te = fp8(g2, w.with_(M=200))
    assert np.array_equal(te, tr[:, 100:300])


def test_determinism_prequantized_and_bf16_output(thr):
    w, x, g = thr
    a_tr, a_te = fp8(g, w)
    b_tr, b_te = fp8(g, w)
    assert np.array_equal(a_tr, b_tr) and np.array_equal(a_te, b_te)
    qz = tfm.tfm_quantize_qkv_per_head(g["q_train"], g["k"], g["v"], g["q_test"])
    p_tr, p_te = tfm.tfm_icl_attention_fp8_prequantized(qz["q8_train"], qz["k8"], qz["v8"], qz["q8_test"],
                                                        qz["s_q"], qz["s_k"], qz["s_v"], alpha=w.alpha)
    assert np.array_equal(p_tr.cpu().numpy(), a_tr) and np.array_equal(p_te.cpu().numpy(), a_te)
    h_tr, h_te = fp8(g, w, out_dtype=torch.bfloat16)
    assert np.array_equal(h_tr, torch.from_numpy(a_tr).to(torch.bfloat16).float().numpy())
    assert np.array_equal(h_te, torch.from_numpy(a_te).to(torch.bfloat16).float().numpy())


def test_train_row_permutation(thr):
    # Permuting the train rows permutes the codes exactly.  The outputs change only
    # through the key-tile order of the P rounding, so both orders stay within T2.
    w, x, g = thr
    perm = torch.from_numpy(np.random.default_rng(23).permutation(w.N)).cuda()
    g2 = {"q_train": g["q_train"][:, perm].contiguous(), "k": g["k"][:, perm].contiguous(),
          "v": g["v"][:, perm].contiguous(), "q_test": g["q_test"]}
    a = tfm.tfm_quantize_qkv_per_head(g["q_train"], g["k"], g["v"], g["q_test"])
    p = tfm.tfm_quantize_qkv_per_head(g2["q_train"], g2["k"], g2["v"], g2["q_test"])
    for key in ("q8_train", "k8", "v8"):
        assert torch.equal(p[key], a[key][:, :, perm])
    assert torch.equal(p["q8_test"], a["q8_test"])
    b_tr, b_te = fp8(g2, w)
    qz = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])
    pc = perm.cpu().numpy()
    rows = sample_rows(w.N, 32, 24)
    # the permuted call's rows are the original rows pc[rows] attending to permuted keys: T2'
    # against O_q of the original rows (Eq. (1) does not depend on the key order)
    qzp = {"q8_train": qz["q8_train"][:, :, pc], "k8": qz["k8"][:, :, pc], "v8": qz["v8"][:, :, pc],
           "q8_test": qz["q8_test"], "s_q": qz["s_q"], "s_k": qz["s_k"], "s_v": qz["s_v"], "s_q_test": qz["s_q_test"]}
    check_fp8_call((b_tr, b_te), qzp, w.alpha, rows, np.arange(32), block_kv=BKV, what="permuted")


# ---------------- bf16 baseline ----------------

@pytest.mark.parametrize("name,B,H,D,N,M", [("tiny", 1, 2, 64, 512, 128), ("edge", 1, 2, 64, 65, 3),
                                            ("edge", 2, 1, 128, 300, 50), ("threshold", 1, 6, 64, 8192, 2048),
                                            ("wide", 1, 8, 128, 8300, 300)])
def test_bf16_kernel_against_exact_attention(name, B, H, D, N, M):
    w = WORKLOADS.get(name, Workload(name, B=B, H=H, D=D, N=N, M=M, dtype="bf16", seed=N)).with_(dtype="bf16")
    x = generate(w)
    g = gpu_inputs(x, torch.bfloat16)
    o_tr, o_te = tfm.tfm_icl_attention_bf16(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
    o_tr, o_te = o_tr.cpu().numpy(), o_te.cpu().numpy()
    rt, re = sample_rows(w.N, 64, 9), sample_rows(w.M, 32, 10)
    for b in range(w.B):
        for h in range(w.H):
            for o, q, rows in ((o_tr, x["q_train"], rt), (o_te, x["q_test"], re)):
                bf16_check(o[b, rows, h], q[b, rows, h].astype(np.float64), x["k"][b, :, h].astype(np.float64),
                           x["v"][b, :, h].astype(np.float64), w.alpha, what=(name, b, h))


@pytest.mark.parametrize("B,H,D,N,M", [(1, 2, 64, 257, 33), (2, 1, 128, 300, 0), (1, 3, 64, 1000, 100)])
def test_bf16_kernel_rounds_fp32_inputs_on_load(B, H, D, N, M):
    # fp32 inputs are rounded to bf16 (nearest even) as the kernel stages them, so the
    # reference is Eq. (1) on the bf16-rounded inputs
    w = Workload("f32in", B=B, H=H, D=D, N=N, M=M, dtype="f32", seed=700 + N)
    x = generate(w)
    g = gpu_inputs(x, torch.float32)
    o_tr, o_te = tfm.tfm_icl_attention_bf16(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
    o_tr, o_te = o_tr.cpu().numpy(), o_te.cpu().numpy()
    r = {k: torch.from_numpy(v).to(torch.bfloat16).double().numpy() for k, v in x.items()}
    for b in range(B):
        for h in range(H):
            for o, q in ((o_tr, r["q_train"]), (o_te, r["q_test"])):
                if q.shape[1]:
                    bf16_check(o[b, :, h], q[b, :, h], r["k"][b, :, h], r["v"][b, :, h], w.alpha, what=(N, b, h))


def test_bf16_workgroup_width_changes_no_bit():
    # B*H*ceil(rows/256) = 280: 8-wave workgroups at head dimension 128; a single head is
    # 35 such workgroups, too few, so it runs 4-wave ones.  A head's outputs depend only on
    # its own inputs, so the two must agree bit for bit.
    w = Workload("wide", B=1, H=8, D=128, N=8300, M=300, dtype="bf16", seed=66)
    g = gpu_inputs(generate(w), torch.bfloat16)
    a_tr, a_te = tfm.tfm_icl_attention_bf16(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
    for h in (0, 5):
        one = {k: t[:, :, h:h + 1].contiguous() for k, t in g.items()}
        b_tr, b_te = tfm.tfm_icl_attention_bf16(one["q_train"], one["k"], one["v"], one["q_test"], alpha=w.alpha)
        assert torch.equal(b_tr[:, :, 0], a_tr[:, :, h]) and torch.equal(b_te[:, :, 0], a_te[:, :, h])


def test_bf16_kernel_invariances(thr):
    w, x, g = thr
    a = tfm.tfm_icl_attention_bf16(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
    b = tfm.tfm_icl_attention_bf16(g["q_train"], g["k"], g["v"], None, alpha=w.alpha)
    c = tfm.tfm_icl_attention_bf16(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha, out_dtype=torch.bfloat16)
    assert torch.equal(a[0], b[0])
    assert torch.equal(c[0], a[0].to(torch.bfloat16)) and torch.equal(c[1], a[1].to(torch.bfloat16))


# ---------------- gate and 16-bit path with fp32 inputs ----------------

@pytest.mark.parametrize("N,expect_fp8", [(8192, False), (8193, True)])
def test_gate_runs_fp8_only_above_8192_train_rows(N, expect_fp8):
    w = Workload("gate", B=1, H=1, D=64, N=N, M=16, dtype="bf16", seed=N)
    g = gpu_inputs(generate(w), torch.bfloat16)
    o_tr, o_te, used = tfm.tfm_icl_attention(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
    assert used == expect_fp8
    direct = (tfm.tfm_icl_attention_fp8 if expect_fp8 else tfm.tfm_icl_attention_bf16)(
        g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
    assert torch.equal(o_tr, direct[0]) and torch.equal(o_te, direct[1])
    # an explicit gate moves the switch
    _, _, used2 = tfm.tfm_icl_attention(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha,
                                        fp8_min_train_rows=N - 1)
    assert used2


def test_bf16_kernel_rounds_fp32_inputs_to_bf16_on_load():
    w = Workload("f32in", B=1, H=2, D=64, N=700, M=33, dtype="f32", seed=31)
    x = generate(w)
    g32 = gpu_inputs(x, torch.float32)
    g16 = {k: v.to(torch.bfloat16) for k, v in g32.items()}
    a = tfm.tfm_icl_attention_bf16(g32["q_train"], g32["k"], g32["v"], g32["q_test"], alpha=w.alpha)
    b = tfm.tfm_icl_attention_bf16(g16["q_train"], g16["k"], g16["v"], g16["q_test"], alpha=w.alpha)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
