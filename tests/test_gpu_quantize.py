"""GPU parity of tfm_quantize_qkv_per_head with the oracle quantizer (Eq. (2)):
codes and scales bit-exact on every element at every workload size, plus every
finite bf16 value against a sweep of scales."""
import concurrent.futures as cf

import numpy as np
import pytest
import torch

from oracle import quantize as OQ
from paper_2609_13031_amd import tfm
from paper_2609_13031_amd.workloads import WORKLOADS, Workload, generate
from parity import gpu_inputs, to_dev, workers

pytestmark = pytest.mark.gpu
KEYS = ("q8_train", "k8", "v8", "q8_test")


def run(x, dtype):
    g = gpu_inputs(x, dtype)
    out = tfm.tfm_quantize_qkv_per_head(g["q_train"], g["k"], g["v"], g["q_test"])
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


@pytest.mark.parametrize("name", ["tiny", "threshold", "many_tables"])
def test_codes_and_scales_bit_exact_full(name):
    w = WORKLOADS[name]
    x = generate(w)
    got = run(x, torch.float32 if w.dtype == "f32" else torch.bfloat16)
    ref = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])
    for k in ("s_q", "s_k", "s_v") + KEYS:
        assert np.array_equal(got[k], ref[k]), (name, k, np.count_nonzero(got[k] != ref[k]))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["mid", "large"])
def test_codes_and_scales_bit_exact_full_size_every_element(name):
    # every code of every tensor against the oracle's quantizer, one (tensor, head) at a time
    # on a pool of threads (the oracle is numpy; the slices are independent)
    w = WORKLOADS[name]
    print("generating", name, flush=True)
    x = generate(w)
    got = run(x, torch.bfloat16)
    s = {"s_q": OQ.scale_from_amax(OQ.absmax_per_head(x["q_train"])),
         "s_k": OQ.scale_from_amax(OQ.absmax_per_head(x["k"])),
         "s_v": OQ.scale_from_amax(OQ.absmax_per_head(x["v"]))}
    for k in s:
        assert np.array_equal(got[k], s[k]), k
    jobs = [(key, src, sc, h) for key, src, sc in (("q8_train", "q_train", "s_q"), ("k8", "k", "s_k"),
                                                    ("v8", "v", "s_v"), ("q8_test", "q_test", "s_q"))
            for h in range(w.H)]

    def one(job):
        key, src, sc, h = job
        ref = OQ.quantize_with_scale(np.ascontiguousarray(x[src][:, :, h:h + 1]), s[sc][:, h:h + 1])
        return job, int(np.count_nonzero(got[key][:, h:h + 1] != ref)), ref.size

    checked = 0
    with cf.ThreadPoolExecutor(workers()) as ex:
        for job, bad, n in ex.map(one, jobs):
            assert bad == 0, (name, job, bad)
            checked += n
    assert checked == (3 * w.N + w.M) * w.B * w.H * w.D
    print("%s: %d codes bit-exact" % (name, checked), flush=True)


BF16_SCALES_AMAX = [1.0, 448.0, 3.0, 0.1, 1e-3, 7.77e5, 2.0 ** -100, 1.5e-38, 3.3e38, 0.0]


@pytest.mark.parametrize("amax", BF16_SCALES_AMAX + [float(np.float32(a)) for a in
                                                     np.random.default_rng(3).uniform(0.01, 1000.0, 6)])
def test_every_finite_bf16_value_against_a_scale(amax):
    # Q_test rows hold every finite bf16 pattern (16384 of them per row-block of 256 x 64);
    # Q_train's absmax sets s_q, so test values beyond it exercise the clamp.
    u = np.arange(1 << 16, dtype=np.uint32) << 16
    allv = u.view(np.float32)
    allv = allv[np.isfinite(allv)]
    pad = (-allv.size) % 64
    q_test = np.concatenate([allv, np.zeros(pad, np.float32)]).reshape(1, -1, 1, 64)
    rng = np.random.default_rng(4)
    q_train = np.clip(rng.standard_normal((1, 100, 1, 64)).astype(np.float32), -1, 1) * np.float32(amax)
    q_train = torch.from_numpy(q_train).to(torch.bfloat16).float().numpy()
    q_train[0, 7, 0, 5] = np.float32(torch.tensor(amax).to(torch.bfloat16).float())
    x = {"q_train": q_train, "k": q_train.copy(), "v": q_train.copy(), "q_test": q_test}
    got = run(x, torch.bfloat16)
    ref = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])
    assert np.array_equal(got["s_q"], ref["s_q"])
    assert np.array_equal(got["q8_test"], ref["q8_test"]), np.count_nonzero(got["q8_test"] != ref["q8_test"])
    assert np.array_equal(got["q8_train"], ref["q8_train"])


def test_random_fp32_patterns_including_subnormals_and_negative_zero():
    rng = np.random.default_rng(5)
    u = rng.integers(0, 1 << 32, size=64 * 4096, dtype=np.uint64).astype(np.uint32)
    x = u.view(np.float32).copy()
    x[~np.isfinite(x)] = -0.0
    x[::97] = -0.0
    x = x.reshape(1, 4096, 1, 64)
    w = {"q_train": x[:, :2048] * np.float32(1e-30), "k": x[:, 2048:], "v": x[:, 1024:3072] * np.float32(1e-40),
         "q_test": x}
    w = {k: np.ascontiguousarray(v, dtype=np.float32) for k, v in w.items()}
    got = run(w, torch.float32)
    ref = OQ.quantize_qkv_per_head(w["q_train"], w["k"], w["v"], w["q_test"])
    for k in ("s_q", "s_k", "s_v") + KEYS:
        assert np.array_equal(got[k], ref[k]), k


@pytest.mark.parametrize("shape", [(1, 1, 1, 64, 1), (3, 5, 2, 128, 0), (2, 200, 3, 64, 77), (1, 64, 33, 128, 5)])
def test_edge_shapes(shape):
    B, N, H, D, M = shape
    w = Workload("edge", B=B, H=H, D=D, N=N, M=M, dtype="f32", seed=N + M)
    x = generate(w)
    got = run(x, torch.float32)
    ref = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"] if M else None)
    for k in ("s_q", "s_k", "s_v", "q8_train", "k8", "v8"):
        assert np.array_equal(got[k], ref[k]), k
    if M:
        assert np.array_equal(got["q8_test"], ref["q8_test"])
    else:
        assert got["q8_test"].shape == (B, H, 0, D)
