"""The no-allocation entry point (tfm_icl_attention_fp8_noalloc) against the fused
entry point it varies: same kernels, the library's fixed scratch instead of a
caller workspace, so the outputs must agree bit for bit, on two calls in a row
(the second smaller, on the scratch the first left behind)."""
import numpy as np
import pytest
import torch

from paper_2609_13031_amd import tfm
from paper_2609_13031_amd.workloads import Workload, generate
from parity import gpu_inputs

pytestmark = pytest.mark.gpu


def both(w, dtype, out_dtype, **opts):
    g = gpu_inputs(generate(w), dtype)
    want = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha, out_dtype=out_dtype,
                                     **opts)
    out = tuple(torch.full_like(o, float("nan")) for o in want)
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    got = tfm.tfm_icl_attention_fp8_noalloc(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha,
                                            out_dtype=out_dtype, out=out, **opts)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == before
    return want, got


def test_noalloc_equals_the_fused_call_on_two_calls_in_a_row():
    big = Workload("noalloc_big", B=2, H=4, D=64, N=5000, M=900, dtype="bf16", seed=90)
    small = Workload("noalloc_small", B=1, H=3, D=128, N=700, M=130, dtype="f32", seed=91)
    for w, dt, odt, opts in ((big, torch.bfloat16, torch.float32, {}),
                             (small, torch.float32, torch.bfloat16, {"q_scale_mode": "per_call", "test_kv_heads": 1})):
        print("noalloc", w, opts, flush=True)
        want, got = both(w, dt, odt, **opts)
        assert torch.equal(got[0], want[0]) and torch.equal(got[1], want[1]), w.name


def test_noalloc_rejects_a_call_beyond_its_scratch():
    w = Workload("noalloc_large", B=1, H=8, D=64, N=65536, M=4096, dtype="bf16", seed=92)
    assert tfm.tfm_icl_attention_fp8_workspace_bytes(w.B, w.H, w.D, w.N, w.M) > 64 << 20
    g = {k: torch.zeros(s, dtype=torch.bfloat16, device="cuda") for k, s in
         (("q_train", (1, w.N, 8, 64)), ("k", (1, w.N, 8, 64)), ("v", (1, w.N, 8, 64)), ("q_test", (1, w.M, 8, 64)))}
    with pytest.raises(tfm.TfmError) as e:
        tfm.tfm_icl_attention_fp8_noalloc(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
    assert e.value.status == 6
