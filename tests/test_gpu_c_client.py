"""The whole FP8 path driven from a plain C program (tests/c_abi_gpu_client.c) that links
libtfm.so and the HIP runtime with the host C compiler, with no Python or torch in its
process.  Its codes and scales must be bit-exact against the oracle's Eq. (2), and its
outputs bitwise equal to the same call made through the Python binding (and within the
parity checks against the oracle)."""
import os
import shutil
import subprocess

import numpy as np
import pytest
import torch

from oracle import quantize as OQ
from paper_2609_13031_amd import tfm
from paper_2609_13031_amd.workloads import Workload, generate
from parity import check_fp8_call, gpu_inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_13031_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

pytestmark = pytest.mark.gpu


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no host C compiler")
def test_c_client_runs_the_fp8_path(tmp_path):
    w = Workload("c_client", B=2, H=3, D=64, N=700, M=130, dtype="bf16", seed=321)
    x = generate(w)
    for name in ("q_train", "k", "v", "q_test"):
        torch.from_numpy(x[name]).to(torch.bfloat16).view(torch.int16).numpy().tofile(str(tmp_path / (name + ".bin")))
    exe = str(tmp_path / "c_abi_gpu_client")
    cc = ["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-D__HIP_PLATFORM_AMD__",
          "-isystem", os.path.join(ROCM, "include"), "-I" + os.path.join(ROOT, "include"),
          os.path.join(ROOT, "tests", "c_abi_gpu_client.c"), "-L" + PKG, "-ltfm", "-L" + os.path.join(ROCM, "lib"),
          "-lamdhip64", "-Wl,-rpath," + PKG, "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", exe]
    r = subprocess.run(cc, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    print("c client built; running it", flush=True)
    r = subprocess.run([exe, str(tmp_path), str(w.B), str(w.H), str(w.D), str(w.N), str(w.M), repr(w.alpha)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "done" in r.stdout, r.stdout + r.stderr

    B, H, D, N, M = w.B, w.H, w.D, w.N, w.M
    rd = lambda n, dt, shape: np.fromfile(str(tmp_path / (n + ".bin")), dtype=dt).reshape(shape)
    # Eq. (2) on the same bf16 values, by the oracle
    qz = OQ.quantize_qkv_per_head(x["q_train"], x["k"], x["v"], x["q_test"])
    for name, rows in (("q8_train", N), ("k8", N), ("v8", N), ("q8_test", M)):
        assert np.array_equal(rd(name, np.uint8, (B, H, rows, D)), qz[name]), name
    sc = rd("scales", np.float32, (4, B, H))
    for i, name in enumerate(("s_q", "s_k", "s_v", "s_q_test")):
        assert np.array_equal(sc[i], qz[name]), name
    o_tr, o_te = rd("o_train", np.float32, (B, N, H, D)), rd("o_test", np.float32, (B, M, H, D))

    # the same call through the Python binding gives the same bits
    g = gpu_inputs(x, torch.bfloat16)
    p_tr, p_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
    assert np.array_equal(p_tr.cpu().numpy(), o_tr) and np.array_equal(p_te.cpu().numpy(), o_te)
    # and the rows are within the parity checks against the oracle
    m = check_fp8_call((o_tr, o_te), qz, w.alpha, None, None, block_kv=tfm.tfm_icl_attention_fp8_block_kv(D),
                       what="c_client")
    print("c client:", m, flush=True)
