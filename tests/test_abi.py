"""C-ABI checks that need no GPU: the library loads, exports every entry point
of include/tfm.h, and rejects bad arguments before enqueuing anything."""
import ctypes
import os
import re
import shutil
import subprocess

import pytest

from paper_2609_13031_amd import tfm

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "tfm.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tfm_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    L = tfm.lib()
    names = header_functions()
    assert len(names) == 19
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(tfm.SIGNATURES)


def test_status_strings_and_version():
    L = tfm.lib()
    assert L.tfm_status_string(0) == b"TFM_OK"
    for st in range(1, 9):
        assert L.tfm_status_string(st).startswith(b"TFM_ERR_")
    assert L.tfm_status_string(99) == b"TFM_ERR_UNKNOWN"
    assert tfm.tfm_version() == 200


def test_block_kv_and_workspace_queries():
    assert tfm.tfm_icl_attention_fp8_block_kv(64) == 128
    assert tfm.tfm_icl_attention_fp8_block_kv(128) == 128
    assert tfm.tfm_icl_attention_fp8_block_kv(96) == 0
    # the slice maxima of the amax pass (4 tensors x B*H heads x 128 slices, uint32) and the
    # scales (4*B*H floats), each 256-aligned
    assert tfm.tfm_quantize_workspace_bytes(2, 6) == 4 * 12 * 128 * 4 + 256
    assert tfm.tfm_quantize_workspace_bytes(0, 6) == 0
    assert tfm.tfm_quantize_workspace_bytes(1, 65536) == 0
    # slice maxima and scales, codes of Q_train, Q_test, K (N or M x D per head), V tiles (ceil(N/64)*64*D)
    B, H, D, N, M = 2, 6, 64, 65536, 16384
    want = 4 * B * H * 128 * 4 + 256 + B * H * (N * D + M * D + N * D + N * D)
    assert tfm.tfm_icl_attention_fp8_workspace_bytes(B, H, D, N, M) == want
    assert tfm.tfm_icl_attention_fp8_workspace_bytes(1, 1, 64, 65, 0) >= 2048 + 256 + 65 * 64 * 2 + 128 * 64
    assert tfm.tfm_icl_attention_fp8_workspace_bytes(1, 1, 96, 10, 0) == 0
    assert tfm.tfm_icl_attention_fp8_prequantized_workspace_bytes(1, 2, 128, 100) == 2 * 128 * 128


FAKE = 0x10000          # aligned, never dereferenced: every call below fails validation first
MIS = 0x10008           # 8-byte aligned only


def opts(mode=0, g=0):
    return ctypes.byref(tfm.tfm_icl_options(mode, g))


def fp8_call(**kw):
    a = dict(in_dtype=1, out_dtype=0, opts=None, B=1, H=2, D=64, N=100, M=10, alpha=0.125, q_train=FAKE, k=FAKE,
             v=FAKE, q_test=FAKE, o_train=FAKE, o_test=FAKE, ws=FAKE, nws=1 << 40)
    a.update(kw)
    return tfm.lib().tfm_icl_attention_fp8(a["in_dtype"], a["out_dtype"], a["opts"], a["B"], a["H"], a["D"], a["N"],
                                           a["M"], a["alpha"], a["q_train"], a["k"], a["v"], a["q_test"],
                                           a["o_train"], a["o_test"], a["ws"], a["nws"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(B=0), 2), (dict(H=0), 2), (dict(N=0), 2), (dict(M=-1), 2), (dict(B=70000), 2),
    (dict(N=2 ** 31 - 100, M=1000), 2), (dict(D=96), 4), (dict(D=32), 4),
    (dict(in_dtype=2), 3), (dict(out_dtype=7), 3),
    (dict(alpha=0.0), 8), (dict(alpha=-1.0), 8), (dict(alpha=float("nan")), 8), (dict(alpha=float("inf")), 8),
    (dict(q_train=None), 1), (dict(k=None), 1), (dict(ws=None), 1), (dict(q_test=None), 1), (dict(o_test=None), 1),
    (dict(v=MIS), 5), (dict(o_train=MIS), 5), (dict(q_test=MIS), 5),
    (dict(nws=1000), 6),
    (dict(opts=opts(mode=3)), 8), (dict(opts=opts(mode=-1)), 8), (dict(opts=opts(g=3, mode=1)), 8),
    (dict(opts=opts(g=-1)), 8), (dict(opts=opts(g=4)), 8), (dict(H=6, opts=opts(g=4)), 8),
    (dict(opts=opts(mode=3), q_train=None), 8),
    (dict(opts=opts(mode=2, g=1), nws=1000), 6), (dict(H=6, opts=opts(mode=1, g=3), nws=1000), 6),
    (dict(opts=opts(g=2), nws=1000), 6),
])
def test_fp8_validation_errors(kw, status):
    assert fp8_call(**kw) == status


def test_grid_limits_are_validated_before_any_launch():
    # A launch holds fewer than 2^32 work-items per grid dimension: at 256 threads per
    # workgroup, at most 16777215 workgroups.  Shapes whose attention or quantize grid
    # would exceed that fail the shape check (the workspace here is always too small,
    # so a shape that passes reports 6 and nothing is launched).
    assert fp8_call(H=1, N=2 ** 29, M=0, q_test=None, o_test=None, nws=1000) == 6   # V: 2^23 tiles of 64 keys
    assert fp8_call(H=1, N=2 ** 30, M=0, q_test=None, o_test=None, nws=1000) == 2   # V: 2^24 tiles
    assert fp8_call(N=2 ** 20, M=2 ** 31 - 2 ** 20 - 1000, nws=1000) == 2      # 2 * 2^24 query tiles
    assert fp8_call(N=2 ** 20, M=2 ** 20, nws=1000) == 6
    assert tfm.tfm_icl_attention_fp8_workspace_bytes(1, 1, 64, 2 ** 30, 0) == 0
    L = tfm.lib()
    n = lambda S: L.tfm_noise_per_head(1, 1, 1, 1, S, 64, FAKE, FAKE, 0.1, FAKE, None, FAKE, 8, None)
    assert n(2 ** 30) == 6            # 2^36 elements: 2^23 workgroups of 8192
    assert n(2 ** 31 - 1) == 2        # just under 2^37 elements: 2^24 workgroups


def test_validation_order_and_m_zero_allows_null_test_pointers():
    # M == 0: NULL test pointers are fine, so the next failing check (workspace) reports
    assert fp8_call(M=0, q_test=None, o_test=None, nws=10) == 6
    # shape errors take precedence over pointer errors
    assert fp8_call(B=0, q_train=None) == 2


def test_quantize_and_bf16_and_prequantized_validation():
    L = tfm.lib()
    q = lambda **kw: L.tfm_quantize_qkv_per_head(kw.get("dt", 0), kw.get("o"), kw.get("B", 1), 2, kw.get("D", 64),
                                                 50, 0, FAKE, FAKE, FAKE, None, FAKE, FAKE, kw.get("v8", FAKE), None,
                                                 FAKE, FAKE, FAKE, kw.get("sqt"), FAKE, kw.get("nws", 1 << 20), None)
    assert q(dt=5) == 3 and q(B=0) == 2 and q(D=100) == 4 and q(v8=None) == 1 and q(v8=MIS) == 5 and q(nws=8) == 6
    assert q(o=opts(mode=5)) == 8 and q(o=opts(g=3)) == 8 and q(sqt=MIS) == 5 and q(sqt=FAKE, nws=8) == 6
    assert q(o=opts(mode=1, g=1), nws=8) == 6
    b = lambda **kw: L.tfm_icl_attention_bf16(kw.get("inp", 1), kw.get("out", 1), kw.get("o"), 1, 2, 64,
                                              kw.get("N", 50), 3, kw.get("alpha", 0.1), FAKE, FAKE, FAKE,
                                              kw.get("qt", FAKE), FAKE, FAKE, None)
    assert b(out=3) == 3 and b(inp=4) == 3 and b(N=0) == 2 and b(alpha=-2.0) == 8 and b(qt=None) == 1
    assert b(qt=MIS) == 5 and b(o=opts(g=3)) == 8 and b(o=opts(g=1), qt=None) == 1
    qs = lambda **kw: L.tfm_icl_attention_fp8_quantize(1, kw.get("o"), 1, 2, 64, 50, kw.get("M", 3), FAKE, FAKE,
                                                       FAKE, kw.get("qt", FAKE), FAKE, kw.get("nws", 1 << 30), None)
    assert qs(qt=None) == 1 and qs(M=0, qt=None, nws=10) == 6 and qs(qt=MIS) == 5 and qs(o=opts(mode=9)) == 8
    at = lambda **kw: L.tfm_icl_attention_fp8_attend(0, kw.get("o"), 1, 2, 64, 50, 3, kw.get("alpha", 0.1), FAKE,
                                                     kw.get("ot", FAKE), FAKE, kw.get("nws", 1 << 30), None)
    assert at(alpha=0.0) == 8 and at(ot=None) == 1 and at(nws=1) == 6 and at(o=opts(g=5)) == 8
    p = lambda **kw: L.tfm_icl_attention_fp8_prequantized(0, kw.get("o"), 1, 2, 64, 50, 0, 0.1, FAKE, FAKE, FAKE,
                                                          None, FAKE, kw.get("sk", FAKE), FAKE, kw.get("sqt"),
                                                          FAKE, None, FAKE, kw.get("nws", 1 << 20), None)
    assert p(sk=None) == 1 and p(nws=100) == 6 and p(o=opts(g=3)) == 8 and p(sqt=MIS) == 5


def test_gate_selects_the_path_before_validating_it():
    L = tfm.lib()
    used = ctypes.c_int(-7)
    g = lambda N, gate, **kw: L.tfm_icl_attention(1, 1, kw.get("o"), 1, 2, 64, N, 3, 0.1, FAKE, FAKE, FAKE, FAKE,
                                                  FAKE, FAKE, gate, ctypes.byref(used), kw.get("ws", FAKE),
                                                  kw.get("nws", 0), None)
    # The FP8 path needs a workspace, the 16-bit path none: the reported error
    # tells which one validated.  (Every call here must fail validation: the
    # pointers are fake and must never reach a kernel.)
    assert g(8193, -1) == 6 and g(9000, 8192) == 6 and g(100, 50) == 6
    assert L.tfm_icl_attention(1, 1, None, 1, 2, 64, 8192, 3, 0.1, FAKE, FAKE, FAKE, None, FAKE, FAKE, -1,
                               ctypes.byref(used), None, 0, None) == 1      # 16-bit path: NULL q_test with M > 0
    assert g(8193, -1, o=opts(g=3)) == 8 and g(100, -1, o=opts(mode=4)) == 8
    assert used.value == -7                        # not written on failure
    assert L.tfm_icl_attention_workspace_bytes(1, 2, 64, 8192, 3, -1) == 0
    assert L.tfm_icl_attention_workspace_bytes(1, 2, 64, 8193, 3, -1) == tfm.tfm_icl_attention_fp8_workspace_bytes(
        1, 2, 64, 8193, 3)
    assert L.tfm_icl_attention_workspace_bytes(1, 2, 64, 100, 3, 99) > 0


def test_noise_validation_and_workspace():
    L = tfm.lib()
    n = lambda **kw: L.tfm_noise_per_head(kw.get("xd", 1), kw.get("zd", 0), kw.get("B", 2), kw.get("H", 3),
                                          kw.get("S", 100), kw.get("D", 64), kw.get("x", FAKE), kw.get("z", FAKE),
                                          kw.get("eps", 0.1), kw.get("out", FAKE), kw.get("rho"), kw.get("ws", FAKE),
                                          kw.get("nws", 8), None)
    # every call here fails validation (the workspace is always too small when nothing else is wrong)
    assert n() == 6
    assert n(B=0) == 2 and n(H=0) == 2 and n(S=-1) == 2 and n(H=300, D=64) == 2 and n(B=70000, H=1) == 2
    assert n(D=12) == 4 and n(D=0) == 4 and n(D=4) == 4
    assert n(xd=2) == 3 and n(zd=5) == 3
    assert n(eps=-0.5) == 8 and n(eps=float("nan")) == 8 and n(eps=float("inf")) == 8
    assert n(x=None) == 1 and n(z=None) == 1 and n(out=None) == 1 and n(ws=None) == 1
    assert n(x=MIS) == 5 and n(out=MIS) == 5 and n(rho=MIS) == 5 and n(rho=MIS, S=0) == 5
    ws = tfm.tfm_noise_per_head_workspace_bytes
    # fixed-order partial sums: one double per (row chunk, b, h), chunks of ceil(32768 / (H D)) rows, then rho
    assert ws(2, 6, 65536, 64) == ((65536 + 85) // 86 * 12 * 8 + 255) // 256 * 256 + 256
    assert ws(1, 1, 1, 8) == 512 and ws(1, 1, 0, 8) == 256 and ws(1, 1, 5, 12) == 0


def test_fit_and_predict_validation():
    L = tfm.lib()
    f = lambda **kw: L.tfm_icl_attention_fp8_fit(1, 0, kw.get("o"), 1, 2, 64, kw.get("N", 300), kw.get("alpha", 0.1),
                                                 FAKE, FAKE, kw.get("v", FAKE), kw.get("ot", FAKE), kw.get("ws", FAKE),
                                                 kw.get("nws", 100), None)
    # every call fails validation: the workspace of 100 bytes is always too small
    assert f() == 6 and f(N=0) == 2 and f(alpha=0.0) == 8 and f(o=opts(mode=2)) == 8 and f(o=opts(g=3)) == 8
    assert f(v=None) == 1 and f(ot=None) == 1 and f(ws=None) == 1 and f(v=MIS) == 5
    need = tfm.tfm_icl_attention_fp8_workspace_bytes(1, 2, 64, 300, 0)
    assert f(nws=need - 1) == 6
    p = lambda **kw: L.tfm_icl_attention_fp8_predict(1, 0, kw.get("o"), 1, 2, 64, 300, kw.get("M", 50), 0.1,
                                                     kw.get("qt", FAKE), kw.get("ot", FAKE), kw.get("ws", FAKE),
                                                     kw.get("nws", 100), None)
    assert p() == 6 and p(M=-1) == 2 and p(o=opts(mode=2)) == 8 and p(qt=None) == 1 and p(ot=MIS) == 5
    assert p(M=0, qt=None, ot=None) == 6 and p(ws=None) == 1
    # one byte short of what M = 50 needs still fails (never a valid call: the pointers are fake)
    need_m = tfm.tfm_icl_attention_fp8_workspace_bytes(1, 2, 64, 300, 50)
    assert need_m > tfm.tfm_icl_attention_fp8_workspace_bytes(1, 2, 64, 300, 0)
    assert p(nws=need_m - 1) == 6


def test_noalloc_validation_before_any_hip_call():
    # every argument error, and a call needing more than the fixed scratch, is reported
    # before the entry point looks up its scratch (no GPU here)
    L = tfm.lib()
    f = L.tfm_icl_attention_fp8_noalloc
    p = ctypes.c_void_p(16)
    args = lambda **kw: [kw.get("ind", 1), kw.get("outd", 1), None, kw.get("B", 1), kw.get("H", 8), kw.get("D", 64),
                         kw.get("N", 4096), kw.get("M", 512), ctypes.c_float(kw.get("alpha", 0.125)),
                         p, p, p, kw.get("qt", p), p, kw.get("ot", p), None]
    assert L.tfm_icl_attention_fp8_workspace_bytes(1, 8, 64, 32768, 4096) <= 64 << 20
    assert L.tfm_icl_attention_fp8_workspace_bytes(1, 8, 64, 65536, 4096) > 64 << 20
    assert f(*args(N=65536)) == 6                      # beyond TFM_NOALLOC_SCRATCH_BYTES
    assert f(*args(D=96)) == 4
    assert f(*args(ind=5)) == 3
    assert f(*args(alpha=float("nan"))) == 8
    assert f(*args(qt=None)) == 1
    assert f(*args(M=0, qt=None, ot=None, N=0)) == 2


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no host C compiler")
def test_plain_c_client_compiles_links_and_runs(tmp_path):
    # the header is plain C99 (no C++ or HIP types in the signatures) and the
    # library links and resolves with the host C toolchain
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    pkg = os.path.join(root, "paper_2609_13031_amd")
    exe = str(tmp_path / "c_abi_client")
    cc = ["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I" + os.path.join(root, "include"),
          os.path.join(root, "tests", "c_abi_client.c"), "-L" + pkg, "-ltfm", "-Wl,-rpath," + pkg, "-o", exe]
    r = subprocess.run(cc, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "all checks passed" in r.stdout, r.stdout + r.stderr
