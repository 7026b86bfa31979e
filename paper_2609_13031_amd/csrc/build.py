"""Build libtfm.so (gfx950) from the HIP sources in this directory.

Usage: python -m paper_2609_13031_amd.csrc.build   (or call build()).
Every source is compiled for gfx950 only, with packed-fp32 instruction
selection disabled, and linked into paper_2609_13031_amd/libtfm.so.
"""
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
OUT = os.path.join(PKG, "libtfm.so")
BUILD_DIR = os.path.join(ROOT, "_build")
SOURCES = ["abi.hip", "quantize.hip", "attn_fp8.hip", "attn_bf16.hip", "noise.hip"]

FLAGS = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I" + os.path.join(ROOT, "include")]


def hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


# The attention kernels take the running max with fmaxf over MFMA results; declaring
# them NaN-free (NaN inputs are outside the documented domain) lets the compiler drop
# the canonicalizing v_max before each of those.
SOURCE_FLAGS = {"attn_fp8.hip": ["-fno-honor-nans"], "attn_bf16.hip": ["-fno-honor-nans"]}


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "not a recognized feature for this target"
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError("command failed: %s\n%s" % (" ".join(cmd), msg))
    return msg


# Test-only GPU code (not part of libtfm): the matrix-instruction probe that the
# precision tests drive, and the shader-clock sampler the benchmark runs beside the
# attention kernel.
PROBE_SRC = os.path.join(ROOT, "tests", "mfma_probe.hip")
PROBE_OUT = os.path.join(ROOT, "tests", "libmfma_probe.so")
CLOCK_SRC = os.path.join(ROOT, "tests", "clock_sampler.hip")
CLOCK_OUT = os.path.join(ROOT, "tests", "libclock_sampler.so")


def _build_test_lib(src, out):
    tmp = out + ".tmp"
    _run([hipcc(), *FLAGS, "-shared", src, "-o", tmp])
    os.replace(tmp, out)
    return out


def build_probe():
    return _build_test_lib(PROBE_SRC, PROBE_OUT)


def build_clock_sampler():
    return _build_test_lib(CLOCK_SRC, CLOCK_OUT)


def build(verbose=False):
    os.makedirs(BUILD_DIR, exist_ok=True)
    cc = hipcc()
    jobs = []
    for src in SOURCES:
        obj = os.path.join(BUILD_DIR, src.replace(".hip", ".o"))
        jobs.append((obj, [cc, *FLAGS, *SOURCE_FLAGS.get(src, []), "-c", os.path.join(HERE, src), "-o", obj]))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        for obj, msg in zip([j[0] for j in jobs], ex.map(lambda j: _run(j[1]), jobs)):
            if verbose and msg.strip():
                print(msg)
    tmp = OUT + ".tmp"
    _run([cc, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + [j[0] for j in jobs])
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
