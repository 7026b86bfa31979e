#!/usr/bin/env python3
"""FP8 ICL attention throughput on one MI355X, with the bf16 kernel beside it.

One step is the whole hot path on one batch: per-head absmax quantization of
Q_train, K, V and Q_test to e4m3 (Eq. (2)), then both ICL attention calls
(train-train and test-train, Sec. 3) in FP8, i.e. one tfm_icl_attention_fp8
call, timed as its two stages with HIP events on the stream the library
launches on.  Inputs are resident in HBM before timing starts.  The headline
workload is two independent tables with 65536 train and 16384 test rows,
6 heads of dimension 64, bf16 in and out.  FLOPs count QK^T and PV of both
calls: 4*B*H*D*N*(N+M).

Prints one JSON line on stdout; progress goes to stderr.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "FP8 ICL attention TFLOP/s + speedup vs bf16 at N_train=65536, 1 MI355X"
FP8_PEAK_TFLOPS = 5000.0          # MI355X dense FP8 MFMA
COUNTERS = os.path.join(ROOT, "profiles", "attn_fp8_mid_counters.txt")
SQ_COUNTERS = os.path.join(ROOT, "profiles", "attn_mid_sq_counters.txt")
CLOCK_LIB = os.path.join(ROOT, "tests", "libclock_sampler.so")   # test-only shader-clock sampler
CSRC = os.path.join(ROOT, "paper_2609_13031_amd", "csrc")
HBM_PEAK_GBS = 8000.0
ORACLE_BLOCK_KV = 128             # key block of the FP8 kernel's running max, checked against the library
# The FP8 kernel's VALU work per (query, key) score is one v_fma_f32, one v_exp_f32, half a
# v_cvt_pk_fp8_f32 and half a v_max3_f32.  Their measured issue costs (2.96, 8.41, 9.94 and
# 5.73 cycles per wave64 instruction, counted in cycles of the shader clock each run got) over
# 1024 SIMDs at the 2.4 GHz peak clock give this many scores per second at most, i.e. 4*D
# times it in FLOP/s.
ALU_SCORES_PER_S = 1024 * 2.4e9 * 64 / (2.96 + 8.41 + 9.94 / 2 + 5.73 / 2)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_digest(name):
    """Hash of a kernel source's code: comments and blank lines do not count."""
    import re
    with open(os.path.join(CSRC, name)) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    lines = [re.sub(r"//.*", "", line).strip() for line in text.splitlines()]
    return hashlib.sha256("\n".join(x for x in lines if x).encode()).hexdigest()[:16]


def counter_value(key, source, path=COUNTERS):
    """A figure from a committed rocprofv3 summary under profiles/, or None when it is
    missing or was taken on a different version of the kernel source it measures."""
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get(source.replace(".hip", "") + "_source_sha256_16") != source_digest(source):
        return None
    try:
        return float(kv[key].split()[0])
    except (KeyError, ValueError, IndexError):
        return None


def sq_figures(w):
    """The FP8 attention kernel's SQ/GRBM counter figures on the headline workload, from the
    committed rocprofv3 summary (None where it is missing or stale): the clock under load,
    MFMA and VALU busy fractions, the FP8 MFMA FLOP the kernel issues per launch and the rate
    they imply at the counted duration, and the share of (wave, key block) pairs skipped
    exactly (their weights all round to e4m3 zero), which issue only the QK^T MFMAs."""
    if w.name != "mid":
        return None
    get = lambda k: counter_value(k, "attn_fp8.hip", SQ_COUNTERS)
    out = {"clock_ghz": get("fp8_clock_ghz"), "mfma_busy": get("fp8_mfma_busy"), "valu_busy": get("fp8_valu_busy"),
           "mfma_flop_per_launch": get("fp8_mfma_flop_per_launch"),
           "mfma_tflops_at_counted_duration": get("fp8_mfma_tflops_at_counted_duration"),
           "valu_instructions_per_wave_and_key_block": get("fp8_valu_insts_per_wave_block"),
           "skipped_block_fraction": get("fp8_skipped_block_fraction"),
           "source": "profiles/attn_mid_sq_counters.txt"}
    return out if any(v is not None for k, v in out.items() if k != "source") else None


def live_clock(run_steps, window_ms):
    """The shader clock while run_steps() runs on the current stream: the test-only sampler
    (one sleeping wave on a second, default-priority stream) reads s_memtime against
    s_memrealtime over a window of window_ms from the start.  None if the sampler library is
    not built or the launch fails."""
    import ctypes
    import torch
    if not os.path.exists(CLOCK_LIB):
        return None
    L = ctypes.CDLL(CLOCK_LIB)
    L.clock_sampler_launch.restype = ctypes.c_int
    L.clock_sampler_launch.argtypes = [ctypes.c_void_p, ctypes.c_ulonglong, ctypes.c_int, ctypes.c_void_p]
    L.clock_sampler_wall_khz.restype = ctypes.c_int
    khz = L.clock_sampler_wall_khz()
    if khz <= 0:
        return None
    out = torch.zeros(2, dtype=torch.int64, device="cuda")
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    if L.clock_sampler_launch(out.data_ptr(), int(window_ms * khz), 1 << 20, side.cuda_stream) != 0:
        return None
    run_steps()
    torch.cuda.synchronize()
    cycles, ticks = out.cpu().tolist()
    return cycles / ticks * khz * 1e3 / 1e9 if ticks > 0 else None


def metrics(got, ref):
    import numpy as np
    d = np.abs(np.asarray(got, np.float64) - ref)
    rms = float(np.sqrt(np.mean(ref ** 2)))
    return {"relF": float(np.linalg.norm(d) / np.linalg.norm(ref)), "max_abs_over_rms": float(d.max() / rms)}


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


_POOL_INPUTS = {}


def _pool_quantize(bh):
    """Worker: the oracle's Eq. (2) for one (table, head) of the workload."""
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle import quantize as OQ
    x = _POOL_INPUTS["x"]
    b, h = bh
    sl = lambda a: np.ascontiguousarray(a[b:b + 1, :, h:h + 1, :])
    with threadpool_limits(limits=1):
        qz = OQ.quantize_qkv_per_head(sl(x["q_train"]), sl(x["k"]), sl(x["v"]), sl(x["q_test"]))
    return bh, qz


def _pool_replay(job):
    """Worker: the oracle's one-pass kernel model on some query rows of one (table, head)."""
    from threadpoolctl import threadpool_limits
    from oracle import attention as OA
    bh, qz, alpha, block_kv, rows_train, rows_test = job
    with threadpool_limits(limits=1):
        o_tr, o_te = OA.icl_attention_fp8_kernel_model(qz, alpha, block_kv, rows_train, rows_test)
    return bh, rows_train, o_tr[0, :, 0]


def cpu_baseline(x, w, rows_train, rows_test, block_kv, workers):
    """The oracle, as it stands, on a bounded sample of the workload, spread over ``workers``
    processes forked before anything touches the GPU: Eq. (2) for every (table, head), then
    the one-pass kernel model for rows_train train and rows_test test rows of each.  Returns
    the report, the oracle's O_qp for train rows [0, accuracy rows) of table 0, head 0, and
    that head's codes."""
    import multiprocessing as mp
    import numpy as np
    _POOL_INPUTS["x"] = x
    heads = [(b, h) for b in range(w.B) for h in range(w.H)]
    ctx = mp.get_context("fork")
    with ctx.Pool(workers) as pool:
        t0 = time.perf_counter()
        qzs = dict(pool.map(_pool_quantize, heads))
        t_quant = time.perf_counter() - t0
        chunk = 512
        jobs = [((b, h), qzs[(b, h)], w.alpha, block_kv, np.arange(r0, min(rows_train, r0 + chunk)), [])
                for (b, h) in heads for r0 in range(0, rows_train, chunk)]
        jobs += [((b, h), qzs[(b, h)], w.alpha, block_kv, [], np.arange(r0, min(rows_test, r0 + chunk)))
                 for (b, h) in heads for r0 in range(0, rows_test, chunk)]
        t0 = time.perf_counter()
        res = pool.map(_pool_replay, jobs, chunksize=1)
        t_attn = time.perf_counter() - t0
    _POOL_INPUTS.clear()
    rows = len(heads) * (rows_train + rows_test)
    flops = 4.0 * w.D * w.N * rows
    head0 = np.concatenate([o for bh, rt, o in res if bh == (0, 0) and len(rt)])
    report = {"value": round(flops / t_attn / 1e12, 5), "unit": "TFLOP/s", "cores": workers, "kind": "oracle",
              "sample": "one-pass FP8 kernel model (fp64 numpy) for train rows 0..%d and test rows 0..%d of every "
                        "one of the %d (table, head) pairs, each against all %d keys, in %d worker processes; "
                        "Eq. (2) for all of the workload's elements took %.2f s more" %
                        (rows_train - 1, rows_test - 1, len(heads), w.N, workers, t_quant),
              "seconds": round(t_attn, 2), "quantize_seconds": round(t_quant, 2), "cpu_model": cpu_model()}
    return report, head0, qzs[(0, 0)]


def cpu_workers():
    """Processes for the CPU baseline: the host cores this process may run on, at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def accuracy(x, w, o_qp, qz, gpu_fp8, gpu_bf16, rows):
    """Errors on train rows [0, rows) of table 0, head 0: the FP8 kernel against the oracle's
    kernel model (O_qp), against Eq. (1) on the dequantized inputs (O_q) and against
    unquantized fp64 attention (O_exact); the method's own error (O_qp and O_q against
    O_exact); and the bf16 kernel against O_exact."""
    import numpy as np
    from oracle import attention as OA

    q = x["q_train"][0, :rows, 0].astype(np.float64)
    exact = OA.softmax_attention(q, x["k"][0, :, 0].astype(np.float64), x["v"][0, :, 0].astype(np.float64),
                                 float(w.alpha))
    o_q = OA.icl_attention_dequantized(qz, w.alpha, np.arange(rows), [])[0][0, :, 0]
    qp = o_qp[:rows]
    out = {"rows": "train rows 0..%d of table 0, head 0 (fp32 outputs)" % (rows - 1),
           "note": "the kernel model here scores with exact dot products; the FP8 MFMA truncates within groups of "
                   "8 products, so the elementwise parity tests compare against the same model fed the hardware's "
                   "scores instead",
           "fp8_kernel_vs_kernel_model": metrics(gpu_fp8, qp),
           "fp8_kernel_vs_dequantized_fp64": metrics(gpu_fp8, o_q),
           "fp8_kernel_vs_fp64_exact": metrics(gpu_fp8, exact),
           "kernel_model_vs_fp64_exact": metrics(qp, exact),
           "dequantized_vs_fp64_exact": metrics(o_q, exact)}
    if gpu_bf16 is not None:
        out["bf16_kernel_vs_fp64_exact"] = metrics(gpu_bf16, exact)
    return out


def time_sdpa(g, w, steps, warmup):
    """torch SDPA (flash backend only), the two ICL calls as two calls: context, not the baseline."""
    import torch
    from torch.nn.attention import SDPBackend, sdpa_kernel
    F = torch.nn.functional
    to_bhsd = lambda t: t.to(torch.bfloat16).transpose(1, 2).contiguous()
    q_tr, k, v, q_te = (to_bhsd(g[n]) for n in ("q_train", "k", "v", "q_test"))
    try:
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
            run = lambda: (F.scaled_dot_product_attention(q_tr, k, v, scale=w.alpha),
                           F.scaled_dot_product_attention(q_te, k, v, scale=w.alpha))
            for _ in range(warmup):
                run()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(steps):
                run()
            e1.record()
            torch.cuda.synchronize()
    except RuntimeError as e:
        log("sdpa flash backend unavailable:", str(e)[:200])
        return None
    ms = e0.elapsed_time(e1) / steps
    log("torch sdpa (flash) %.3f ms" % ms)
    return {"ms": round(ms, 4), "tflops": round(w.flops / ms / 1e9, 2), "backend": "flash"}


def crossover(max_n):
    """FP8 vs bf16 for a single train-train call (B=1, H=8, M=0, bf16 in/out), the shape of the
    paper's kernel tables, on synthetic tables drawn like the headline workload."""
    import torch
    from paper_2609_13031_amd import tfm
    from paper_2609_13031_amd.workloads import Workload, generate

    rows = []
    for D in (64, 128):
        N = 1024
        while N <= max_n:
            w = Workload("crossover", B=1, H=8, D=D, N=N, M=0, dtype="bf16", seed=N + D)
            g = {k: torch.from_numpy(v).to(torch.bfloat16).cuda() for k, v in generate(w).items() if k != "q_test"}
            o = torch.empty((1, N, 8, D), dtype=torch.bfloat16, device="cuda")
            ws = torch.empty(tfm.tfm_icl_attention_fp8_workspace_bytes(1, 8, D, N, 0), dtype=torch.uint8,
                             device="cuda")
            reps = max(3, min(50, int(2e12 / w.flops)))
            runs = {
                "fp8": lambda: tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], None, alpha=w.alpha,
                                                         out_dtype=torch.bfloat16, out=(o, None), workspace=ws),
                "bf16": lambda: tfm.tfm_icl_attention_bf16(g["q_train"], g["k"], g["v"], None, alpha=w.alpha,
                                                           out_dtype=torch.bfloat16, out=(o, None)),
            }
            res = {"D": D, "N": N}
            for name, fn in runs.items():
                fn()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(reps):
                    fn()
                e1.record()
                torch.cuda.synchronize()
                res[name + "_ms"] = round(e0.elapsed_time(e1) / reps, 4)
            res["fp8_tflops"] = round(w.flops / res["fp8_ms"] / 1e9, 1)
            res["bf16_tflops"] = round(w.flops / res["bf16_ms"] / 1e9, 1)
            res["speedup"] = round(res["bf16_ms"] / res["fp8_ms"], 3)
            log("crossover", res)
            rows.append(res)
            del g, o, ws
            N *= 2
    return {"crossover": rows, "call": "train-train only, B=1, H=8, bf16 in/out, FP8 time includes quantization"}


def noise_op(w, steps, warmup):
    """Eq. (3) on the K tensor of the workload (bf16 x, bf16 z), timed per call with HIP events on
    the stream the library launches on; HBM roofline on the algorithmic bytes x + z + out."""
    import torch
    from paper_2609_13031_amd import tfm

    shape = (w.B, w.N, w.H, w.D)
    gen = torch.Generator(device="cuda").manual_seed(5)
    x = torch.randn(shape, generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    z = torch.randn(shape, generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    out = torch.empty_like(x)
    ws = torch.empty(tfm.tfm_noise_per_head_workspace_bytes(w.B, w.H, w.N, w.D), dtype=torch.uint8, device="cuda")
    run = lambda: tfm.tfm_noise_per_head(x, z, 0.0265, out=out, workspace=ws)
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    algo = 3 * x.numel() * 2
    gbs = algo / ms / 1e6
    log("noise op %.4f ms, %.1f GB/s" % (ms, gbs))
    return {"noise_op": {"tensor": "K of %s: (B=%d, S=%d, H=%d, D=%d) bf16, z bf16" % (w.name, *shape),
                         "ms_per_call": round(ms, 4), "algorithmic_bytes": algo,
                         "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": 8000.0, "unit": "GB/s",
                                      "frac": round(gbs / 8000.0, 4)},
                         "design_bytes": 4 * x.numel() * 2, "steps": steps, "warmup": warmup}}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mid")
    ap.add_argument("--cpu-train-rows", type=int, default=4096,
                    help="train query rows per (table, head) of the oracle sample")
    ap.add_argument("--cpu-test-rows", type=int, default=1024,
                    help="test query rows per (table, head) of the oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--accuracy-rows", type=int, default=1024,
                    help="rows of the oracle sample also compared with fp64 attention (with the CPU baseline)")
    ap.add_argument("--no-bf16", action="store_true")
    ap.add_argument("--sdpa", action="store_true",
                    help="also time torch's scaled_dot_product_attention (flash backend, bf16) as context")
    ap.add_argument("--crossover", action="store_true",
                    help="instead of the headline step: FP8 (quantization included) vs bf16 for one train-train "
                         "call, B=1, H=8, N=1k..512k, D=64 and 128; prints one JSON line with the table")
    ap.add_argument("--crossover-max-n", type=int, default=1 << 19)
    ap.add_argument("--noise", action="store_true",
                    help="instead of the headline step: the Eq. (3) noise operator on the workload's K tensor; "
                         "prints one JSON line")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a 1 GiB device copy (for scaling HBM counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the FP8 ICL attention of each (table, head) is independent, "
              "and the library has no multi-GPU path (asked for --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    from paper_2609_13031_amd.workloads import WORKLOADS, generate

    w = WORKLOADS[args.workload]
    cpu = None
    if not (args.crossover or args.noise):
        log("generating", w)
        x = generate(w)
        if not args.no_cpu_baseline:
            # before anything touches the GPU: the pool's workers are forked from this process
            n = cpu_workers()
            log("cpu baseline (oracle) in %d processes" % n)
            cpu = cpu_baseline(x, w, min(args.cpu_train_rows, w.N), min(args.cpu_test_rows, w.M), ORACLE_BLOCK_KV, n)
            log("cpu baseline: %s" % cpu[0])

    import torch
    from paper_2609_13031_amd import tfm

    tfm.lib()
    if args.crossover:
        print(json.dumps(crossover(args.crossover_max_n)), flush=True)
        return
    if args.noise:
        print(json.dumps(noise_op(w, args.steps, args.warmup)), flush=True)
        return
    in_dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    dev = torch.device("cuda:0")
    g = {k: torch.from_numpy(v).to(in_dt).to(dev) for k, v in x.items()}
    out_dt = torch.bfloat16
    o_tr = torch.empty((w.B, w.N, w.H, w.D), dtype=out_dt, device=dev)
    o_te = torch.empty((w.B, w.M, w.H, w.D), dtype=out_dt, device=dev)
    ws = torch.empty(tfm.tfm_icl_attention_fp8_workspace_bytes(w.B, w.H, w.D, w.N, w.M), dtype=torch.uint8,
                     device=dev)

    def quantize():
        tfm.tfm_icl_attention_fp8_quantize(g["q_train"], g["k"], g["v"], g["q_test"], workspace=ws)

    def attend():
        tfm.tfm_icl_attention_fp8_attend(ws, w.B, w.H, w.D, w.N, w.M, alpha=w.alpha, out_dtype=out_dt,
                                         out=(o_tr, o_te))

    log("warmup", args.warmup)
    for _ in range(args.warmup):
        quantize()
        attend()
    torch.cuda.synchronize()

    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    begin, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    begin.record()
    for i in range(K):
        ev[i][0].record()
        quantize()
        ev[i][1].record()
        attend()
        ev[i][2].record()
    end.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_wall) * 1e3
    total_ms = begin.elapsed_time(end)
    ms_step = total_ms / K
    q_ms = [e[0].elapsed_time(e[1]) for e in ev]
    a_ms = [e[1].elapsed_time(e[2]) for e in ev]
    attn_ms = sum(a_ms) / K
    quant_ms = sum(q_ms) / K
    log("fp8 step %.3f ms (quantize %.3f, attention %.3f), wall %.1f ms for %d steps" %
        (ms_step, quant_ms, attn_ms, wall_ms, K))

    # the shader clock over the first 60% of a second, identical run of the K steps
    def steps():
        for _ in range(K):
            quantize()
            attend()
    clock_ghz = live_clock(steps, 0.6 * K * ms_step)
    log("shader clock during the FP8 steps: %s GHz" % clock_ghz)

    bf16 = None
    if not args.no_bf16:
        gb = g if in_dt == torch.bfloat16 else {k: v.to(torch.bfloat16) for k, v in g.items()}
        b_tr, b_te = torch.empty_like(o_tr), torch.empty_like(o_te)
        run_bf16 = lambda: tfm.tfm_icl_attention_bf16(gb["q_train"], gb["k"], gb["v"], gb["q_test"], alpha=w.alpha,
                                                      out_dtype=out_dt, out=(b_tr, b_te))
        for _ in range(args.warmup):
            run_bf16()
        torch.cuda.synchronize()
        b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        b0.record()
        for _ in range(K):
            run_bf16()
        b1.record()
        torch.cuda.synchronize()
        bf16_ms = b0.elapsed_time(b1) / K
        bf16 = {"ms": round(bf16_ms, 4), "tflops": round(w.flops / bf16_ms / 1e9, 2)}
        log("bf16 %.3f ms" % bf16_ms)

    sdpa = None
    if args.sdpa:
        sdpa = time_sdpa(g, w, K, args.warmup)

    if args.copy_calibration:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        log("copy calibration: 3 x 1 GiB device copies done")

    value = w.flops / ms_step / 1e9                      # TFLOP/s
    achieved = w.flops / attn_ms / 1e9
    # the HBM counter summaries were taken on the headline workload only
    counted = w.name == "mid"
    traffic = counter_value("hbm_bytes_per_launch", "attn_fp8.hip") if counted else None
    in_bytes = 4 if w.dtype == "f32" else 2
    q_elems = (3 * w.N + w.M) * w.B * w.H * w.D
    q_algo = q_elems * (in_bytes + 1)                    # inputs read once, e4m3 codes written
    q_gbs = q_algo / quant_ms / 1e6
    result = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "fp8_e4m3", "data": "synthetic",
        "config": {"workload": "%s: B=%d tables, H=%d heads, D=%d, N_train=%d, N_test=%d, %s in, bf16 out"
                               % (w.name, w.B, w.H, w.D, w.N, w.M, w.dtype),
                   "B": w.B, "H": w.H, "D": w.D, "N_train": w.N, "N_test": w.M, "in_dtype": w.dtype,
                   "out_dtype": "bf16", "parallelism": "single GPU"},
        "stages_ms": {"quantize": round(quant_ms, 4), "attention": round(attn_ms, 4),
                      "quantize_median": round(float(np.median(q_ms)), 4),
                      "attention_median": round(float(np.median(a_ms)), 4)},
        "speedup_vs_bf16": round(bf16["ms"] / ms_step, 3) if bf16 else None,
        "attention_only_speedup_vs_bf16": round(bf16["ms"] / attn_ms, 3) if bf16 else None,
        "bf16": bf16,
        "torch_sdpa_bf16_context": sdpa,
        "roofline": {"kernel": "attn_fp8_kernel", "bound": "mfma", "achieved": round(achieved, 2),
                     "peak": FP8_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / FP8_PEAK_TFLOPS, 4),
                     "traffic": traffic, "counters": sq_figures(w),
                     "live_clock": None if clock_ghz is None else {
                         "shader_ghz": round(clock_ghz, 3), "tflops_per_ghz": round(achieved / clock_ghz, 1),
                         "how": "s_memtime over s_memrealtime, read by one sleeping wave beside a second run of the "
                                "timed steps"}},
        "alu_roofline": {"kernel": "attn_fp8_kernel", "bound": "alu", "achieved": round(achieved, 2),
                         "peak": round(ALU_SCORES_PER_S * 4 * w.D / 1e12, 1), "unit": "TFLOP/s",
                         "frac": round(achieved / (ALU_SCORES_PER_S * 4 * w.D / 1e12), 4),
                         "note": "VALU issue ceiling of the softmax work per score (exp, fma, e4m3 convert, max)"},
        "quantize_hbm": {"stage": "slice maxima, then scales and codes of Q_train, K, V, Q_test (2 launches)",
                         "ms": round(quant_ms, 4), "algorithmic_bytes": q_algo, "achieved": round(q_gbs, 1),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(q_gbs / HBM_PEAK_GBS, 4),
                         "traffic": counter_value("quantize_stage_hbm_bytes_per_step", "quantize.hip") if counted else None},
    }
    if cpu is not None:
        if tfm.tfm_icl_attention_fp8_block_kv(w.D) != ORACLE_BLOCK_KV:
            raise RuntimeError("the oracle sample replayed key blocks of %d; the library uses %d"
                               % (ORACLE_BLOCK_KV, tfm.tfm_icl_attention_fp8_block_kv(w.D)))
        result["cpu_baseline"], o_qp, qz = cpu
        # one more FP8 call (and bf16 call) with fp32 outputs, outside the timed region
        f_tr, f_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha,
                                               workspace=ws)
        r = min(args.accuracy_rows, len(o_qp))
        gpu_fp8 = f_tr[0, :r, 0].cpu().numpy()
        gpu_bf16 = None
        if not args.no_bf16:
            gpu_bf16 = tfm.tfm_icl_attention_bf16(gb["q_train"][:1], gb["k"][:1], gb["v"][:1], None,
                                                  alpha=w.alpha)[0][0, :r, 0].cpu().numpy()
        del f_tr, f_te
        log("accuracy on %d rows" % r)
        result["accuracy"] = accuracy(x, w, o_qp, qz, gpu_fp8, gpu_bf16, r)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
