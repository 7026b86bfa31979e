"""Execution models of the library's entry points: HIP graphs and concurrent streams.

The library never allocates and enqueues only kernels (no memset or copy nodes),
so a caller can capture a call into a HIP graph, for example the predict step of
a serving loop, and replay it.  Every replay must equal the eager call on the
same buffers bit for bit, with eager work of the program between replays, and a
replay must follow inputs changed in place (the graph reads the same addresses).
It keeps no state outside the caller's buffers, so calls on different streams
with their own workspaces may run concurrently.  The eager calls are checked
against the oracle in the other GPU tests."""
import pytest
import torch

from paper_2609_13031_amd import tfm
from paper_2609_13031_amd.workloads import Workload, generate
from parity import gpu_inputs

pytestmark = pytest.mark.gpu


def capture(fn):
    """Capture fn() into a CUDAGraph (HIP graph) after one warm-up call on a side stream."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fn()
    torch.cuda.synchronize()
    return graph


def test_fused_call_replays_equal_eager():
    w = Workload("graph", B=2, H=3, D=64, N=2000, M=300, dtype="bf16", seed=70)
    g = gpu_inputs(generate(w), torch.bfloat16)
    ws = torch.empty(tfm.tfm_icl_attention_fp8_workspace_bytes(w.B, w.H, w.D, w.N, w.M), dtype=torch.uint8,
                     device="cuda")
    o_tr = torch.empty((w.B, w.N, w.H, w.D), dtype=torch.bfloat16, device="cuda")
    o_te = torch.empty((w.B, w.M, w.H, w.D), dtype=torch.bfloat16, device="cuda")
    call = lambda: tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha,
                                             out_dtype=torch.bfloat16, out=(o_tr, o_te), workspace=ws)
    graph = capture(call)
    for rep in range(4):
        # the eager reference, into other buffers, between replays
        e_tr, e_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha,
                                               out_dtype=torch.bfloat16)
        o_tr.zero_()
        o_te.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_tr, e_tr) and torch.equal(o_te, e_te), rep
        # new inputs in place: the next replay must follow them
        g["q_test"].mul_(-1.5)
        g["v"].add_(0.25)


def test_fit_once_predict_replays_follow_new_test_batches():
    w = Workload("graph_fp", B=1, H=4, D=128, N=1500, M=256, dtype="bf16", seed=71)
    x = generate(w)
    g = gpu_inputs(x, torch.bfloat16)
    _, ws = tfm.tfm_icl_attention_fp8_fit(g["q_train"], g["k"], g["v"], alpha=w.alpha, m_max=w.M)
    q_static = g["q_test"].clone()
    o_static = torch.empty((w.B, w.M, w.H, w.D), dtype=torch.float32, device="cuda")
    graph = capture(lambda: tfm.tfm_icl_attention_fp8_predict(ws, q_static, w.N, alpha=w.alpha, out=o_static))
    gen = torch.Generator(device="cuda").manual_seed(72)
    for rep in range(4):
        batch = (torch.randn(q_static.shape, generator=gen, device="cuda") * (rep + 1)).to(torch.bfloat16)
        q_static.copy_(batch)
        graph.replay()
        torch.cuda.synchronize()
        want = tfm.tfm_icl_attention_fp8_predict(ws, batch, w.N, alpha=w.alpha)
        assert torch.equal(o_static, want), rep
        # and the same rows through the fused entry point (same fit state, same scales)
        _, f_te = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], batch, alpha=w.alpha)
        assert torch.equal(o_static, f_te), rep


def test_two_streams_with_their_own_workspaces_match_sequential_calls():
    # No state outside the caller's buffers: the same calls enqueued on two streams at once,
    # each with its own workspace and outputs, give the sequential results bit for bit.
    ws_args = []
    for seed in (73, 74):
        w = Workload("streams", B=1, H=4, D=64, N=5000, M=600, dtype="bf16", seed=seed)
        ws_args.append((w, gpu_inputs(generate(w), torch.bfloat16)))
    want = [tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
            for w, g in ws_args]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    got = [None, None]
    for rep in range(3):
        for i, ((w, g), s) in enumerate(zip(ws_args, streams)):
            with torch.cuda.stream(s):
                got[i] = tfm.tfm_icl_attention_fp8(g["q_train"], g["k"], g["v"], g["q_test"], alpha=w.alpha)
        torch.cuda.synchronize()
        for i in range(2):
            assert torch.equal(got[i][0], want[i][0]) and torch.equal(got[i][1], want[i][1]), (rep, i)
