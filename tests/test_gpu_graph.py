"""The library calls record into a HIP graph (torch.cuda.CUDAGraph): they
launch kernels only (no allocation, memset or synchronisation), so a captured
forward + backward replays to the eager results. Each graph is replayed
several times with eager work on the outputs in between."""
import pytest

from paper_2606_20005_amd import inputs
from parity_utils import to_gpu_f32, upload

pytestmark = pytest.mark.gpu

ALL = ("dq1", "dk1", "dq2", "dk2")


def _capture(fn):
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()   # warm-up on a side stream, as capture requires
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fn()
    return graph


def _replays(graph, outputs, check, n=4):
    import torch
    for _ in range(n):
        for t in outputs:
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        check()


def test_graph_separate_path(gpu_lib):
    """Single-pass forward and the separate backward kernels, all four
    gradients, causal with ragged extents: every replay is bitwise equal to the
    eager call (these kernels have a fixed summation order)."""
    import torch
    d = inputs.make("tiny", B=2, H=2, n_q=300, n_k=700)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    ref_f = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, True, 0)
    ref_b = gpu_lib.bwd(q1, k1, q2, k2, *ref_f, g, w.s1, w.s2, True, 0, want=ALL)
    torch.cuda.synchronize()
    fo = tuple(torch.empty_like(t) for t in ref_f)
    bo = {n: torch.empty_like(t) for n, t in zip(ALL, ref_b)}

    def step():
        gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, True, 0, out=fo)
        gpu_lib.bwd(q1, k1, q2, k2, *fo, g, w.s1, w.s2, True, 0, want=ALL, out=bo)

    def check():
        for a, b in zip(fo, ref_f):
            assert torch.equal(a, b)
        for n, t in zip(ALL, ref_b):
            assert torch.equal(bo[n], t), n

    _replays(_capture(step), list(fo) + list(bo.values()), check)


def test_graph_adaptive_paths(gpu_lib):
    """Split-K forward (caller-owned workspace) and the fused backward (its dQ
    zeroed by a fill kernel inside the graph): replays match the eager call,
    dQ up to the order of its atomic adds."""
    import torch
    d = inputs.make("tiny", B=2, H=2, n_q=16, n_k=4000)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    W = gpu_lib.split_count(2, 2, 16, 4000, w.d1, w.d2)
    assert W > 1 and gpu_lib.bwd_choose(2, 2, 16, 4000, w.d1, w.d2) == "fused"
    ws = torch.empty(gpu_lib.split_workspace_bytes(2, 2, 16, W) // 4, dtype=torch.float32, device="cuda")
    ref_f = gpu_lib.fwd_split(q1, k1, q2, k2, w.s1, w.s2, False, 0, splits=W, workspace=ws)
    ref_b = gpu_lib.bwd(q1, k1, q2, k2, *ref_f, g, w.s1, w.s2, False, 0, want=("dq2", "dk2"), strategy="fused")
    torch.cuda.synchronize()
    fo = tuple(torch.empty_like(t) for t in ref_f)
    bo = {"dq2": torch.empty_like(ref_b[2]), "dk2": torch.empty_like(ref_b[3])}

    def step():
        gpu_lib.fwd_split(q1, k1, q2, k2, w.s1, w.s2, False, 0, splits=W, workspace=ws, out=fo)
        gpu_lib.bwd(q1, k1, q2, k2, *fo, g, w.s1, w.s2, False, 0, want=("dq2", "dk2"), out=bo, strategy="fused")

    def check():
        for a, b in zip(fo, ref_f):
            assert torch.equal(a, b)
        assert torch.equal(bo["dk2"], ref_b[3])
        assert torch.allclose(bo["dq2"], ref_b[2], rtol=1e-5, atol=1e-7)

    _replays(_capture(step), list(fo) + list(bo.values()), check)
