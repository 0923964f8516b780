"""The allocation-free split-K forward (streamkl_fwd_split_noalloc) against
the split-K forward with a caller workspace (streamkl_fwd_split), through the
C ABI, on two calls in a row, the second with a smaller input: the static
scratch keeps the first call's partials, and every partial the second call
reads must be its own. Both share their kernels, so the results must agree
bit for bit (which implies the row tolerance of the parity tests), and they
are checked against the oracle on sampled rows as well."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2606_20005_amd import inputs
from parity_utils import check_rows, upload

pytestmark = pytest.mark.gpu


def _split_with_workspace(sk, q1, k1, q2, k2, w, causal, splits):
    import torch
    B, H, NQ, NK = q1.shape[0], q1.shape[1], q1.shape[2], k1.shape[2]
    need = sk.split_workspace_bytes(B, H, NQ, splits)
    ws = torch.full((need // 4,), float("nan"), dtype=torch.float32, device="cuda")
    return sk.fwd_split(q1, k1, q2, k2, w.s1, w.s2, causal, 0, splits=splits, workspace=ws)


def _noalloc_c_abi(sk, q1, k1, q2, k2, w, causal, splits):
    import torch
    B, H, NQ, NK = q1.shape[0], q1.shape[1], q1.shape[2], k1.shape[2]
    out = [torch.full((B, H, NQ), float("nan"), dtype=torch.float32, device="cuda") for _ in range(3)]
    p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    st = sk.lib.streamkl_fwd_split_noalloc(p(q1), p(k1), p(q2), p(k2), B, H, NQ, NK, w.d1, w.d2, w.s1, w.s2,
                                           int(causal), 0, splits, p(out[0]), p(out[1]), p(out[2]),
                                           ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == sk.OK, sk.lib.streamkl_strerror(st)
    return out


@pytest.mark.parametrize("causal", [False, True])
def test_noalloc_matches_workspace_split_twice(gpu_lib, causal):
    import torch
    cases = (dict(B=16, H=1, n_q=64, n_k=8192), dict(B=3, H=2, n_q=20, n_k=1000))
    for i, over in enumerate(cases):
        d = inputs.make("mid", **over)
        w = d["w"]
        print(f"[noalloc] call {i}: causal={causal} {over}", flush=True)
        q1, k1, q2, k2 = upload(d)
        splits = gpu_lib.split_count(w.B, w.H, w.n_q, w.n_k, w.d1, w.d2)
        assert splits > 1
        assert gpu_lib.split_workspace_bytes(w.B, w.H, w.n_q, splits) <= gpu_lib.NOALLOC_SCRATCH_BYTES
        ref = _split_with_workspace(gpu_lib, q1, k1, q2, k2, w, causal, splits)
        got = _noalloc_c_abi(gpu_lib, q1, k1, q2, k2, w, causal, splits)
        torch.cuda.synchronize()
        for name, a, b in zip(("kl", "lse1", "lse2"), got, ref):
            assert torch.equal(a, b), name
        rows = np.array([0, 1, w.n_q // 2, w.n_q - 1])
        args = (d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, 0)
        for b_ in (0, w.B - 1):
            rk, r1, r2 = oracle.forward_rows(*args, b_, w.H - 1, rows)
            ridx = torch.as_tensor(rows, device="cuda")
            check_rows("kl", got[0][b_, w.H - 1, ridx].cpu().numpy(), rk)
            check_rows("lse1", got[1][b_, w.H - 1, ridx].cpu().numpy(), r1)
            check_rows("lse2", got[2][b_, w.H - 1, ridx].cpu().numpy(), r2)


def test_noalloc_allocates_nothing(gpu_lib):
    import torch
    d = inputs.make("mid", B=16, H=1, n_q=16, n_k=4096)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    out = tuple(torch.empty((w.B, w.H, w.n_q), dtype=torch.float32, device="cuda") for _ in range(3))
    gpu_lib.fwd_split_noalloc(q1, k1, q2, k2, w.s1, w.s2, False, 0, out=out)
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    alloc0 = torch.cuda.memory_allocated()
    for _ in range(3):
        gpu_lib.fwd_split_noalloc(q1, k1, q2, k2, w.s1, w.s2, False, 0, out=out)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == alloc0
    assert torch.cuda.mem_get_info()[0] == free0
    assert float(out[0].min()) >= -1e-3
