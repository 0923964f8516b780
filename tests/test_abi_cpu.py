"""The C-ABI library loads on a host without a GPU, exports every entry point
declared in include/streamkl.h, and rejects bad arguments before enqueuing
anything (no compute call is made here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "streamkl.h")


@pytest.fixture(scope="module")
def sk():
    from paper_2606_20005_amd import streamkl
    return streamkl


def declared_entry_points():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(streamkl_\w+)\s*\(", text)))


def test_header_declares_expected_entry_points(sk):
    assert declared_entry_points() == sorted(sk.ENTRY_POINTS)


def test_library_exports_every_declared_symbol(sk):
    for name in declared_entry_points():
        assert hasattr(sk.lib, name), name


def test_version_and_strerror(sk):
    assert sk.version().startswith("streamkl ") and "gfx950" in sk.version()
    for st in range(5):
        assert sk.lib.streamkl_strerror(st)
    assert b"unknown" in sk.lib.streamkl_strerror(99)
    assert [d for d in range(0, 300) if sk.supported_head_dim(d)] == list(range(32, 257, 32))


FAKE = ctypes.c_void_p(0x100000)        # 16-byte aligned, never dereferenced on error paths
MIS = ctypes.c_void_p(0x100008)         # 8-byte aligned only


def fwd_call(sk, **kw):
    a = dict(Q1=FAKE, K1=FAKE, Q2=FAKE, K2=FAKE, B=1, H=2, NQ=64, NK=64, d1=64, d2=64, s1=0.125, s2=0.125,
             causal=0, direction=0, kl=FAKE, lse1=FAKE, lse2=FAKE, stream=None)
    a.update(kw)
    return sk.lib.streamkl_fwd(a["Q1"], a["K1"], a["Q2"], a["K2"], a["B"], a["H"], a["NQ"], a["NK"], a["d1"],
                               a["d2"], a["s1"], a["s2"], a["causal"], a["direction"], a["kl"], a["lse1"],
                               a["lse2"], a["stream"])


def bwd_call(sk, **kw):
    a = dict(Q1=FAKE, K1=FAKE, Q2=FAKE, K2=FAKE, B=1, H=2, NQ=64, NK=64, d1=64, d2=64, s1=0.125, s2=0.125,
             causal=0, direction=0, kl=FAKE, lse1=FAKE, lse2=FAKE, dkl=None, dQ1=None, dK1=None, dQ2=FAKE,
             dK2=FAKE, stream=None)
    a.update(kw)
    return sk.lib.streamkl_bwd(a["Q1"], a["K1"], a["Q2"], a["K2"], a["B"], a["H"], a["NQ"], a["NK"], a["d1"],
                               a["d2"], a["s1"], a["s2"], a["causal"], a["direction"], a["kl"], a["lse1"],
                               a["lse2"], a["dkl"], a["dQ1"], a["dK1"], a["dQ2"], a["dK2"], a["stream"])


@pytest.mark.parametrize("call", [fwd_call, bwd_call])
@pytest.mark.parametrize("kw,expect", [
    (dict(Q1=None), 1), (dict(K2=None), 1), (dict(kl=None), 1), (dict(lse2=None), 1),
    (dict(B=-1), 1), (dict(NQ=-3), 1), (dict(NK=-1), 1), (dict(causal=2), 1), (dict(direction=5), 1),
    (dict(s1=0.0), 1), (dict(s2=-0.5), 1), (dict(s1=float("inf")), 1), (dict(s2=float("nan")), 1),
    (dict(Q1=MIS), 1), (dict(K1=MIS), 1),
    (dict(d1=80), 2), (dict(d2=16), 2), (dict(d2=288), 2), (dict(d1=512), 2), (dict(B=70000, H=70000), 2),
    (dict(B=0), 0), (dict(H=0), 0), (dict(NQ=0, Q1=None, Q2=None, kl=None, lse1=None, lse2=None,
                                          dQ2=None, dK2=None, dK1=FAKE), None),
])
def test_argument_checks(sk, call, kw, expect):
    if expect is None:          # N_Q = 0: forward is a no-op; backward would zero-fill dK (a launch)
        if call is fwd_call:
            assert call(sk, **kw) == 0
        return
    assert call(sk, **kw) == expect


def bwd_ex_call(sk, strategy=0, **kw):
    a = dict(Q1=FAKE, K1=FAKE, Q2=FAKE, K2=FAKE, B=1, H=2, NQ=64, NK=64, d1=64, d2=64, s1=0.125, s2=0.125,
             causal=0, direction=0, kl=FAKE, lse1=FAKE, lse2=FAKE, dkl=None, dQ1=None, dK1=None, dQ2=FAKE,
             dK2=FAKE, stream=None)
    a.update(kw)
    return sk.lib.streamkl_bwd_ex(a["Q1"], a["K1"], a["Q2"], a["K2"], a["B"], a["H"], a["NQ"], a["NK"], a["d1"],
                                  a["d2"], a["s1"], a["s2"], a["causal"], a["direction"], a["kl"], a["lse1"],
                                  a["lse2"], a["dkl"], a["dQ1"], a["dK1"], a["dQ2"], a["dK2"], strategy, a["stream"])


@pytest.mark.parametrize("strategy", [0, 1, 2])
@pytest.mark.parametrize("kw,expect", [
    (dict(Q1=None), 1), (dict(kl=None), 1), (dict(NK=-1), 1), (dict(causal=2), 1), (dict(s2=0.0), 1),
    (dict(K2=MIS), 1), (dict(dQ2=ctypes.c_void_p(0x100002)), 1), (dict(dQ2=None, dK2=None), 1),
    (dict(d1=100), 2), (dict(B=0), 0), (dict(NK=5_000_000, d1=256), 2),
])
def test_bwd_ex_argument_checks(sk, strategy, kw, expect):
    assert bwd_ex_call(sk, strategy, **kw) == expect


def test_bwd_ex_rejects_unknown_strategy(sk):
    assert bwd_ex_call(sk, 3) == 1
    assert bwd_ex_call(sk, -1) == 1


def test_bwd_ex_fused_needs_lds_room(sk):
    # all four gradients at d1 = d2 = 256: the fused kernel's LDS working set
    # exceeds 160 KiB, so the explicit request is unsupported (nothing launched)
    four = dict(d1=256, d2=256, dQ1=FAKE, dK1=FAKE, dQ2=FAKE, dK2=FAKE)
    assert bwd_ex_call(sk, 2, **four) == 2


def test_extent_limit_of_32_bit_slabs(sk):
    # N * max(d) * 4 must stay below 2^32 bytes per head
    assert fwd_call(sk, NK=4_194_304, d1=256) == 2
    assert bwd_call(sk, NQ=4_194_304, d2=256) == 2
    assert fwd_call(sk, NQ=0, NK=4_194_303, d1=256, Q1=None, Q2=None) == 0


def test_bwd_choose_follows_the_adaptive_rule(sk):
    """Fused when T_Q * 8 <= T_K and T_Q <= 4 (128-row tiles), the fused kernel
    exists for the request, and some dQ is requested."""
    assert sk.bwd_choose(16, 1, 16, 65536, 128, 128) == "fused"       # decode: T_Q = 1, T_K = 512
    assert sk.bwd_choose(1, 32, 16384, 16384, 128, 128) == "separate"  # T_Q = T_K = 128
    assert sk.bwd_choose(1, 8, 8192, 131072, 192, 64, True) == "separate"  # T_Q = 64 > 4
    assert sk.bwd_choose(1, 1, 512, 4096, 64, 64) == "fused"          # 4 * 8 <= 32 (boundary)
    assert sk.bwd_choose(1, 1, 512, 3968, 64, 64) == "separate"       # 4 * 8 > 31
    assert sk.bwd_choose(1, 1, 513, 1 << 20, 64, 64) == "separate"    # T_Q = 5 > 4
    assert sk.bwd_choose(1, 1, 16, 65536, 64, 64, want=("dk2",)) == "separate"   # no dQ: dK kernel only
    assert sk.bwd_choose(1, 1, 16, 65536, 256, 256, want=("dq1", "dk1", "dq2", "dk2")) == "separate"
    assert sk.bwd_choose(1, 1, 16, 65536, 128, 128, want=("dq1", "dk1", "dq2", "dk2")) == "fused"
    for bad in (dict(B=-1), dict(n_k=-5), dict(d1=48), dict(want=())):
        a = dict(B=1, H=1, n_q=16, n_k=4096, d1=64, d2=64, causal=False, direction=0, want=("dq2", "dk2"))
        a.update(bad)
        with pytest.raises(sk.StreamKLError):
            sk.bwd_choose(**a)
    assert sk.lib.streamkl_bwd_choose(1, 1, 16, 4096, 64, 64, 2, 0, 12) == 0    # causal flag
    assert sk.lib.streamkl_bwd_choose(1, 1, 16, 4096, 64, 64, 0, 2, 12) == 0    # direction
    assert sk.lib.streamkl_bwd_choose(1, 1, 16, 4096, 64, 64, 0, 0, 16) == 0    # unknown gradient bit


def test_bwd_needs_one_gradient(sk):
    assert bwd_call(sk, dQ2=None, dK2=None) == 1


def test_bwd_misaligned_fp32(sk):
    assert bwd_call(sk, dQ2=ctypes.c_void_p(0x100002)) == 1
    assert bwd_call(sk, dkl=ctypes.c_void_p(0x100001)) == 1


def test_python_binding_rejects_cpu_tensors(sk):
    import torch
    x = torch.zeros((1, 1, 4, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        sk.fwd(x, x, x, x)


def split_call(sk, **kw):
    a = dict(Q1=FAKE, K1=FAKE, Q2=FAKE, K2=FAKE, B=1, H=2, NQ=16, NK=4096, d1=64, d2=64, s1=0.125, s2=0.125,
             causal=0, direction=0, splits=4, ws=FAKE, ws_bytes=1 << 20, kl=FAKE, lse1=FAKE, lse2=FAKE,
             stream=None)
    a.update(kw)
    return sk.lib.streamkl_fwd_split(a["Q1"], a["K1"], a["Q2"], a["K2"], a["B"], a["H"], a["NQ"], a["NK"], a["d1"],
                                     a["d2"], a["s1"], a["s2"], a["causal"], a["direction"], a["splits"], a["ws"],
                                     a["ws_bytes"], a["kl"], a["lse1"], a["lse2"], a["stream"])


@pytest.mark.parametrize("kw,expect", [
    (dict(splits=0), 1), (dict(splits=-2), 1), (dict(ws=None), 1), (dict(ws=ctypes.c_void_p(0x100002)), 1),
    (dict(ws_bytes=20 * 4 * 2 * 16 - 1), 1), (dict(kl=None), 1), (dict(Q1=None), 1), (dict(d2=72), 2),
    (dict(B=0), 0), (dict(NQ=0, ws=None, Q1=None, Q2=None, kl=None, lse1=None, lse2=None), 0),
])
def test_split_argument_checks(sk, kw, expect):
    assert split_call(sk, **kw) == expect


def test_split_workspace_bytes(sk):
    # five fp32 row statistics per split, per row (m1, l1, m2, l2, acc)
    assert sk.split_workspace_bytes(2, 3, 17, 5) == 20 * 5 * 2 * 3 * 17
    assert sk.split_workspace_bytes(2, 3, 17, 1) == 0
    assert sk.split_workspace_bytes(-1, 3, 17, 4) == 0


def test_split_count_follows_the_adaptive_rule(sk):
    """W = 1 once the single-pass grid reaches the target of 512 workgroups,
    otherwise floor(512 / P_base) capped by the number of 32-key tiles."""
    # 16 heads of 16 query rows (one 32-row workgroup each) over 64K keys: 512 / 16
    assert sk.split_count(16, 1, 16, 65536, 128, 128) == 32
    # one query row, 4 heads: 512 / 4 = 128 chunks
    assert sk.split_count(1, 4, 1, 1 << 20, 64, 64) == 128
    # a 16K x 16K head set already launches 2048 workgroups of 256 rows
    assert sk.split_count(1, 32, 16384, 16384, 128, 128) == 1
    # 8 heads of 8192 rows: 256 workgroups of 256 rows -> 2
    assert sk.split_count(1, 8, 8192, 131072, 192, 64) == 2
    # capped by the tiles of a short key range: 40 keys are 2 tiles
    assert sk.split_count(1, 1, 1, 40, 128, 128) == 2
    assert sk.split_count(1, 1, 1, 0, 128, 128) == 1
    # invalid or unsupported
    assert sk.split_count(-1, 1, 1, 1, 128, 128) == 0
    assert sk.split_count(1, 1, 1, 1, 80, 128) == 0


def test_split_merge_grid_limit(sk):
    """2^34 rows split in two: every per-head extent and the partial grid are
    within limits, but one merge workgroup per four rows would exceed the
    launch grid; the call is refused before anything is launched."""
    big = dict(B=1024, H=1024, NQ=16384, NK=64, splits=2, ws_bytes=1 << 62)
    assert split_call(sk, **big) == 2
    # 2^31 rows pass the grid checks and stop at the next one (no output pointer): nothing is launched
    assert split_call(sk, **dict(big, B=128, kl=None)) == 1


def noalloc_call(sk, **kw):
    a = dict(Q1=FAKE, K1=FAKE, Q2=FAKE, K2=FAKE, B=16, H=1, NQ=64, NK=65536, d1=128, d2=128, s1=0.125, s2=0.125,
             causal=0, direction=0, splits=32, kl=FAKE, lse1=FAKE, lse2=FAKE, stream=None)
    a.update(kw)
    return sk.lib.streamkl_fwd_split_noalloc(a["Q1"], a["K1"], a["Q2"], a["K2"], a["B"], a["H"], a["NQ"], a["NK"],
                                             a["d1"], a["d2"], a["s1"], a["s2"], a["causal"], a["direction"],
                                             a["splits"], a["kl"], a["lse1"], a["lse2"], a["stream"])


@pytest.mark.parametrize("kw,expect", [
    (dict(Q1=None), 1), (dict(kl=None), 1), (dict(splits=0), 1), (dict(causal=3), 1), (dict(d2=40), 2),
    (dict(B=0), 0), (dict(NQ=0), 0),
    # partials of 20 * W * B * H * N_Q bytes must fit the static scratch
    (dict(NQ=8192, splits=32), 4), (dict(B=1, NQ=1 << 20, splits=2), 4),
])
def test_noalloc_argument_checks(sk, kw, expect):
    assert noalloc_call(sk, **kw) == expect


def test_noalloc_scratch_limit_is_the_header_constant(sk):
    text = open(HEADER).read()
    m = re.search(r"#define STREAMKL_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == sk.NOALLOC_SCRATCH_BYTES == 16 << 20
    # largest W for B*H*N_Q = 1024 rows that still fits: 20 * W * 1024 <= 16 MiB
    w_max = sk.NOALLOC_SCRATCH_BYTES // (20 * 1024)
    assert sk.split_workspace_bytes(16, 1, 64, w_max) <= sk.NOALLOC_SCRATCH_BYTES
    assert noalloc_call(sk, splits=w_max + 1) == sk.ERR_SCRATCH_LIMIT


def act_fwd_call(sk, **kw):
    a = dict(Q1=FAKE, K1=FAKE, Q2=FAKE, K2=FAKE, B=1, H=2, NQ=64, NK=64, d1=64, d2=64, s1=0.125, s2=0.125,
             causal=0, direction=0, act=1, kl=FAKE, st1=None, st2=None, stream=None)
    a.update(kw)
    return sk.lib.streamkl_fwd_act(a["Q1"], a["K1"], a["Q2"], a["K2"], a["B"], a["H"], a["NQ"], a["NK"], a["d1"],
                                   a["d2"], a["s1"], a["s2"], a["causal"], a["direction"], a["act"], a["kl"],
                                   a["st1"], a["st2"], a["stream"])


def act_bwd_call(sk, **kw):
    a = dict(Q1=FAKE, K1=FAKE, Q2=FAKE, K2=FAKE, B=1, H=2, NQ=64, NK=64, d1=64, d2=64, s1=0.125, s2=0.125,
             causal=0, direction=0, act=1, kl=None, st1=None, st2=None, dkl=None, dQ1=None, dK1=None, dQ2=FAKE,
             dK2=FAKE, stream=None)
    a.update(kw)
    return sk.lib.streamkl_bwd_act(a["Q1"], a["K1"], a["Q2"], a["K2"], a["B"], a["H"], a["NQ"], a["NK"], a["d1"],
                                   a["d2"], a["s1"], a["s2"], a["causal"], a["direction"], a["act"], a["kl"],
                                   a["st1"], a["st2"], a["dkl"], a["dQ1"], a["dK1"], a["dQ2"], a["dK2"], a["stream"])


@pytest.mark.parametrize("call", [act_fwd_call, act_bwd_call])
@pytest.mark.parametrize("kw,expect", [
    (dict(act=2), 1), (dict(act=-1), 1), (dict(Q1=None), 1), (dict(K2=None), 1), (dict(NQ=-1), 1),
    (dict(s1=0.0), 1), (dict(causal=2), 1), (dict(Q2=MIS), 1), (dict(d1=112), 2), (dict(B=0), 0),
])
def test_activation_argument_checks(sk, call, kw, expect):
    assert call(sk, **kw) == expect


def test_activation_specific_checks(sk):
    # sigmoid forward: kl required, the masses optional but aligned when given
    assert act_fwd_call(sk, kl=None) == 1
    assert act_fwd_call(sk, st1=ctypes.c_void_p(0x100002)) == 1
    # softmax through the act entry points keeps streamkl_fwd / streamkl_bwd's requirements
    assert act_fwd_call(sk, act=0, st1=None) == 1
    assert act_bwd_call(sk, act=0) == 1          # kl, lse1, lse2 missing
    # sigmoid backward: no saved statistic needed, one gradient needed
    assert act_bwd_call(sk, dQ2=None, dK2=None) == 1


def test_padded_head_dims_rules(sk):
    """Head dims 32, 96, 160, 224 run the kernels of the next multiple of 64:
    the split-K rule counts 128-row workgroups for them, and the adaptive
    backward rule never picks the fused kernel (its dQ wait counts every
    atomic of a 64-multiple head)."""
    assert sk.bwd_choose(16, 1, 16, 65536, 128, 128) == "fused"
    for d1, d2 in ((96, 128), (128, 32), (160, 224)):
        assert sk.bwd_choose(16, 1, 16, 65536, d1, d2) == "separate"
    # 16 heads of 16 rows: one 32-row workgroup each for 64-multiples, one
    # 128-row workgroup each for padded dims: the same P_base = 16 here
    assert sk.split_count(16, 1, 16, 65536, 96, 96) == 32
    assert sk.split_count(1, 1, 512, 65536, 96, 96) == 128          # 4 workgroups of 128 rows
    assert sk.split_count(1, 1, 512, 65536, 128, 128) == 256        # 2 workgroups of 256 rows
