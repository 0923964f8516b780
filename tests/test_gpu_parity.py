"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle, element
by element, on identical seeded bf16 inputs, at sizes that span several tiles
and a ragged tail. Full-size workloads are in test_gpu_fullsize.py."""
import numpy as np
import pytest

import oracle
from paper_2606_20005_amd import inputs
from parity_utils import check_grad, check_rows, to_gpu_f32, upload

pytestmark = pytest.mark.gpu

ALL = ("dq1", "dk1", "dq2", "dk2")


def run_case(sk, d, causal, direction, want=ALL, use_g=True, strategy="separate"):
    import torch
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    kl, l1, l2 = sk.fwd(q1, k1, q2, k2, w.s1, w.s2, causal, direction)
    g_np = d["g"] if use_g else None
    g = to_gpu_f32(g_np) if use_g else None
    grads = sk.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, direction, want=want, strategy=strategy)
    torch.cuda.synchronize()
    ref = oracle.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, direction, g_np)
    check_rows("kl", kl.cpu().numpy(), ref[0])
    check_rows("lse1", l1.cpu().numpy(), ref[1])
    check_rows("lse2", l2.cpu().numpy(), ref[2])
    out = {}
    for name, got, r in zip(ALL, grads, ref[3:]):
        if name in want:
            out[name] = check_grad(name, got.cpu().numpy(), r)
        else:
            assert got is None
    return out


@pytest.mark.parametrize("direction", [0, 1])
@pytest.mark.parametrize("causal", [False, True])
def test_tiny_all_outputs(gpu_lib, causal, direction):
    run_case(gpu_lib, inputs.make("tiny"), causal, direction)


def test_tiny_identical_exact_zero(gpu_lib):
    import torch
    d = inputs.make("tiny", "identical")
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    for causal in (False, True):
        kl, l1, l2 = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, causal, 0)
        grads = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, None, w.s1, w.s2, causal, 0, want=ALL)
        torch.cuda.synchronize()
        assert float(kl.abs().max()) <= 1e-6
        for t in grads:
            assert float(t.abs().max()) <= 1e-6


def test_tiny_q1_zero_uniform(gpu_lib):
    for causal in (False, True):
        run_case(gpu_lib, inputs.make("tiny", "q1zero"), causal, 0)


@pytest.mark.parametrize("nq,nk,causal", [
    (257, 257, False), (257, 257, True), (1000, 1000, True), (100, 300, True), (100, 300, False),
    (300, 100, True), (1, 1, False), (1, 200, True), (129, 33, False), (33, 129, True), (64, 1, True),
])
def test_ragged_shapes(gpu_lib, nq, nk, causal):
    d = inputs.make("tiny", B=1, H=2, n_q=nq, n_k=nk)
    run_case(gpu_lib, d, causal, 0)


@pytest.mark.parametrize("H,nq,nk,d1,d2", [(3, 400, 650, 128, 64), (2, 513, 513, 64, 128), (1, 129, 1000, 64, 64),
                                           (2, 700, 300, 128, 64)])
def test_causal_key_split_grids(gpu_lib, H, nq, nk, d1, d2):
    """Causal grids of at most 512 workgroups of 128 rows with d1 + d2 <= 192
    take the key-split forward (two wave halves over alternate key tiles of
    each ring stage, merged at the end): odd numbers of key tiles, ragged key
    tails, N_Q above and below N_K (rows with no key), all gradients."""
    d = inputs.make("tiny", B=1, H=H, n_q=nq, n_k=nk, d1=d1, d2=d2)
    run_case(gpu_lib, d, True, 0)
    run_case(gpu_lib, d, True, 1, want=("dq2", "dk2"))


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("late", [False, True])
def test_exponent_reference_moves_far_mid_row(gpu_lib, causal, late):
    """Key rows scaled by 64 (exact in bf16) put the logits of some query rows
    about 90 doublings per standard deviation away from everything else, in
    either direction depending on the row: rows whose dot product with them
    is positive have to move their exponent reference far up in the middle of
    the pass (late: keys 200-215, after six tiles), lane by lane, while other
    rows of the same waves do not; with the big keys first (late = False) the
    later keys fall far below the reference. The single-pass forward, the
    split forward (three chunks) and the gradients match the oracle."""
    import torch
    d = inputs.make("tiny", B=1, H=2, n_q=96, n_k=320)
    big = slice(200, 216) if late else slice(0, 16)
    d["K1"][:, :, big] *= np.float32(64.0)
    d["K2"][:, :, 100:104] *= np.float32(64.0)
    run_case(gpu_lib, d, causal, 0)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    kl, l1, l2 = gpu_lib.fwd_split(q1, k1, q2, k2, w.s1, w.s2, causal, 0, splits=3)
    torch.cuda.synchronize()
    ref = oracle.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, causal, 0, d["g"])
    check_rows("kl split", kl.cpu().numpy(), ref[0])
    check_rows("lse1 split", l1.cpu().numpy(), ref[1])
    check_rows("lse2 split", l2.cpu().numpy(), ref[2])


@pytest.mark.parametrize("d1", [64, 128, 192, 256])
@pytest.mark.parametrize("d2", [64, 128, 192, 256])
def test_every_head_dim_pair(gpu_lib, d1, d2):
    d = inputs.make("tiny", B=1, H=1, n_q=160, n_k=200, d1=d1, d2=d2, s1=d1 ** -0.5, s2=d2 ** -0.5)
    run_case(gpu_lib, d, True, 0)
    run_case(gpu_lib, d, False, 1)


@pytest.mark.parametrize("want", [("dq2", "dk2"), ("dq1", "dk1"), ("dq2",), ("dk1",), ("dq1", "dk2")])
@pytest.mark.parametrize("direction", [0, 1])
def test_gradient_subsets(gpu_lib, want, direction):
    d = inputs.make("tiny", B=1, H=1, n_q=200, n_k=230, d1=128, d2=64, s1=128 ** -0.5)
    run_case(gpu_lib, d, True, direction, want=want)


def test_upstream_gradient_none_is_ones(gpu_lib):
    run_case(gpu_lib, inputs.make("tiny", n_q=130, n_k=190), True, 0, use_g=False)


def _signed_g(shape, pattern):
    rng = np.random.default_rng(11)
    g = rng.uniform(0.5, 1.5, size=shape).astype(np.float32)
    if pattern == "mixed":            # random signs: almost every 32-row tile holds a negative g
        g *= rng.choice(np.float32([-1, 1]), size=shape)
    elif pattern == "some_tiles":     # one negative row in every other 32-row tile, zeros elsewhere
        g[..., 40::64] *= -1
        g[..., 3::50] = 0.0
        g[..., 7::64] = -0.0
    elif pattern == "magnitudes":     # |g| over many binades, zeros, signs
        g *= np.float32(2.0) ** rng.integers(-60, 40, size=shape).astype(np.float32)
        g[..., 5::9] *= -1
        g[..., ::13] = 0.0
    return g


@pytest.mark.parametrize("strategy", ["separate", "fused"])
@pytest.mark.parametrize("pattern", ["mixed", "some_tiles", "magnitudes"])
def test_upstream_gradient_signs(gpu_lib, pattern, strategy):
    """The kernels fold |g| of a row into its exponent offsets when they can
    (dQ: every row, the sign applied when written; dK: tiles whose g are all
    >= 0) and multiply by g otherwise: negative, zero and widely scaled g
    give the oracle's gradients on either side of that choice."""
    d = inputs.make("tiny", B=1, H=2, n_q=200, n_k=700)
    d["g"] = _signed_g(d["g"].shape, pattern)
    for causal in (False, True):
        run_case(gpu_lib, d, causal, 0, strategy=strategy)


@pytest.mark.parametrize("pattern", ["ones", "none", "mixed", "some_tiles", "magnitudes"])
@pytest.mark.parametrize("n_q,n_k,d1,d2,causal,direction", [
    (200, 700, 64, 64, True, 0), (1000, 300, 128, 64, False, 1), (33, 129, 64, 128, True, 0),
    (3, 300, 32, 32, False, 0), (257, 257, 96, 160, True, 1),
])
def test_dk_prepared_statistics_match_in_kernel_staging(gpu_lib, pattern, n_q, n_k, d1, d2, causal, direction):
    """When a dQ is requested too, the dK kernel streams row statistics that a
    prep kernel wrote into that dQ output beforehand; alone, it forms them
    itself. Same arithmetic: dK bit for bit equal either way, for every g
    pattern (folded and unfolded tiles, g absent), ragged tails, both
    directions, padded dims and a dQ too small to hold them (3 rows of d = 32:
    in-kernel path on both sides). The dQ written over the prepared values
    equals a dQ-only call bit for bit."""
    import torch
    d = inputs.make("tiny", B=1, H=2, n_q=n_q, n_k=n_k, d1=d1, d2=d2, s1=d1 ** -0.5, s2=d2 ** -0.5)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    g = None if pattern == "none" else to_gpu_f32(np.ones_like(d["g"]) if pattern == "ones"
                                                   else _signed_g(d["g"].shape, pattern))
    kl, l1, l2 = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, causal, direction)
    args = (q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, causal, direction)
    for pair in (("dq2", "dk2"), ("dq1", "dk1"), ALL):
        both = gpu_lib.bwd(*args, want=pair)
        dk_only = gpu_lib.bwd(*args, want=tuple(n for n in pair if n.startswith("dk")))
        dq_only = gpu_lib.bwd(*args, want=tuple(n for n in pair if n.startswith("dq")))
        torch.cuda.synchronize()
        for x, y, z in zip(both, dk_only, dq_only):
            if x is None:
                continue
            ref = y if y is not None else z
            assert torch.equal(x, ref), pair


@pytest.mark.parametrize("name,over,causal", [
    ("distill", dict(H=2, n_q=512, n_k=512), True),
    ("mid", dict(H=2, n_q=512, n_k=512), False),
    ("mid", dict(H=2, n_q=512, n_k=512), True),
    ("long", dict(H=2, n_q=640, n_k=640), True),
    ("indexer", dict(H=2, n_q=128, n_k=2048), True),
])
def test_workload_structures_reduced(gpu_lib, name, over, causal):
    """Each workload's value distribution and masking at a size the full oracle covers."""
    run_case(gpu_lib, inputs.make(name, **over), causal, 0)


@pytest.mark.parametrize("H,n,d1,d2", [(8, 640, 128, 64), (16, 333, 64, 64), (24, 300, 128, 128)])
def test_causal_rank_order_grids(gpu_lib, H, n, d1, d2):
    """Causal grids whose heads split evenly over the 8 XCDs and that fit in a
    few rounds of resident workgroups are handed out rank by rank per XCD (1,
    2 and 3 heads per XCD here, ragged row counts): every row and key of every
    head against the oracle, all four gradients, both directions."""
    d = inputs.make("distill", B=1, H=H, n_q=n, n_k=n, d1=d1, d2=d2, s1=d1 ** -0.5, s2=d2 ** -0.5)
    run_case(gpu_lib, d, True, 0)
    run_case(gpu_lib, d, True, 1, want=("dq1", "dk1", "dq2", "dk2"))


def test_causal_eight_wave_forward_reduced(gpu_lib):
    """1024 heads of 256 rows: B*H*ceil(N_Q/256) = 1024 workgroups, enough that
    the causal forward takes its eight-wave, 256-row configuration (the one the
    full causal mid workload runs) rather than the four-wave one for small
    grids. Every row of four heads against the oracle, and the four-wave
    configuration (two heads, same values) must agree with it."""
    import torch
    d = inputs.make("mid", H=1024, n_q=256, n_k=256)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    kl, l1, l2 = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, True, 0)
    _, _, dq2, dk2 = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, True, 0, want=("dq2", "dk2"))
    small = gpu_lib.fwd(q1[:, :2].contiguous(), k1[:, :2].contiguous(), q2[:, :2].contiguous(),
                        k2[:, :2].contiguous(), w.s1, w.s2, True, 0)
    torch.cuda.synchronize()
    for h in (0, 1, 517, 1023):
        sl = lambda x: x[:, h:h + 1]  # noqa: E731
        ref = oracle.backward(sl(d["Q1"]), sl(d["K1"]), sl(d["Q2"]), sl(d["K2"]), w.s1, w.s2, True, 0,
                              sl(d["g"]))
        check_rows("kl", kl[:, h:h + 1].cpu().numpy(), ref[0])
        check_rows("lse1", l1[:, h:h + 1].cpu().numpy(), ref[1])
        check_rows("lse2", l2[:, h:h + 1].cpu().numpy(), ref[2])
        check_grad("dq2", dq2[:, h:h + 1].cpu().numpy(), ref[5])
        check_grad("dk2", dk2[:, h:h + 1].cpu().numpy(), ref[6])
    for a, b in zip(small, (kl, l1, l2)):
        assert torch.allclose(a, b[:, :2], rtol=1e-5, atol=1e-5)


def test_deterministic_and_inputs_untouched(gpu_lib):
    import torch
    d = inputs.make("distill", H=2, n_q=384, n_k=384)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    before = [t.clone() for t in (q1, k1, q2, k2)]
    runs = []
    for _ in range(2):
        kl, l1, l2 = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, True, 0)
        g = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, None, w.s1, w.s2, True, 0, want=ALL)
        torch.cuda.synchronize()
        runs.append([t.cpu() for t in (kl, l1, l2, *g)])
    for a, b in zip(*runs):
        assert torch.equal(a, b)
    for a, b in zip(before, (q1, k1, q2, k2)):
        assert torch.equal(a, b)


def test_no_device_allocation_in_library(gpu_lib):
    import torch
    d = inputs.make("tiny", n_q=512, n_k=512)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    kl, l1, l2 = (torch.empty((1, 1, 512), dtype=torch.float32, device="cuda") for _ in range(3))
    grads = {n: torch.empty((1, 1, 512, 64), dtype=torch.float32, device="cuda") for n in ALL}
    gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, True, 0, out=(kl, l1, l2))
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    alloc0 = torch.cuda.memory_allocated()
    for _ in range(3):
        gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, True, 0, out=(kl, l1, l2))
        gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, None, w.s1, w.s2, True, 0, want=ALL, out=grads)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert torch.cuda.memory_allocated() == alloc0
    assert free1 == free0


def test_autograd_mean_objective(gpu_lib):
    """loss = mean over (b, h, i) of KL (the paper's objective); grads of q2, k2 only."""
    import torch
    d = inputs.make("distill", H=2, n_q=256, n_k=256)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    q2.requires_grad_(True)
    k2.requires_grad_(True)
    kl = gpu_lib.attention_kl(q1, k1, q2, k2, s1=w.s1, s2=w.s2, causal=True)
    loss = kl.mean()
    loss.backward()
    torch.cuda.synchronize()
    n = kl.numel()
    ref = oracle.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, True, 0, np.full(kl.shape, 1.0 / n))
    check_rows("kl", kl.detach().cpu().numpy(), ref[0])
    assert q1.grad is None and k1.grad is None
    # the autograd path returns bf16 gradients (the input dtype)
    check_grad("dq2", q2.grad.float().cpu().numpy(), ref[5])
    check_grad("dk2", k2.grad.float().cpu().numpy(), ref[6])


def test_invalid_arguments_raise(gpu_lib):
    d = inputs.make("tiny", n_q=64, n_k=64)
    q1, k1, q2, k2 = upload(d)
    with pytest.raises(gpu_lib.StreamKLError):
        gpu_lib.fwd(q1, k1, q2, k2, -1.0, 0.1)
    with pytest.raises(ValueError):
        gpu_lib.fwd(q1.float(), k1, q2, k2)


DIMS = (32, 64, 96, 128, 160, 192, 224, 256)


@pytest.mark.parametrize("d1", DIMS)
@pytest.mark.parametrize("d2", DIMS)
def test_every_head_dim_pair_multiple_of_32(gpu_lib, d1, d2):
    """Every pair of head dims {32, 64, ..., 256}: the ones that are not a
    multiple of 64 run the kernels of the next multiple of 64 on rows of their
    real length (the extra columns read as zeros). Causal FWD and non-causal
    REV alternate over the pairs; all four gradients, ragged extents."""
    d = inputs.make("tiny", B=1, H=1, n_q=150, n_k=190, d1=d1, d2=d2, s1=d1 ** -0.5, s2=d2 ** -0.5)
    k = DIMS.index(d1) + DIMS.index(d2)
    run_case(gpu_lib, d, k % 2 == 0, k // 2 % 2)


@pytest.mark.parametrize("d1,d2", [(32, 32), (96, 96), (160, 64), (224, 32)])
def test_padded_dims_split_and_strategies(gpu_lib, d1, d2):
    """Padded head dims through the split-K forward (decode-like shape) and the
    backward strategy rule, which keeps them on the separate kernels; asking
    for the fused kernel is refused."""
    import torch
    d = inputs.make("tiny", B=8, H=1, n_q=16, n_k=3000, d1=d1, d2=d2, s1=d1 ** -0.5, s2=d2 ** -0.5)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    W = gpu_lib.split_count(w.B, w.H, w.n_q, w.n_k, d1, d2)
    assert W > 1
    kl, l1, l2 = gpu_lib.fwd_split(q1, k1, q2, k2, w.s1, w.s2, True, 0, splits=W)
    one = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, True, 0)
    g = to_gpu_f32(d["g"])
    grads = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, True, 0, want=("dq2", "dk2"), strategy="auto")
    with pytest.raises(gpu_lib.StreamKLError):
        gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, True, 0, want=("dq2", "dk2"), strategy="fused")
    torch.cuda.synchronize()
    ref = oracle.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, True, 0, d["g"])
    for got in (kl, one[0]):
        check_rows("kl", got.cpu().numpy(), ref[0])
    check_rows("lse1", l1.cpu().numpy(), ref[1])
    check_rows("lse2", l2.cpu().numpy(), ref[2])
    check_grad("dq2", grads[2].cpu().numpy(), ref[5])
    check_grad("dk2", grads[3].cpu().numpy(), ref[6])


@pytest.mark.parametrize("d1,d2", [(32, 224), (96, 160)])
def test_padded_dims_sigmoid(gpu_lib, d1, d2):
    """The sigmoid-score path on padded head dims, all four gradients."""
    import torch
    from oracle import sigmoid_oracle as so
    d = inputs.make("tiny", B=1, H=2, n_q=140, n_k=170, d1=d1, d2=d2, s1=d1 ** -0.5, s2=d2 ** -0.5)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    kl, m1, m2 = gpu_lib.fwd_act(q1, k1, q2, k2, w.s1, w.s2, True, 1, "sigmoid")
    grads = gpu_lib.bwd(q1, k1, q2, k2, None, None, None, g, w.s1, w.s2, True, 1, want=ALL, activation="sigmoid")
    torch.cuda.synchronize()
    ref = so.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2, True, 1, d["g"])
    check_rows("kl", kl.cpu().numpy(), ref[0])
    check_rows("mass1", m1.cpu().numpy(), ref[1])
    check_rows("mass2", m2.cpu().numpy(), ref[2])
    for name, got, r in zip(ALL, grads, ref[3:]):
        check_grad(name, got.cpu().numpy(), r)


def test_padded_dims_eight_wave_grid(gpu_lib):
    """Padded head dims with enough rows that 64-multiples would take the
    eight-wave configuration (they take the four-wave padded one): 64 heads of
    384 rows, d1 = 96, d2 = 32, causal, four heads against the oracle."""
    import torch
    d = inputs.make("tiny", B=1, H=64, n_q=384, n_k=384, d1=96, d2=32, s1=96 ** -0.5, s2=32 ** -0.5)
    w = d["w"]
    q1, k1, q2, k2 = upload(d)
    g = to_gpu_f32(d["g"])
    kl, l1, l2 = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, True, 0)
    grads = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, g, w.s1, w.s2, True, 0, want=ALL)
    torch.cuda.synchronize()
    for h in (0, 17, 63):
        sl = lambda x: x[:, h:h + 1]  # noqa: E731
        ref = oracle.backward(sl(d["Q1"]), sl(d["K1"]), sl(d["Q2"]), sl(d["K2"]), w.s1, w.s2, True, 0, sl(d["g"]))
        check_rows("kl", kl[:, h:h + 1].cpu().numpy(), ref[0])
        check_rows("lse1", l1[:, h:h + 1].cpu().numpy(), ref[1])
        for name, got, r in zip(ALL, grads, ref[3:]):
            check_grad(name, got[:, h:h + 1].cpu().numpy(), r)


@pytest.mark.parametrize("where", ["query", "key"])
def test_nonfinite_inputs_stay_in_the_rows_that_see_them(gpu_lib, where):
    """The documented reach of a non-finite input. An infinity in query row 7
    of head 0 (or in column 5 of key row 20, causal, so that rows 0-19 never
    attend it): the forward outputs of the rows that do not see it are bit
    for bit those of finite inputs; their dQ rows too, except, for the key
    case, column 5 of dQ1 (a masked zero weight times the key row of the
    same tile); head 1 is untouched in every output, dK included."""
    import torch
    n = 120
    d = inputs.make("tiny", B=1, H=2, n_q=n, n_k=n)
    w = d["w"]
    clean = upload(d)
    bad_np = {k: d[k].copy() for k in ("Q1", "K1", "Q2", "K2")}
    cols = np.ones(d["Q1"].shape[-1], dtype=bool)
    if where == "query":
        bad_np["Q1"][0, 0, 7, 3] = np.inf
        causal, affected = False, np.zeros(n, dtype=bool)
        affected[7] = True
    else:
        bad_np["K1"][0, 0, 20, 5] = np.inf
        causal, affected = True, np.arange(n) >= 20
        cols[5] = False
    bad = upload(bad_np)
    outs = []
    for q1, k1, q2, k2 in (clean, bad):
        kl, l1, l2 = gpu_lib.fwd(q1, k1, q2, k2, w.s1, w.s2, causal, 0)
        grads = gpu_lib.bwd(q1, k1, q2, k2, kl, l1, l2, None, w.s1, w.s2, causal, 0, want=ALL)
        torch.cuda.synchronize()
        outs.append([t.cpu().numpy() for t in (kl, l1, l2, *grads)])
    (kl0, a0, b0, q10, k10, q20, k20), (kl1, a1, b1, q11, k11, q21, k21) = outs
    for x, y in zip(outs[0], outs[1]):   # head 1
        assert np.array_equal(x[0, 1], y[0, 1])
    keep = ~affected
    for x, y in ((kl0, kl1), (a0, a1), (b0, b1), (q20, q21)):
        assert np.array_equal(x[0, 0, keep], y[0, 0, keep])
    assert np.array_equal(q10[0, 0, keep][:, cols], q11[0, 0, keep][:, cols])
    assert not np.isfinite(kl1[0, 0, affected]).any()
    assert not np.isfinite(q11[0, 0, affected]).all(axis=-1).any()
