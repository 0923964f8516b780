"""Python binding of libstreamkl.so (the C ABI declared in include/streamkl.h).

Argument marshalling only: every step of the forward and backward pass runs
in the library's gfx950 kernels. PyTorch provides device memory and the
current HIP stream. Importing this module fails loudly when the library has
not been built; there is no fallback implementation.

    kl, lse1, lse2 = fwd(q1, k1, q2, k2, s1, s2, causal, direction)
    kl, lse1, lse2 = fwd_split(q1, k1, q2, k2, s1, s2, causal, direction, splits="auto")
    dQ1, dK1, dQ2, dK2 = bwd(q1, k1, q2, k2, kl, lse1, lse2, dkl, ..., want=("dq2", "dk2"), strategy="auto")
    loss = attention_kl(q1, k1, q2, k2, causal=True).mean(); loss.backward()
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libstreamkl.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_HIP, ERR_SCRATCH_LIMIT = 0, 1, 2, 3, 4
NOALLOC_SCRATCH_BYTES = 16 << 20
FWD, REV = 0, 1
BWD_AUTO, BWD_SEPARATE, BWD_FUSED = 0, 1, 2
GRAD_BITS = {"dq1": 1, "dk1": 2, "dq2": 4, "dk2": 8}
ACT_SOFTMAX, ACT_SIGMOID = 0, 1
ENTRY_POINTS = ("streamkl_fwd", "streamkl_bwd", "streamkl_bwd_ex", "streamkl_bwd_choose", "streamkl_fwd_split",
                "streamkl_fwd_split_noalloc", "streamkl_fwd_split_workspace_bytes", "streamkl_fwd_split_count",
                "streamkl_fwd_act", "streamkl_bwd_act", "streamkl_strerror", "streamkl_version",
                "streamkl_supported_head_dim")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_20005_amd.build` "
                          "(the attention-KL primitive has no non-HIP implementation)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i, f = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
    lib.streamkl_fwd.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, f, f, i, i, vp, vp, vp, vp]
    lib.streamkl_fwd.restype = i
    lib.streamkl_bwd.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, f, f, i, i, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.streamkl_bwd.restype = i
    lib.streamkl_bwd_ex.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, f, f, i, i, vp, vp, vp, vp, vp, vp, vp, vp, i,
                                    vp]
    lib.streamkl_bwd_ex.restype = i
    lib.streamkl_fwd_act.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, f, f, i, i, i, vp, vp, vp, vp]
    lib.streamkl_fwd_act.restype = i
    lib.streamkl_bwd_act.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, f, f, i, i, i, vp, vp, vp, vp, vp, vp, vp,
                                     vp, vp]
    lib.streamkl_bwd_act.restype = i
    lib.streamkl_bwd_choose.argtypes = [i, i, i, i, i, i, i, i, i]
    lib.streamkl_bwd_choose.restype = i
    sz = ctypes.c_size_t
    lib.streamkl_fwd_split.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, f, f, i, i, i, vp, sz, vp, vp, vp, vp]
    lib.streamkl_fwd_split.restype = i
    lib.streamkl_fwd_split_noalloc.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, f, f, i, i, i, vp, vp, vp, vp]
    lib.streamkl_fwd_split_noalloc.restype = i
    lib.streamkl_fwd_split_workspace_bytes.argtypes = [i, i, i, i]
    lib.streamkl_fwd_split_workspace_bytes.restype = sz
    lib.streamkl_fwd_split_count.argtypes = [i, i, i, i, i, i]
    lib.streamkl_fwd_split_count.restype = i
    lib.streamkl_strerror.argtypes = [i]
    lib.streamkl_strerror.restype = ctypes.c_char_p
    lib.streamkl_version.argtypes = []
    lib.streamkl_version.restype = ctypes.c_char_p
    lib.streamkl_supported_head_dim.argtypes = [i]
    lib.streamkl_supported_head_dim.restype = i
    return lib


lib = _load()


class StreamKLError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {lib.streamkl_strerror(status).decode()} (status {status})")


def version() -> str:
    return lib.streamkl_version().decode()


def supported_head_dim(d: int) -> bool:
    return bool(lib.streamkl_supported_head_dim(int(d)))


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(dev):
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _direction(direction) -> int:
    if direction in (FWD, "fwd", "forward"):
        return FWD
    if direction in (REV, "rev", "reverse"):
        return REV
    raise ValueError(f"direction must be 'fwd' (KL(P1||P2)) or 'rev' (KL(P2||P1)), got {direction!r}")


def _check_inputs(q1, k1, q2, k2):
    for n, t in (("q1", q1), ("k1", k1), ("q2", q2), ("k2", k2)):
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise ValueError(f"{n} must be a GPU tensor")
        if t.dtype != torch.bfloat16:
            raise ValueError(f"{n} must be bfloat16, got {t.dtype}")
        if t.dim() != 4 or not t.is_contiguous():
            raise ValueError(f"{n} must be a contiguous [B, H, N, d] tensor")
    B, H, NQ, d1 = q1.shape
    NK = k1.shape[2]
    d2 = q2.shape[3]
    if tuple(k1.shape) != (B, H, NK, d1) or tuple(q2.shape) != (B, H, NQ, d2) or tuple(k2.shape) != (B, H, NK, d2):
        raise ValueError(f"inconsistent shapes q1{tuple(q1.shape)} k1{tuple(k1.shape)} "
                         f"q2{tuple(q2.shape)} k2{tuple(k2.shape)}")
    if len({q1.device, k1.device, q2.device, k2.device}) != 1:
        raise ValueError("all inputs must be on one device")
    return B, H, NQ, NK, d1, d2


def _scales(s1, s2, d1, d2):
    return (1.0 / math.sqrt(d1) if s1 is None else float(s1)), (1.0 / math.sqrt(d2) if s2 is None else float(s2))


def _f32_rows(t, shape, dev, name):
    if t is None:
        return None
    if t.dtype != torch.float32 or tuple(t.shape) != shape or not t.is_contiguous() or t.device != dev:
        raise ValueError(f"{name} must be a contiguous float32 tensor of shape {shape} on {dev}")
    return t


def fwd(q1, k1, q2, k2, s1=None, s2=None, causal=False, direction=FWD, out=None):
    """streamkl_fwd: returns (kl, lse1, lse2), float32 [B, H, N_Q].

    s_t defaults to 1/sqrt(d_t). ``out`` may hold three preallocated tensors.
    """
    B, H, NQ, NK, d1, d2 = _check_inputs(q1, k1, q2, k2)
    s1, s2 = _scales(s1, s2, d1, d2)
    dev = q1.device
    if out is None:
        out = tuple(torch.empty((B, H, NQ), dtype=torch.float32, device=dev) for _ in range(3))
    kl, lse1, lse2 = (_f32_rows(t, (B, H, NQ), dev, n) for t, n in zip(out, ("kl", "lse1", "lse2")))
    with torch.cuda.device(dev):
        st = lib.streamkl_fwd(_p(q1), _p(k1), _p(q2), _p(k2), B, H, NQ, NK, d1, d2, s1, s2,
                              int(bool(causal)), _direction(direction), _p(kl), _p(lse1), _p(lse2), _stream(dev))
    if st != OK:
        raise StreamKLError(st, "streamkl_fwd")
    return kl, lse1, lse2


def _activation(activation) -> int:
    if activation in (ACT_SOFTMAX, "softmax"):
        return ACT_SOFTMAX
    if activation in (ACT_SIGMOID, "sigmoid"):
        return ACT_SIGMOID
    raise ValueError(f"activation must be 'softmax' or 'sigmoid', got {activation!r}")


def fwd_act(q1, k1, q2, k2, s1=None, s2=None, causal=False, direction=FWD, activation="sigmoid", out=None):
    """streamkl_fwd_act: returns (kl, stat1, stat2), float32 [B, H, N_Q].

    activation "softmax": exactly fwd (the stats are the LSEs). "sigmoid":
    unnormalised sigmoid scores, kl is the generalized KL of the two score
    rows and the stats are the row masses sum_j sigmoid(S_t[j]).
    """
    B, H, NQ, NK, d1, d2 = _check_inputs(q1, k1, q2, k2)
    s1, s2 = _scales(s1, s2, d1, d2)
    dev = q1.device
    if out is None:
        out = tuple(torch.empty((B, H, NQ), dtype=torch.float32, device=dev) for _ in range(3))
    kl, st1, st2 = (_f32_rows(t, (B, H, NQ), dev, n) for t, n in zip(out, ("kl", "stat1", "stat2")))
    with torch.cuda.device(dev):
        st = lib.streamkl_fwd_act(_p(q1), _p(k1), _p(q2), _p(k2), B, H, NQ, NK, d1, d2, s1, s2, int(bool(causal)),
                                  _direction(direction), _activation(activation), _p(kl), _p(st1), _p(st2),
                                  _stream(dev))
    if st != OK:
        raise StreamKLError(st, "streamkl_fwd_act")
    return kl, st1, st2


def split_count(B, H, n_q, n_k, d1, d2) -> int:
    """streamkl_fwd_split_count: the adaptive split count of Sec. 3.3 (0 for invalid arguments)."""
    return int(lib.streamkl_fwd_split_count(int(B), int(H), int(n_q), int(n_k), int(d1), int(d2)))


def split_workspace_bytes(B, H, n_q, splits) -> int:
    """streamkl_fwd_split_workspace_bytes: workspace the split-K forward needs."""
    return int(lib.streamkl_fwd_split_workspace_bytes(int(B), int(H), int(n_q), int(splits)))


def fwd_split(q1, k1, q2, k2, s1=None, s2=None, causal=False, direction=FWD, splits="auto", out=None,
              workspace=None):
    """streamkl_fwd_split: the split-K forward; returns (kl, lse1, lse2) like fwd.

    splits: an int >= 1 or "auto" (split_count). The workspace is allocated
    here unless ``workspace`` (a device tensor of at least split_workspace_bytes
    bytes) is given.
    """
    B, H, NQ, NK, d1, d2 = _check_inputs(q1, k1, q2, k2)
    s1, s2 = _scales(s1, s2, d1, d2)
    dev = q1.device
    w = split_count(B, H, NQ, NK, d1, d2) if splits == "auto" else int(splits)
    if out is None:
        out = tuple(torch.empty((B, H, NQ), dtype=torch.float32, device=dev) for _ in range(3))
    kl, lse1, lse2 = (_f32_rows(t, (B, H, NQ), dev, n) for t, n in zip(out, ("kl", "lse1", "lse2")))
    need = split_workspace_bytes(B, H, NQ, w)
    if workspace is None:
        workspace = torch.empty(max(need, 4), dtype=torch.uint8, device=dev)
    ws_bytes = workspace.numel() * workspace.element_size()
    with torch.cuda.device(dev):
        st = lib.streamkl_fwd_split(_p(q1), _p(k1), _p(q2), _p(k2), B, H, NQ, NK, d1, d2, s1, s2,
                                    int(bool(causal)), _direction(direction), w, _p(workspace), ws_bytes,
                                    _p(kl), _p(lse1), _p(lse2), _stream(dev))
    if st != OK:
        raise StreamKLError(st, "streamkl_fwd_split")
    return kl, lse1, lse2


def fwd_split_noalloc(q1, k1, q2, k2, s1=None, s2=None, causal=False, direction=FWD, splits="auto", out=None):
    """streamkl_fwd_split_noalloc: the split-K forward with its partial row
    statistics in the library's static per-GPU scratch (nothing is allocated
    for them); returns (kl, lse1, lse2) like fwd_split. Outputs are allocated
    here unless ``out`` is given."""
    B, H, NQ, NK, d1, d2 = _check_inputs(q1, k1, q2, k2)
    s1, s2 = _scales(s1, s2, d1, d2)
    dev = q1.device
    w = split_count(B, H, NQ, NK, d1, d2) if splits == "auto" else int(splits)
    if out is None:
        out = tuple(torch.empty((B, H, NQ), dtype=torch.float32, device=dev) for _ in range(3))
    kl, lse1, lse2 = (_f32_rows(t, (B, H, NQ), dev, n) for t, n in zip(out, ("kl", "lse1", "lse2")))
    with torch.cuda.device(dev):
        st = lib.streamkl_fwd_split_noalloc(_p(q1), _p(k1), _p(q2), _p(k2), B, H, NQ, NK, d1, d2, s1, s2,
                                            int(bool(causal)), _direction(direction), w, _p(kl), _p(lse1),
                                            _p(lse2), _stream(dev))
    if st != OK:
        raise StreamKLError(st, "streamkl_fwd_split_noalloc")
    return kl, lse1, lse2


_STRATEGIES = {"auto": BWD_AUTO, "separate": BWD_SEPARATE, "fused": BWD_FUSED}


def _strategy(strategy) -> int:
    if isinstance(strategy, str):
        if strategy not in _STRATEGIES:
            raise ValueError(f"strategy must be one of {sorted(_STRATEGIES)}, got {strategy!r}")
        return _STRATEGIES[strategy]
    return int(strategy)


def bwd_choose(B, H, n_q, n_k, d1, d2, causal=False, direction=FWD, want=("dq2", "dk2")) -> str:
    """streamkl_bwd_choose: the strategy ("separate" or "fused") the adaptive rule picks."""
    bits = 0
    for n in want:
        bits |= GRAD_BITS[n]
    r = lib.streamkl_bwd_choose(B, H, n_q, n_k, d1, d2, int(bool(causal)), _direction(direction), bits)
    if r == 0:
        raise StreamKLError(ERR_INVALID_ARG, "streamkl_bwd_choose")
    return "fused" if r == BWD_FUSED else "separate"


def bwd(q1, k1, q2, k2, kl, lse1, lse2, dkl=None, s1=None, s2=None, causal=False, direction=FWD,
        want=("dq2", "dk2"), out=None, strategy="separate", activation="softmax"):
    """streamkl_bwd / streamkl_bwd_ex / streamkl_bwd_act: returns (dQ1, dK1, dQ2, dK2), float32, None where not
    requested.

    want: any of "dq1", "dk1", "dq2", "dk2". dkl: per-row upstream gradient
    (float32 [B, H, N_Q]) or None for all ones. ``out`` may map those names to
    preallocated tensors. strategy: "separate" (streamkl_bwd, reproducible),
    "fused" (one kernel, dQ by atomics) or "auto" (the adaptive rule).
    activation "sigmoid" (streamkl_bwd_act, separate kernels): kl, lse1, lse2
    are not needed and may be None.
    """
    act = _activation(activation)
    B, H, NQ, NK, d1, d2 = _check_inputs(q1, k1, q2, k2)
    s1, s2 = _scales(s1, s2, d1, d2)
    dev = q1.device
    rows = (B, H, NQ)
    kl, lse1, lse2 = (_f32_rows(t, rows, dev, n) for t, n in ((kl, "kl"), (lse1, "lse1"), (lse2, "lse2")))
    dkl = _f32_rows(dkl, rows, dev, "dkl")
    shapes = {"dq1": (B, H, NQ, d1), "dk1": (B, H, NK, d1), "dq2": (B, H, NQ, d2), "dk2": (B, H, NK, d2)}
    unknown = set(want) - set(shapes)
    if unknown:
        raise ValueError(f"unknown gradient names {sorted(unknown)}")
    out = dict(out or {})
    grads = {}
    for n in ("dq1", "dk1", "dq2", "dk2"):
        if n in want:
            t = out.get(n)
            grads[n] = _f32_rows(t, shapes[n], dev, n) if t is not None else \
                torch.empty(shapes[n], dtype=torch.float32, device=dev)
        else:
            grads[n] = None
    strat = _strategy(strategy)
    args = (_p(q1), _p(k1), _p(q2), _p(k2), B, H, NQ, NK, d1, d2, s1, s2, int(bool(causal)), _direction(direction),
            _p(kl), _p(lse1), _p(lse2), _p(dkl), _p(grads["dq1"]), _p(grads["dk1"]), _p(grads["dq2"]),
            _p(grads["dk2"]))
    with torch.cuda.device(dev):
        if act == ACT_SIGMOID:
            if strat != BWD_SEPARATE:
                raise ValueError("sigmoid scores run the separate backward kernels only")
            st, where = lib.streamkl_bwd_act(*args[:14], act, *args[14:], _stream(dev)), "streamkl_bwd_act"
        elif strat == BWD_SEPARATE:
            st, where = lib.streamkl_bwd(*args, _stream(dev)), "streamkl_bwd"
        else:
            st, where = lib.streamkl_bwd_ex(*args, strat, _stream(dev)), "streamkl_bwd_ex"
    if st != OK:
        raise StreamKLError(st, where)
    return grads["dq1"], grads["dk1"], grads["dq2"], grads["dk2"]


class _AttentionKL(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q1, k1, q2, k2, s1, s2, causal, direction, bwd_strategy, act):
        if act == ACT_SIGMOID:
            kl, st1, st2 = fwd_act(q1, k1, q2, k2, s1, s2, causal, direction, ACT_SIGMOID)
        else:
            # the adaptive split count is 1 (the single-pass kernel) unless the heads have few query rows
            kl, st1, st2 = fwd_split(q1, k1, q2, k2, s1, s2, causal, direction, splits="auto")
        ctx.save_for_backward(q1, k1, q2, k2, kl, st1, st2)
        ctx.cfg = (s1, s2, causal, direction, bwd_strategy, act)
        ctx.mark_non_differentiable(st1, st2)
        return kl, st1, st2

    @staticmethod
    def backward(ctx, gkl, _g1, _g2):
        q1, k1, q2, k2, kl, st1, st2 = ctx.saved_tensors
        s1, s2, causal, direction, strategy, act = ctx.cfg
        names = [n for n, need in zip(("dq1", "dk1", "dq2", "dk2"), ctx.needs_input_grad[:4]) if need]
        if not names:
            return (None,) * 10
        g = gkl.to(torch.float32).contiguous()
        dq1, dk1, dq2, dk2 = bwd(q1, k1, q2, k2, kl, st1, st2, g, s1, s2, causal, direction, want=names,
                                 strategy="separate" if act == ACT_SIGMOID else strategy, activation=act)
        cast = lambda t, ref: None if t is None else t.to(ref.dtype)   # noqa: E731
        return cast(dq1, q1), cast(dk1, k1), cast(dq2, q2), cast(dk2, k2), None, None, None, None, None, None


def attention_kl(q1, k1, q2, k2, *, s1=None, s2=None, causal=False, direction="fwd", return_lse=False,
                 bwd_strategy="auto", activation="softmax"):
    """Per-row KL between softmax(s1 q1 k1^T) and softmax(s2 q2 k2^T), differentiable.

    Returns kl [B, H, N_Q] (and the two row statistics if ``return_lse``:
    lse1, lse2 for softmax, the row masses for sigmoid). The paper's training
    objective is ``attention_kl(...).mean()``. Gradients flow to the inputs
    that require them: (q2, k2) in standard distillation (Setting 1),
    (q1, k1) when the first distribution is trained (Setting 2), or both.
    bwd_strategy: "auto" (the adaptive rule of streamkl_bwd_choose), "fused"
    or "separate" (bitwise reproducible gradients). activation "sigmoid":
    unnormalised sigmoid scores and the generalized KL (streamkl_fwd_act).
    """
    d1, d2 = q1.shape[-1], q2.shape[-1]
    s1, s2 = _scales(s1, s2, d1, d2)
    _strategy(bwd_strategy)
    kl, st1, st2 = _AttentionKL.apply(q1, k1, q2, k2, s1, s2, bool(causal), _direction(direction), bwd_strategy,
                                      _activation(activation))
    return (kl, st1, st2) if return_lse else kl
