"""Distilled modal recurrence (Laughing Hyena) on AMD MI355X.

Thin Python binding of ``liblh.so`` (C ABI in ``include/lh.h``): it checks
tensor shapes and dtypes, marshals pointers and the current HIP stream, and
calls the library.  Every step of the computation runs in the library's HIP
kernels; there is no fallback.  PyTorch provides device memory and streams.

    prefill(lam, R, h0, u, state, y)   # y[b,t,c], t < T, and state = x_T
    prefill_plan(B, D, d, T, io="bf16")  # which plan prefill takes ("scan", "mfma", "mfma_seg")
    prefill_with_plan(lam, R, h0, u, state, y, plan=PLAN_MFMA)  # a named plan (tests, benchmarks)
    prefill_fft(lam, R, h0, u, state, y)  # the same results by FFT convolution
    step(lam, R, h0, state, u_t, y_t)  # y_t from x_t, then x_{t+1} in place

``lam``, ``R``: complex64 ``[D, d]``; ``h0``: float32 ``[D]``; ``u``, ``y``:
float32 or bfloat16 ``[B, T, D]``; ``state``: complex64 ``[B, D, d]``;
``u_t``, ``y_t``: ``[B, D]``.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

__all__ = [
    "LH_F32",
    "LH_BF16",
    "LHError",
    "lib",
    "library_path",
    "workspace_bytes",
    "prefill_plan",
    "PREFILL_PLANS",
    "PLAN_AUTO",
    "PLAN_MFMA",
    "PLAN_MFMA_SEG",
    "prefill",
    "prefill_with_plan",
    "prefill_noalloc",
    "NOALLOC_SCRATCH_BYTES",
    "fft_workspace_bytes",
    "prefill_fft",
    "step",
    "mh_step",
    "distill",
    "companion_coeffs",
    "companion_step",
    "companion_init_workspace_bytes",
    "companion_init",
    "STATUS",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liblh.so")

LH_F32 = 0
LH_BF16 = 1
# plan requests of prefill_with_plan (values > 0 are VALU chunk lengths)
PLAN_AUTO = 0
PLAN_MFMA = -1
PLAN_MFMA_SEG = -2
# scratch that lh_prefill_noalloc holds per GPU
NOALLOC_SCRATCH_BYTES = 64 << 20
STATUS = {
    0: "LH_OK",
    1: "LH_ERR_INVALID_ARG",
    2: "LH_ERR_OVERLAP",
    3: "LH_ERR_UNSUPPORTED_DTYPE",
    4: "LH_ERR_NO_DEVICE",
    5: "LH_ERR_WORKSPACE",
    6: "LH_ERR_HIP",
}

_lib: Optional[ctypes.CDLL] = None


class LHError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        self.name = STATUS.get(status, f"status {status}")
        super().__init__(f"{self.name}: {detail}")


def library_path() -> str:
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            f"{_LIB_PATH} is missing: build it with `python -m paper_2310_18780_amd.build` "
            "(or __graft_entry__.build()); there is no fallback implementation")
    # torch first: it brings its own HIP runtime, and the library's dependency
    # on the HIP runtime then resolves to that same, already loaded copy.
    # Loaded the other way round, the process would hold two HIP runtimes and
    # torch's memory and streams would be unknown to the library's.
    import torch  # noqa: F401

    L = ctypes.CDLL(_LIB_PATH)
    i64, vp, sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t
    L.lh_abi_version.argtypes = []
    L.lh_abi_version.restype = ctypes.c_int
    L.lh_status_string.argtypes = [ctypes.c_int]
    L.lh_status_string.restype = ctypes.c_char_p
    L.lh_last_error.argtypes = []
    L.lh_last_error.restype = ctypes.c_char_p
    L.lh_prefill_workspace_bytes.argtypes = [i64, i64, i64, i64]
    L.lh_prefill_workspace_bytes.restype = sz
    L.lh_prefill_with_plan_workspace_bytes.argtypes = [i64, i64, i64, i64, i64]
    L.lh_prefill_with_plan_workspace_bytes.restype = sz
    L.lh_prefill_plan.argtypes = [i64, i64, i64, i64, i64, ctypes.c_int]
    L.lh_prefill_plan.restype = ctypes.c_int
    L.lh_prefill.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, ctypes.c_int, vp, vp, vp, sz, vp]
    L.lh_prefill.restype = ctypes.c_int
    L.lh_prefill_with_plan.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, ctypes.c_int, vp, vp,
                                       i64, vp, sz, vp]
    L.lh_prefill_with_plan.restype = ctypes.c_int
    L.lh_prefill_noalloc.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, ctypes.c_int, vp, vp, vp]
    L.lh_prefill_noalloc.restype = ctypes.c_int
    L.lh_prefill_fft_workspace_bytes.argtypes = [i64, i64, i64, i64]
    L.lh_prefill_fft_workspace_bytes.restype = sz
    L.lh_prefill_fft.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, ctypes.c_int, vp, vp, vp, sz,
                                 vp]
    L.lh_prefill_fft.restype = ctypes.c_int
    L.lh_step.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, ctypes.c_int, vp]
    L.lh_step.restype = ctypes.c_int
    L.lh_mh_step.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, ctypes.c_int, vp]
    L.lh_mh_step.restype = ctypes.c_int
    L.lh_distill.argtypes = [vp, vp, vp, vp, i64, i64, i64, vp, vp, vp, vp, vp, vp]
    L.lh_distill.restype = ctypes.c_int
    L.lh_companion_coeffs.argtypes = [vp, vp, i64, i64, vp, vp, vp]
    L.lh_companion_coeffs.restype = ctypes.c_int
    L.lh_companion_step.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, ctypes.c_int, vp]
    L.lh_companion_step.restype = ctypes.c_int
    L.lh_companion_init_workspace_bytes.argtypes = [i64, i64, i64]
    L.lh_companion_init_workspace_bytes.restype = sz
    L.lh_companion_init.argtypes = [vp, vp, i64, i64, i64, i64, ctypes.c_int, vp, vp, sz, vp]
    L.lh_companion_init.restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int) -> None:
    if status != 0:
        raise LHError(status, lib().lh_last_error().decode(errors="replace"))


def workspace_bytes(B: int, D: int, d: int, T: int, plan: int = PLAN_AUTO) -> int:
    """Workspace bytes of ``prefill`` (``lh_prefill_workspace_bytes``), or of
    ``prefill_with_plan`` with this plan request
    (``lh_prefill_with_plan_workspace_bytes``)."""
    if plan == PLAN_AUTO:
        n = lib().lh_prefill_workspace_bytes(B, D, d, T)
    else:
        n = lib().lh_prefill_with_plan_workspace_bytes(B, D, d, T, plan)
    if n == ctypes.c_size_t(-1).value:
        raise LHError(1, f"invalid sizes B={B} D={D} d={d} T={T} plan={plan}")
    return int(n)


PREFILL_PLANS = ("scan", "mfma", "mfma_seg")


def prefill_plan(B: int, D: int, d: int, T: int, plan: int = PLAN_AUTO, io: str = "f32") -> str:
    """The plan a prefill takes for 16-byte aligned u and y (``lh_prefill_plan``):
    "scan" (VALU), "mfma" (matrix cores, whole prompt) or "mfma_seg" (segmented)."""
    k = lib().lh_prefill_plan(B, D, d, T, plan, {"f32": 0, "bf16": 1}[io])
    if k < 0:
        raise LHError(1, f"no prefill plan for B={B} D={D} d={d} T={T} plan={plan} io={io}")
    return PREFILL_PLANS[k]


def _io_dtype(t) -> int:
    import torch

    if t.dtype == torch.float32:
        return LH_F32
    if t.dtype == torch.bfloat16:
        return LH_BF16
    raise TypeError(f"u / y must be float32 or bfloat16, got {t.dtype}")


def _need(t, name, dtype, shape):
    import torch

    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a HIP device, got {t.device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _stream(dev, stream):
    """(torch stream object, raw hipStream_t handle) of ``stream``: None is the
    device's current stream; a raw handle is wrapped as an external stream."""
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(dev)
    elif not isinstance(stream, torch.cuda.Stream):
        stream = torch.cuda.ExternalStream(int(stream), device=dev)
    return stream, int(stream.cuda_stream)


def _scratch(need: int, workspace, dev, stream):
    """The caller's workspace, or a new one when ``workspace`` is None.  A
    workspace allocated here comes from torch's caching allocator, whose blocks
    belong to the current stream; the library enqueues on ``stream``, so the
    block is marked as used there (record_stream) and is not handed out again
    before that stream's work on it has completed."""
    import torch

    if need > 0 and workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
        if stream.cuda_stream != torch.cuda.current_stream(dev).cuda_stream:
            workspace.record_stream(stream)
    if workspace is None:
        return workspace, None, 0
    return workspace, workspace.data_ptr(), workspace.numel() * workspace.element_size()


def _prefill_args(lam, R, h0, u, state, y):
    import torch

    B, T, D = u.shape
    d = lam.shape[1]
    _need(lam, "lam", torch.complex64, (D, d))
    _need(R, "R", torch.complex64, (D, d))
    _need(h0, "h0", torch.float32, (D,))
    _need(u, "u", u.dtype, (B, T, D))
    _need(state, "state", torch.complex64, (B, D, d))
    _need(y, "y", u.dtype, (B, T, D))
    return B, D, d, T, _io_dtype(u)


def prefill(lam, R, h0, u, state, y, workspace=None, stream=None) -> None:
    """Prompt outputs ``y`` and post-prompt state ``state`` (both overwritten),
    with the library's automatic plan (``lh_prefill``).

    ``workspace``: a uint8 CUDA tensor of at least ``workspace_bytes(...)``
    bytes, or None to have one allocated here with torch."""
    B, D, d, T, io = _prefill_args(lam, R, h0, u, state, y)
    st, handle = _stream(u.device, stream)
    workspace, ws_ptr, ws_len = _scratch(workspace_bytes(B, D, d, T), workspace, u.device, st)
    _check(lib().lh_prefill(lam.data_ptr(), R.data_ptr(), h0.data_ptr(), u.data_ptr(), B, D, d, T,
                            io, state.data_ptr(), y.data_ptr(), ws_ptr, ws_len, handle))


def prefill_with_plan(lam, R, h0, u, state, y, plan: int, workspace=None, stream=None) -> None:
    """``prefill`` with a named plan (``lh_prefill_with_plan``): ``PLAN_AUTO``,
    ``PLAN_MFMA``, ``PLAN_MFMA_SEG`` or a VALU chunk length > 0."""
    B, D, d, T, io = _prefill_args(lam, R, h0, u, state, y)
    st, handle = _stream(u.device, stream)
    workspace, ws_ptr, ws_len = _scratch(workspace_bytes(B, D, d, T, plan), workspace, u.device, st)
    _check(lib().lh_prefill_with_plan(lam.data_ptr(), R.data_ptr(), h0.data_ptr(), u.data_ptr(), B,
                                      D, d, T, io, state.data_ptr(), y.data_ptr(), plan, ws_ptr,
                                      ws_len, handle))


def prefill_noalloc(lam, R, h0, u, state, y, stream=None) -> None:
    """``prefill`` without a workspace (``lh_prefill_noalloc``): the library's
    static per-GPU scratch serves the plan, so nothing is allocated.  Sizes
    needing more than ``NOALLOC_SCRATCH_BYTES`` of scratch raise; calls that
    overlap on one GPU race on that scratch."""
    B, D, d, T, io = _prefill_args(lam, R, h0, u, state, y)
    _check(lib().lh_prefill_noalloc(lam.data_ptr(), R.data_ptr(), h0.data_ptr(), u.data_ptr(), B,
                                    D, d, T, io, state.data_ptr(), y.data_ptr(),
                                    _stream(u.device, stream)[1]))


def fft_workspace_bytes(B: int, D: int, d: int, T: int) -> int:
    n = lib().lh_prefill_fft_workspace_bytes(B, D, d, T)
    if n == ctypes.c_size_t(-1).value:
        raise LHError(1, f"invalid sizes for the FFT prefill B={B} D={D} d={d} T={T}")
    return int(n)


def prefill_fft(lam, R, h0, u, state, y, workspace=None, stream=None) -> None:
    """``prefill``'s results by FFT convolution with the materialised filter
    and a Vandermonde contraction for the state (``lh_prefill_fft``)."""
    B, D, d, T, io = _prefill_args(lam, R, h0, u, state, y)
    st, handle = _stream(u.device, stream)
    workspace, ws_ptr, ws_len = _scratch(fft_workspace_bytes(B, D, d, T), workspace, u.device, st)
    _check(lib().lh_prefill_fft(lam.data_ptr(), R.data_ptr(), h0.data_ptr(), u.data_ptr(), B, D,
                                d, T, io, state.data_ptr(), y.data_ptr(), ws_ptr, ws_len, handle))


def step(lam, R, h0, state, u_t, y_t, stream=None) -> None:
    """One decode step: ``y_t`` from the current state, then the state update
    in place."""
    import torch

    B, D = u_t.shape
    d = lam.shape[1]
    _need(lam, "lam", torch.complex64, (D, d))
    _need(R, "R", torch.complex64, (D, d))
    _need(h0, "h0", torch.float32, (D,))
    _need(state, "state", torch.complex64, (B, D, d))
    _need(u_t, "u_t", u_t.dtype, (B, D))
    _need(y_t, "y_t", u_t.dtype, (B, D))
    io = _io_dtype(u_t)
    _check(lib().lh_step(lam.data_ptr(), R.data_ptr(), h0.data_ptr(), state.data_ptr(),
                         u_t.data_ptr(), y_t.data_ptr(), B, D, d, io,
                         _stream(u_t.device, stream)[1]))


def mh_step(lam, R, h0, state, q, k, v, y, stream=None) -> None:
    """One multi-head decode step (``lh_mh_step``): ``y`` from the current
    per-entry states of the ``M`` heads, then the state update in place.

    ``lam``, ``R``: ``[M, d]`` complex64; ``h0``: ``[M]``; ``state``:
    ``[B, M, N, N, d]`` complex64; ``q``, ``k``, ``v``, ``y``: ``[B, M N]``.
    """
    import torch

    B, M, N, _, d = state.shape
    _need(lam, "lam", torch.complex64, (M, d))
    _need(R, "R", torch.complex64, (M, d))
    _need(h0, "h0", torch.float32, (M,))
    _need(state, "state", torch.complex64, (B, M, N, N, d))
    for name, t in (("q", q), ("k", k), ("v", v), ("y", y)):
        _need(t, name, q.dtype, (B, M * N))
    io = _io_dtype(q)
    _check(lib().lh_mh_step(lam.data_ptr(), R.data_ptr(), h0.data_ptr(), state.data_ptr(),
                            q.data_ptr(), k.data_ptr(), v.data_ptr(), y.data_ptr(), B, M, N, d,
                            io, _stream(q.device, stream)[1]))


def distill(A, theta, R, target, loss, dA, dtheta, dR, hhat=None, stream=None) -> None:
    """Distillation objective (``lh_distill``): ``loss [D]`` and the gradients
    ``dA, dtheta [D, d]`` (float32), ``dR [D, d]`` (complex64,
    ``d/dRe R + i d/dIm R``) of the squared l2 error between the modal filter
    of polar poles ``A e^{i theta}`` and residues ``R`` and ``target [D, L]``;
    optionally the materialised filter ``hhat [D, L]``."""
    import torch

    D, d = A.shape
    L = target.shape[1]
    _need(A, "A", torch.float32, (D, d))
    _need(theta, "theta", torch.float32, (D, d))
    _need(R, "R", torch.complex64, (D, d))
    _need(target, "target", torch.float32, (D, L))
    _need(loss, "loss", torch.float32, (D,))
    _need(dA, "dA", torch.float32, (D, d))
    _need(dtheta, "dtheta", torch.float32, (D, d))
    _need(dR, "dR", torch.complex64, (D, d))
    if hhat is not None:
        _need(hhat, "hhat", torch.float32, (D, L))
    _check(lib().lh_distill(A.data_ptr(), theta.data_ptr(), R.data_ptr(), target.data_ptr(), D, d,
                            L, loss.data_ptr(), dA.data_ptr(), dtheta.data_ptr(), dR.data_ptr(),
                            hhat.data_ptr() if hhat is not None else None,
                            _stream(A.device, stream)[1]))


def companion_coeffs(lam, R, a, beta, stream=None) -> None:
    """Rational coefficients of the filters' companion form
    (``lh_companion_coeffs``): ``a, beta [D, 2d]`` float64 from ``lam, R [D, d]``."""
    import torch

    D, d = lam.shape
    _need(lam, "lam", torch.complex64, (D, d))
    _need(R, "R", torch.complex64, (D, d))
    _need(a, "a", torch.float64, (D, 2 * d))
    _need(beta, "beta", torch.float64, (D, 2 * d))
    _check(lib().lh_companion_coeffs(lam.data_ptr(), R.data_ptr(), D, d, a.data_ptr(),
                                     beta.data_ptr(), _stream(lam.device, stream)[1]))


def companion_step(a, beta, h0, state, u_t, y_t, stream=None) -> None:
    """One companion decode step (``lh_companion_step``); ``state [B, D, 2d]``
    float64 in place."""
    import torch

    B, D, order = state.shape
    _need(a, "a", torch.float64, (D, order))
    _need(beta, "beta", torch.float64, (D, order))
    _need(h0, "h0", torch.float32, (D,))
    _need(state, "state", torch.float64, (B, D, order))
    _need(u_t, "u_t", u_t.dtype, (B, D))
    _need(y_t, "y_t", u_t.dtype, (B, D))
    if order % 2:
        raise ValueError(f"companion order must be even (2d), got {order}")
    _check(lib().lh_companion_step(a.data_ptr(), beta.data_ptr(), h0.data_ptr(), state.data_ptr(),
                                   u_t.data_ptr(), y_t.data_ptr(), B, D, order // 2,
                                   _io_dtype(u_t), _stream(u_t.device, stream)[1]))


def companion_init_workspace_bytes(D: int, d: int, T: int) -> int:
    n = lib().lh_companion_init_workspace_bytes(D, d, T)
    if n == ctypes.c_size_t(-1).value:
        raise LHError(1, f"invalid sizes for the companion initialisation D={D} d={d} T={T}")
    return int(n)


def companion_init(a, u, state, workspace=None, stream=None) -> None:
    """Companion state after the prompt ``u [B, T, D]`` (``lh_companion_init``,
    Proposition "fast_init")."""
    import torch

    B, T, D = u.shape
    order = a.shape[1]
    _need(a, "a", torch.float64, (D, order))
    _need(u, "u", u.dtype, (B, T, D))
    _need(state, "state", torch.float64, (B, D, order))
    if order % 2:
        raise ValueError(f"companion order must be even (2d), got {order}")
    st, handle = _stream(u.device, stream)
    workspace, ws_ptr, ws_len = _scratch(companion_init_workspace_bytes(D, order // 2, T), workspace,
                                         u.device, st)
    _check(lib().lh_companion_init(a.data_ptr(), u.data_ptr(), B, D, order // 2, T, _io_dtype(u),
                                   state.data_ptr(), ws_ptr, ws_len, handle))
