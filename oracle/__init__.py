"""CPU oracle for the distilled modal recurrence -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run anything in this package.  The product path (the
HIP library and its Python binding) never calls it and shares no code with it.

What it computes, in float64, from the definitions of the paper:

* the filter of a distilled channel, materialised: ``h_0 = h0`` and
  ``h_t = Re sum_n R_n lambda_n^(t-1)`` for ``t >= 1`` (eq. "modal_impulse",
  Sec. 3.2, with the real part taken as for real target filters, and the
  pass-through ``h0`` of the state-space form eq. "dtssm", Sec. 2);
* outputs by direct causal convolution ``y_t = sum_{j<=t} h_{t-j} u_j``
  (eq. "cnn", Sec. 2), with no blocking, FFT or recurrence;
* states by their definition as the response of ``x_{t+1} = A x_t + B u_t``,
  ``A = diag(lambda)``, ``B = 1`` from ``x_0 = 0`` (Proposition
  "modal_realization", Sec. 3.4; eq. "dtssm"):
  ``x_T[n] = sum_{k<T} lambda_n^(T-1-k) u_k``, evaluated as a dot product with a
  table of powers.

Inputs are taken exactly as the GPU receives them (complex64 / float32, or
bfloat16-exact float32) and promoted to float64.  Powers are running float64
products, ``lambda^0 = 1`` even for ``lambda = 0``.

Conventions fixed here (readings of the paper):

* ``y_t`` reads the state *before* it absorbs ``u_t`` (eq. "dtssm"), so a decode
  step after a prefill of ``T`` tokens yields ``y_T``;
* ``C = (R_1 .. R_d)`` is a plain row vector: no conjugation and no 1/2 factor in
  ``R x`` (the 1/2 of the conjugate-pair form of App. B.1 cancels);
* the post-prompt state is ``x_T``, the state after ``u_0 .. u_{T-1}``.

Parity of every function here is pinned by ``tests/test_oracle_pins.py``
against closed forms, library routines and brute force.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

__all__ = [
    "filter_taps",
    "power_table",
    "causal_conv",
    "conv_at",
    "state_after",
    "run",
    "run_rows",
    "native_available",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle_conv.so")
_lib: Optional[ctypes.CDLL] = None


def _load_native() -> Optional[ctypes.CDLL]:
    global _lib
    if _lib is None and os.path.exists(_LIB_PATH):
        lib = ctypes.CDLL(_LIB_PATH)
        lib.oracle_causal_conv_rows.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64]
        lib.oracle_causal_conv_rows.restype = None
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def native_available() -> bool:
    return _load_native() is not None


def native_threads() -> int:
    lib = _load_native()
    return int(lib.oracle_num_threads()) if lib is not None else 1


def power_table(lam: np.ndarray, m: int) -> np.ndarray:
    """``P[..., k] = lam^k`` for ``k = 0 .. m-1`` as running float64 products
    (``np.cumprod`` multiplies left to right: ``lam^k = lam^(k-1) * lam``).

    ``lam``: complex array of any shape; returns complex128 ``lam.shape + (m,)``.
    """
    lam = np.asarray(lam).astype(np.complex128)
    P = np.empty(lam.shape + (m,), np.complex128)
    if m > 0:
        P[..., 0] = 1.0
    if m > 1:
        P[..., 1:] = np.cumprod(np.broadcast_to(lam[..., None], lam.shape + (m - 1,)), axis=-1)
    return P


def filter_taps(lam: np.ndarray, R: np.ndarray, h0: np.ndarray, L: int) -> np.ndarray:
    """Materialised filters ``h[c, t]``, ``t < L``, float64 ``[D, L]``.

    ``h[c, 0] = h0[c]``; ``h[c, t] = Re sum_n R[c, n] lam[c, n]^(t-1)`` for
    ``t >= 1`` (eq. "modal_impulse" and the pass-through of eq. "dtssm").
    """
    lam = np.atleast_2d(np.asarray(lam)).astype(np.complex128)
    R = np.atleast_2d(np.asarray(R)).astype(np.complex128)
    h0 = np.atleast_1d(np.asarray(h0)).astype(np.float64)
    D = lam.shape[0]
    h = np.empty((D, L), np.float64)
    if L == 0:
        return h
    h[:, 0] = h0
    p = np.ones(lam.shape, np.complex128)  # lam^(t-1) at t = 1
    for t in range(1, L):
        h[:, t] = np.real(np.sum(R * p, axis=1))
        p = p * lam
    return h


def conv_at(h: np.ndarray, u: np.ndarray, t: int) -> float:
    """One output of the causal convolution: ``sum_{j=0}^{t} h[t-j] u[j]``."""
    h = np.asarray(h, np.float64)
    u = np.asarray(u, np.float64)
    return float(np.dot(h[t::-1], u[: t + 1]))


def causal_conv(h: np.ndarray, u: np.ndarray) -> np.ndarray:
    """Direct causal convolution of matching rows (eq. "cnn").

    ``h``: ``[..., L]`` filters, ``u``: ``[..., L]`` inputs (same leading shape
    or broadcastable); returns float64 ``[..., L]`` with
    ``y[..., t] = sum_{j<=t} h[..., t-j] u[..., j]``.
    """
    h = np.asarray(h, np.float64)
    u = np.asarray(u, np.float64)
    h, u = np.broadcast_arrays(h, u)
    shape = u.shape
    L = shape[-1]
    if L == 0 or u.size == 0:
        return np.zeros(shape, np.float64)
    hr =np.ascontiguousarray(h.reshape(-1, L))
    ur = np.ascontiguousarray(u.reshape(-1, L))
    y = np.empty_like(ur)
    lib = _load_native()
    if lib is not None and ur.shape[0] > 0 and L > 0:
        lib.oracle_causal_conv_rows(hr.ctypes.data, ur.ctypes.data, y.ctypes.data,
                                    ur.shape[0], L)
    else:
        for i in range(ur.shape[0]):
            for t in range(L):
                y[i, t] = np.dot(hr[i, t::-1], ur[i, : t + 1])
    return y.reshape(shape)


def state_after(lam: np.ndarray, u: np.ndarray, T: int) -> np.ndarray:
    """``x_T[n] = sum_{k<T} lam[n]^(T-1-k) u[k]`` for one channel's modes.

    ``lam``: ``[d]`` complex; ``u``: ``[>=T]`` real.  Returns complex128 ``[d]``.
    """
    lam = np.asarray(lam).astype(np.complex128).reshape(-1)
    u = np.asarray(u, np.float64)[:T]
    if T == 0:
        return np.zeros(lam.shape, np.complex128)
    P = power_table(lam, T)  # P[n, m] = lam^m
    return P @ u[::-1]  # m = T-1-k


def run_rows(lam, R, h0, u_prompt, u_dec, rows: Sequence) -> Dict[str, np.ndarray]:
    """Oracle results for selected ``(b, c)`` rows of a workload.

    ``u_prompt``: ``[B, T, D]``, ``u_dec``: ``[B, K, D]`` (any float dtype);
    ``rows``: iterable of ``(b, c)``.  Returns, per selected row ``i``:
    ``y_prefill[i, T]``, ``x_T[i, d]``, ``y_dec[i, K]``, ``x_end[i, d]``.
    """
    rows = list(rows)
    T = u_prompt.shape[1]
    K = u_dec.shape[1]
    L = T + K
    chans = sorted({c for _, c in rows})
    cidx = {c: i for i, c in enumerate(chans)}
    lam = np.asarray(lam)
    R = np.asarray(R)
    h0 = np.asarray(h0)
    h = filter_taps(lam[chans], R[chans], h0[chans], L)
    uf = np.empty((len(rows), L), np.float64)
    for i, (b, c) in enumerate(rows):
        uf[i, :T] = u_prompt[b, :, c]
        uf[i, T:] = u_dec[b, :, c]
    hr = np.stack([h[cidx[c]] for _, c in rows]) if rows else np.empty((0, L))
    y = causal_conv(hr, uf)
    xT = np.stack([state_after(lam[c], uf[i], T) for i, (_, c) in enumerate(rows)])
    xE = np.stack([state_after(lam[c], uf[i], L) for i, (_, c) in enumerate(rows)])
    return {"y_prefill": y[:, :T], "x_T": xT, "y_dec": y[:, T:], "x_end": xE}


def run(lam, R, h0, u_prompt, u_dec) -> Dict[str, np.ndarray]:
    """Full oracle of a (small) workload.

    Returns ``y_prefill [B,T,D]``, ``x_T [B,D,d]``, ``y_dec [B,K,D]`` and
    ``x_end [B,D,d]`` (float64 / complex128).
    """
    B, T, D = u_prompt.shape
    K = u_dec.shape[1]
    d = np.asarray(lam).shape[1]
    rows = [(b, c) for b in range(B) for c in range(D)]
    out = run_rows(lam, R, h0, u_prompt, u_dec, rows)
    return {
        "y_prefill": out["y_prefill"].reshape(B, D, T).transpose(0, 2, 1),
        "x_T": out["x_T"].reshape(B, D, d),
        "y_dec": out["y_dec"].reshape(B, D, K).transpose(0, 2, 1),
        "x_end": out["x_end"].reshape(B, D, d),
    }
