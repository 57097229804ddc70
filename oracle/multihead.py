"""CPU oracle for the multi-head (head-tied) distilled decode -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run anything in this package.  The product path
never calls it and shares no code with it.

The multi-head long convolution of Sec. 5 ("Multi-head Long Convolutions"):
the projections ``q, k, v`` of width ``D`` are split into ``M`` heads of
``N = D / M`` channels; per head ``m`` and step ``t`` the outer product
``z_t = k_t (x) v_t`` (``z_t[i, j] = k_t[i] v_t[j]``) is convolved, every one of
its ``N x N`` entries independently, with the head's filter ``h^m``, and the
result multiplies ``q_t``:

    w_t[i, j] = sum_{s <= t} h^m_{t-s} z_s[i, j]          (eq. "cnn" per entry)
    y_t[i]    = sum_j w_t[i, j] q_t[j]                      (matrix times vector)

With the head's filter distilled to modes (``lambda``, ``R``, ``h0``; eq.
"modal_impulse"), each entry carries the state of Proposition
"modal_realization": ``x_{t+1}[i, j, n] = lambda_n x_t[i, j, n] + z_t[i, j]``
from ``x_0 = 0``, so that the state after ``T`` steps is
``x_T[i, j, n] = sum_{s<T} lambda_n^(T-1-s) z_s[i, j]``.

This module evaluates those definitions in float64: the filter materialised
by ``oracle.filter_taps``, the outputs by direct causal convolution of every
entry (``oracle.causal_conv``) followed by the contraction with ``q``, and the
states by direct power sums -- no recurrence, blocking or FFT.

Reading (where the paper leaves a choice): the ``q`` contraction runs over the
second (value) index of ``z``, the literal matrix-vector product of the
paper's formula.  The other orientation (``q`` against the key index, as in
the multi-head state-space layer the design is adapted from) is the same
computation with ``k`` and ``v`` exchanged.

Parity of every function here is pinned by ``tests/test_multihead_pins.py``.
"""
from __future__ import annotations

from typing import Dict, Sequence

import numpy as np

from . import causal_conv, filter_taps, power_table

__all__ = ["mh_filters", "mh_outputs", "mh_outputs_rows", "mh_state", "mh_state_rows", "mh_run"]


def mh_filters(lam, R, h0, L: int) -> np.ndarray:
    """Materialised head filters ``h[m, t]``, ``t < L`` (float64 ``[M, L]``)."""
    return filter_taps(lam, R, h0, L)


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def mh_outputs_rows(lam, R, h0, q, k, v, rows: Sequence) -> np.ndarray:
    """Outputs ``y[t]`` of selected ``(b, m, i)`` rows for every step.

    ``q, k, v``: ``[B, L, M, N]`` (any float dtype), the inputs of steps
    ``0 .. L-1`` (a prompt followed by decode steps: the formula does not
    distinguish them).  Returns float64 ``[len(rows), L]``.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, L, M, N = q.shape
    h = mh_filters(lam, R, h0, L)
    out = np.empty((len(rows), L), np.float64)
    for r, (b, m, i) in enumerate(rows):
        z = k[b, :, m, i][None, :] * v[b, :, m, :].T  # z[j, s] = k_s[i] v_s[j]
        w = causal_conv(np.broadcast_to(h[m], z.shape), z)  # w[j, t]
        out[r] = np.sum(w * q[b, :, m, :].T, axis=0)
    return out


def mh_outputs(lam, R, h0, q, k, v) -> np.ndarray:
    """All outputs ``y[b, t, m, i]`` (float64 ``[B, L, M, N]``)."""
    B, L, M, N = np.shape(q)
    rows = [(b, m, i) for b in range(B) for m in range(M) for i in range(N)]
    y = mh_outputs_rows(lam, R, h0, q, k, v, rows)
    return y.reshape(B, M, N, L).transpose(0, 3, 1, 2)


def mh_state_rows(lam, k, v, T: int, rows: Sequence) -> np.ndarray:
    """States ``x_T[i, j, n]`` of selected ``(b, m, i)`` rows: complex128
    ``[len(rows), N, d]`` with ``x_T[j, n] = sum_{s<T} lambda_n^(T-1-s) k_s[i] v_s[j]``."""
    k, v = _f64(k), _f64(v)
    lam = np.asarray(lam).astype(np.complex128)
    M, d = lam.shape
    N = k.shape[3]
    out = np.zeros((len(rows), N, d), np.complex128)
    if T == 0:
        return out
    P = power_table(lam, T)  # P[m, n, e] = lambda^e
    for r, (b, m, i) in enumerate(rows):
        z = k[b, :T, m, i][:, None] * v[b, :T, m, :]  # z[s, j]
        out[r] = (P[m][:, ::-1] @ z).T  # e = T-1-s
    return out


def mh_state(lam, k, v, T: int) -> np.ndarray:
    """All states after ``T`` steps: complex128 ``[B, M, N, N, d]``."""
    B, _, M, N = np.shape(k)
    d = np.shape(lam)[1]
    rows = [(b, m, i) for b in range(B) for m in range(M) for i in range(N)]
    return mh_state_rows(lam, k, v, T, rows).reshape(B, M, N, N, d)


def mh_run(lam, R, h0, q, k, v, T0: int) -> Dict[str, np.ndarray]:
    """Oracle of a decode run: the state after the first ``T0`` steps (the
    prompt), the outputs of the remaining steps and the final state."""
    L = np.shape(q)[1]
    y = mh_outputs(lam, R, h0, q, k, v)
    return {"x_T0": mh_state(lam, k, v, T0), "y_dec": y[:, T0:], "x_end": mh_state(lam, k, v, L)}
