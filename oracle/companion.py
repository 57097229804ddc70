"""CPU oracle for the companion (rational) form of a distilled filter -- TEST
INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run anything in this package.  The product path
never calls it and shares no code with it.

The real filter of a distilled channel, ``h_0 = h0`` and
``h_t = Re sum_n R_n lambda_n^(t-1)`` (eq. "modal_impulse"), is the impulse
response of a real system of order ``2d`` whose poles are the ``d`` poles and
their conjugates, with residues ``R_n / 2`` and ``conj(R_n) / 2`` (the
conjugate-pair form of App. B.1).  Its transfer function in ``w = z^-1`` is
rational (eq. "dtssm_tf"; delay-free path eq. "delay_free_tf"):

    H(w) = b0 + (beta_1 w + ... + beta_2d w^2d) / (1 + a_1 w + ... + a_2d w^2d),

``b0 = h0``, the denominator ``p(w) = prod_k (1 - rho_k w)`` over the ``2d``
poles ``rho_k`` and the numerator ``sum_k r_k w prod_{j != k} (1 - rho_j w)``
(the partial fractions ``sum_k r_k w / (1 - rho_k w)`` brought to the common
denominator).  Its companion canonical realisation (eq. "ssm_canon",
Lemma "efficient_recurrence") steps a real state of ``2d`` entries:

    y_t        = beta . x_t + b0 u_t
    x_{t+1}[0] = u_t - a . x_t,     x_{t+1}[m] = x_t[m-1]  (m >= 1)

and Proposition "fast_init" gives the state after a prompt without stepping:
``x_T = (v_{T-1}, ..., v_{T-2d})`` with ``v = g * u`` and ``g`` the impulse
response of ``1 / p(w)`` (``g_0 = 1``, ``g_t = -sum_m a_m g_{t-m}``).

Everything is float64 (coefficients from the complex128 roots through numpy
polynomial products).  Parity is pinned by ``tests/test_companion_pins.py``.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

__all__ = ["from_modal", "companion_matrix", "companion_run", "inverse_denominator_response", "fast_init"]


def _pair_poles(lam, R):
    lam = np.asarray(lam).astype(np.complex128)
    R = np.asarray(R).astype(np.complex128)
    rho = np.concatenate([lam, np.conj(lam)])
    r = np.concatenate([R / 2.0, np.conj(R) / 2.0])
    return rho, r


def from_modal(lam, R, h0) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Rational coefficients of every channel: ``a [D, 2d]`` (``a_1 .. a_2d``),
    ``beta [D, 2d]`` (``beta_1 .. beta_2d``) and ``b0 [D]`` (float64)."""
    lam = np.atleast_2d(lam)
    R = np.atleast_2d(R)
    D, d = lam.shape
    a = np.empty((D, 2 * d))
    beta = np.empty((D, 2 * d))
    for c in range(D):
        rho, r = _pair_poles(lam[c], R[c])
        # np.poly: coefficients of prod_k (x - rho_k), highest power first; in
        # w = 1/x the same list is p(w) = prod_k (1 - rho_k w), lowest first
        p = np.poly(rho)
        num = np.zeros(2 * d + 1, np.complex128)  # coefficients of w^0 .. w^2d
        for k in range(2 * d):
            others = np.poly(np.delete(rho, k))  # prod_{j != k} (1 - rho_j w), w^0 first
            num[1:] += r[k] * others
        a[c] = np.real(p[1:])
        beta[c] = np.real(num[1:])
    return a, beta, np.asarray(h0, np.float64).reshape(D).copy()


def companion_matrix(a) -> np.ndarray:
    """The ``2d x 2d`` state matrix of the companion canonical form
    (eq. "ssm_canon"): first row ``-a``, ones on the subdiagonal."""
    a = np.asarray(a, np.float64)
    n = a.shape[0]
    A = np.zeros((n, n))
    A[0, :] = -a
    A[np.arange(1, n), np.arange(n - 1)] = 1.0
    return A


def companion_run(a, beta, b0, u, x0=None) -> Tuple[np.ndarray, np.ndarray]:
    """Run the companion state-space system ``(A_c, e_1, beta, b0)`` of one
    channel over ``u [L]`` from ``x0`` (zeros by default): ``y_t = beta . x_t
    + b0 u_t`` and ``x_{t+1} = A_c x_t + e_1 u_t`` with the explicit matrix of
    ``companion_matrix``.  Returns ``y [L]`` and the final state ``[2d]``."""
    A = companion_matrix(a)
    beta = np.asarray(beta, np.float64)
    u = np.asarray(u, np.float64)
    n = A.shape[0]
    e1 = np.zeros(n)
    e1[0] = 1.0
    x = np.zeros(n) if x0 is None else np.asarray(x0, np.float64).copy()
    y = np.empty(u.shape[0])
    for t in range(u.shape[0]):
        y[t] = float(np.dot(beta, x)) + float(b0) * u[t]
        x = A @ x + e1 * u[t]
    return y, x


def inverse_denominator_response(a, L: int) -> np.ndarray:
    """``g_t``, ``t < L``: impulse response of ``1 / p(w)``."""
    a = np.asarray(a, np.float64)
    g = np.zeros(L)
    for t in range(L):
        acc = 1.0 if t == 0 else 0.0
        for m in range(1, min(t, a.shape[0]) + 1):
            acc -= a[m - 1] * g[t - m]
        g[t] = acc
    return g


def fast_init(a, u) -> np.ndarray:
    """State after the prompt ``u [T]`` of one channel by Proposition
    "fast_init": ``x_T[j] = v_{T-1-j}`` with ``v = g * u`` (``v_t = 0`` for
    ``t < 0``)."""
    a = np.asarray(a, np.float64)
    u = np.asarray(u, np.float64)
    T = u.shape[0]
    n = a.shape[0]
    g = inverse_denominator_response(a, T)
    x = np.zeros(n)
    for j in range(n):
        t = T - 1 - j
        if t >= 0:
            x[j] = np.dot(g[t::-1], u[:t + 1])  # sum_k g_{t-k} u_k
    return x
