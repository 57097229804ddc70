"""CPU oracle for the distillation objective -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run anything in this package.  The product path
never calls it and shares no code with it.

The step before the deployed recurrence (Sec. 3.2, "Modal canonical form"):
each channel's filter is fitted by the modal impulse response (eq.
"modal_impulse") with poles in polar form ``lambda_n = A_n e^{i theta_n}`` and
residues ``R_n`` in cartesian form, minimising the squared l2 interpolation
error against a real target over ``t = 1 .. L``:

    hhat_t = Re sum_n R_n lambda_n^(t-1),       loss = sum_{t=1}^{L} (hhat_t - h_t)^2

(the pass-through ``h0`` is matched exactly by ``h_0`` and is not part of the
objective).  The gradients follow from differentiating that definition, with
``e_t = hhat_t - h_t``:

    d loss / d Re R_n  =  2 sum_t e_t Re(lambda_n^(t-1))
    d loss / d Im R_n  = -2 sum_t e_t Im(lambda_n^(t-1))
    d loss / d A_n     =  2 sum_t e_t Re(R_n (t-1) lambda_n^(t-2) e^{i theta_n})
    d loss / d theta_n =  2 sum_t e_t Re(R_n i (t-1) lambda_n^(t-1))

(``d lambda / d A = e^{i theta}``, ``d lambda / d theta = i lambda``; the
``t = 1`` terms of the pole gradients vanish).  Everything is evaluated in
float64 from the float32 parameters, powers as running products.

Parity is pinned by ``tests/test_distill_pins.py``.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from . import power_table

__all__ = ["modal_filter", "distill_loss_grad"]


def _poles(A, theta) -> np.ndarray:
    A = np.asarray(A, np.float64)
    theta = np.asarray(theta, np.float64)
    return A * np.exp(1j * theta)


def modal_filter(A, theta, R, L: int) -> np.ndarray:
    """``hhat[c, t-1] = Re sum_n R[c,n] lambda[c,n]^(t-1)`` for ``t = 1 .. L``
    (float64 ``[D, L]``)."""
    lam = _poles(A, theta)
    R = np.asarray(R).astype(np.complex128)
    P = power_table(lam, L)  # [D, d, L]: lambda^(t-1) at index t-1
    return np.real(np.einsum("cn,cnt->ct", R, P))


def distill_loss_grad(A, theta, R, target) -> Dict[str, np.ndarray]:
    """Loss ``[D]`` and gradients ``dA, dtheta [D, d]`` (float64), ``dR
    [D, d]`` (complex128: ``d/dRe R + i d/dIm R``) for targets ``[D, L]``."""
    target = np.asarray(target, np.float64)
    L = target.shape[1]
    lam = _poles(A, theta)
    R = np.asarray(R).astype(np.complex128)
    P = power_table(lam, L)  # lambda^(t-1)
    hhat = np.real(np.einsum("cn,cnt->ct", R, P))
    e = hhat - target
    loss = np.sum(e * e, axis=1)
    g = np.einsum("ct,cnt->cn", e, P)  # sum_t e_t lambda^(t-1)
    dR = 2.0 * (g.real - 1j * g.imag)
    # lambda^(t-2) (t - 1): zero at t = 1, lambda^0 = 1 at t = 2
    tm1 = np.arange(L, dtype=np.float64)  # t - 1
    Pm = np.zeros_like(P)
    if L > 1:
        Pm[..., 1:] = P[..., :-1]  # lambda^(t-2) for t >= 2
    S = np.einsum("ct,t,cnt->cn", e, tm1, Pm)  # sum_t e_t (t-1) lambda^(t-2)
    unit = np.exp(1j * np.asarray(theta, np.float64))
    dA = 2.0 * np.real(R * S * unit)
    dtheta = 2.0 * np.real(R * 1j * S * lam)
    return {"loss": loss, "dA": dA, "dtheta": dtheta, "dR": dR, "hhat": hhat}
