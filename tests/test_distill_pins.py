"""Pins of the distillation-objective oracle (``oracle.distill``): the polar
closed form of the modal filter printed in Sec. 3.2, zero loss and gradient at
an exactly representable target, the geometric-series closed forms of a single
real mode, and central finite differences of the loss for every gradient.
Planted mistakes in the oracle must fail at least one pin.
"""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle.distill as od


def rand_params(rng, D, d, L, a=(0.3, 0.98)):
    A = rng.uniform(*a, (D, d)).astype(np.float32)
    th = rng.uniform(0, math.pi, (D, d)).astype(np.float32)
    R = (rng.standard_normal((D, d)) + 1j * rng.standard_normal((D, d))).astype(np.complex64)
    tgt = rng.standard_normal((D, L)).astype(np.float32) * 0.3
    return A, th, R, tgt


def pin_polar_form():
    # Re hhat_t = sum_n A_n^(t-1) [Re R_n cos(theta_n (t-1)) - Im R_n sin(theta_n (t-1))]
    rng = np.random.default_rng(1)
    A, th, R, _ = rand_params(rng, 3, 4, 50)
    h = od.modal_filter(A, th, R, 50)
    for c in range(3):
        for t in range(1, 51):
            ref = sum(float(A[c, n]) ** (t - 1) * (float(R[c, n].real) * math.cos(float(th[c, n]) * (t - 1))
                                                   - float(R[c, n].imag) * math.sin(float(th[c, n]) * (t - 1)))
                      for n in range(4))
            assert abs(h[c, t - 1] - ref) <= 1e-12 * max(1.0, abs(ref)), (c, t)


def pin_exact_target_is_stationary():
    rng = np.random.default_rng(2)
    A, th, R, _ = rand_params(rng, 4, 3, 40)
    tgt = od.modal_filter(A, th, R, 40)
    out = od.distill_loss_grad(A, th, R, tgt)
    assert np.all(out["loss"] <= 1e-24)
    for k in ("dA", "dtheta", "dR"):
        assert np.max(np.abs(out[k])) <= 1e-11, k


def pin_single_real_mode_closed_form():
    # theta = 0, R = r real, target 0: e_t = r a^(t-1), loss = r^2 (1 - a^(2L)) / (1 - a^2),
    # dA = 2 r^2 sum_k k a^(2k-1) = (2 r^2 / a) x (1 - L x^(L-1) + (L-1) x^L) / (1 - x)^2, x = a^2,
    # dR = 2 r (1 - x^L) / (1 - x) (real), dtheta = 0 (the imaginary parts vanish)
    a, r, L = 0.8, 1.5, 37
    x = a * a
    out = od.distill_loss_grad(np.array([[a]]), np.array([[0.0]]), np.array([[r + 0j]]), np.zeros((1, L)))
    assert abs(out["loss"][0] - r * r * (1 - x ** L) / (1 - x)) <= 1e-12
    dA = 2 * r * r / a * x * (1 - L * x ** (L - 1) + (L - 1) * x ** L) / (1 - x) ** 2
    assert abs(out["dA"][0, 0] - dA) <= 1e-11 * abs(dA)
    assert abs(out["dR"][0, 0] - 2 * r * (1 - x ** L) / (1 - x)) <= 1e-11
    assert abs(out["dtheta"][0, 0]) <= 1e-12


def pin_finite_differences():
    rng = np.random.default_rng(3)
    D, d, L = 2, 3, 29
    A, th, R, tgt = rand_params(rng, D, d, L)
    A, th = A.astype(np.float64), th.astype(np.float64)
    R = R.astype(np.complex128)
    out = od.distill_loss_grad(A, th, R, tgt)

    def loss(A_, th_, R_):
        e = od.modal_filter(A_, th_, R_, L) - tgt.astype(np.float64)
        return np.sum(e * e, axis=1)

    eps = 1e-6
    for c in range(D):
        for n in range(d):
            for name, grad in (("A", out["dA"][c, n]), ("theta", out["dtheta"][c, n]),
                               ("ReR", out["dR"][c, n].real), ("ImR", out["dR"][c, n].imag)):
                Ap, Am, tp, tm, Rp, Rm = A.copy(), A.copy(), th.copy(), th.copy(), R.copy(), R.copy()
                if name == "A":
                    Ap[c, n] += eps; Am[c, n] -= eps
                elif name == "theta":
                    tp[c, n] += eps; tm[c, n] -= eps
                elif name == "ReR":
                    Rp[c, n] += eps; Rm[c, n] -= eps
                else:
                    Rp[c, n] += 1j * eps; Rm[c, n] -= 1j * eps
                fd = (loss(Ap, tp, Rp)[c] - loss(Am, tm, Rm)[c]) / (2 * eps)
                assert abs(fd - grad) <= 1e-6 * max(1.0, abs(grad)), (name, c, n, fd, grad)


PINS = [pin_polar_form, pin_exact_target_is_stationary, pin_single_real_mode_closed_form,
        pin_finite_differences]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin()


def test_loss_matches_filter():
    rng = np.random.default_rng(4)
    A, th, R, tgt = rand_params(rng, 3, 2, 17)
    out = od.distill_loss_grad(A, th, R, tgt)
    np.testing.assert_array_equal(out["hhat"], od.modal_filter(A, th, R, 17))


# ----------------------------------------------------------------------------
# planted mistakes
# ----------------------------------------------------------------------------
_orig = od.distill_loss_grad
_orig_filter = od.modal_filter


def _m_no_two(*a):
    o = dict(_orig(*a)); o["dA"] = o["dA"] / 2; return o


def _m_imr_sign(*a):
    o = dict(_orig(*a)); o["dR"] = np.conj(o["dR"]); return o


def _m_theta_no_lambda(A, th, R, tgt):
    o = dict(_orig(A, th, R, tgt))
    lam = np.asarray(A, float) * np.exp(1j * np.asarray(th, float))
    o["dtheta"] = o["dtheta"] / np.where(np.abs(lam) > 0, np.abs(lam), 1)
    return o


def _m_filter_power_t(A, th, R, L):
    lam = np.asarray(A, float) * np.exp(1j * np.asarray(th, float))
    return np.real(_orig_filter(A, th, np.asarray(R) * lam, L))  # lambda^t instead of lambda^(t-1)


MUTANTS = {
    "gradient_missing_factor_two": ("distill_loss_grad", _m_no_two),
    "imaginary_residue_sign": ("distill_loss_grad", _m_imr_sign),
    "theta_gradient_scaled": ("distill_loss_grad", _m_theta_no_lambda),
    "filter_power_off_by_one": ("modal_filter", _m_filter_power_t),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(od, attr, fn)
    caught = []
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"
