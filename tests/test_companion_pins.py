"""Pins of the companion-form oracle (``oracle.companion``): the transfer
function identity against the partial fractions of the modal form, the
impulse response of the rational filter through scipy's difference-equation
filter against the modal filter, the closed form of the transfer function's
numerator through the matrix determinant lemma (the canonization recipe of the
paper, computed with numpy eigenvalues), the closed form of one real mode, the
companion recurrence against direct convolution and a difference-equation
route for its state, and the fast initialisation against the recurrence.
Planted mistakes in the oracle must fail at least one pin.
"""
from __future__ import annotations

import numpy as np
import pytest
import scipy.signal

import oracle
import oracle.companion as oc


def rand_modal(rng, D, d, r=(0.3, 0.9)):
    lam = (rng.uniform(*r, (D, d)) * np.exp(1j * rng.uniform(0, np.pi, (D, d)))).astype(np.complex64)
    R = ((rng.standard_normal((D, d)) + 1j * rng.standard_normal((D, d))) / np.sqrt(2 * d)).astype(np.complex64)
    h0 = rng.standard_normal(D).astype(np.float32)
    return lam, R, h0


def full_coeffs(a, beta, b0):
    """Numerator and denominator of H(w) = b0 + beta(w) / p(w) as one fraction."""
    den = np.concatenate([[1.0], a])
    num = b0 * den
    num[1:] += beta
    return num, den


def pin_transfer_function_identity():
    # H(w) = b0 + sum_k r_k w / (1 - rho_k w) over the 2d conjugate-paired poles
    rng = np.random.default_rng(1)
    lam, R, h0 = rand_modal(rng, 3, 4)
    a, beta, b0 = oc.from_modal(lam, R, h0)
    for c in range(3):
        rho = np.concatenate([lam[c], np.conj(lam[c])]).astype(np.complex128)
        res = np.concatenate([R[c] / 2, np.conj(R[c]) / 2]).astype(np.complex128)
        num, den = full_coeffs(a[c], beta[c], b0[c])
        for w in rng.standard_normal(6) * 0.7 + 1j * rng.standard_normal(6) * 0.7:
            ref = float(h0[c]) + np.sum(res * w / (1 - rho * w))
            got = np.polyval(num[::-1], w) / np.polyval(den[::-1], w)
            assert abs(got - ref) <= 1e-10 * max(1.0, abs(ref)), (c, w)


def pin_impulse_response_is_the_modal_filter():
    rng = np.random.default_rng(2)
    lam, R, h0 = rand_modal(rng, 4, 3)
    a, beta, b0 = oc.from_modal(lam, R, h0)
    L = 60
    h = oracle.filter_taps(lam, R, h0, L)
    imp = np.zeros(L)
    imp[0] = 1.0
    for c in range(4):
        num, den = full_coeffs(a[c], beta[c], b0[c])
        got = scipy.signal.lfilter(num, den, imp)
        assert np.max(np.abs(got - h[c])) <= 1e-10 * np.max(np.abs(h[c])), c


def pin_determinant_lemma_numerator():
    # A = diag(rho), B = 1, C = r: by the matrix determinant lemma
    # det(zI - A + B C) = det(zI - A) (1 + C (zI - A)^-1 B), so the order-2d
    # numerator of H in z is det(zI - A + B C) + (h0 - 1) det(zI - A) and its
    # denominator det(zI - A).  Both determinants are evaluated numerically
    # (np.linalg.det of the explicit matrices) at points z and compared with
    # the oracle's polynomials, read in z (w = 1/z, times z^2d).
    rng = np.random.default_rng(3)
    lam, R, h0 = rand_modal(rng, 3, 3)
    a, beta, b0 = oc.from_modal(lam, R, h0)
    for c in range(3):
        rho = np.concatenate([lam[c], np.conj(lam[c])]).astype(np.complex128)
        res = np.concatenate([R[c] / 2, np.conj(R[c]) / 2]).astype(np.complex128)
        n2 = rho.shape[0]
        A = np.diag(rho)
        BC = np.outer(np.ones(n2), res)
        num, den = full_coeffs(a[c], beta[c], b0[c])
        for z in (1.3, -0.8 + 0.9j, 2.0j, 0.4 - 1.7j):
            I = np.eye(n2)
            num_ref = np.linalg.det(z * I - A + BC) + (float(h0[c]) - 1.0) * np.linalg.det(z * I - A)
            den_ref = np.linalg.det(z * I - A)
            num_z = np.polyval(num, z)  # sum_m num[m] z^(2d-m)
            den_z = np.polyval(den, z)
            assert abs(num_z - num_ref) <= 1e-9 * max(1.0, abs(num_ref)), (c, z)
            assert abs(den_z - den_ref) <= 1e-10 * max(1.0, abs(den_ref)), (c, z)


def pin_single_real_mode_closed_form():
    # lambda = l real, R = q real: p(w) = (1 - l w)^2, beta(w) = q w - q l w^2
    l, q, h0 = 0.6, 1.25, 0.5
    a, beta, b0 = oc.from_modal(np.array([[l]]), np.array([[q + 0j]]), np.array([h0]))
    np.testing.assert_allclose(a[0], [-2 * l, l * l], rtol=0, atol=1e-15)
    np.testing.assert_allclose(beta[0], [q, -q * l], rtol=0, atol=1e-15)
    assert b0[0] == h0


def pin_recurrence_outputs_and_state():
    rng = np.random.default_rng(5)
    lam, R, h0 = rand_modal(rng, 3, 2)
    a, beta, b0 = oc.from_modal(lam, R, h0)
    L = 80
    u = rng.standard_normal((3, L))
    h = oracle.filter_taps(lam, R, h0, L)
    y_ref = oracle.causal_conv(h, u)
    for c in range(3):
        y, x = oc.companion_run(a[c], beta[c], b0[c], u[c])
        assert np.max(np.abs(y - y_ref[c])) <= 1e-10 * np.max(np.abs(y_ref[c])), c
        # state by the difference equation of 1 / p: x_L = (v_{L-1}, ..., v_{L-2d})
        v = scipy.signal.lfilter([1.0], np.concatenate([[1.0], a[c]]), u[c])
        np.testing.assert_allclose(x, v[::-1][: a.shape[1]], rtol=1e-10, atol=1e-12)


def pin_fast_init_matches_recurrence():
    rng = np.random.default_rng(6)
    lam, R, h0 = rand_modal(rng, 2, 3)
    a, beta, b0 = oc.from_modal(lam, R, h0)
    for T in (0, 1, 3, 6, 7, 50):
        u = rng.standard_normal(T)
        for c in range(2):
            _, x = oc.companion_run(a[c], beta[c], b0[c], u)
            np.testing.assert_allclose(oc.fast_init(a[c], u), x, rtol=1e-10, atol=1e-12)


PINS = [pin_transfer_function_identity, pin_impulse_response_is_the_modal_filter,
        pin_determinant_lemma_numerator, pin_single_real_mode_closed_form,
        pin_recurrence_outputs_and_state, pin_fast_init_matches_recurrence]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin()


def test_decode_continues_prompt():
    # stepping the companion state after a fast initialisation continues the
    # convolution with the modal filter (the decode after a prefill)
    rng = np.random.default_rng(7)
    lam, R, h0 = rand_modal(rng, 2, 2)
    a, beta, b0 = oc.from_modal(lam, R, h0)
    T, K = 30, 12
    u = rng.standard_normal((2, T + K))
    y_ref = oracle.causal_conv(oracle.filter_taps(lam, R, h0, T + K), u)
    for c in range(2):
        x = oc.fast_init(a[c], u[c, :T])
        y, _ = oc.companion_run(a[c], beta[c], b0[c], u[c, T:], x)
        assert np.max(np.abs(y - y_ref[c, T:])) <= 1e-10 * np.max(np.abs(y_ref[c])), c


# ----------------------------------------------------------------------------
# planted mistakes
# ----------------------------------------------------------------------------
_from = oc.from_modal
_run = oc.companion_run
_init = oc.fast_init


def _m_no_conjugate_half(lam, R, h0):
    # residue R instead of the pair (R/2, conj(R)/2): twice the filter's real part
    a, beta, b0 = _from(lam, R, h0)
    return a, 2 * beta, b0


def _m_beta_shift(lam, R, h0):
    a, beta, b0 = _from(lam, R, h0)
    return a, np.concatenate([beta[:, 1:], np.zeros_like(beta[:, :1])], axis=1), b0


def _m_feedback_sign(a, beta, b0, u, x0=None):
    return _run(-np.asarray(a), beta, b0, u, x0)


def _m_init_off_by_one(a, u):
    x = _init(a, np.concatenate([np.asarray(u, float), [0.0]]))  # (v_T, ..., v_{T-2d+1})
    return x


MUTANTS = {
    "residue_not_halved": ("from_modal", _m_no_conjugate_half),
    "numerator_shifted": ("from_modal", _m_beta_shift),
    "feedback_sign": ("companion_run", _m_feedback_sign),
    "fast_init_off_by_one": ("fast_init", _m_init_off_by_one),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(oc, attr, fn)
    caught = []
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"
