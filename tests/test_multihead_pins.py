"""Pins of the multi-head oracle (``oracle.multihead``) against what the paper
and the mathematics fix: a hand-derived worked example, the one-channel head
(a library convolution), a plain-Python recurrence, the rank-one closed form
and the constant-input (partial Neumann series) closed form.  Planted mistakes
in the oracle must fail at least one pin.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import pytest

import oracle
import oracle.multihead as mh

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "multihead", "tiny.json")


def rand_heads(rng, B, L, M, N, d, r=(0.5, 0.97)):
    lam = (rng.uniform(*r, (M, d)) * np.exp(1j * rng.uniform(0, math.pi, (M, d)))).astype(np.complex64)
    R = (rng.standard_normal((M, d)) + 1j * rng.standard_normal((M, d))).astype(np.complex64)
    h0 = rng.standard_normal(M).astype(np.float32)
    q, k, v = (rng.standard_normal((B, L, M, N)).astype(np.float32) for _ in range(3))
    return lam, R, h0, q, k, v


def brute_heads(lam, R, h0, q, k, v):
    """Plain-Python recurrence per entry (Proposition "modal_realization"):
    w_t[i,j] = Re(sum_n R_n x[i,j,n]) + h0 z_t[i,j], y_t[i] = sum_j w_t[i,j] q_t[j],
    then x[i,j,n] <- lam_n x[i,j,n] + z_t[i,j].  Returns (y[B,L,M,N], x[B,M,N,N,d])."""
    B, L, M, N = q.shape
    d = lam.shape[1]
    y = [[[[0.0] * N for _ in range(M)] for _ in range(L)] for _ in range(B)]
    X = [[[[[0j] * d for _ in range(N)] for _ in range(N)] for _ in range(M)] for _ in range(B)]
    for b in range(B):
        for m in range(M):
            lm = [complex(z) for z in lam[m]]
            rm = [complex(z) for z in R[m]]
            hm = float(h0[m])
            for t in range(L):
                for i in range(N):
                    acc = 0.0
                    for j in range(N):
                        z = float(k[b, t, m, i]) * float(v[b, t, m, j])
                        x = X[b][m][i][j]
                        w = sum(r * xn for r, xn in zip(rm, x)).real + hm * z
                        acc += w * float(q[b, t, m, j])
                        X[b][m][i][j] = [l * xn + z for l, xn in zip(lm, x)]
                    y[b][t][m][i] = acc
    return np.array(y), np.array(X)


def pin_golden():
    g = json.load(open(GOLDEN))
    lam = np.array([[complex(*p) for p in row] for row in g["lambda"]], np.complex64)
    R = np.array([[complex(*p) for p in row] for row in g["R"]], np.complex64)
    h0 = np.array(g["h0"], np.float32)
    q = np.array(g["q"], np.float32)[None, :, None, :]
    k = np.array(g["k"], np.float32)[None, :, None, :]
    v = np.array(g["v"], np.float32)[None, :, None, :]
    y = mh.mh_outputs(lam, R, h0, q, k, v)
    np.testing.assert_allclose(y[0, :, 0, :], np.array(g["y"], float), rtol=0, atol=1e-12)
    for T, xs in g["x"].items():
        x = mh.mh_state(lam, k, v, int(T))
        np.testing.assert_allclose(x[0, 0, :, :, 0], np.array(xs, complex), rtol=0, atol=1e-12)


def pin_scalar_head_is_library_convolution():
    # N = 1: y_t = q_t (h * (k v))_t with np.convolve taking the library route
    rng = np.random.default_rng(3)
    lam, R, h0, q, k, v = rand_heads(rng, 2, 37, 3, 1, 4)
    y = mh.mh_outputs(lam, R, h0, q, k, v)
    L = q.shape[1]
    for m in range(3):
        t = np.arange(L)
        pw = lam[m].astype(np.complex128)[:, None] ** np.maximum(t - 1, 0)[None, :]
        h = np.where(t == 0, float(h0[m]), np.real(R[m].astype(np.complex128) @ pw))
        for b in range(2):
            zk = k[b, :, m, 0].astype(float) * v[b, :, m, 0].astype(float)
            ref = np.convolve(h, zk)[:L] * q[b, :, m, 0].astype(float)
            np.testing.assert_allclose(y[b, :, m, 0], ref, rtol=1e-11, atol=1e-11)


def pin_brute_recurrence():
    rng = np.random.default_rng(4)
    lam, R, h0, q, k, v = rand_heads(rng, 2, 9, 2, 3, 3)
    yb, xb = brute_heads(lam, R, h0, q, k, v)
    np.testing.assert_allclose(mh.mh_outputs(lam, R, h0, q, k, v), yb, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(mh.mh_state(lam, k, v, 9), xb, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(mh.mh_state(lam, k[:, :4], v[:, :4], 4),
                               brute_heads(lam, R, h0, q[:, :4], k[:, :4], v[:, :4])[1],
                               rtol=1e-10, atol=1e-10)


def pin_rank_one_closed_form():
    # k_s = a_s e, v_s = c_s f: w_t = (h * (a c))_t e f^T, so y_t = (h * (a c))_t (f . q_t) e
    rng = np.random.default_rng(5)
    M, N, L, d = 2, 5, 23, 3
    lam, R, h0, q, _, _ = rand_heads(rng, 1, L, M, N, d)
    e = rng.standard_normal(N).astype(np.float32)
    f = rng.standard_normal(N).astype(np.float32)
    a = rng.standard_normal(L).astype(np.float32)
    c = rng.standard_normal(L).astype(np.float32)
    # float64 products of float32 factors are exact, so k and v factor exactly
    a64, c64, e64, f64 = (x.astype(np.float64) for x in (a, c, e, f))
    k = np.broadcast_to(a64[None, :, None, None] * e64[None, None, None, :], (1, L, M, N))
    v = np.broadcast_to(c64[None, :, None, None] * f64[None, None, None, :], (1, L, M, N))
    y = mh.mh_outputs(lam, R, h0, q, k, v)
    for m in range(M):
        t = np.arange(L)
        h = [float(h0[m])] + [sum((complex(r) * complex(l) ** (s - 1)).real
                                  for r, l in zip(R[m], lam[m])) for s in range(1, L)]
        g = np.convolve(np.array(h), a.astype(float) * c.astype(float))[:L]
        fq = q[0, :, m, :].astype(float) @ f.astype(float)
        ref = (g * fq)[:, None] * e.astype(float)[None, :]
        np.testing.assert_allclose(y[0, :, m, :], ref, rtol=1e-9, atol=1e-9)


def pin_constant_inputs_neumann():
    # k = v = q = 1: z = 1 everywhere, w_t = h0 + Re sum_n R_n (1 - lam_n^t)/(1 - lam_n),
    # y_t = N w_t and x_T = (1 - lam^T) / (1 - lam) in every entry
    M, N, L, d = 2, 3, 40, 2
    lam = np.array([[0.9 * np.exp(0.3j), 0.5 * np.exp(-1.1j)], [0.7, -0.6 + 0.2j]], np.complex64)
    R = np.array([[1 + 2j, -0.5 + 0.25j], [0.75, 2 - 1j]], np.complex64)
    h0 = np.array([0.5, -1.5], np.float32)
    ones = np.ones((1, L, M, N), np.float32)
    y = mh.mh_outputs(lam, R, h0, ones, ones, ones)
    for m in range(M):
        lm = lam[m].astype(np.complex128)
        rm = R[m].astype(np.complex128)
        for t in range(L):
            w = float(h0[m]) + (rm * (1 - lm ** t) / (1 - lm)).sum().real
            np.testing.assert_allclose(y[0, t, m, :], N * w, rtol=1e-10)
    x = mh.mh_state(lam, ones, ones, 17)
    for m in range(M):
        lm = lam[m].astype(np.complex128)
        np.testing.assert_allclose(x[0, m], np.broadcast_to((1 - lm ** 17) / (1 - lm), (N, N, d)),
                                   rtol=1e-10)


def pin_bilinear_and_zero():
    rng = np.random.default_rng(6)
    lam, R, h0, q, k, v = rand_heads(rng, 1, 11, 2, 4, 2)
    k2 = rng.standard_normal(k.shape).astype(np.float32)
    y1 = mh.mh_outputs(lam, R, h0, q, k, v)
    y2 = mh.mh_outputs(lam, R, h0, q, k2, v)
    y12 = mh.mh_outputs(lam, R, h0, q, (k.astype(float) + 2 * k2.astype(float)), v)
    np.testing.assert_allclose(y12, y1 + 2 * y2, rtol=1e-9, atol=1e-9)
    assert np.all(mh.mh_outputs(lam, R, h0, q, k, np.zeros_like(v)) == 0)
    assert np.all(mh.mh_state(lam, k, v, 0) == 0)


PINS = [pin_golden, pin_scalar_head_is_library_convolution, pin_brute_recurrence,
        pin_rank_one_closed_form, pin_constant_inputs_neumann, pin_bilinear_and_zero]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin()


def test_rows_match_full():
    rng = np.random.default_rng(7)
    lam, R, h0, q, k, v = rand_heads(rng, 2, 13, 3, 4, 2)
    full = mh.mh_outputs(lam, R, h0, q, k, v)
    rows = [(1, 2, 3), (0, 0, 0), (1, 1, 2)]
    part = mh.mh_outputs_rows(lam, R, h0, q, k, v, rows)
    for r, (b, m, i) in enumerate(rows):
        np.testing.assert_array_equal(part[r], full[b, :, m, i])
    xs = mh.mh_state_rows(lam, k, v, 9, rows)
    xf = mh.mh_state(lam, k, v, 9)
    for r, (b, m, i) in enumerate(rows):
        np.testing.assert_array_equal(xs[r], xf[b, m, i])


# ----------------------------------------------------------------------------
# planted mistakes: each mutant of the oracle must fail at least one pin
# ----------------------------------------------------------------------------

def _mut_transposed(lam, R, h0, q, k, v, rows):
    # contracts q with the key index instead of the value index
    return _orig_rows(lam, R, h0, q, v, k, rows)


def _mut_no_h0(lam, R, h0, q, k, v, rows):
    return _orig_rows(lam, R, np.zeros_like(np.asarray(h0)), q, k, v, rows)


def _mut_conj(lam, R, h0, q, k, v, rows):
    return _orig_rows(lam, np.conj(np.asarray(R)), h0, q, k, v, rows)


def _mut_state_off_by_one(lam, k, v, T, rows):
    return _orig_state(lam, k, v, T + 1 if T > 0 else 0, rows) if T + 1 <= np.shape(k)[1] else \
        _orig_state(lam, k, v, T, rows) * np.asarray(lam).astype(complex)[rows[0][1]][None, None, :]


def _mut_state_no_reverse(lam, k, v, T, rows):
    k, v = np.asarray(k, float), np.asarray(v, float)
    out = _orig_state(lam, k[:, :T][:, ::-1], v[:, :T][:, ::-1], T, rows)
    return out


_orig_rows = mh.mh_outputs_rows
_orig_state = mh.mh_state_rows
MUTANTS = {
    "transposed_contraction": ("mh_outputs_rows", _mut_transposed),
    "dropped_h0": ("mh_outputs_rows", _mut_no_h0),
    "conjugated_residues": ("mh_outputs_rows", _mut_conj),
    "state_off_by_one": ("mh_state_rows", _mut_state_off_by_one),
    "state_time_reversed": ("mh_state_rows", _mut_state_no_reverse),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(mh, attr, fn)
    caught = []
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"
