"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own formula: each compares it with a
closed form, a library routine that takes another route, a brute-force
recurrence in plain Python, or a hand-derived worked example under
``tests/golden/``.  ``test_planted_mistakes_are_caught`` plants plausible
mistakes in the oracle (on the CPU) and checks that some pin fails for each.
"""
from __future__ import annotations

import cmath
import glob
import json
import math
import os

import numpy as np
import pytest
import scipy.signal

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ----------------------------------------------------------------------------
# helpers that are independent of the oracle
# ----------------------------------------------------------------------------

def brute_recurrence(lam, R, h0, u):
    """Plain-Python diagonal recurrence of Proposition "modal_realization":
    y_t = Re(sum_n R_n x_t[n]) + h0 u_t, then x_{t+1}[n] = lam_n x_t[n] + u_t.
    Returns (list of y_t, list of states x_0..x_L)."""
    lam = [complex(v) for v in lam]
    R = [complex(v) for v in R]
    x = [0j] * len(lam)
    ys, xs = [], [list(x)]
    for ut in u:
        ut = float(ut)
        ys.append(sum(r * xn for r, xn in zip(R, x)).real + float(h0) * ut)
        x = [ln * xn + ut for ln, xn in zip(lam, x)]
        xs.append(list(x))
    return ys, xs


def rand_case(rng, B, D, d, T, K, r=(0.5, 0.97), th=math.pi):
    lam = (rng.uniform(*r, (D, d)) * np.exp(1j * rng.uniform(0, th, (D, d)))).astype(np.complex64)
    R = (rng.standard_normal((D, d)) + 1j * rng.standard_normal((D, d))).astype(np.complex64)
    h0 = rng.standard_normal(D).astype(np.float32)
    up = rng.standard_normal((B, T, D)).astype(np.float32)
    ud = rng.standard_normal((B, K, D)).astype(np.float32)
    return lam, R, h0, up, ud


def polar_taps(lam, R, h0, L):
    """Real filter from the polar closed form of Sec. 3.2, with math.cos/sin."""
    h = [float(h0)]
    for t in range(1, L):
        s = 0.0
        for ln, rn in zip(lam, R):
            ln, rn = complex(ln), complex(rn)
            A, th = abs(ln), cmath.phase(ln)
            s += A ** (t - 1) * (rn.real * math.cos(th * (t - 1)) - rn.imag * math.sin(th * (t - 1)))
        h.append(s)
    return np.array(h)


def relerr(a, b):
    a = np.asarray(a)
    b = np.asarray(b)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ----------------------------------------------------------------------------
# pins (each raises AssertionError on failure)
# ----------------------------------------------------------------------------

def pin_golden(path):
    g = json.load(open(path))
    lam = np.array([[complex(*z) for z in row] for row in g["lambda"]], np.complex64)
    R = np.array([[complex(*z) for z in row] for row in g["R"]], np.complex64)
    h0 = np.array(g["h0"], np.float32)
    u = np.array(g["u"], np.float32)
    T = g["T"]
    up = u[None, :T, None]
    ud = u[None, T:, None]
    out = oracle.run(lam, R, h0, up, ud)
    y = np.concatenate([out["y_prefill"][0, :, 0], out["y_dec"][0, :, 0]])
    np.testing.assert_allclose(y, np.array(g["y"], float), rtol=0, atol=1e-12)
    xT = np.array([complex(*z) for z in g["x_T"]])
    xE = np.array([complex(*z) for z in g["x_end"]])
    np.testing.assert_allclose(out["x_T"][0, 0], xT, rtol=0, atol=1e-12)
    np.testing.assert_allclose(out["x_end"][0, 0], xE, rtol=0, atol=1e-12)


def pin_impulse_polar():
    rng = np.random.default_rng(11)
    lam, R, h0, _, _ = rand_case(rng, 1, 2, 3, 1, 1)
    L = 300
    up = np.zeros((1, L, 2), np.float32)
    up[0, 0, :] = 1.0
    out = oracle.run(lam, R, h0, up, np.zeros((1, 0, 2), np.float32))
    for c in range(2):
        ref = polar_taps(lam[c], R[c], h0[c], L)
        assert relerr(out["y_prefill"][0, :, c], ref) < 1e-12


def pin_impulse_polar_long():
    # poles of the long-prompt workload (r up to 0.99999, near-DC angles) at
    # the last lag the workload reaches, t = T + K - 1
    w = workloads.workload("c5")
    lam, R, h0 = workloads.make_params(w)
    L = w.T + w.K
    chans = [0, 517]
    h = oracle.filter_taps(lam[chans], R[chans], h0[chans], L)
    for i, c in enumerate(chans):
        for t in (1, 2, 4097, L - 1):
            s = 0.0
            for ln, rn in zip(lam[c], R[c]):
                ln, rn = complex(ln), complex(rn)
                A, th = abs(ln), cmath.phase(ln)
                s += A ** (t - 1) * (rn.real * math.cos(th * (t - 1)) - rn.imag * math.sin(th * (t - 1)))
            scale = float(np.sum(np.abs(R[c])))
            assert abs(h[i, t] - s) <= 1e-9 * scale, (c, t, h[i, t], s)


def pin_step_response():
    # u = 1: partial Neumann series (App. A.4): x_T = (1 - lam^T)/(1 - lam),
    # y_t = h0 + Re sum_n R_n (1 - lam_n^t)/(1 - lam_n)
    rng = np.random.default_rng(5)
    lam, R, h0, _, _ = rand_case(rng, 1, 3, 4, 1, 1)
    T, K = 150, 40
    up = np.ones((1, T, 3), np.float32)
    ud = np.ones((1, K, 3), np.float32)
    out = oracle.run(lam, R, h0, up, ud)
    y = np.concatenate([out["y_prefill"][0], out["y_dec"][0]], axis=0)
    for c in range(3):
        l = lam[c].astype(np.complex128)
        r = R[c].astype(np.complex128)
        for t in range(T + K):
            ref = h0[c] + np.real(np.sum(r * (1 - l ** t) / (1 - l)))
            assert abs(y[t, c] - ref) <= 1e-10 * max(1.0, abs(ref))
        np.testing.assert_allclose(out["x_T"][0, c], (1 - l ** T) / (1 - l), rtol=1e-11)
        np.testing.assert_allclose(out["x_end"][0, c], (1 - l ** (T + K)) / (1 - l), rtol=1e-11)


def pin_sinusoid_state_long():
    # u_k = cos(w k), k < T = 65536 with the long-prompt poles:
    # x_T = 1/2 [(e^{iwT} - lam^T)/(e^{iw} - lam) + (e^{-iwT} - lam^T)/(e^{-iw} - lam)]
    w = workloads.workload("c5")
    lam, _, _ = workloads.make_params(w)
    T = w.T
    om = 0.0123
    u = np.cos(om * np.arange(T))
    for c in (3, 900):
        x = oracle.state_after(lam[c], u, T)
        for n in range(0, w.d, 7):
            l = complex(lam[c, n])
            lT = cmath.exp(T * cmath.log(l))
            z = cmath.exp(1j * om)
            ref = 0.5 * ((z ** T - lT) / (z - l) + (z.conjugate() ** T - lT) / (z.conjugate() - l))
            assert abs(x[n] - ref) <= 1e-9 * abs(ref), (c, n, x[n], ref)


def pin_brute_force():
    rng = np.random.default_rng(1)
    for (B, D, d, T, K) in [(1, 1, 1, 7, 3), (2, 3, 2, 20, 5), (1, 2, 4, 64, 16), (2, 2, 3, 33, 0),
                            (1, 1, 2, 0, 9)]:
        lam, R, h0, up, ud = rand_case(rng, B, D, d, T, K)
        out = oracle.run(lam, R, h0, up, ud)
        for b in range(B):
            for c in range(D):
                u = np.concatenate([up[b, :, c], ud[b, :, c]])
                ys, xs = brute_recurrence(lam[c], R[c], h0[c], u)
                ys = np.array(ys)
                np.testing.assert_allclose(out["y_prefill"][b, :, c], ys[:T], rtol=1e-11, atol=1e-11)
                np.testing.assert_allclose(out["y_dec"][b, :, c], ys[T:], rtol=1e-11, atol=1e-11)
                np.testing.assert_allclose(out["x_T"][b, c], np.array(xs[T]), rtol=1e-11, atol=1e-11)
                np.testing.assert_allclose(out["x_end"][b, c], np.array(xs[T + K]), rtol=1e-11, atol=1e-11)


def pin_lfilter_modal():
    # each mode is the first-order system R/(z - lam) = R z^-1 / (1 - lam z^-1)
    # (partial fractions, Proposition "modal_form"), filtered by scipy.signal.lfilter
    rng = np.random.default_rng(2)
    lam, R, h0, up, ud = rand_case(rng, 2, 3, 4, 90, 20)
    out = oracle.run(lam, R, h0, up, ud)
    T, K = 90, 20
    for b in range(2):
        for c in range(3):
            u = np.concatenate([up[b, :, c], ud[b, :, c]]).astype(np.float64)
            acc = np.zeros(T + K, np.complex128)
            for n in range(4):
                l = complex(lam[c, n])
                r = complex(R[c, n])
                acc += scipy.signal.lfilter([0.0, r], [1.0, -l], u.astype(np.complex128))
            y = np.real(acc) + float(h0[c]) * u
            np.testing.assert_allclose(out["y_prefill"][b, :, c], y[:T], rtol=1e-10, atol=1e-10)
            np.testing.assert_allclose(out["y_dec"][b, :, c], y[T:], rtol=1e-10, atol=1e-10)
            # state after T inputs = output at index T of the filter z^-1/(1 - lam z^-1)
            upad = np.concatenate([u[:T], [0.0]]).astype(np.complex128)
            xs = np.array([scipy.signal.lfilter([0.0, 1.0], [1.0, -complex(lam[c, n])], upad)[T]
                           for n in range(4)])
            np.testing.assert_allclose(out["x_T"][b, c], xs, rtol=1e-10, atol=1e-10)


def pin_transfer_function_route():
    # the same system as one rational transfer function in w = z^-1: the
    # partial fractions h0 + sum_n R_n w / (1 - lam_n w) brought over the
    # common denominator prod_n (1 - lam_n w) (expanded with np.convolve),
    # checked against the residue form on the unit circle and then run as a
    # difference equation by scipy.signal.lfilter; the real part of its
    # output is y (the real part of the modal filter's output)
    rng = np.random.default_rng(3)
    d = 3
    lam, R, h0, up, ud = rand_case(rng, 1, 2, d, 60, 10)
    out = oracle.run(lam, R, h0, up, ud)
    for c in range(2):
        ls = lam[c].astype(np.complex128)
        rs = R[c].astype(np.complex128)
        den = np.array([1.0 + 0j])
        for l in ls:
            den = np.convolve(den, [1.0, -l])
        num = float(h0[c]) * den
        for n in range(d):
            others = np.array([1.0 + 0j])
            for j in range(d):
                if j != n:
                    others = np.convolve(others, [1.0, -ls[j]])
            num[1:] += rs[n] * others
        for om in (0.0, 0.7, 2.1, np.pi):
            w = np.exp(-1j * om)
            ref = float(h0[c]) + np.sum(rs * w / (1 - ls * w))
            got = np.polyval(num[::-1], w) / np.polyval(den[::-1], w)
            assert abs(got - ref) <= 1e-11 * max(1.0, abs(ref)), (c, om)
        u = np.concatenate([up[0, :, c], ud[0, :, c]]).astype(np.complex128)
        y = np.real(scipy.signal.lfilter(num, den, u))
        ref = np.concatenate([out["y_prefill"][0, :, c], out["y_dec"][0, :, c]])
        assert relerr(ref, y) < 1e-8


def pin_fftconvolve():
    rng = np.random.default_rng(4)
    lam, R, h0, up, ud = rand_case(rng, 1, 2, 5, 700, 100, r=(0.9, 0.995))
    out = oracle.run(lam, R, h0, up, ud)
    L = 800
    for c in range(2):
        h = polar_taps(lam[c], R[c], h0[c], L)
        u = np.concatenate([up[0, :, c], ud[0, :, c]]).astype(np.float64)
        y = scipy.signal.fftconvolve(h, u)[:L]
        ref = np.concatenate([out["y_prefill"][0, :, c], out["y_dec"][0, :, c]])
        assert relerr(ref, y) < 1e-10


def pin_conjugate_pair():
    # App. B.1: poles (lam, lam*) with C = 1/2 [R, R*] give a real output equal
    # to the d-mode system's Re(R x) output.
    rng = np.random.default_rng(6)
    lam, R, h0, up, ud = rand_case(rng, 1, 1, 3, 40, 8)
    out = oracle.run(lam, R, h0, up, ud)
    u = np.concatenate([up[0, :, 0], ud[0, :, 0]])
    l2 = [complex(v) for v in lam[0]] + [complex(v).conjugate() for v in lam[0]]
    c2 = [0.5 * complex(v) for v in R[0]] + [0.5 * complex(v).conjugate() for v in R[0]]
    x = [0j] * 6
    ys = []
    for ut in u:
        ut = float(ut)
        yc = sum(cc * xn for cc, xn in zip(c2, x)) + float(h0[0]) * ut
        assert abs(yc.imag) < 1e-12 * max(1.0, abs(yc))
        ys.append(yc.real)
        x = [ln * xn + ut for ln, xn in zip(l2, x)]
    ref = np.concatenate([out["y_prefill"][0, :, 0], out["y_dec"][0, :, 0]])
    np.testing.assert_allclose(ref, np.array(ys), rtol=1e-11, atol=1e-11)


def pin_invariants():
    rng = np.random.default_rng(7)
    lam, R, h0, up, ud = rand_case(rng, 2, 3, 4, 50, 10)
    o1 = oracle.run(lam, R, h0, up, ud)
    # linearity in u
    up2 = rng.standard_normal(up.shape).astype(np.float32)
    ud2 = rng.standard_normal(ud.shape).astype(np.float32)
    o2 = oracle.run(lam, R, h0, up2, ud2)
    f = lambda a: a.astype(np.float64)
    o3 = oracle.run(lam, R, h0, 2 * f(up) - 3 * f(up2), 2 * f(ud) - 3 * f(ud2))
    for k in o1:
        np.testing.assert_allclose(o3[k], 2 * o1[k] - 3 * o2[k], rtol=1e-10, atol=1e-10)
    # time invariance: s leading zeros shift the output by s
    s = 7
    upz = np.concatenate([np.zeros((2, s, 3), np.float32), up], axis=1)
    o4 = oracle.run(lam, R, h0, upz, ud)
    np.testing.assert_allclose(o4["y_prefill"][:, s:], o1["y_prefill"], rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(o4["y_prefill"][:, :s], 0.0, atol=0)
    np.testing.assert_allclose(o4["x_T"], o1["x_T"], rtol=1e-11, atol=1e-11)
    # mode permutation
    perm = np.array([2, 0, 3, 1])
    o5 = oracle.run(lam[:, perm], R[:, perm], h0, up, ud)
    np.testing.assert_allclose(o5["y_dec"], o1["y_dec"], rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(o5["x_end"], o1["x_end"][:, :, perm], rtol=1e-11, atol=1e-11)
    # channel and batch independence
    up6 = up.copy()
    up6[1, :, 2] += 5.0
    o6 = oracle.run(lam, R, h0, up6, ud)
    np.testing.assert_allclose(o6["y_prefill"][0], o1["y_prefill"][0], rtol=0, atol=0)
    np.testing.assert_allclose(o6["y_prefill"][1, :, :2], o1["y_prefill"][1, :, :2], rtol=0, atol=0)
    # prefill(T) then K decode outputs == outputs of a prefill over T + K
    full = oracle.run(lam, R, h0, np.concatenate([up, ud], axis=1), ud[:, :0])
    np.testing.assert_allclose(full["y_prefill"][:, 50:], o1["y_dec"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(full["x_T"], o1["x_end"], rtol=1e-12, atol=1e-12)


def pin_conv_at():
    # one output of eq. "cnn" against numpy's full convolution (a library
    # route that shares nothing with the oracle), at the first lags, a middle
    # one and the last, on random rows, plus a hand-worked example:
    # h = (1, 2, 3), u = (4, 5, 6): y_0 = 4, y_1 = 2*4 + 5 = 13,
    # y_2 = 3*4 + 2*5 + 6 = 28
    assert oracle.conv_at([1.0, 2.0, 3.0], [4.0, 5.0, 6.0], 0) == 4.0
    assert oracle.conv_at([1.0, 2.0, 3.0], [4.0, 5.0, 6.0], 1) == 13.0
    assert oracle.conv_at([1.0, 2.0, 3.0], [4.0, 5.0, 6.0], 2) == 28.0
    rng = np.random.default_rng(12)
    for L in (1, 2, 7, 300, 4097):
        h = rng.standard_normal(L)
        u = rng.standard_normal(L)
        full = np.convolve(h, u)
        for t in sorted({0, 1 % L, L // 2, L - 1}):
            got = oracle.conv_at(h, u, t)
            assert abs(got - full[t]) <= 1e-12 * max(1.0, float(np.sum(np.abs(h[: t + 1]))) *
                                                      float(np.max(np.abs(u)))), (L, t)


def pin_run_rows_subset():
    # run_rows on a shuffled subset with repeated channels and batch rows must
    # return, in the order asked, each row's results as the plain-Python
    # recurrence gives them (no reference to the oracle's own helpers)
    rng = np.random.default_rng(13)
    B, D, d, T, K = 3, 5, 3, 25, 6
    lam, R, h0, up, ud = rand_case(rng, B, D, d, T, K)
    rows = [(2, 4), (0, 1), (2, 4), (1, 0), (0, 3), (1, 1), (2, 0)]
    out = oracle.run_rows(lam, R, h0, up, ud, rows)
    for i, (b, c) in enumerate(rows):
        u = np.concatenate([up[b, :, c], ud[b, :, c]])
        ys, xs = brute_recurrence(lam[c], R[c], h0[c], u)
        ys = np.array(ys)
        np.testing.assert_allclose(out["y_prefill"][i], ys[:T], rtol=1e-11, atol=1e-11)
        np.testing.assert_allclose(out["y_dec"][i], ys[T:], rtol=1e-11, atol=1e-11)
        np.testing.assert_allclose(out["x_T"][i], np.array(xs[T]), rtol=1e-11, atol=1e-11)
        np.testing.assert_allclose(out["x_end"][i], np.array(xs[T + K]), rtol=1e-11, atol=1e-11)


PINS = [pin_impulse_polar, pin_step_response, pin_brute_force, pin_lfilter_modal,
        pin_transfer_function_route, pin_fftconvolve, pin_conjugate_pair, pin_invariants,
        pin_conv_at, pin_run_rows_subset]
GOLDEN_FILES = sorted(glob.glob(os.path.join(GOLDEN, "*.json")))


# ----------------------------------------------------------------------------
# tests
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("path", GOLDEN_FILES, ids=[os.path.basename(p) for p in GOLDEN_FILES])
def test_golden(path):
    pin_golden(path)


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()


def test_impulse_polar_long():
    pin_impulse_polar_long()


def test_sinusoid_state_long():
    pin_sinusoid_state_long()


def test_power_table_matches_polar_form():
    w = workloads.workload("c5")
    lam, _, _ = workloads.make_params(w)
    m = w.T + w.K
    P = oracle.power_table(lam[5], m)
    for n in range(w.d):
        l = complex(lam[5, n])
        A, th = abs(l), cmath.phase(l)
        ref = A ** (m - 1) * complex(math.cos(th * (m - 1)), math.sin(th * (m - 1)))
        assert abs(P[n, m - 1] - ref) <= 1e-10 * abs(ref)
    # lam = 0: lam^0 = 1 and every later power 0
    P0 = oracle.power_table(np.zeros(2, np.complex64), 4)
    np.testing.assert_array_equal(P0, [[1, 0, 0, 0], [1, 0, 0, 0]])


def test_native_conv_matches_numpy_path():
    if not oracle.native_available():
        pytest.skip("oracle C helper not built (run __graft_entry__.build())")
    rng = np.random.default_rng(9)
    h = rng.standard_normal((5, 300))
    u = rng.standard_normal((5, 300))
    y = oracle.causal_conv(h, u)
    ref = np.stack([np.convolve(h[i], u[i])[:300] for i in range(5)])
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_degenerate_shapes():
    lam = np.full((2, 1), 0.5, np.complex64)
    R = np.ones((2, 1), np.complex64)
    h0 = np.zeros(2, np.float32)
    out = oracle.run(lam, R, h0, np.zeros((1, 0, 2), np.float32), np.zeros((1, 0, 2), np.float32))
    assert out["y_prefill"].shape == (1, 0, 2) and out["y_dec"].shape == (1, 0, 2)
    np.testing.assert_array_equal(out["x_T"], 0)


# ----------------------------------------------------------------------------
# planted mistakes: each mutant of the oracle must fail at least one pin
# ----------------------------------------------------------------------------

def _taps_power_t(lam, R, h0, L):  # lam^t instead of lam^(t-1)
    h = _orig_taps(lam, R, h0, L + 1)
    return np.concatenate([h[:, :1], h[:, 2:]], axis=1)


def _taps_conj(lam, R, h0, L):  # conjugated residues
    return _orig_taps(lam, np.conj(np.asarray(R)), h0, L)


def _taps_no_h0(lam, R, h0, L):  # dropped pass-through
    return _orig_taps(lam, R, np.zeros_like(np.asarray(h0)), L)


def _taps_imag(lam, R, h0, L):  # imaginary instead of real part
    return _orig_taps(lam, -1j * np.asarray(R), h0, L)


def _taps_post_update(lam, R, h0, L):  # output read after the state update
    h = _orig_taps(lam, R, h0, L + 1)
    out = h[:, 1:].copy()
    out[:, 0] += np.asarray(h0, np.float64).reshape(-1)
    return out


def _state_off_by_one(lam, u, T):  # x_{T-1} instead of x_T
    return _orig_state(lam, u, max(T - 1, 0))


def _state_reversed(lam, u, T):  # lam^k u_k instead of lam^(T-1-k) u_k
    u = np.asarray(u, np.float64)[:T]
    return _orig_state(lam, u[::-1], T)


def _conv_no_lag0(h, u):  # drops the j = t term
    y = _orig_conv(h, u)
    return y - np.asarray(h)[..., :1] * np.asarray(u)


def _conv_at_lag_shift(h, u, t):  # one lag off: sum_j h[t-1-j] u[j]
    h = np.asarray(h, np.float64)
    u = np.asarray(u, np.float64)
    return float(np.dot(h[t - 1::-1], u[:t])) if t > 0 else 0.0


def _run_rows_state_compact_index(lam, R, h0, u_prompt, u_dec, rows):
    # states from the poles at the row's position among the distinct channels
    # instead of its own channel (the same on full, in-order row sets)
    rows = list(rows)
    out = _orig_run_rows(lam, R, h0, u_prompt, u_dec, rows)
    chans = sorted({c for _, c in rows})
    cidx = {c: i for i, c in enumerate(chans)}
    lam = np.asarray(lam)
    T = u_prompt.shape[1]
    for i, (b, c) in enumerate(rows):
        uf = np.concatenate([u_prompt[b, :, c], u_dec[b, :, c]]).astype(np.float64)
        out["x_T"][i] = oracle.state_after(lam[cidx[c]], uf, T)
        out["x_end"][i] = oracle.state_after(lam[cidx[c]], uf, len(uf))
    return out


def _run_rows_sorted(lam, R, h0, u_prompt, u_dec, rows):  # rows returned sorted, not as asked
    return _orig_run_rows(lam, R, h0, u_prompt, u_dec, sorted(set(rows)) if rows else rows)


_orig_taps = oracle.filter_taps
_orig_state = oracle.state_after
_orig_conv = oracle.causal_conv
_orig_run_rows = oracle.run_rows

MUTANTS = {
    "power_t": ("filter_taps", _taps_power_t),
    "conj_R": ("filter_taps", _taps_conj),
    "no_h0": ("filter_taps", _taps_no_h0),
    "imag_part": ("filter_taps", _taps_imag),
    "post_update_output": ("filter_taps", _taps_post_update),
    "state_T_minus_1": ("state_after", _state_off_by_one),
    "state_reversed": ("state_after", _state_reversed),
    "conv_no_lag0": ("causal_conv", _conv_no_lag0),
    "conv_at_lag_shift": ("conv_at", _conv_at_lag_shift),
    "run_rows_state_compact_index": ("run_rows", _run_rows_state_compact_index),
    "run_rows_sorted": ("run_rows", _run_rows_sorted),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(oracle, attr, fn)
    caught = []
    for pin in PINS + [lambda: [pin_golden(p) for p in GOLDEN_FILES]]:
        try:
            pin()
        except AssertionError:
            caught.append(getattr(pin, "__name__", "golden"))
    assert caught, f"mutant {name} passed every pin"
