"""GPU parity of the companion form (``lh_companion_coeffs``,
``lh_companion_step``, ``lh_companion_init``) against the CPU oracle
(``oracle.companion`` for the coefficients and states, the modal direct
convolution of ``oracle`` for the outputs) on the same seeded inputs.

Tolerances.  Coefficients: per channel, ``max |c_gpu - c_ref| <= 1e-11
max(1, max |c_ref|)`` (float64 along two different routes: real quadratic
factors on the GPU, complex roots in the oracle).  States: per (b, c),
``max_m |x_gpu - x_ref| <= 1e-8 max_m |x_ref|`` (float64 recurrences and sums
whose terms exceed the result by at most ~1e6 in the cases below).  Outputs:
the modal path's row tolerance (1e-4, plus one rounding for bfloat16).  The
cases keep the orders and pole radii where the companion form is accurate
(it is not near the unit circle at d = 16; see ``include/lh.h``).
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import oracle.companion as oc
import workloads
from parity_util import _np, check_x, check_y, seq_rowmax

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    import paper_2310_18780_amd as lh

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    lh.lib()
    yield


def inputs(B, D, d, T, K, io, r, seed=0):
    w = workloads.Workload("case", B, D, d, T, K, io, r[0], r[1], np.pi, 1.0 / d, seed)
    return workloads.make_inputs(w)


def gpu_coeffs(lam, R):
    import torch

    import paper_2310_18780_amd as lh

    D, d = lam.shape
    a = torch.full((D, 2 * d), float("nan"), dtype=torch.float64, device="cuda")
    beta = torch.full_like(a, float("nan"))
    lh.companion_coeffs(torch.from_numpy(lam).cuda(), torch.from_numpy(R).cuda(), a, beta)
    torch.cuda.synchronize()
    return a, beta


def check_state(xg, xr, what):
    err = np.max(np.abs(xg - xr), axis=-1)
    scale = np.max(np.abs(xr), axis=-1)
    bad = err > 1e-8 * np.maximum(scale, 1e-300)
    assert not np.any(bad), f"{what}: rows {np.nonzero(bad)} err {err[bad]} scale {scale[bad]}"


COEFF_CASES = [(5, 1, (0.5, 0.99)), (7, 2, (0.5, 0.999)), (3, 4, (0.3, 0.99)), (4, 8, (0.5, 0.95)),
               (2, 16, (0.3, 0.9)), (300, 3, (0.5, 0.99))]


@pytest.mark.parametrize("case", COEFF_CASES, ids=[f"D{c[0]}_d{c[1]}" for c in COEFF_CASES])
def test_coefficients(case):
    D, d, r = case
    lam, R, h0, _, _ = inputs(1, D, d, 0, 0, "f32", r)
    a, beta = gpu_coeffs(lam, R)
    ar, br, _ = oc.from_modal(lam, R, h0)
    for name, g, ref in (("a", a.cpu().numpy(), ar), ("beta", beta.cpu().numpy(), br)):
        err = np.max(np.abs(g - ref), axis=1)
        scale = np.maximum(1.0, np.max(np.abs(ref), axis=1))
        assert np.all(err <= 1e-11 * scale), (name, np.max(err / scale))


def test_coefficients_special_poles():
    # lambda = 0 (factor 1), real poles (theta = 0: a double real root), R = 0
    lam = np.array([[0, 0.5, -0.25], [0.9, 0.9, 0.3j]], np.complex64)
    R = np.array([[1 + 1j, 0.5, 2], [0, 1 - 2j, 1j]], np.complex64)
    a, beta = gpu_coeffs(lam, R)
    ar, br, _ = oc.from_modal(lam, R, np.zeros(2, np.float32))
    np.testing.assert_allclose(a.cpu().numpy(), ar, rtol=0, atol=1e-14)
    np.testing.assert_allclose(beta.cpu().numpy(), br, rtol=0, atol=1e-14)


# (B, D, d, T0, K, io, r)
STEP_CASES = [
    (2, 70, 1, 30, 10, "f32", (0.5, 0.99)),
    (3, 33, 2, 50, 8, "bf16", (0.5, 0.99)),
    (1, 65, 4, 100, 12, "f32", (0.5, 0.95)),
    (2, 20, 8, 200, 6, "f32", (0.5, 0.9)),
    (1, 9, 16, 64, 5, "f32", (0.3, 0.6)),
    (2, 300, 4, 0, 7, "f32", (0.5, 0.95)),   # from the zero state
    (1, 5, 3, 2, 4, "bf16", (0.5, 0.9)),     # prompt shorter than the order
    (4, 257, 2, 1000, 3, "f32", (0.9, 0.999)),
    (5, 1, 4, 80, 4, "bf16", (0.5, 0.95)),   # a single channel
]


@pytest.mark.parametrize("case", STEP_CASES, ids=[
    f"B{c[0]}_D{c[1]}_d{c[2]}_T{c[3]}_K{c[4]}_{c[5]}" for c in STEP_CASES])
def test_coeffs_init_and_steps(case):
    """The product path end to end: coefficients, fast initialisation from the
    prompt, then K steps; states against the oracle's companion recurrence,
    outputs against the modal filter's direct convolution."""
    import torch

    import paper_2310_18780_amd as lh

    B, D, d, T0, K, io, r = case
    _log(f"[companion] {case}")
    lam, R, h0, up, ud = inputs(B, D, d, T0, K, io, r)
    iot = torch.bfloat16 if io == "bf16" else torch.float32
    a, beta = gpu_coeffs(lam, R)
    ar, br, b0 = oc.from_modal(lam, R, h0)
    u_t = torch.from_numpy(np.ascontiguousarray(up)).cuda().to(iot)
    state = torch.full((B, D, 2 * d), float("nan"), dtype=torch.float64, device="cuda")
    lh.companion_init(a, u_t, state)
    torch.cuda.synchronize()
    x0 = state.cpu().numpy()
    x0_ref = np.stack([np.stack([oc.fast_init(ar[c], up[b, :, c]) for c in range(D)])
                       for b in range(B)])
    check_state(x0.reshape(-1, 2 * d), x0_ref.reshape(-1, 2 * d), "fast initialisation")
    h0_t = torch.from_numpy(h0).cuda()
    ud_t = torch.from_numpy(np.ascontiguousarray(ud.transpose(1, 0, 2))).cuda().to(iot)
    y = torch.full((K, B, D), float("nan"), dtype=iot, device="cuda")
    for k in range(K):
        lh.companion_step(a, beta, h0_t, state, ud_t[k], y[k])
    torch.cuda.synchronize()
    xe = state.cpu().numpy()
    xe_ref = np.empty_like(xe)
    for b in range(B):
        for c in range(D):
            _, xe_ref[b, c] = oc.companion_run(ar[c], br[c], b0[c], ud[b, :, c], x0_ref[b, c])
    check_state(xe.reshape(-1, 2 * d), xe_ref.reshape(-1, 2 * d), "state after the steps")
    ref = oracle.run(lam, R, h0, up, ud)
    yg = _np(y).transpose(1, 2, 0).reshape(B * D, K)
    yr = ref["y_dec"].transpose(0, 2, 1).reshape(B * D, K)
    rm = seq_rowmax(ref["y_prefill"].transpose(0, 2, 1).reshape(B * D, T0), yr)
    e = check_y(yg, yr, io, "companion decode y", rowmax=rm)
    _log(f"[companion] {case} max row-relative output error {e:.2e}")


def test_init_t0_zeroes_the_state():
    import torch

    import paper_2310_18780_amd as lh

    a = torch.zeros((6, 4), dtype=torch.float64, device="cuda")
    u = torch.empty((2, 0, 6), device="cuda")
    state = torch.full((2, 6, 4), 3.0, dtype=torch.float64, device="cuda")
    lh.companion_init(a, u, state)
    torch.cuda.synchronize()
    assert torch.count_nonzero(state).item() == 0


def test_matches_modal_decode_on_a_workload():
    """A prompt of 2048 steps at the 125M width with 4 modes: the companion
    decode's outputs against the modal decode's (GPU against GPU, both
    within tolerance of the same filter)."""
    import torch

    import paper_2310_18780_amd as lh

    B, D, d, T, K = 8, 768, 4, 2048, 16
    lam, R, h0, up, ud = inputs(B, D, d, T, K, "f32", (0.8, 0.99), seed=3)
    a, beta = gpu_coeffs(lam, R)
    t = {k: torch.from_numpy(np.ascontiguousarray(v)).cuda() for k, v in
         dict(lam=lam, R=R, h0=h0, u=up, ud=ud.transpose(1, 0, 2)).items()}
    xc = torch.empty((B, D, 2 * d), dtype=torch.float64, device="cuda")
    xm = torch.empty((B, D, d), dtype=torch.complex64, device="cuda")
    lh.companion_init(a, t["u"], xc)
    lh.prefill(t["lam"], t["R"], t["h0"], t["u"], xm, torch.empty_like(t["u"]))
    yc = torch.empty((K, B, D), device="cuda")
    ym = torch.empty_like(yc)
    for k in range(K):
        lh.companion_step(a, beta, t["h0"], xc, t["ud"][k], yc[k])
        lh.step(t["lam"], t["R"], t["h0"], xm, t["ud"][k], ym[k])
    torch.cuda.synchronize()
    d_ = (yc - ym).abs().amax(dim=0)
    m_ = ym.abs().amax(dim=0)
    assert bool(torch.all(d_ <= 2e-4 * m_)), float((d_ / m_).max())


def test_batch_past_the_grid_limit():
    """B = 4 * 65535 + 1 rows: the step runs in two launches (65535 row groups
    of 4, then one row); sampled rows, including both sides of the cut,
    against the oracle's companion recurrence and modal outputs."""
    import torch

    import paper_2310_18780_amd as lh

    B, D, d, T0, K = 4 * 65535 + 1, 1, 1, 3, 2
    w = workloads.Workload("case", B, D, d, T0, K, "f32", 0.5, 0.95, np.pi, 1.0, 0)
    lam, R, h0 = workloads.make_params(w)
    rng = np.random.default_rng(12)
    up = rng.standard_normal((B, T0, D)).astype(np.float32)
    ud = rng.standard_normal((B, K, D)).astype(np.float32)
    a, beta = gpu_coeffs(lam, R)
    ar, br, b0 = oc.from_modal(lam, R, h0)
    state = torch.full((B, D, 2 * d), float("nan"), dtype=torch.float64, device="cuda")
    lh.companion_init(a, torch.from_numpy(up).cuda(), state)
    h0_t = torch.from_numpy(h0).cuda()
    ud_t = torch.from_numpy(np.ascontiguousarray(ud.transpose(1, 0, 2))).cuda()
    y = torch.full((K, B, D), float("nan"), device="cuda")
    for k in range(K):
        lh.companion_step(a, beta, h0_t, state, ud_t[k], y[k])
    torch.cuda.synchronize()
    cut = 4 * 65535
    bs = sorted({0, 1, cut - 2, cut - 1, cut, *rng.integers(B, size=100).tolist()})
    xe = state[bs, 0].cpu().numpy()
    yg = y[:, bs, 0].cpu().numpy().T
    xr = np.empty_like(xe)
    for i, b in enumerate(bs):
        x0 = oc.fast_init(ar[0], up[b, :, 0])
        _, xr[i] = oc.companion_run(ar[0], br[0], b0[0], ud[b, :, 0], x0)
    check_state(xe, xr, "state after the steps")
    ref = oracle.run_rows(lam, R, h0, up, ud, [(b, 0) for b in bs])
    e = check_y(yg, ref["y_dec"], "f32", "companion decode y",
                rowmax=seq_rowmax(ref["y_prefill"], ref["y_dec"]))
    _log(f"[companion grid limit] max row-relative output error {e:.2e}")
