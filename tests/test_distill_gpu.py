"""GPU parity of the distillation objective (``lh_distill``) against the CPU
oracle ``oracle.distill`` on the same seeded inputs.

Tolerances: the loss relative 1e-4; gradients per channel on the infinity norm
over the channel's 4 d gradient entries, ``max |g_gpu - g_ref| <= 1e-4 *
max |g_ref|``; the materialised filter per channel, ``max_t |hhat_gpu -
hhat_ref| <= 1e-4 * max_t |hhat_ref|``.  At an exactly representable target
the loss and gradients are float32 rounding noise, checked against the scale
of the same channel's gradient at a random target.
"""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest

import oracle.distill as od
import workloads

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


def params(D, d, seed=0, a=(0.5, 0.999)):
    w = workloads.Workload("case", 1, D, d, 1, 1, "f32", a[0], a[1], math.pi, 1.0 / d, seed)
    return workloads.distill_params(w), w


def run_gpu(A, th, R, tgt, want_h=True):
    import torch

    import paper_2310_18780_amd as lh

    D, d = A.shape
    L = tgt.shape[1]
    tl = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    At, tht, Rt, tgt_t = tl(A), tl(th), tl(R), tl(tgt)
    loss = torch.full((D,), float("nan"), device="cuda")
    dA = torch.full((D, d), float("nan"), device="cuda")
    dth = torch.full((D, d), float("nan"), device="cuda")
    dR = torch.full((D, d), complex(float("nan"), 0), dtype=torch.complex64, device="cuda")
    hh = torch.full((D, L), float("nan"), device="cuda") if want_h else None
    lh.distill(At, tht, Rt, tgt_t, loss, dA, dth, dR, hh)
    torch.cuda.synchronize()
    out = dict(loss=loss.cpu().numpy(), dA=dA.cpu().numpy(), dtheta=dth.cpu().numpy(),
               dR=dR.cpu().numpy())
    if want_h:
        out["hhat"] = hh.cpu().numpy()
    return out


def grads_matrix(o):
    return np.concatenate([o["dA"], o["dtheta"], o["dR"].real, o["dR"].imag], axis=1)


def compare(got, ref, what=""):
    np.testing.assert_array_less(np.abs(got["loss"] - ref["loss"]), 1e-4 * np.abs(ref["loss"]) + 1e-30)
    g, r = grads_matrix(got), grads_matrix(ref)
    assert np.all(np.isfinite(g)), what
    err = np.max(np.abs(g - r), axis=1)
    scale = np.max(np.abs(r), axis=1)
    bad = err > 1e-4 * scale
    assert not np.any(bad), f"{what}: gradient rows {np.nonzero(bad)[0]} err {err[bad]} scale {scale[bad]}"
    if "hhat" in got:
        eh = np.max(np.abs(got["hhat"] - ref["hhat"]), axis=1)
        sh = np.max(np.abs(ref["hhat"]), axis=1)
        assert np.all(eh <= 1e-4 * sh), f"{what}: hhat {eh / sh}"
    return float(np.max(err / np.maximum(scale, 1e-300)))


# (D, d, L)
CASES = [
    (3, 4, 50),
    (5, 16, 4096),     # one full segment (256 threads x 16 steps)
    (2, 7, 5000),      # two segments, ragged; d not a multiple of the 8-mode chunk
    (1, 1, 1),
    (4, 33, 300),      # five mode chunks, the last with one mode
    (2, 16, 20000),    # five segments
]


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_random_targets(case):
    D, d, L = case
    _log(f"distill case {case}")
    (A, th, R), w = params(D, d)
    tgt = workloads.distill_target(w, L, tau=max(8.0, L / 8))
    got = run_gpu(A, th, R, tgt)
    ref = od.distill_loss_grad(A, th, R, tgt)
    e = compare(got, ref, str(case))
    _log(f"  max rel gradient error {e:.2e}")


def test_zero_modulus_and_unit_circle_poles():
    (A, th, R), w = params(3, 8, seed=3)
    A = A.copy()
    A[0, :3] = 0.0        # lambda = 0: a one-tap filter (0^0 = 1)
    A[1, 2] = 1.0         # on the unit circle
    A[2, :] = 1.0
    tgt = workloads.distill_target(w, 700, tau=100.0)
    got = run_gpu(A, th, R, tgt)
    ref = od.distill_loss_grad(A, th, R, tgt)
    compare(got, ref, "zero / unit poles")


def test_exact_target_is_stationary_up_to_rounding():
    (A, th, R), w = params(4, 16, seed=5)
    L = 2000
    tgt = od.modal_filter(A, th, R, L).astype(np.float32)
    got = run_gpu(A, th, R, tgt)
    ref_random = od.distill_loss_grad(A, th, R, workloads.distill_target(w, L, tau=250.0))
    hh = od.modal_filter(A, th, R, L)
    assert np.all(got["loss"] <= 1e-9 * np.sum(hh * hh, axis=1))
    gscale = np.max(np.abs(grads_matrix(ref_random)), axis=1)
    assert np.all(np.max(np.abs(grads_matrix(got)), axis=1) <= 1e-4 * gscale)


def test_without_filter_output_and_determinism():
    (A, th, R), w = params(6, 16, seed=7)
    tgt = workloads.distill_target(w, 3000, tau=400.0)
    a = run_gpu(A, th, R, tgt, want_h=False)
    b = run_gpu(A, th, R, tgt, want_h=True)
    for k in ("loss", "dA", "dtheta"):
        assert np.array_equal(a[k].view(np.uint32), b[k].view(np.uint32)), k
    assert np.array_equal(a["dR"].view(np.uint64), b["dR"].view(np.uint64))
