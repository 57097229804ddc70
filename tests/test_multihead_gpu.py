"""GPU parity of the multi-head decode step (``lh_mh_step``) against the CPU
oracle ``oracle.multihead`` on the same seeded inputs.

Every case starts from the oracle's state after ``T0`` prompt steps (rounded to
complex64, as a caller would hold it), runs the ``K`` remaining steps on the GPU
one launch per step, and compares each step's outputs and the final state with
the oracle's direct convolution and power sums over all ``T0 + K`` steps.

Tolerances: float32 outputs per (b, m, i) row over the steps,
``max_t |y_gpu - y_ref| <= 1e-4 * max_t |y_ref|``; bfloat16 outputs add the
bfloat16 rounding (2^-8 relative); states per entry (b, m, i, j) over the modes,
``max_n |x_gpu - x_ref| <= 1e-4 * max_n |x_ref|``.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle.multihead as mh
import workloads
from parity_util import _np, check_x, check_y

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


def case_inputs(B, M, N, d, T0, K, io, seed=0):
    w = workloads.MHWorkload("case", B, M, N, d, T0, K, io, 0.5, 0.999, np.pi, 1.0 / d, seed)
    lam, R, h0 = workloads.mh_params(w)
    rows = [workloads.mh_row(w, b) for b in range(B)]
    q, k, v = (np.stack([r[i] for r in rows]) for i in range(3))  # [B, L, M, N]
    return w, lam, R, h0, q, k, v


def run_gpu(lam, R, h0, q, k, v, x0, T0, io):
    """K = L - T0 GPU steps from the state x0 [B,M,N,N,d]; returns y [B,K,M,N]
    (float32 numpy) and the final state (complex64 numpy)."""
    import torch

    import paper_2310_18780_amd as lh

    B, L, M, N = q.shape
    K = L - T0
    iot = torch.bfloat16 if io == "bf16" else torch.float32
    dev = "cuda"
    tl = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    lam_t, R_t, h0_t = tl(lam), tl(R), tl(h0)
    state = tl(x0.astype(np.complex64))
    # inputs step-major so that step t reads contiguous [B, M N] slices
    qs, ks, vs = (tl(a.transpose(1, 0, 2, 3).reshape(L, B, M * N)).to(iot) for a in (q, k, v))
    y = torch.full((K, B, M * N), float("nan"), dtype=iot, device=dev)
    for t in range(K):
        lh.mh_step(lam_t, R_t, h0_t, state, qs[T0 + t], ks[T0 + t], vs[T0 + t], y[t])
    torch.cuda.synchronize()
    return _np(y).reshape(K, B, M, N).transpose(1, 0, 2, 3), state.cpu().numpy()


def compare(y_gpu, x_gpu, lam, R, h0, q, k, v, T0, io, rows=None):
    B, L, M, N = q.shape
    d = lam.shape[1]
    if rows is None:
        rows = [(b, m, i) for b in range(B) for m in range(M) for i in range(N)]
    y_ref = mh.mh_outputs_rows(lam, R, h0, q, k, v, rows)[:, T0:]
    x_ref = mh.mh_state_rows(lam, k, v, L, rows)
    yg = np.stack([y_gpu[b, :, m, i] for b, m, i in rows])
    xg = np.stack([x_gpu[b, m, i] for b, m, i in rows])
    ey = check_y(yg, y_ref, io, "multi-head y")
    ex = check_x(xg.reshape(-1, d), x_ref.reshape(-1, d), "multi-head state")
    return ey, ex


# (B, M, N, d, T0, K, io)
SMALL = [
    (2, 2, 8, 16, 5, 4, "f32"),     # 8 lanes per entry, N = one access per wave
    (1, 3, 13, 16, 3, 3, "f32"),    # ragged N (not a multiple of the 32 entries a pass covers)
    (2, 1, 70, 4, 2, 3, "f32"),     # 2 lanes per entry, N > 64, rows not a multiple of 4
    (1, 2, 5, 3, 4, 2, "f32"),      # odd d: generic path
    (3, 2, 9, 32, 2, 3, "bf16"),    # bfloat16 q/k/v/y, 16 lanes per entry
    (1, 1, 1, 2, 0, 3, "f32"),      # one entry, one lane, empty prompt
    (2, 4, 17, 64, 1, 2, "f32"),    # 32 lanes per entry
    (1, 1, 3, 128, 1, 2, "f32"),    # 64 lanes per entry
    (1, 2, 6, 1, 3, 3, "bf16"),     # d = 1: generic path, bfloat16
    (2, 3, 33, 16, 0, 5, "bf16"),   # empty prompt, bfloat16, ragged rows
]


@pytest.mark.parametrize("case", SMALL, ids=[str(c) for c in SMALL])
def test_small_case(case):
    B, M, N, d, T0, K, io = case
    _log(f"multi-head case {case}")
    w, lam, R, h0, q, k, v = case_inputs(*case)
    x0 = mh.mh_state(lam, k, v, T0)
    y, x = run_gpu(lam, R, h0, q, k, v, x0, T0, io)
    ey, ex = compare(y, x, lam, R, h0, q, k, v, T0, io)
    _log(f"  max rel err y {ey:.2e}, state {ex:.2e}")


def test_key_value_exchange_gives_the_other_orientation():
    # exchanging k and v contracts q with the key index: y'_i = sum_j q_j w_ji
    B, M, N, d, T0, K, io = 1, 2, 6, 16, 2, 3, "f32"
    w, lam, R, h0, q, k, v = case_inputs(B, M, N, d, T0, K, io, seed=5)
    x0 = mh.mh_state(lam, v, k, T0)
    y, _ = run_gpu(lam, R, h0, q, v, k, x0, T0, io)
    h = mh.mh_filters(lam, R, h0, T0 + K)
    for m in range(M):
        for t in range(T0, T0 + K):
            z = k[0, : t + 1, m, :, None].astype(float) * v[0, : t + 1, m, None, :].astype(float)
            wt = np.tensordot(h[m, t::-1], z, axes=(0, 0))  # w_t[i, j] = sum_s h_{t-s} k_s[i] v_s[j]
            ref = wt.T @ q[0, t, m].astype(float)
            err = np.max(np.abs(y[0, t - T0, m] - ref))
            assert err <= 1e-4 * np.max(np.abs(ref)), (m, t, err)


def test_bench_workload_sampled_rows():
    """The multi-head bench workload at full size from an empty prompt, in the
    launch configuration the benchmark times; outputs and final states of
    sampled rows against the oracle."""
    import torch

    import paper_2310_18780_amd as lh

    w = workloads.mh_workload("mh").with_(K=8)
    _log(f"multi-head workload {w.name} K={w.K}")
    lam, R, h0 = workloads.mh_params(w)
    dev = "cuda"
    state = torch.zeros((w.B, w.M, w.N, w.N, w.d), dtype=torch.complex64, device=dev)
    q = np.empty((w.B, w.K, w.M, w.N), np.float32)
    k, v = np.empty_like(q), np.empty_like(q)
    for b in range(w.B):
        q[b], k[b], v[b] = workloads.mh_row(w, b)
    tl = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    qs, ks, vs = (tl(a.transpose(1, 0, 2, 3).reshape(w.K, w.B, w.D)) for a in (q, k, v))
    y = torch.empty((w.K, w.B, w.D), dtype=torch.float32, device=dev)
    lam_t, R_t, h0_t = tl(lam), tl(R), tl(h0)
    for t in range(w.K):
        lh.mh_step(lam_t, R_t, h0_t, state, qs[t], ks[t], vs[t], y[t])
    torch.cuda.synchronize()
    rng = np.random.default_rng(11)
    rows = {(0, 0, 0), (w.B - 1, w.M - 1, w.N - 1)}
    while len(rows) < 24:
        rows.add((int(rng.integers(w.B)), int(rng.integers(w.M)), int(rng.integers(w.N))))
    rows = sorted(rows)
    yn = y.cpu().numpy().reshape(w.K, w.B, w.M, w.N).transpose(1, 0, 2, 3)
    bs = torch.tensor([r[0] for r in rows], device=dev)
    ms = torch.tensor([r[1] for r in rows], device=dev)
    is_ = torch.tensor([r[2] for r in rows], device=dev)
    xs = state[bs, ms, is_].cpu().numpy()  # [rows, N, d]
    x_full = np.zeros((w.B, w.M, w.N, w.N, w.d), np.complex64)
    for r, (b, m, i) in enumerate(rows):
        x_full[b, m, i] = xs[r]
    ey, ex = compare(yn, x_full, lam, R, h0, q, k, v, 0, "f32", rows)
    _log(f"  max rel err y {ey:.2e}, state {ex:.2e}")


def test_bitwise_determinism():
    import torch

    B, M, N, d, T0, K, io = 2, 2, 40, 16, 3, 2, "f32"
    w, lam, R, h0, q, k, v = case_inputs(B, M, N, d, T0, K, io, seed=9)
    x0 = mh.mh_state(lam, k, v, T0)
    y1, x1 = run_gpu(lam, R, h0, q, k, v, x0, T0, io)
    y2, x2 = run_gpu(lam, R, h0, q, k, v, x0, T0, io)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))
    assert np.array_equal(x1.view(np.uint64), x2.view(np.uint64))
