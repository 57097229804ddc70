"""Full-size parity of the benchmarked prefill plan against an independent
kernel: at the bench workload (B = 64, D = 2048, d = 16, T = 4096, bfloat16
u/y) and the wide d = 64 workload (B = 256, D = 2048, T = 1024, float32 u/y),
the automatic plan (the matrix-core chunked scan) is compared over every
(b, c) row of the outputs and every state with the VALU chunked scan
(``lh_prefill_with_plan`` with a chunk length: other kernels, another
association of the same sums).  Each result is within its 1e-4 row tolerance
of the exact one (checked against the oracle on sampled rows elsewhere), so
the two may differ by twice that: row-relative 2e-4 on float32, plus one
bfloat16 rounding on each side for bfloat16 outputs.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import workloads
from parity_util import BF16_REL, to_device

pytestmark = pytest.mark.gpu

PAIR_TOL = 2e-4  # two results, each within 1e-4 of the exact one


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def _compare_outputs(ya, ys, io):
    """Row-relative check of y [B, T, D] (rows (b, c) over t), batch row by
    batch row on the device; returns the worst row-relative difference."""
    import torch

    worst = 0.0
    for b in range(ya.shape[0]):
        a = ya[b].float()
        s = ys[b].float()
        rowmax = s.abs().amax(dim=0, keepdim=True)  # [1, D]
        err = (a - s).abs()
        bound = PAIR_TOL * rowmax
        if io == "bf16":
            bound = bound + 2 * BF16_REL * s.abs()
        bad = err > bound
        if bool(bad.any()):
            idx = torch.nonzero(bad)[0].tolist()
            t, c = idx
            raise AssertionError(
                f"y[{b}, {t}, {c}]: {int(bad.sum())} outputs of batch row {b} differ; "
                f"auto={a[t, c].item()!r} scan={s[t, c].item()!r} rowmax={rowmax[0, c].item():.4g}")
        worst = max(worst, float((err / rowmax.clamp_min(1e-30)).amax()))
    return worst


def _compare_states(xa, xs):
    """Per (b, c): max over modes of |x_auto - x_scan| <= 2e-4 max |x_scan|."""
    import torch

    err = (xa - xs).abs()  # [B, D, d]
    rowmax = xs.abs().amax(dim=2, keepdim=True)
    bad = err > PAIR_TOL * rowmax
    if bool(bad.any()):
        b, c, n = torch.nonzero(bad)[0].tolist()
        raise AssertionError(f"x_T[{b}, {c}, {n}]: {int(bad.sum())} modes differ; "
                             f"auto={xa[b, c, n].item()!r} scan={xs[b, c, n].item()!r}")
    return float((err / rowmax.clamp_min(1e-30)).amax())


@pytest.mark.parametrize("name,chunk", [("c3", 512), ("c4", 256)])
def test_automatic_plan_against_vector_scan_on_every_row(name, chunk):
    import torch

    import paper_2310_18780_amd as lh

    w = workloads.workload(name)
    _log(f"[full plans] {w} scan chunk {chunk}")
    auto = lh.prefill_plan(w.B, w.D, w.d, w.T, io=w.io)
    assert auto == "mfma", auto
    assert lh.prefill_plan(w.B, w.D, w.d, w.T, plan=chunk, io=w.io) == "scan"
    lam, R, h0 = workloads.make_params(w)
    iot = torch.bfloat16 if w.io == "bf16" else torch.float32
    u = torch.empty((w.B, w.T, w.D), dtype=iot, device="cuda")
    for b in range(w.B):
        u[b].copy_(torch.from_numpy(workloads.prompt_row(w, b)))
    t = to_device(lam, R, h0, np.zeros((1, 1, w.D), np.float32), np.zeros((1, 0, w.D), np.float32),
                  "f32")
    res = {}
    for plan in (0, chunk):
        y = torch.full_like(u, float("nan"))
        x = torch.full((w.B, w.D, w.d), complex(float("nan"), 0), dtype=torch.complex64,
                       device="cuda")
        if plan == 0:
            lh.prefill(t["lam"], t["R"], t["h0"], u, x, y)
        else:
            lh.prefill_with_plan(t["lam"], t["R"], t["h0"], u, x, y, plan)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(y.float()).all()) and bool(torch.isfinite(x.real).all())
        res[plan] = (y, x)
    ey = _compare_outputs(res[0][0], res[chunk][0], w.io)
    ex = _compare_states(res[0][1], res[chunk][1])
    _log(f"[full plans] {name}: every row, worst row-relative difference y {ey:.3g}, x_T {ex:.3g}")
