"""Seeded sweep of small random shapes through every prefill plan that
applies (automatic, VALU chunks of a random length, matrix cores over the
whole prompt, segmented matrix cores) followed by decode steps, each against
the oracle with the tolerances of ``parity_util``.  The shapes mix ragged
sizes, odd and power-of-two mode counts, short and long prompts and both
input types; pole radii span slow and fast decay."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import workloads
from parity_util import compare_full, run_gpu, to_device

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def _cases(n=160, seed=2026):
    """Every other case has a shape the matrix-core plans take (d = 16 or 32,
    D a multiple of 8, prompts that split into segments); eight more take
    d = 64 with float32 u/y and D a multiple of 4."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        if i % 2:
            d = int(rng.choice([16, 32]))
            D = int(rng.choice([8, 16, 24, 40, 64, 72, 136]))
            T = int(rng.choice([1, 31, 33, 96, 257, 512, 576, 1024, 2048]))
        else:
            d = int(rng.choice([1, 2, 3, 4, 5, 8, 15, 16, 17, 31, 32, 33, 64]))
            D = int(rng.choice([1, 3, 8, 16, 24, 40, 64, 72, 130]))
            T = int(rng.choice([0, 1, 5, 31, 32, 33, 100, 256, 300, 512, 576, 1024]))
        B = int(rng.integers(1, 7))
        K = int(rng.integers(1, 5))
        io = "bf16" if rng.random() < 0.4 else "f32"
        r_lo = float(rng.choice([0.3, 0.8, 0.99]))
        out.append((i, B, D, d, T, K, io, r_lo))
    for j in range(8):  # d = 64 on the matrix-core plans: float32 u/y, D % 4 == 0
        D = int(rng.choice([4, 8, 12, 20, 36, 68]))
        T = int(rng.choice([1, 31, 33, 96, 257, 512, 576]))
        B = int(rng.integers(1, 21))
        K = int(rng.integers(1, 5))
        r_lo = float(rng.choice([0.3, 0.8, 0.99]))
        out.append((n + j, B, D, 64, T, K, "f32", r_lo))
    return out


def _plans(lh, B, D, d, T, io, rng):
    plans = [0, int(rng.integers(1, max(2, T + 1)))]
    for ch in (-1, -2):
        try:
            lh.prefill_plan(B, D, d, T, plan=ch, io=io)
        except Exception:
            continue
        plans.append(ch)
    return plans


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    import paper_2310_18780_amd as lh

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    lh.lib()
    yield


@pytest.mark.parametrize("case", _cases(), ids=lambda c: f"{c[0]}_B{c[1]}_D{c[2]}_d{c[3]}_T{c[4]}_{c[6]}")
def test_random_shape(case):
    import paper_2310_18780_amd as lh

    i, B, D, d, T, K, io, r_lo = case
    w = workloads.Workload("case", B, D, d, T, K, io, r_lo, 0.999, np.pi, 1.0 / d, 100 + i)
    lam, R, h0, up, ud = workloads.make_inputs(w)
    ref = oracle.run(lam, R, h0, up, ud)
    t = to_device(lam, R, h0, up, ud, io)
    rng = np.random.default_rng(1000 + i)
    for ch in _plans(lh, B, D, d, T, io, rng):
        _log(f"[random] {case} plan={ch}")
        out = run_gpu(t, plan=ch)
        errs = compare_full(out, ref, io)
        _log(f"[random] {case} plan={ch} errors {errs}")
