"""lh_prefill_noalloc (the prefill without a workspace argument, serving its
plan from the library's static per-GPU scratch) against lh_prefill on the
same inputs, through the C ABI: calls in a row on one GPU, each later one
smaller than the one before (the scratch keeps the earlier call's contents),
covering the whole-prompt matrix-core plan at the bench workload's full size,
the segmented matrix-core plan and the VALU chunked scan.  The two entry
points run the same kernels with the same plan, so results must agree bit
for bit.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import workloads
from parity_util import to_device

pytestmark = pytest.mark.gpu

# (B, D, d, T, io, plan the automatic choice takes), largest first
CASES = [
    (64, 2048, 16, 4096, "bf16", "mfma"),     # bench workload, 38 MB of scratch
    (4, 256, 32, 4096, "f32", "mfma_seg"),    # segments + matrix-core tables, 12 MB
    (2, 70, 16, 300, "f32", "scan"),          # VALU chunked scan, 99 KB
]


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def test_noalloc_matches_prefill_on_calls_in_a_row():
    import torch

    import paper_2310_18780_amd as lh

    assert torch.cuda.is_available()
    lh.lib()
    for B, D, d, T, io, plan in CASES:
        _log(f"[noalloc] B={B} D={D} d={d} T={T} io={io}")
        assert lh.prefill_plan(B, D, d, T, io=io) == plan
        assert 0 < lh.workspace_bytes(B, D, d, T) <= lh.NOALLOC_SCRATCH_BYTES
        w = workloads.Workload("case", B, D, d, T, 0, io, 0.9, 0.9999, np.pi, 1.0 / d, 0)
        lam, R, h0 = workloads.make_params(w)
        iot = torch.bfloat16 if io == "bf16" else torch.float32
        g = torch.Generator(device="cuda").manual_seed(B * 131 + d)
        u = torch.randn((B, T, D), generator=g, device="cuda").to(iot)
        t = to_device(lam, R, h0, np.zeros((1, 1, D), np.float32),
                      np.zeros((1, 0, D), np.float32), "f32")
        out = {}
        for name in ("prefill", "noalloc"):
            y = torch.full_like(u, float("nan"))
            x = torch.full((B, D, d), complex(float("nan"), 0), dtype=torch.complex64,
                           device="cuda")
            if name == "prefill":
                lh.prefill(t["lam"], t["R"], t["h0"], u, x, y)
            else:
                lh.prefill_noalloc(t["lam"], t["R"], t["h0"], u, x, y)
            torch.cuda.synchronize()
            out[name] = (y, x)
        assert torch.equal(out["prefill"][0], out["noalloc"][0]), (B, D, d, T, io)
        assert torch.equal(out["prefill"][1], out["noalloc"][1]), (B, D, d, T, io)
        assert bool(torch.isfinite(out["noalloc"][0].float()).all())
        del out, u
        torch.cuda.empty_cache()


def test_noalloc_refuses_sizes_beyond_its_scratch():
    import torch

    import paper_2310_18780_amd as lh

    B, D, d, T = 16, 4096, 64, 128  # matrix-core tables of 4096 channels: 229 MB
    assert lh.workspace_bytes(B, D, d, T) > lh.NOALLOC_SCRATCH_BYTES
    lam = torch.zeros((D, d), dtype=torch.complex64, device="cuda")
    h0 = torch.zeros((D,), dtype=torch.float32, device="cuda")
    u = torch.zeros((B, T, D), dtype=torch.float32, device="cuda")
    y = torch.zeros_like(u)
    x = torch.zeros((B, D, d), dtype=torch.complex64, device="cuda")
    with pytest.raises(lh.LHError) as e:
        lh.prefill_noalloc(lam, lam.clone(), h0, u, x, y)
    assert e.value.status == 5 and "scratch" in str(e.value)
    assert bool((y == 0).all())  # nothing was enqueued
