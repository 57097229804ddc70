"""HIP-graph capture of the library's entry points (the way a serving loop
replays them): each call sequence is captured once and replayed several times
with unrelated eager work and synchronisations in between; every replay must
equal the eager run bit for bit.  The library enqueues kernels only (no
allocation, no memset nodes), so its calls are capturable as they are.
"""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from parity_util import to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    import paper_2310_18780_amd as lh

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    lh.lib()
    yield


def check_graph(run, outputs, reset, reps=3):
    """run(): the call sequence; outputs: tensors it writes; reset(): puts the
    outputs (and any in/out state) back to the starting point."""
    import torch

    reset()
    run()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outputs]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm-up on a side stream before capture
        reset()
        run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    for rep in range(reps):
        reset()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        junk = torch.randn(1 << 20, device="cuda").sum()  # unrelated eager work
        torch.cuda.synchronize()
        for i, (o, r) in enumerate(zip(outputs, ref)):
            assert torch.equal(o, r), (rep, i)
        del junk


def inputs(B, D, d, T, K, io, seed=0, r=(0.5, 0.999)):
    w = workloads.Workload("case", B, D, d, T, K, io, r[0], r[1], np.pi, 1.0 / d, seed)
    lam, R, h0, up, ud = workloads.make_inputs(w)
    return to_device(lam, R, h0, up, ud, io)


@pytest.mark.parametrize("kind", ["segmented", "fft", "noalloc"])
def test_prefill_plans(kind):
    import torch

    import paper_2310_18780_amd as lh

    t = inputs(2, 64, 16, 1024, 8, "f32")
    B, T, D = t["u"].shape
    d = t["lam"].shape[1]
    y = torch.empty_like(t["u"])
    state = torch.empty((B, D, d), dtype=torch.complex64, device="cuda")
    if kind == "segmented":
        assert lh.workspace_bytes(B, D, d, T) > lh.workspace_bytes(B, D, d, T, plan=256)
        ws = torch.empty(lh.workspace_bytes(B, D, d, T), dtype=torch.uint8, device="cuda")

        def run():
            lh.prefill(t["lam"], t["R"], t["h0"], t["u"], state, y, workspace=ws)
    elif kind == "fft":
        ws = torch.empty(lh.fft_workspace_bytes(B, D, d, T), dtype=torch.uint8, device="cuda")

        def run():
            lh.prefill_fft(t["lam"], t["R"], t["h0"], t["u"], state, y, workspace=ws)
    else:  # the segmented plan on the library's static scratch: nothing allocated
        assert 0 < lh.workspace_bytes(B, D, d, T) <= lh.NOALLOC_SCRATCH_BYTES

        def run():
            lh.prefill_noalloc(t["lam"], t["R"], t["h0"], t["u"], state, y)

    def reset():
        y.fill_(float("nan"))
        state.fill_(float("nan"))

    check_graph(run, [y, state], reset)


def test_multihead_steps():
    import torch

    import paper_2310_18780_amd as lh

    B, M, N, d, K = 2, 2, 24, 16, 6
    g = torch.Generator().manual_seed(3)
    lam = (torch.rand((M, d), generator=g) * 0.9 * torch.exp(1j * torch.rand((M, d), generator=g) * 3)).to(torch.complex64).cuda()
    R = torch.randn((M, d), dtype=torch.complex64, generator=g).cuda()
    h0 = torch.randn(M, generator=g).cuda()
    q, k, v = (torch.randn((K, B, M * N), generator=g).cuda() for _ in range(3))
    state = torch.empty((B, M, N, N, d), dtype=torch.complex64, device="cuda")
    y = torch.empty((K, B, M * N), device="cuda")

    def run():
        for i in range(K):
            lh.mh_step(lam, R, h0, state, q[i], k[i], v[i], y[i])

    def reset():
        state.zero_()
        y.fill_(float("nan"))

    check_graph(run, [y, state], reset)


def test_companion_init_and_steps():
    import torch

    import paper_2310_18780_amd as lh

    t = inputs(3, 40, 4, 300, 6, "f32", r=(0.5, 0.95))
    B, T, D = t["u"].shape
    d = t["lam"].shape[1]
    a = torch.empty((D, 2 * d), dtype=torch.float64, device="cuda")
    beta = torch.empty_like(a)
    lh.companion_coeffs(t["lam"], t["R"], a, beta)
    ws = torch.empty(lh.companion_init_workspace_bytes(D, d, T), dtype=torch.uint8, device="cuda")
    state = torch.empty((B, D, 2 * d), dtype=torch.float64, device="cuda")
    K = t["ud"].shape[0]
    y = torch.empty((K, B, D), device="cuda")

    def run():
        lh.companion_init(a, t["u"], state, workspace=ws)
        for i in range(K):
            lh.companion_step(a, beta, t["h0"], state, t["ud"][i], y[i])

    def reset():
        state.fill_(float("nan"))
        y.fill_(float("nan"))

    check_graph(run, [y, state], reset)


def test_distillation():
    import torch

    import paper_2310_18780_amd as lh

    w = workloads.Workload("case", 1, 32, 16, 1, 1, "f32", 0.5, 0.999, np.pi, 1.0 / 16, 0)
    A, th, R = workloads.distill_params(w)
    tgt = workloads.distill_target(w, 2000, tau=300.0)
    tl = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    At, tht, Rt, tg = tl(A), tl(th), tl(R), tl(tgt)
    D, d = A.shape
    loss = torch.empty(D, device="cuda")
    dA = torch.empty((D, d), device="cuda")
    dth = torch.empty_like(dA)
    dR = torch.empty((D, d), dtype=torch.complex64, device="cuda")
    hh = torch.empty((D, tgt.shape[1]), device="cuda")

    def run():
        lh.distill(At, tht, Rt, tg, loss, dA, dth, dR, hh)

    def reset():
        for o in (loss, dA, dth, hh):
            o.fill_(float("nan"))
        dR.fill_(complex(float("nan"), 0))

    check_graph(run, [loss, dA, dth, dR, hh], reset)
