"""GPU parity: the HIP path, called through the C ABI, against the CPU oracle
on the same seeded inputs (tolerances in ``parity_util``).

* small cases: every output and state, over shapes that span several
  wavefronts, chunks and ragged tails, both I/O dtypes, odd and large mode
  counts, T = 0, single-step chunks;
* the five workloads at their full sizes, in the launch configuration the
  benchmark uses: all outputs and states of sampled (b, c) rows, which the
  oracle computes one by one;
* properties that hold at any size: prefill(T) + K steps == prefill(T + K),
  bitwise determinism, HIP-graph replay == eager, state save / restore.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import workloads
from parity_util import (compare_full, compare_rows, gather_rows, run_gpu, sample_rows,
                         to_device, check_y, check_x, _np)

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    import paper_2310_18780_amd as lh

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    lh.lib()  # fails loudly when the library is missing
    yield


def small_case(B, D, d, T, K, io, seed=0, r=(0.5, 0.999), theta=np.pi):
    w = workloads.Workload("case", B, D, d, T, K, io, r[0], r[1], theta, 1.0 / d, seed)
    return w, workloads.make_inputs(w)


# (B, D, d, T, K, io, plan)
SMALL = [
    (1, 4, 4, 64, 16, "f32", 0),       # the tiny workload's shape, automatic plan
    (2, 70, 16, 300, 20, "f32", 0),    # one sequential pass, D not a multiple of 64
    (2, 70, 16, 300, 20, "f32", 64),   # chunked, ragged last chunk (300 = 4*64 + 44)
    (3, 130, 3, 257, 9, "bf16", 32),   # odd d (masked modes), bf16 I/O, ragged
    (1, 65, 32, 200, 5, "f32", 48),    # two lanes per row
    (2, 33, 64, 129, 7, "f32", 16),    # four lanes per row
    (2, 33, 64, 129, 7, "bf16", 0),
    (1, 7, 1, 100, 3, "f32", 0),       # d = 1
    (1, 7, 1, 100, 3, "f32", 7),
    (1, 5, 17, 50, 4, "f32", 8),       # d = 17: 2 lanes x 16 modes, 15 masked
    (2, 9, 100, 40, 3, "f32", 0),      # d = 100: 8 lanes per row
    (1, 3, 1024, 20, 2, "f32", 0),     # the largest d: 64 lanes per row
    (1, 3, 1024, 20, 2, "f32", 6),
    (1, 4, 6, 64, 4, "f32", 0),        # step: 3 mode pairs per lane
    (1, 4, 5, 64, 4, "bf16", 0),       # step: single modes, 8 lanes per row
    (2, 10, 4, 0, 5, "f32", 0),        # T = 0: zero state, decode from zero
    (2, 10, 4, 1, 3, "f32", 0),        # T = 1
    (1, 8, 4, 40, 3, "f32", 1),        # every step its own chunk
    (1, 8, 4, 40, 3, "f32", 39),       # two chunks, last of length 1
    (4, 256, 16, 512, 8, "bf16", 64),  # many waves, bf16, chunked
    (3, 20, 128, 60, 5, "f32", 0),     # d = 128: step with 64 lanes per row
    # matrix-core prefill (plan = -1 = LH_PREFILL_MFMA; d = 16 / 32, D % 8 == 0)
    (2, 64, 16, 300, 20, "f32", -1),   # ragged last chunk (300 = 9*32 + 12), 14 idle columns
    (3, 136, 16, 257, 9, "bf16", -1),  # 17 channel groups (partial line group), 257 = 8*32 + 1
    (17, 16, 32, 100, 5, "f32", -1),   # d = 32, second batch block of one row
    (1, 8, 32, 31, 3, "bf16", -1),     # T < 32: one partial chunk
    (2, 8, 16, 32, 2, "f32", -1),      # exactly one full chunk
    (2, 8, 16, 64, 2, "bf16", -1),     # two full chunks
    (1, 8, 16, 1, 3, "f32", -1),       # T = 1
    (4, 256, 16, 512, 8, "bf16", -1),  # many workgroups
    (33, 72, 32, 160, 4, "f32", -1),   # three batch blocks, 9 channel groups
    (70, 24, 16, 97, 3, "bf16", -1),   # 4 batch groups per workgroup, 2 blocks, 6 rows in the last
    (40, 16, 16, 200, 3, "f32", -1),   # 2 batch groups per workgroup (float32), ragged
    (20, 8, 16, 65, 2, "bf16", -1),    # 2 batch groups per workgroup (bfloat16)
    # bfloat16, d = 16: two u tiles in flight (the loop runs two chunks per pass)
    (2, 16, 16, 20, 3, "bf16", -1),    # only a partial chunk
    (2, 16, 16, 32, 3, "bf16", -1),    # one full chunk, nothing after it
    (3, 24, 16, 33, 3, "bf16", -1),    # one full chunk and a partial one
    (2, 16, 16, 96, 3, "bf16", -1),    # three full chunks (odd count, no partial)
    (3, 16, 16, 20, 3, "f32", -1),     # float32: only a partial chunk
    (2, 24, 16, 96, 3, "f32", -1),     # float32: three full chunks
    (20, 16, 16, 33, 3, "f32", -1),    # float32, 2 batch groups per wave: a full and a partial chunk
    (5, 67, 2, 33, 6, "bf16", 0),      # d = 2: one lane per row, B not a multiple of 4
    (3, 1, 16, 90, 5, "f32", 0),       # a single channel
    (2, 1, 5, 70, 4, "bf16", 16),      # a single channel, chunked, generic decode
    # segmented matrix-core prefill (plan = -2 = LH_PREFILL_MFMA_SEG: T cut into
    # 2^k segments of >= 256 steps; each (batch row, segment) pair is a matrix column)
    (2, 64, 16, 512, 5, "f32", -2),    # two segments of 256 steps
    (3, 136, 16, 1024, 5, "bf16", -2), # four segments, 17 channel groups, bfloat16
    (1, 16, 32, 2048, 4, "f32", -2),   # d = 32, eight segments
    (5, 40, 32, 4096, 3, "bf16", -2),  # d = 32, bfloat16, 16 segments, 5 rows
    (40, 16, 16, 1024, 3, "f32", -2),  # 2 column groups per wave (float32, d = 16)
    (2, 24, 16, 576, 3, "bf16", -2),   # two segments of 9 chunks (odd count), bfloat16
    (2, 24, 32, 576, 3, "f32", -2),    # the same with float32, d = 32
    # d = 64: 4 channels per workgroup, one group of 16 rows per wave
    (2, 12, 64, 96, 3, "f32", -1),     # three channel groups, three full chunks
    (20, 8, 64, 70, 3, "f32", -1),     # second batch group of 4 rows; 70 = 2*32 + 6
    (1, 4, 64, 20, 2, "f32", -1),      # only a partial chunk
    (3, 4, 64, 1, 2, "f32", -1),       # T = 1
    (2, 12, 64, 512, 3, "f32", -2),    # two segments of 256 steps
    (3, 4, 64, 1024, 2, "f32", -2),    # four segments
]


@pytest.mark.parametrize("case", SMALL, ids=[
    f"B{c[0]}_D{c[1]}_d{c[2]}_T{c[3]}_K{c[4]}_{c[5]}_C{c[6]}" for c in SMALL])
def test_small_case(case):
    B, D, d, T, K, io, chunk = case
    _log(f"[small] {case}")
    w, (lam, R, h0, up, ud) = small_case(B, D, d, T, K, io)
    ref = oracle.run(lam, R, h0, up, ud)
    out = run_gpu(to_device(lam, R, h0, up, ud, io), plan=chunk)
    errs = compare_full(out, ref, io)
    _log(f"[small] {case} max row-relative errors {errs}")


def test_tiny_workload():
    w = workloads.workload("tiny")
    lam, R, h0, up, ud = workloads.make_inputs(w)
    ref = oracle.run(lam, R, h0, up, ud)
    out = run_gpu(to_device(lam, R, h0, up, ud, w.io))
    _log(f"[tiny] {compare_full(out, ref, w.io)}")


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_full_workload_sampled_rows(name):
    """Full-size workload, automatic plan (as benchmarked): every output and
    state of at least 128 sampled (b, c) rows against the oracle, among them
    the first and last rows and channels of several matrix-core tiles."""
    import torch

    w = workloads.workload(name)
    _log(f"[full] {w}")
    lam, R, h0, up, ud = workloads.make_inputs(w)
    t = to_device(lam, R, h0, up, ud, w.io)
    out = run_gpu(t)
    rows = sample_rows(w.B, w.D, 128)
    got = gather_rows(out, rows)
    del out, t
    torch.cuda.empty_cache()
    ref = oracle.run_rows(lam, R, h0, up, ud, rows)
    _log(f"[full] {name} rows={len(rows)} errors {compare_rows(got, ref, w.io)}")


@pytest.mark.parametrize("name", ["c2", "c3", "c5"])
def test_decode_continues_prefill(name):
    """prefill(T) followed by K steps gives the outputs and state of a single
    prefill over the T + K inputs (any size; GPU against GPU)."""
    import torch

    import paper_2310_18780_amd as lh

    w = workloads.workload(name)
    if name == "c5":
        w = w.with_(T=8192)  # keep the concatenated copy small
    lam, R, h0, up, ud = workloads.make_inputs(w)
    t = to_device(lam, R, h0, up, ud, w.io)
    out = run_gpu(t)
    ucat = torch.cat([t["u"], t["ud"].transpose(0, 1)], dim=1).contiguous()
    y2 = torch.empty_like(ucat)
    st2 = torch.empty_like(out["x_end"])
    lh.prefill(t["lam"], t["R"], t["h0"], ucat, st2, y2)
    torch.cuda.synchronize()
    B, D, d = w.B, w.D, w.d
    yd = _np(out["y_dec"]).transpose(1, 2, 0).reshape(B * D, -1)
    y2d = _np(y2[:, w.T:]).transpose(0, 2, 1).reshape(B * D, -1).astype(np.float64)
    check_y(yd, y2d, w.io, "decode vs long prefill", ref_rounded=True)
    check_x(_np(out["x_end"]).reshape(-1, d), _np(st2).reshape(-1, d).astype(np.complex128),
            "state after decode vs long prefill")


def _bits(x):
    import torch

    if x.is_complex():
        x = torch.view_as_real(x)
    return x.contiguous().view(torch.int16 if x.element_size() == 2 else torch.int32)


def test_bitwise_determinism():
    """Two runs on the same inputs give identical bits (the kernels use no
    atomics and a fixed reduction order)."""
    import torch

    w = workloads.workload("c2")
    lam, R, h0, up, ud = workloads.make_inputs(w.with_(K=32))
    t = to_device(lam, R, h0, up, ud, w.io)
    for chunk in (0, 100):
        a = run_gpu(t, plan=chunk)
        b = run_gpu(t, plan=chunk)
        for k in a:
            assert torch.equal(_bits(a[k]), _bits(b[k])), (chunk, k)


def test_graph_replay_matches_eager():
    """K decode steps (and a prefill) captured in a HIP graph; every replay,
    with eager work in between, equals the eager run bit for bit."""
    import torch

    import paper_2310_18780_amd as lh

    w = workloads.workload("c3").with_(B=8, T=256, K=24)
    lam, R, h0, up, ud = workloads.make_inputs(w)
    t = to_device(lam, R, h0, up, ud, w.io)
    eager = run_gpu(t)

    B, T, D, d, K = w.B, w.T, w.D, w.d, w.K
    y = torch.empty_like(t["u"])
    state = torch.empty((B, D, d), dtype=torch.complex64, device="cuda")
    y_dec = torch.empty((K, B, D), dtype=t["u"].dtype, device="cuda")
    x_T = torch.empty_like(state)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm-up on a side stream before capture
        lh.prefill(t["lam"], t["R"], t["h0"], t["u"], state, y)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lh.prefill(t["lam"], t["R"], t["h0"], t["u"], state, y)
        x_T.copy_(state)
        for k in range(K):
            lh.step(t["lam"], t["R"], t["h0"], state, t["ud"][k], y_dec[k])
    for rep in range(4):
        y.fill_(float("nan"))
        y_dec.fill_(float("nan"))
        state.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        junk = torch.randn(1 << 20, device="cuda").sum()  # unrelated eager work
        torch.cuda.synchronize()
        assert torch.equal(y, eager["y_prefill"]), rep
        assert torch.equal(x_T, eager["x_T"]), rep
        assert torch.equal(y_dec, eager["y_dec"]), rep
        assert torch.equal(state, eager["x_end"]), rep
        del junk


def test_state_save_restore():
    """The state is the checkpoint: copy it to the host mid-decode, restore it
    into a fresh buffer and continue; outputs are bitwise identical."""
    import torch

    import paper_2310_18780_amd as lh

    w = workloads.workload("c2").with_(K=40)
    lam, R, h0, up, ud = workloads.make_inputs(w)
    t = to_device(lam, R, h0, up, ud, w.io)
    ref = run_gpu(t)
    state = torch.empty((w.B, w.D, w.d), dtype=torch.complex64, device="cuda")
    y = torch.empty_like(t["u"])
    lh.prefill(t["lam"], t["R"], t["h0"], t["u"], state, y)
    yk = torch.empty((w.B, w.D), dtype=t["u"].dtype, device="cuda")
    for k in range(17):
        lh.step(t["lam"], t["R"], t["h0"], state, t["ud"][k], yk)
    host = state.cpu()
    del state
    fresh = host.to("cuda")
    for k in range(17, w.K):
        lh.step(t["lam"], t["R"], t["h0"], fresh, t["ud"][k], yk)
        assert torch.equal(yk, ref["y_dec"][k]), k
    assert torch.equal(fresh, ref["x_end"])


def test_chunk_plans_agree_with_oracle_on_long_prompt():
    """The long-prompt poles (r up to 0.99999, near-DC) over 16k steps with
    several explicit chunk lengths, all rows checked."""
    w = workloads.workload("c5").with_(B=1, D=96, T=16384, K=8)
    lam, R, h0, up, ud = workloads.make_inputs(w)
    ref = oracle.run(lam, R, h0, up, ud)
    t = to_device(lam, R, h0, up, ud, w.io)
    for chunk in (0, 256, 1000, 4096, 16384):
        out = run_gpu(t, plan=chunk)
        _log(f"[long] chunk={chunk} {compare_full(out, ref, w.io)}")


def test_bf16_outputs_round_half_to_even():
    """With lambda = 0 and R = 0 the output is h0 * u exactly in float32; with
    h0 = 1 + 2^-8 and bfloat16 inputs every product lies exactly halfway
    between two bfloat16 values, so the stored outputs must be the
    ties-to-even rounding (torch's float32 -> bfloat16 conversion)."""
    import torch

    import paper_2310_18780_amd as lh

    B, T, D, d = 2, 40, 96, 2
    lam = torch.zeros((D, d), dtype=torch.complex64, device="cuda")
    R = torch.zeros((D, d), dtype=torch.complex64, device="cuda")
    h0 = torch.full((D,), 1.0 + 2.0 ** -8, dtype=torch.float32, device="cuda")
    g = torch.Generator().manual_seed(0)
    # bfloat16 values with random exponents and mantissas (odd and even)
    u = (torch.randn((B, T, D), generator=g) * 4.0).to(torch.bfloat16)
    ref = (u.float() * h0.cpu()).to(torch.bfloat16)
    ud = u.cuda()
    state = torch.empty((B, D, d), dtype=torch.complex64, device="cuda")
    y = torch.empty_like(ud)
    lh.prefill(lam, R, h0, ud, state, y)
    yt = torch.empty((B, D), dtype=torch.bfloat16, device="cuda")
    lh.step(lam, R, h0, state, ud[:, 0].contiguous(), yt)
    torch.cuda.synchronize()
    assert torch.equal(y.cpu().view(torch.int16), ref.view(torch.int16))
    assert torch.equal(yt.cpu().view(torch.int16), ref[:, 0].contiguous().view(torch.int16))
    # the ties really are ties: the float32 product is not a bfloat16 value
    prod = u.float() * h0.cpu()
    assert bool((prod.to(torch.bfloat16).float() != prod).float().mean() > 0.9)


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_unaligned_io_falls_back_to_the_vector_scan(io):
    """u and y one element past a 16-byte boundary: the automatic matrix-core
    plans (whole prompt, and segmented) run the VALU chunked scan instead,
    with the same workspace, and still match the oracle."""
    import torch

    import paper_2310_18780_amd as lh

    for B, D, d, T in ((2, 64, 16, 1024), (32, 4096, 16, 8)):  # segmented / whole-prompt plans
        w, (lam, R, h0, up, ud) = small_case(B, D, d, T, 0, io)
        ref = oracle.run(lam, R, h0, up, ud)
        t = to_device(lam, R, h0, up, ud, io)
        n = B * T * D
        ubuf = torch.empty(n + 1, dtype=t["u"].dtype, device="cuda")
        ybuf = torch.full((n + 1,), float("nan"), dtype=t["u"].dtype, device="cuda")
        u = ubuf[1:].view(B, T, D)
        u.copy_(t["u"])
        y = ybuf[1:].view(B, T, D)
        assert u.data_ptr() % 16 != 0 and y.data_ptr() % 16 != 0
        state = torch.empty((B, D, d), dtype=torch.complex64, device="cuda")
        lh.prefill(t["lam"], t["R"], t["h0"], u, state, y)
        torch.cuda.synchronize()
        yp = _np(y).transpose(0, 2, 1).reshape(B * D, T)
        check_y(yp, ref["y_prefill"].transpose(0, 2, 1).reshape(B * D, T), io, "unaligned prefill y")
        check_x(_np(state).reshape(-1, d), ref["x_T"].reshape(-1, d), "unaligned prefill x_T")


@pytest.mark.parametrize("case", [
    # (B, D, d, T, io, plan the automatic choice must equal)
    (16, 768, 16, 2048, "f32", -1),  # the 768-wide workload: the whole-prompt plan
    (2, 512, 32, 8192, "f32", -2),   # few rows, long prompt: the segmented plan
    (2, 512, 16, 8192, "bf16", -2),
    (64, 2048, 16, 256, "bf16", -1),
    (4, 768, 64, 1024, "f32", -2),   # d = 64, few rows: segments
    (32, 768, 64, 1000, "f32", -1),  # d = 64, no segments, 384 workgroups: whole prompt
])
def test_automatic_plan_choice(case):
    """The automatic plan's outputs and state equal, bit for bit, those of the
    matrix-core plan its chunk-step estimate picks (whole prompt or
    segmented) for these shapes."""
    import torch

    import paper_2310_18780_amd as lh

    B, D, d, T, io, want = case
    assert lh.prefill_plan(B, D, d, T, io=io) == {-1: "mfma", -2: "mfma_seg"}[want]
    w, (lam, R, h0, up, ud) = small_case(B, D, d, T, 0, io)
    t = to_device(lam, R, h0, up, ud, io)
    res = {}
    for ch in (0, want):
        y = torch.full_like(t["u"], float("nan"))
        st = torch.full((B, D, d), complex(float("nan"), 0), dtype=torch.complex64, device="cuda")
        lh.prefill_with_plan(t["lam"], t["R"], t["h0"], t["u"], st, y, ch)
        torch.cuda.synchronize()
        res[ch] = (y, st)
    assert torch.equal(res[0][0], res[want][0]) and torch.equal(res[0][1], res[want][1])


def test_batch_past_the_grid_limit():
    """B = 8 * 65535 + 1 rows: the decode step's fast path (8 batch rows per
    thread) would need 65536 row groups in the grid's y dimension, so the step
    takes the generic path; B = 8 * 65535 is the largest fast-path batch.
    Sampled rows (both ends and the rows around the row-group boundaries)
    against the oracle."""
    import torch

    import paper_2310_18780_amd as lh

    for B in (8 * 65535, 8 * 65535 + 1):
        D, d, T, K = 1, 2, 3, 2
        w = workloads.Workload("case", B, D, d, T, K, "f32", 0.5, 0.999, np.pi, 1.0 / d, 0)
        lam, R, h0 = workloads.make_params(w)
        rng = np.random.default_rng(11)
        up = rng.standard_normal((B, T, D)).astype(np.float32)
        ud = rng.standard_normal((B, K, D)).astype(np.float32)
        out = run_gpu(to_device(lam, R, h0, up, ud, "f32"))
        bs = sorted({0, 1, 2, 7, 8, 9, B - 9, B - 8, B - 7, B - 2, B - 1,
                     *rng.integers(B, size=200).tolist()})
        rows = [(b, 0) for b in bs]
        got = gather_rows(out, rows)
        del out
        torch.cuda.empty_cache()
        ref = oracle.run_rows(lam, R, h0, up, ud, rows)
        _log(f"[grid limit] B={B} errors {compare_rows(got, ref, 'f32')}")


def test_prefill_on_a_side_stream_under_allocator_churn():
    """A prefill enqueued on a stream other than the current one, with its
    workspace allocated by the binding, keeps that workspace while it runs:
    allocations and writes on the current stream right after the call (which
    the caching allocator would serve from a block it thinks free) change no
    result.  Compared bit for bit with the same call on the current stream,
    and sampled rows with the oracle."""
    import torch

    import paper_2310_18780_amd as lh

    B, D, d, T = 16, 512, 16, 2048  # matrix-core plan with a 6 MB workspace
    w, (lam, R, h0, up, ud) = small_case(B, D, d, T, 0, "f32")
    t = to_device(lam, R, h0, up, ud, "f32")
    need = lh.workspace_bytes(B, D, d, T)
    assert need > 0
    ref_y = torch.empty_like(t["u"])
    ref_x = torch.empty((B, D, d), dtype=torch.complex64, device="cuda")
    lh.prefill(t["lam"], t["R"], t["h0"], t["u"], ref_x, ref_y)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()  # default priority
    for rep in range(3):
        y = torch.full_like(t["u"], float("nan"))
        x = torch.full((B, D, d), complex(float("nan"), 0), dtype=torch.complex64, device="cuda")
        torch.cuda.synchronize()
        lh.prefill(t["lam"], t["R"], t["h0"], t["u"], x, y, stream=side)
        for _ in range(8):  # churn on the current stream while the prefill runs
            junk = torch.empty(need, dtype=torch.uint8, device="cuda")
            junk.fill_(0x7F)
            del junk
        side.synchronize()
        torch.cuda.synchronize()
        assert torch.equal(y, ref_y) and torch.equal(x, ref_x), f"repetition {rep}"
    rows = [(0, 0), (3, 17), (15, 511), (8, 256)]
    ref = oracle.run_rows(lam, R, h0, up, ud, rows)
    yg = np.stack([_np(y[b, :, c]) for b, c in rows])
    xg = np.stack([_np(x[b, c]) for b, c in rows])
    errs = (check_y(yg, ref["y_prefill"], "f32", "side-stream prefill y"),
            check_x(xg, ref["x_T"], "side-stream x_T"))
    _log(f"[side stream] row errors {errs}")
