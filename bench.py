#!/usr/bin/env python3
"""Benchmark of the distilled modal recurrence on one MI355X.

One step = one pass of the whole hot path over one batch of the workload:
prefill of the B x T prompt (all outputs + post-prompt state) followed by K
decode steps (one lh_step launch per token, replayed from a HIP graph).
Inputs are resident in HBM before the timed region starts.

Prints ONE JSON line: decode tokens/s (B * K / decode time) as ``value``,
prefill tokens/s, the decode kernel's roofline (HBM) and the prefill's (HBM
for the matrix-core plans at d = 16 and 32, the bfloat16 MFMA peak at d = 64,
the VALU peak for the VALU scan; the declared flop rate beside it), and the
CPU oracle timed on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--workload c3]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode tokens/s (B·steps/s) + HBM GB/s at D=2048,d=16; prefill tokens/s"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
FP32_VALU_PEAK_TFLOPS = 157.3  # MI355X fp32 vector (with packed FP32 FMA)
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix (no sparsity)
PROFILES = os.path.join(ROOT, "profiles")


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="c3")
    p.add_argument("--decode-launch", choices=["graph", "eager"], default="graph")
    p.add_argument("--no-cpu-baseline", action="store_true",
                   help="leave out the oracle timing (cpu_baseline is then null)")
    p.add_argument("--cpu-rows", type=int, default=0,
                   help="(b, c) rows of the oracle sample (0: sized for ~15 s)")
    p.add_argument("--stream-pool", type=int, default=64,
                   help="state buffers of the HBM-streaming decode measurement (0: skip)")
    p.add_argument("--decode-pool-only", action="store_true",
                   help="run only the HBM-streaming decode over the state pool (for counter "
                        "passes of that kernel)")
    p.add_argument("--copy-calibration", action="store_true",
                   help="run only a plain device copy of known size (counter calibration)")
    p.add_argument("--multihead", action="store_true",
                   help="time the multi-head decode step (lh_mh_step) instead, on --mh-workload")
    p.add_argument("--mh-workload", default="mh")
    p.add_argument("--fft", action="store_true",
                   help="time the FFT prefill (lh_prefill_fft) beside the scan prefill on "
                        "--fft-workload")
    p.add_argument("--fft-workload", default="c5")
    p.add_argument("--companion", action="store_true",
                   help="time the companion-form decode step and fast initialisation beside the "
                        "modal ones on --companion-workload")
    p.add_argument("--companion-workload", default="cp")
    p.add_argument("--launch-floor", action="store_true",
                   help="time plain kernels with the decode step's footprint on --workload "
                        "(an empty launch, an in-place update and a copy of the state's bytes), "
                        "graph-replayed like the decode steps")
    p.add_argument("--distill", action="store_true",
                   help="time the distillation objective (lh_distill) on --workload's filter "
                        "bank with L = its T")
    return p.parse_args()


def src_digest(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2310_18780_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def profile_value(summary_name, key, digest):
    """A figure from a committed rocprofv3 counter summary, if the summary was
    taken on the current kernel source (else None)."""
    path = os.path.join(PROFILES, summary_name)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_src = re.search(r"^source_sha256_16:\s*([0-9a-f]+)", text, re.M)
    m_v = re.search(r"^" + key + r":\s*([0-9.eE+-]+)", text, re.M)
    if not m_src or not m_v or m_src.group(1) != digest:
        return None
    return float(m_v.group(1))


def counter_traffic(summary_name, digest):
    """HBM bytes per launch from a committed rocprofv3 counter summary."""
    return profile_value(summary_name, "hbm_bytes_per_launch", digest)


def copy_calibration():
    import torch

    n = 256 << 20
    a = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "launches": 5}))


def make_device_inputs(w):
    import numpy as np
    import torch

    import workloads

    lam, R, h0 = workloads.make_params(w)
    iot = torch.bfloat16 if w.io == "bf16" else torch.float32
    u = torch.empty((w.B, w.T, w.D), dtype=iot, device="cuda")
    ud = torch.empty((w.K, w.B, w.D), dtype=iot, device="cuda")
    for b in range(w.B):
        u[b].copy_(torch.from_numpy(workloads.prompt_row(w, b)))
        ud[:, b].copy_(torch.from_numpy(workloads.decode_row(w, b)))
    return dict(lam=torch.from_numpy(lam).cuda(), R=torch.from_numpy(R).cuda(),
                h0=torch.from_numpy(h0).cuda(), u=u, ud=ud)


def decode_bytes(w):
    es = 2 if w.io == "bf16" else 4
    return 16 * w.B * w.D * w.d + 2 * es * w.B * w.D + 16 * w.D * w.d + 4 * w.D


def prefill_bytes(w):
    es = 2 if w.io == "bf16" else 4
    return 2 * es * w.B * w.T * w.D + 8 * w.B * w.D * w.d + 16 * w.D * w.d + 4 * w.D


def prefill_flops(w):
    return 12 * w.d * w.B * w.T * w.D + 2 * w.B * w.T * w.D


def mfma64_flops(w):
    """Flops the d = 64 matrix-core plan executes (16x16x32 bfloat16
    products, 16384 flops each; float32 operands in three bfloat16 terms, six
    term products per contraction): per channel, 16-row column block and
    32-step chunk, 48 products for the chunk's end state (8 row tiles of P U),
    12 for the outputs from the chunk's inputs (2 row tiles of T U) and 32 for
    those from its entry state (W X: 2 row tiles x 4 K tiles x 4 term
    products); a partial last chunk takes the 44 output products only."""
    full, part = w.T // 32, int(w.T % 32 != 0)
    return 16384 * w.D * -(-w.B // 16) * (92 * full + 44 * part)


def dtype_detail(w, plan):
    """What the arithmetic of the path is, beyond the float32 label."""
    io = "bfloat16 u/y (widened exactly, outputs rounded to nearest even)" if w.io == "bf16" \
        else "float32 u/y"
    if plan == "scan":
        pre = "prefill on the float32 VALU"
    elif w.io == "bf16":
        pre = ("prefill contractions on bfloat16 matrix cores with float32 accumulation: "
               "float32 operands split into bfloat16 terms, two for the outputs, three for "
               "the chunk end states; carry in float32")
    else:
        pre = ("prefill contractions on bfloat16 matrix cores with float32 accumulation: "
               "float32 operands split into three bfloat16 terms; carry in float32")
    return f"complex float32 state; {io}; {pre}; decode on the float32 VALU"


def cpu_baseline(w, rows_wanted):
    """The oracle (as it stands) on a bounded sample: complete rows (prompt
    outputs, decode outputs, both states) of (b, c) pairs of the workload."""
    import numpy as np

    import oracle
    import workloads

    lam, R, h0 = workloads.make_params(w)
    L = w.T + w.K
    if rows_wanted <= 0:
        # about 15 s of oracle work (the sizing assumes direct convolution at
        # L^2/2 multiply-adds per row and 0.5e9 per core; measured runs land at
        # about 0.7 of the target)
        rate = 0.5e9 * max(1, oracle.native_threads())
        rows_wanted = int(max(64, min(w.B * w.D, 20.0 * rate / (L * L / 2))))
    nb = max(1, min(w.B, -(-rows_wanted // w.D)))
    per_b = -(-rows_wanted // nb)
    rng = np.random.default_rng(7)
    bs = rng.choice(w.B, size=nb, replace=False)
    up = np.empty((w.B, w.T, w.D), np.float32)  # only rows in bs are filled
    ud = np.empty((w.B, w.K, w.D), np.float32)
    for b in bs:
        up[b] = workloads.prompt_row(w, int(b))
        ud[b] = workloads.decode_row(w, int(b))
    rows = [(int(b), int(c)) for b in bs for c in range(min(per_b, w.D))][:rows_wanted]
    t0 = time.perf_counter()
    oracle.run_rows(lam, R, h0, up, ud, rows)
    dt = time.perf_counter() - t0
    seqs = len(rows) / w.D  # whole-width sequences' worth of rows
    return {
        "value": seqs * w.K / dt,
        "unit": "tokens/s",
        "cores": oracle.native_threads(),
        **host_cpu(),
        "kind": "oracle",
        "sample": (f"{len(rows)} (b,c) rows of {w.name} ({seqs:.2f} sequences' worth), each fully "
                   f"computed (T={w.T} prompt + K={w.K} decode outputs by direct float64 "
                   f"convolution, plus both states) in {dt:.2f} s; value = decode outputs "
                   f"per second scaled to whole sequences (rows / D * K / time); the oracle "
                   f"also produced the prompt outputs in that time"),
        "seconds": dt,
    }


def host_cpu():
    """The host CPUs the oracle may run on: the affinity set's size and the CPU
    model (``cores`` beside it is the OpenMP thread count the oracle used)."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"affinity_cpus": len(os.sched_getaffinity(0)), "cpu_model": model}


def mh_decode_bytes(w):
    es = 2 if w.io == "bf16" else 4
    return 16 * w.B * w.M * w.N * w.N * w.d + 4 * es * w.B * w.D + 16 * w.M * w.d + 4 * w.M


def mh_cpu_baseline(w, seconds=10.0):
    """The multi-head oracle on a bounded sample: complete output rows (all
    K steps of one (b, m, i)), added in batches until about ``seconds``."""
    import numpy as np

    import oracle
    import oracle.multihead as mho
    import workloads

    lam, R, h0 = workloads.mh_params(w)
    q = np.empty((w.B, w.T0 + w.K, w.M, w.N), np.float32)
    k, v = np.empty_like(q), np.empty_like(q)
    done, bs, dt = 0, [], 0.0
    for b in np.random.default_rng(7).permutation(w.B):
        b = int(b)
        q[b], k[b], v[b] = workloads.mh_row(w, b)  # input generation is not timed
        bs.append(b)
        order = [(b, m, i) for m in range(w.M) for i in range(w.N)]
        for j in range(0, len(order), 64):
            t0 = time.perf_counter()
            mho.mh_outputs_rows(lam, R, h0, q, k, v, order[j:j + 64])
            dt += time.perf_counter() - t0
            done += len(order[j:j + 64])
            if dt >= seconds:
                break
        if dt >= seconds:
            break
    return {
        "value": done / w.D * w.K / dt,
        "unit": "tokens/s",
        "cores": oracle.native_threads(),
        **host_cpu(),
        "kind": "oracle",
        "sample": (f"{done} output rows (b, m, i) of {w.name} (batch rows {bs}), each all "
                   f"T0+K={w.T0 + w.K} steps by direct float64 convolution of its N={w.N} "
                   f"outer-product entries, in {dt:.2f} s; value = rows / D * K / time"),
        "seconds": dt,
    }


def multihead_main(args):
    import torch

    import paper_2310_18780_amd as lh
    import workloads

    lh.lib()
    w = workloads.mh_workload(args.mh_workload)
    lam, R, h0 = (torch.from_numpy(a).cuda() for a in workloads.mh_params(w))
    iot = torch.bfloat16 if w.io == "bf16" else torch.float32
    L = w.T0 + w.K
    q = torch.empty((L, w.B, w.D), dtype=iot, device="cuda")
    k, v = torch.empty_like(q), torch.empty_like(q)
    for b in range(w.B):
        for dst, src in zip((q, k, v), workloads.mh_row(w, b)):
            dst[:, b].copy_(torch.from_numpy(src.reshape(L, w.D)))
    state = torch.zeros((w.B, w.M, w.N, w.N, w.d), dtype=torch.complex64, device="cuda")
    y = torch.empty((w.K, w.B, w.D), dtype=iot, device="cuda")
    for t in range(w.T0):  # the prompt's state, by stepping
        lh.mh_step(lam, R, h0, state, q[t], k[t], v[t], y[0])

    def decode_eager():
        for t in range(w.K):
            lh.mh_step(lam, R, h0, state, q[w.T0 + t], k[w.T0 + t], v[w.T0 + t], y[t])

    decode_eager()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        decode_eager()
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        graph.replay()
    stream = torch.cuda.current_stream()
    a, c = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    a.record(stream)
    for _ in range(args.steps):
        graph.replay()
    c.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = a.elapsed_time(c) / args.steps  # per K-step decode
    us = ms * 1e3 / w.K
    dbytes = mh_decode_bytes(w)
    gbs = dbytes / (us * 1e-6) / 1e9
    cpu = None if args.no_cpu_baseline else mh_cpu_baseline(w)
    out = {
        "metric": "multi-head decode tokens/s (B·steps/s) + HBM GB/s",
        "value": w.B * w.K / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "M": w.M, "N": w.N, "D": w.D, "d": w.d,
                   "T0": w.T0, "K": w.K, "io": w.io, "decode_launch": "graph"},
        "decode_us_per_token_step": us,
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS,
                     "traffic": counter_traffic(f"mh_step_{w.name}_counters.txt",
                                                src_digest("multihead.hip", "lh_internal.hpp")),
                     "kernel": "mh_step_kernel", "bytes_per_launch": dbytes},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


# declared flops of the distillation objective per (t, n): the running power
# (complex product, 6), the filter term Re(R p) (2 FMA, 4); then the powers
# again (6) and the two gradient sums e p and e (t-1) p (4 FMA, 8)
DISTILL_FLOPS_PER_TAP_MODE = 24


def distill_main(args):
    import numpy as np
    import torch

    import paper_2310_18780_amd as lh
    import workloads

    lh.lib()
    w = workloads.workload(args.workload)
    L = w.T
    A, th, R = workloads.distill_params(w)
    tgt = workloads.distill_target(w, L)
    tl = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    At, tht, Rt, tg = tl(A), tl(th), tl(R), tl(tgt)
    loss = torch.empty((w.D,), device="cuda")
    dA = torch.empty((w.D, w.d), device="cuda")
    dth = torch.empty_like(dA)
    dR = torch.empty((w.D, w.d), dtype=torch.complex64, device="cuda")

    def call():
        lh.distill(At, tht, Rt, tg, loss, dA, dth, dR)

    for _ in range(max(1, args.warmup)):
        call()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    a, c = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    a.record(stream)
    for _ in range(args.steps):
        call()
    c.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = a.elapsed_time(c) / args.steps
    flops = DISTILL_FLOPS_PER_TAP_MODE * w.D * L * w.d
    tf = flops / (ms * 1e-3) / 1e12
    nbytes = 4 * w.D * L + (4 + 4 + 8) * w.D * w.d * 2 + 4 * w.D
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        import oracle.distill as od

        done, dt = 0, 0.0
        while dt < 10.0 and done < w.D:
            sl = slice(done, min(w.D, done + 16))
            t1 = time.perf_counter()
            od.distill_loss_grad(A[sl], th[sl], R[sl], tgt[sl])
            dt += time.perf_counter() - t1
            done = sl.stop
        cpu = {"value": done * L / dt, "unit": "taps/s", "cores": oracle.native_threads(),
               **host_cpu(), "kind": "oracle",
               "sample": f"{done} of {w.D} channels (loss and gradients over L={L} taps, "
                         f"d={w.d}, float64 numpy) in {dt:.2f} s",
               "seconds": dt}
    out = {
        "metric": "distillation objective taps/s (loss + gradients, per channel and tap)",
        "value": w.D * L / (ms * 1e-3),
        "unit": "taps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"distill_{w.name}", "D": w.D, "d": w.d, "L": L},
        "ms_per_call": ms,
        "roofline": {"bound": "alu", "achieved": tf, "peak": FP32_VALU_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": tf / FP32_VALU_PEAK_TFLOPS, "traffic": None,
                     "kernel": "distill_kernel", "flops_per_launch": flops,
                     "bytes_per_launch": nbytes, "gbps": nbytes / (ms * 1e-3) / 1e9},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def fft_pass_bytes(w):
    """HBM bytes the FFT prefill's passes move by design (each pass reads and
    writes its arrays once): filter [T, D] written and read, its spectrum
    written by the column pass and read and written by the row pass, the input
    pairs' spectra written, read and written in the row pass and read by the
    inverse column pass, the spectrum read once per pair, u read twice (the
    transform and the state contraction), y and the state written."""
    es = 2 if w.io == "bf16" else 4
    N = 1
    while N < 2 * w.T - 1:
        N *= 2
    npair = (w.B + 1) // 2
    spec = 8 * N * w.D
    return (2 * 4 * w.T * w.D + 3 * spec + 4 * npair * spec + npair * spec
            + 2 * es * w.B * w.T * w.D + es * w.B * w.T * w.D + 8 * w.B * w.D * w.d)


def fft_cpu_baseline(w, seconds=40.0):
    """The oracle (direct float64 convolution and Vandermonde sums) on complete
    prompt rows of the workload, sized by ``seconds`` at an assumed rate
    (measured runs take about a third of it: some 13 s)."""
    import numpy as np

    import oracle
    import workloads

    lam, R, h0 = workloads.make_params(w)
    rate = 0.5e9 * max(1, oracle.native_threads())
    rows_wanted = int(max(8, min(w.B * w.D, seconds * rate / (w.T * w.T / 2))))
    up = np.empty((1, w.T, w.D), np.float32)
    up[0] = workloads.prompt_row(w, 0)
    ud = np.empty((1, 0, w.D), np.float32)
    rows = [(0, c) for c in range(min(rows_wanted, w.D))]
    t0 = time.perf_counter()
    oracle.run_rows(lam, R, h0, up, ud, rows)
    dt = time.perf_counter() - t0
    return {"value": len(rows) / w.D * w.T / dt, "unit": "tokens/s",
            "cores": oracle.native_threads(), **host_cpu(), "kind": "oracle",
            "sample": (f"{len(rows)} (b,c) rows of {w.name} (T={w.T} prompt outputs by direct "
                       f"float64 convolution and the state by direct sums) in {dt:.2f} s; value "
                       f"= prompt tokens per second scaled to whole sequences (rows / D * T / "
                       f"time)"),
            "seconds": dt}


def fft_main(args):
    import torch

    import paper_2310_18780_amd as lh
    import workloads

    lh.lib()
    w = workloads.workload(args.fft_workload).with_(K=1)
    t = make_device_inputs(w)
    B, T, D, d = w.B, w.T, w.D, w.d
    state = torch.empty((B, D, d), dtype=torch.complex64, device="cuda")
    y = torch.empty_like(t["u"])
    wsf = lh.fft_workspace_bytes(B, D, d, T)
    ws_fft = torch.empty(max(wsf, 1), dtype=torch.uint8, device="cuda")
    wss = lh.workspace_bytes(B, D, d, T)
    ws_scan = torch.empty(max(wss, 1), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def fft():
        lh.prefill_fft(t["lam"], t["R"], t["h0"], t["u"], state, y, workspace=ws_fft)

    def scan():
        lh.prefill(t["lam"], t["R"], t["h0"], t["u"], state, y, workspace=ws_scan)

    def timed(fn):
        for _ in range(max(1, args.warmup)):
            fn()
        torch.cuda.synchronize()
        marks = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                 for _ in range(args.steps)]
        t0 = time.perf_counter()
        for a, c in marks:
            a.record(stream)
            fn()
            c.record(stream)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1e3 / args.steps
        ms = sorted(a.elapsed_time(c) for a, c in marks)
        return ms[len(ms) // 2], wall

    fft_ms, fft_wall = timed(fft)
    scan_ms, _ = timed(scan)
    alg = prefill_bytes(w)
    gbs = alg / (fft_ms * 1e-3) / 1e9
    pbytes = fft_pass_bytes(w)
    cpu = None if args.no_cpu_baseline else fft_cpu_baseline(w)
    out = {
        "metric": "prefill tokens/s (FFT convolution prefill)",
        "value": B * T / (fft_ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": fft_wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"fft_prefill_{w.name}", "B": B, "D": D, "d": d, "T": T,
                   "io": w.io, "workspace_bytes": wsf},
        "prefill_ms": fft_ms,
        "scan_prefill_ms": scan_ms,
        "scan_prefill_tokens_per_s": B * T / (scan_ms * 1e-3),
        "fft_over_scan_time": fft_ms / scan_ms,
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "lh_prefill_fft (all passes)", "bytes_per_launch": alg,
                     "pass_bytes_per_launch": pbytes,
                     "pass_gbps": pbytes / (fft_ms * 1e-3) / 1e9},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def companion_step_bytes(w):
    """Algorithmic bytes of one companion step: the float64 state [B, D, 2d]
    read and written, u_t and y_t, the coefficients a, beta [D, 2d] and h0."""
    es = 2 if w.io == "bf16" else 4
    return 2 * 8 * w.B * w.D * 2 * w.d + 2 * es * w.B * w.D + 2 * 8 * w.D * 2 * w.d + 4 * w.D


def companion_main(args):
    import numpy as np
    import torch

    import paper_2310_18780_amd as lh
    import workloads

    lh.lib()
    w = workloads.workload(args.companion_workload)
    t = make_device_inputs(w)
    B, T, D, d, K = w.B, w.T, w.D, w.d, w.K
    a = torch.empty((D, 2 * d), dtype=torch.float64, device="cuda")
    beta = torch.empty_like(a)
    xc = torch.empty((B, D, 2 * d), dtype=torch.float64, device="cuda")
    xm = torch.empty((B, D, d), dtype=torch.complex64, device="cuda")
    ws = torch.empty(max(lh.companion_init_workspace_bytes(D, d, T), 1), dtype=torch.uint8,
                     device="cuda")
    y_dec = torch.empty((K, B, D), dtype=t["u"].dtype, device="cuda")
    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        s, e = ev(), ev()
        s.record(stream)
        for _ in range(reps):
            fn()
        e.record(stream)
        torch.cuda.synchronize()
        return s.elapsed_time(e) / reps

    coeff_ms = timed(lambda: lh.companion_coeffs(t["lam"], t["R"], a, beta), 5)
    init_ms = timed(lambda: lh.companion_init(a, t["u"], xc, workspace=ws), max(3, args.steps // 4))

    def graph_of(step):
        step()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        return g

    gc = graph_of(lambda: [lh.companion_step(a, beta, t["h0"], xc, t["ud"][k], y_dec[k])
                           for k in range(K)])
    gm = graph_of(lambda: [lh.step(t["lam"], t["R"], t["h0"], xm, t["ud"][k], y_dec[k])
                           for k in range(K)])
    for _ in range(args.warmup):
        gc.replay()
        gm.replay()
    t0 = time.perf_counter()
    comp_ms = timed(gc.replay, args.steps)
    wall = (time.perf_counter() - t0) * 1e3 / args.steps
    modal_ms = timed(gm.replay, args.steps)
    us = comp_ms * 1e3 / K
    nbytes = companion_step_bytes(w)
    gbs = nbytes / (us * 1e-6) / 1e9
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        import oracle.companion as oc

        lam, R, h0 = workloads.make_params(w)
        ar, br, b0 = oc.from_modal(lam, R, h0)
        done, t1 = 0, time.perf_counter()
        x0 = np.zeros(2 * d)
        for b in range(B):
            ud = workloads.decode_row(w, b)
            for c in range(D):
                oc.companion_run(ar[c], br[c], b0[c], ud[:, c], x0)
                done += 1
                if time.perf_counter() - t1 > 10.0:
                    break
            if time.perf_counter() - t1 > 10.0:
                break
        dt = time.perf_counter() - t1
        cpu = {"value": done / D * K / dt, "unit": "tokens/s", "cores": 1, **host_cpu(),
               "kind": "oracle",
               "sample": f"{done} (b,c) rows of {w.name}, K={K} companion steps each (float64 "
                         f"numpy, one process) in {dt:.2f} s; value = steps per second scaled "
                         f"to whole sequences (rows / D * K / time)",
               "seconds": dt}
    out = {
        "metric": "decode tokens/s (companion-form recurrence)",
        "value": B * K / (comp_ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": w.name, "B": B, "D": D, "d": d, "order": 2 * d, "T": T, "K": K,
                   "io": w.io},
        "companion_us_per_token_step": us,
        "modal_us_per_token_step": modal_ms * 1e3 / K,
        "modal_tokens_per_s": B * K / (modal_ms * 1e-3),
        "init_ms": init_ms,
        "init_tokens_per_s": B * T / (init_ms * 1e-3),
        "coeffs_ms": coeff_ms,
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "companion_step_kernel", "bytes_per_launch": nbytes},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def decode_pool(w, t, npool, reps, floors=True):
    """The decode step over a pool of ``npool`` state buffers (``npool`` x the
    state, larger than the 256 MB Infinity Cache), one launch per buffer in
    turn, replayed from a graph: every launch reads and writes its state in
    HBM (each buffer was last touched ``npool`` launches earlier).  u_t and
    y_t are one slice each, so the launch moves the step's algorithmic bytes
    with only the state coming from HBM.  With ``floors``, plain torch kernels
    moving the same state bytes over the same pool are timed the same way: an
    in-place update of each buffer, and a copy of each buffer into the one half
    a pool away (last touched ``npool / 2`` launches, 0.5 GiB, earlier)."""
    import torch

    import paper_2310_18780_amd as lh

    B, D, d = w.B, w.D, w.d
    pool = [torch.zeros((B, D, d), dtype=torch.complex64, device="cuda") for _ in range(npool)]
    yk = torch.empty((B, D), dtype=t["u"].dtype, device="cuda")
    stream = torch.cuda.current_stream()

    def graph_of(fn):
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        g.replay()
        torch.cuda.synchronize()
        return g

    def per_launch_us(g):
        a, c = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            g.replay()
        c.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(c) * 1e3 / (reps * npool)

    g = graph_of(lambda: [lh.step(t["lam"], t["R"], t["h0"], s, t["ud"][0], yk) for s in pool])
    out = {"launch_us": per_launch_us(g), "pool_buffers": npool,
           "pool_bytes": npool * 8 * B * D * d, "replays": reps}
    del g
    if floors:
        fl = [s.view(torch.float32) for s in pool]
        g = graph_of(lambda: [f.add_(1.0) for f in fl])
        out["inplace_add_floor_us"] = per_launch_us(g)
        del g
        g = graph_of(lambda: [fl[(i + npool // 2) % npool].copy_(fl[i]) for i in range(npool)])
        out["copy_floor_us"] = per_launch_us(g)
        del g
    del pool
    torch.cuda.synchronize()
    return out


def len_pool(r):
    return r["pool_buffers"]


def decode_pool_only_main(args):
    """Only the HBM-streaming decode (``decode_pool`` without the floors), for
    counter passes of the decode kernel on that pattern."""
    import paper_2310_18780_amd as lh
    import workloads

    lh.lib()
    w = workloads.workload(args.workload)
    t = make_device_inputs(w.with_(T=1, K=1))
    r = decode_pool(w, t, args.stream_pool, max(1, args.steps), floors=False)
    us = r["launch_us"]
    print(json.dumps({"workload": w.name, "decode_pool": r,
                      "gbps": decode_bytes(w) / (us * 1e-6) / 1e9}), flush=True)


def launch_floor_main(args):
    """Reference points for the decode step: per-launch times of plain torch
    kernels with the step's footprint (the state's bytes), replayed K at a time
    from a graph exactly as the decode steps are."""
    import torch

    import workloads

    w = workloads.workload(args.workload)
    nbytes = 8 * w.B * w.D * w.d
    a = torch.zeros(nbytes // 4, device="cuda")
    b = torch.zeros_like(a)
    K = w.K

    def per_launch_us(fn):
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(K):
                fn()
        g.replay()
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t = []
        for _ in range(max(3, args.steps // 4)):
            s.record()
            g.replay()
            e.record()
            torch.cuda.synchronize()
            t.append(s.elapsed_time(e) * 1e3 / K)
        return sorted(t)[len(t) // 2]

    out = {
        "metric": "per-launch time of reference kernels with the decode step's footprint",
        "config": {"workload": w.name, "state_bytes": nbytes, "launches_per_graph": K},
        "empty_launch_us": per_launch_us(lambda: a[:1].add_(1.0)),
        "inplace_add_state_bytes_us": per_launch_us(lambda: a.add_(1.0)),
        "copy_state_bytes_us": per_launch_us(lambda: b.copy_(a)),
        "decode_step_bytes": decode_bytes(w),
    }
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this benchmark runs on exactly one GPU; --gpus {args.gpus} is not "
              f"supported (every (b, c) row is independent, so batch/channel sharding needs "
              f"no exchange; it is not built here).", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.multihead:
        multihead_main(args)
        return
    if args.distill:
        distill_main(args)
        return
    if args.fft:
        fft_main(args)
        return
    if args.companion:
        companion_main(args)
        return
    if args.launch_floor:
        launch_floor_main(args)
        return
    if args.decode_pool_only:
        decode_pool_only_main(args)
        return

    import torch

    import paper_2310_18780_amd as lh
    import workloads

    lh.lib()
    w = workloads.workload(args.workload)
    t_setup = time.perf_counter()
    t = make_device_inputs(w)
    B, T, D, d, K = w.B, w.T, w.D, w.d, w.K
    state = torch.empty((B, D, d), dtype=torch.complex64, device="cuda")
    y = torch.empty_like(t["u"])
    y_dec = torch.empty((K, B, D), dtype=t["u"].dtype, device="cuda")
    wsb = lh.workspace_bytes(B, D, d, T)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def prefill():
        lh.prefill(t["lam"], t["R"], t["h0"], t["u"], state, y, workspace=ws)

    def decode_eager():
        for k in range(K):
            lh.step(t["lam"], t["R"], t["h0"], state, t["ud"][k], y_dec[k])

    prefill()
    decode_eager()
    torch.cuda.synchronize()
    graph = None
    if args.decode_launch == "graph":
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            decode_eager()
        torch.cuda.synchronize()

        def decode():
            graph.replay()
    else:
        decode = decode_eager
    setup_s = time.perf_counter() - t_setup

    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    for _ in range(args.warmup):
        prefill()
        decode()
    torch.cuda.synchronize()

    marks = [(ev(), ev(), ev()) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for (a, b_, c) in marks:
        a.record(stream)
        prefill()
        b_.record(stream)
        decode()
        c.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    pre_ms = [a.elapsed_time(b_) for a, b_, _ in marks]
    dec_ms = [b_.elapsed_time(c) for _, b_, c in marks]
    pre_avg = sorted(pre_ms)[len(pre_ms) // 2]  # median of the timed prefills
    dec_avg = sum(dec_ms) / len(dec_ms)
    step_ms = wall * 1e3 / args.steps
    dec_launch_us = dec_avg * 1e3 / K

    dbytes = decode_bytes(w)
    dec_gbs = dbytes / (dec_launch_us * 1e-6) / 1e9
    pre_tf = prefill_flops(w) / (pre_avg * 1e-3) / 1e12
    traffic = counter_traffic(f"decode_step_{w.name}_counters.txt",
                              src_digest("decode.hip", "lh_internal.hpp"))
    pre_digest = src_digest("prefill.hip", "prefill_mfma.hip", "lh_internal.hpp")
    traffic_pre = counter_traffic(f"prefill_{w.name}_counters.txt", pre_digest)
    # The matrix-core plans at d = 16 and 32 execute their split-term
    # contractions far below the bfloat16 MFMA ridge (at most 208 flops per
    # byte of u and y against 2500 / 8 = 312), so their roofline is HBM; at
    # d = 64 the 92 products per channel, 16 rows and 32 steps come to 368
    # flops per byte, above the ridge, so its roofline is the bfloat16 MFMA
    # peak; the VALU scan executes about the declared flops at high
    # intensity, so its roofline is the VALU peak.
    plan = lh.prefill_plan(w.B, w.D, w.d, w.T, io=w.io)
    pre_gbs = prefill_bytes(w) / (pre_avg * 1e-3) / 1e9
    if plan == "scan":
        roofline_prefill = {"bound": "alu", "achieved": pre_tf, "peak": FP32_VALU_PEAK_TFLOPS,
                            "unit": "TFLOP/s", "frac": pre_tf / FP32_VALU_PEAK_TFLOPS}
    elif w.d == 64:  # matrix-core plan above the MFMA ridge: bound by the bf16 MFMA rate
        mf = mfma64_flops(w) / (pre_avg * 1e-3) / 1e12
        roofline_prefill = {"bound": "mfma", "achieved": mf, "peak": BF16_MFMA_PEAK_TFLOPS,
                            "unit": "TFLOP/s", "frac": mf / BF16_MFMA_PEAK_TFLOPS,
                            "mfma_flops_per_launch": mfma64_flops(w),
                            "hbm_frac": pre_gbs / HBM_PEAK_GBS}
    else:
        roofline_prefill = {"bound": "hbm", "achieved": pre_gbs, "peak": HBM_PEAK_GBS,
                            "unit": "GB/s", "frac": pre_gbs / HBM_PEAK_GBS}
    roofline_prefill.update({
        "plan": plan, "traffic": traffic_pre,
        "traffic_gbps": (traffic_pre / (pre_avg * 1e-3) / 1e9 if traffic_pre is not None else None),
        "flops_per_launch": prefill_flops(w), "bytes_per_launch": prefill_bytes(w),
        "gbps": pre_gbs, "declared_tflops": pre_tf,
        "declared_frac_of_fp32_valu_peak": pre_tf / FP32_VALU_PEAK_TFLOPS,
        "mfma_busy": profile_value(f"prefill_{w.name}_sq_counters.txt", "mfma_busy_fraction",
                                   pre_digest),
        "valu_busy": profile_value(f"prefill_{w.name}_sq_counters.txt", "valu_busy_fraction",
                                   pre_digest)})

    # Eager decode: K launches through the binding, one per token (host
    # argument checks and marshalling included), timed like the graph replay.
    for k in range(min(K, 8)):
        lh.step(t["lam"], t["R"], t["h0"], state, t["ud"][k], y_dec[k])
    torch.cuda.synchronize()
    a_e, c_e = ev(), ev()
    t_e = time.perf_counter()
    a_e.record(stream)
    decode_eager()
    c_e.record(stream)
    torch.cuda.synchronize()
    eager_us = a_e.elapsed_time(c_e) * 1e3 / K
    eager_host_us = (time.perf_counter() - t_e) * 1e6 / K

    # HBM-streaming decode: the same kernel over a pool of state buffers larger
    # than the 256 MB Infinity Cache (as the states of a model's layers
    # together are), so that every launch reads and writes its state in HBM;
    # plain copy and in-place update kernels over the same pool beside it.
    streaming = None
    if args.stream_pool > 0:
        streaming = decode_pool(w, t, args.stream_pool, 8)
        streaming["gbps"] = dbytes / (streaming["launch_us"] * 1e-6) / 1e9
        streaming["frac"] = streaming["gbps"] / HBM_PEAK_GBS
        streaming["state_bytes_gbps_of_copy_floor"] = (
            16 * B * D * d / (streaming["copy_floor_us"] * 1e-6) / 1e9)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args.cpu_rows)

    # The decode kernel's roofline: HBM, taken on the pool pass where the state
    # streams from HBM; the timed workload's own decode (one 16 MiB state
    # stepped K times) keeps its state in the Infinity Cache, so its rate is
    # reported beside it, labelled with that residency.
    dig = src_digest("decode.hip", "lh_internal.hpp")
    resident = {"bound": "hbm", "achieved": dec_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": dec_gbs / HBM_PEAK_GBS, "traffic": traffic,
                "traffic_gbps": (traffic / (dec_launch_us * 1e-6) / 1e9
                                 if traffic is not None else None),
                "kernel": "step_pairs_kernel", "bytes_per_launch": dbytes,
                "launch_us": dec_launch_us,
                "residency": "infinity-cache: the workload's one state is stepped K times in a "
                             "row and stays in the 256 MB cache; counters include cache hits"}
    if streaming is not None:
        traffic_pool = counter_traffic(f"decode_step_{w.name}_pool_counters.txt", dig)
        roofline = {"bound": "hbm", "achieved": streaming["gbps"], "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": streaming["frac"], "traffic": traffic_pool,
                    "kernel": "step_pairs_kernel", "bytes_per_launch": dbytes,
                    "launch_us": streaming["launch_us"],
                    "copy_floor_us": streaming["copy_floor_us"],
                    "inplace_add_floor_us": streaming["inplace_add_floor_us"],
                    "residency": f"hbm: one launch per buffer of a {len_pool(streaming)}-buffer "
                                 f"state pool ({streaming['pool_bytes'] / 2**30:.2f} GiB), timed "
                                 f"over {streaming['replays']} graph replays"}
    else:
        roofline = resident

    out = {
        "metric": METRIC,
        "value": B * K / (dec_avg * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "dtype_detail": dtype_detail(w, plan),
        "data": "synthetic",
        "config": {"workload": w.name, "B": B, "D": D, "d": d, "T": T, "K": K, "io": w.io,
                   "decode_launch": args.decode_launch, "prefill_workspace_bytes": wsb},
        "prefill_tokens_per_s": B * T / (pre_avg * 1e-3),
        "prefill_ms": pre_avg,
        "decode_ms_per_step_total": dec_avg,
        "decode_us_per_token_step": dec_launch_us,
        "decode_gbps": dec_gbs,
        "decode_eager_us_per_token_step": eager_us,
        "decode_eager_host_us_per_token_step": eager_host_us,
        "roofline": roofline,
        "roofline_cache_resident": resident,
        "roofline_prefill": roofline_prefill,
        "decode_hbm_streaming": streaming,
        "cpu_baseline": cpu,
        "setup_s": setup_s,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
