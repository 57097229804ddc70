"""C ABI checks that need no GPU: the library loads, exports every function
``include/lh.h`` declares, and rejects bad arguments on the host with the
documented status before touching any device.

Calls here pass made-up addresses; they are only made where the library
returns before any device work (argument errors), and the "all arguments
valid" case runs only when no GPU is visible (it must then report
LH_ERR_NO_DEVICE).
"""
from __future__ import annotations

import ctypes
import os
import re

import pytest

import paper_2310_18780_amd as lh

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lh.h")

pytestmark = pytest.mark.skipif(not os.path.exists(lh.library_path()),
                                reason="liblh.so not built (run __graft_entry__.build())")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lh_[a-z_0-9]+)\s*\(", text)))


def header_enum(name):
    text = open(HEADER).read()
    m = re.search(r"#define\s+" + name + r"\s+(\d+)", text)
    return int(m.group(1))


def no_gpu():
    import torch

    return torch.cuda.device_count() == 0


def test_exports_every_declared_symbol():
    L = lh.lib()
    names = header_functions()
    assert {"lh_prefill", "lh_step", "lh_prefill_workspace_bytes", "lh_status_string",
            "lh_prefill_with_plan", "lh_prefill_with_plan_workspace_bytes"} <= set(names)
    for n in names:
        assert hasattr(L, n), f"{n} declared in lh.h but not exported"


def test_exported_symbols_are_c_linkage():
    out = os.popen(f"nm -D --defined-only {lh.library_path()}").read()
    for n in header_functions():
        assert re.search(r"\bT " + n + r"$", out, flags=re.M), n


def test_abi_version_and_status_strings():
    L = lh.lib()
    assert L.lh_abi_version() == header_enum("LH_ABI_VERSION")
    for code, name in lh.STATUS.items():
        assert L.lh_status_string(code).decode().startswith(name)
    assert L.lh_status_string(99).decode() == "unknown lh_status"


def test_workspace_sizes():
    # no workspace for T = 0 or a single chunk
    assert lh.workspace_bytes(2, 8, 4, 0) == 0
    assert lh.workspace_bytes(2, 8, 4, 100, plan=100) == 0
    assert lh.workspace_bytes(2, 8, 4, 100, plan=500) == 0
    # chunked: lambda^C table (256-byte aligned) + [B, nchunks, D, d] entry states
    B, D, d, T, C = 3, 10, 4, 100, 30
    nch = -(-T // C)
    pow_bytes = -(-(D * d * 8) // 256) * 256
    assert lh.workspace_bytes(B, D, d, T, plan=C) == pow_bytes + B * nch * D * d * 8
    # automatic plans: matrix-core tables for d = 16 / 32 with D % 8 == 0 and
    # d = 64 with D % 4 == 0 (bfloat16 fragments of P, T, W: (4 d/16 + 2) x 3 x
    # 64 x 16 B per channel, plus lambda^C), the VALU plan otherwise
    frag = lambda D, d: D * (4 * (d // 16) + 2) * 3 * 64 * 16  # noqa: E731
    assert lh.workspace_bytes(64, 2048, 16, 4096) == -(-frag(2048, 16) // 256) * 256 + 2048 * 16 * 8
    # the explicit matrix-core plan needs the same tables
    assert lh.workspace_bytes(4, 1024, 32, 65536, plan=-1) == frag(1024, 32) + 1024 * 32 * 8
    # long prompt, few rows: the automatic plan cuts the prompt into 32 segments
    # of 2048 steps on the matrix cores (lambda^C, segment entry states, then
    # the matrix-core tables)
    up = lambda x: -(-x // 256) * 256  # noqa: E731
    seg_ws = up(1024 * 32 * 8) + up(4 * 32 * 1024 * 32 * 8) + frag(1024, 32) + 1024 * 32 * 8
    assert lh.workspace_bytes(4, 1024, 32, 65536) == seg_ws
    assert lh.workspace_bytes(4, 1024, 32, 65536, plan=-2) == seg_ws
    # the VALU chunked scan when asked for (32 chunks of 2048 steps)
    assert lh.workspace_bytes(4, 1024, 32, 65536, plan=2048) == 1024 * 32 * 8 + 4 * 32 * 1024 * 32 * 8
    # the segmented plan needs segments of >= 256 steps, a multiple of 32
    assert lh.lib().lh_prefill_with_plan_workspace_bytes(4, 1024, 32, 500, -2) == ctypes.c_size_t(-1).value
    # the matrix-core plan needs d = 16 / 32 and D % 8 == 0, or d = 64 and D % 4 == 0
    bad = ctypes.c_size_t(-1).value
    assert lh.lib().lh_prefill_with_plan_workspace_bytes(2, 12, 16, 64, -1) == bad
    assert lh.lib().lh_prefill_with_plan_workspace_bytes(2, 18, 64, 64, -1) == bad
    assert lh.lib().lh_prefill_with_plan_workspace_bytes(2, 8, 48, 64, -1) == bad
    # d = 64: the same fragments (18 per channel), then lambda^C
    assert lh.workspace_bytes(2, 12, 64, 64, plan=-1) == up(frag(12, 64)) + 12 * 64 * 8
    # the wide d = 64 workload: the matrix-core plan; with bfloat16 u/y (no
    # matrix-core plan at d = 64) one VALU pass
    assert lh.workspace_bytes(256, 2048, 64, 1024) == up(frag(2048, 64)) + 2048 * 64 * 8
    assert lh.prefill_plan(256, 2048, 64, 1024, io="bf16") == "scan"
    # D % 8 != 0: VALU plan, few rows -> 5 chunks of 64 steps
    assert lh.workspace_bytes(2, 70, 16, 300) == 70 * 16 * 8 + 2 * 5 * 70 * 16 * 8
    # invalid sizes
    L = lh.lib()
    bad = ctypes.c_size_t(-1).value
    for args in [(0, 1, 1, 1, 0), (1, 0, 1, 1, 0), (1, 1, 0, 1, 0), (1, 1, 1025, 1, 0),
                 (1, 1, 1, -1, 0), (1, 1, 1, 1, -1), (1, 1, 1, 1, -3),
                 (1 << 40, 1 << 20, 64, 1 << 20, 0)]:
        assert L.lh_prefill_with_plan_workspace_bytes(*args) == bad, args
        if args[4] == 0:
            assert L.lh_prefill_workspace_bytes(*args[:4]) == bad, args
    # the automatic request of the planned call is lh_prefill's own size
    for args in [(2, 8, 4, 0), (64, 2048, 16, 4096), (4, 1024, 32, 65536), (2, 70, 16, 300)]:
        assert L.lh_prefill_with_plan_workspace_bytes(*args, 0) == L.lh_prefill_workspace_bytes(*args)


def test_prefill_plan_query():
    """lh_prefill_plan: the plan lh_prefill takes (host only, no device)."""
    P = lh.prefill_plan
    assert P(1, 4, 4, 64) == "scan"                    # d = 4: no matrix-core plan
    assert P(256, 2048, 64, 1024) == "mfma"            # d = 64: matrix-core plan, float32 u/y
    assert P(256, 2048, 64, 1024, io="bf16") == "scan"  # d = 64 needs float32 u/y
    assert P(1, 768, 64, 1024) == "scan"               # d = 64, B < 4 and B T <= 1024
    assert P(4, 768, 64, 1024) == "mfma_seg"           # d = 64, few rows
    assert P(16, 768, 64, 1000) == "mfma"              # no segments, 4 rows or more
    assert P(2, 768, 64, 1000) == "scan"               # no segments, fewer than 4 rows, 192 workgroups
    assert P(4, 768, 64, 256) == "mfma"                # no segments, 4 rows
    assert P(64, 768, 64, 1000) == "mfma"              # no segments, 768 workgroups
    assert P(64, 2048, 16, 4096, io="bf16") == "mfma"  # enough (channel, row) tiles
    assert P(4, 1024, 32, 65536) == "mfma_seg"         # 4 rows, long prompt
    assert P(16, 768, 16, 2048) == "mfma"              # chunk-step estimate: whole prompt
    assert P(2, 512, 32, 8192) == "mfma_seg"           # chunk-step estimate: segments
    assert P(2, 70, 16, 300) == "scan"                 # D % 8 != 0
    assert P(4, 1024, 32, 500) == "scan"               # T does not split into segments
    # explicit plans
    assert P(4, 1024, 32, 65536, plan=2048) == "scan"
    assert P(2, 16, 16, 64, plan=-1) == "mfma"
    assert P(2, 16, 16, 1024, plan=-2) == "mfma_seg"
    assert P(2, 12, 64, 64, plan=-1) == "mfma"    # d = 64, float32 u/y
    L = lh.lib()
    for args in [(2, 12, 16, 64, -1, 0), (2, 12, 64, 64, -1, 1), (2, 18, 64, 64, -1, 0), (4, 1024, 32, 500, -2, 0), (0, 1, 1, 1, 0, 0),
                 (1, 1, 1, 1, -3, 0), (1, 1, 1, 1, 0, 2), (1, 1, 1, -1, 0, 1)]:
        assert L.lh_prefill_plan(*args) == -1, args


# made-up, well-separated, aligned addresses (never dereferenced)
A = 0x7F0000000000
MB = 1 << 20


def prefill_args(**kw):
    """Arguments of lh_prefill_with_plan (with the plan request ``chunk``)."""
    a = dict(lam=A, R=A + MB, h0=A + 2 * MB, u=A + 3 * MB, B=2, D=8, d=4, T=16, io=lh.LH_F32,
             state=A + 64 * MB, y=A + 128 * MB, chunk=0, ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    return [a[k] for k in ("lam", "R", "h0", "u", "B", "D", "d", "T", "io", "state", "y", "chunk",
                           "ws", "ws_bytes", "stream")]


def auto_args(**kw):
    """Arguments of lh_prefill (no plan request)."""
    args = prefill_args(**kw)
    return args[:11] + args[12:]


def step_args(**kw):
    a = dict(lam=A, R=A + MB, h0=A + 2 * MB, state=A + 64 * MB, u=A + 3 * MB, y=A + 128 * MB,
             B=2, D=8, d=4, io=lh.LH_F32, stream=None)
    a.update(kw)
    return [a[k] for k in ("lam", "R", "h0", "state", "u", "y", "B", "D", "d", "io", "stream")]


@pytest.mark.parametrize("kw,status", [
    (dict(lam=None), 1), (dict(R=None), 1), (dict(h0=None), 1), (dict(state=None), 1),
    (dict(u=None), 1), (dict(y=None), 1),
    (dict(B=0), 1), (dict(D=-3), 1), (dict(d=0), 1), (dict(d=1025), 1), (dict(T=-1), 1),
    (dict(chunk=-3), 1),
    (dict(chunk=-2), 1),                 # segmented plan: d = 4 unsupported
    (dict(B=1 << 40, D=1 << 20), 1),  # element count overflow
    (dict(io=7), 3),
    (dict(u=A + 3 * MB + 2), 1),  # misaligned float32 input
    (dict(lam=A + 4), 1),  # misaligned complex64
    (dict(y=A + 3 * MB + 64), 2),  # y overlaps u
    (dict(state=A + MB + 8), 2),  # state overlaps R
    (dict(y=A + 64 * MB + 16), 2),  # y overlaps state
    (dict(chunk=4), 5),  # chunked plan needs a workspace
    (dict(chunk=4, ws=A + 256 * MB, ws_bytes=16), 5),  # too small
    (dict(chunk=4, ws=A + 256 * MB + 8, ws_bytes=1 << 20), 1),  # misaligned workspace
    (dict(chunk=4, ws=A + 64 * MB, ws_bytes=1 << 20), 2),  # workspace overlaps state
])
def test_prefill_rejects_bad_arguments(kw, status):
    L = lh.lib()
    assert L.lh_prefill_with_plan(*prefill_args(**kw)) == status
    assert L.lh_last_error().decode() != ""
    if "chunk" not in kw:  # the automatic call checks the same way
        assert L.lh_prefill(*auto_args(**kw)) == status
        assert L.lh_last_error().decode() != ""


def test_prefill_t0_allows_null_io():
    if not no_gpu():
        pytest.skip("made-up addresses are only passed through when no GPU is visible")
    L = lh.lib()
    assert L.lh_prefill(*auto_args(T=0, u=None, y=None)) == 4  # reaches the device check
    assert L.lh_prefill_with_plan(*prefill_args(T=0, u=None, y=None)) == 4


@pytest.mark.parametrize("kw,status", [
    (dict(lam=None), 1), (dict(y=None), 1), (dict(u=None), 1), (dict(state=None), 1),
    (dict(B=0), 1), (dict(d=2000), 1), (dict(io=2), 3),
    (dict(y=A + 3 * MB), 2),  # y_t aliases u_t
    (dict(state=A + 2 * MB), 2),  # state overlaps h0
    (dict(y=A + 64 * MB + 8), 2),  # y_t overlaps state
    (dict(h0=A + 2 * MB + 2), 1),
])
def test_step_rejects_bad_arguments(kw, status):
    L = lh.lib()
    assert L.lh_step(*step_args(**kw)) == status


def test_valid_arguments_report_no_device_without_gpu():
    if not no_gpu():
        pytest.skip("made-up addresses are only passed through when no GPU is visible")
    L = lh.lib()
    assert L.lh_prefill(*auto_args()) == 4
    assert "device" in L.lh_last_error().decode()
    assert L.lh_prefill_with_plan(*prefill_args()) == 4
    assert L.lh_step(*step_args()) == 4
    assert L.lh_step(*step_args(io=lh.LH_BF16)) == 4


def test_binding_raises_when_library_missing(monkeypatch, tmp_path):
    monkeypatch.setattr(lh, "_LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(lh, "_lib", None)
    with pytest.raises(ImportError):
        lh.lib()


def mh_args(**kw):
    a = dict(lam=A, R=A + MB, h0=A + 2 * MB, state=A + 64 * MB, q=A + 3 * MB, k=A + 4 * MB,
             v=A + 5 * MB, y=A + 128 * MB, B=2, M=2, N=4, d=4, io=lh.LH_F32, stream=None)
    a.update(kw)
    return [a[k] for k in ("lam", "R", "h0", "state", "q", "k", "v", "y", "B", "M", "N", "d", "io",
                           "stream")]


@pytest.mark.parametrize("kw,status", [
    (dict(lam=None), 1), (dict(state=None), 1), (dict(q=None), 1), (dict(k=None), 1),
    (dict(v=None), 1), (dict(y=None), 1),
    (dict(B=0), 1), (dict(M=0), 1), (dict(N=-1), 1), (dict(d=0), 1), (dict(d=1025), 1),
    (dict(B=1 << 20, M=1 << 10, N=1 << 16), 1),  # state size overflow (2^63 bytes)
    (dict(io=5), 3),
    (dict(y=A + 4 * MB), 2),            # y aliases k
    (dict(state=A + 5 * MB + 8), 2),    # state overlaps v
    (dict(y=A + 64 * MB + 64), 2),      # y overlaps state
    (dict(q=A + 3 * MB + 2), 1),        # misaligned float32
    (dict(R=A + MB + 4), 1),            # misaligned complex64
])
def test_mh_step_rejects_bad_arguments(kw, status):
    L = lh.lib()
    assert L.lh_mh_step(*mh_args(**kw)) == status
    assert L.lh_last_error().decode() != ""


def test_mh_step_reports_no_device_without_gpu():
    if not no_gpu():
        pytest.skip("made-up addresses are only passed through when no GPU is visible")
    L = lh.lib()
    assert L.lh_mh_step(*mh_args()) == 4
    assert L.lh_mh_step(*mh_args(io=lh.LH_BF16, d=3)) == 4


def distill_args(**kw):
    a = dict(A=A, th=A + MB, R=A + 2 * MB, tg=A + 3 * MB, D=4, d=4, L=16, loss=A + 64 * MB,
             dA=A + 65 * MB, dth=A + 66 * MB, dR=A + 67 * MB, h=None, stream=None)
    a.update(kw)
    return [a[k] for k in ("A", "th", "R", "tg", "D", "d", "L", "loss", "dA", "dth", "dR", "h",
                           "stream")]


@pytest.mark.parametrize("kw,status", [
    (dict(A=None), 1), (dict(th=None), 1), (dict(R=None), 1), (dict(tg=None), 1),
    (dict(loss=None), 1), (dict(dA=None), 1), (dict(dth=None), 1), (dict(dR=None), 1),
    (dict(D=0), 1), (dict(d=0), 1), (dict(d=1025), 1), (dict(L=0), 1),
    (dict(D=1 << 40, L=1 << 30), 1),    # size overflow
    (dict(dA=A + MB), 2),               # output overlaps theta
    (dict(dth=A + 65 * MB + 4), 2),     # dtheta overlaps dA
    (dict(h=A + 3 * MB + 16), 2),       # hhat overlaps the target
    (dict(R=A + 2 * MB + 4), 1),        # misaligned complex64
])
def test_distill_rejects_bad_arguments(kw, status):
    L = lh.lib()
    assert L.lh_distill(*distill_args(**kw)) == status
    assert L.lh_last_error().decode() != ""


def test_distill_reports_no_device_without_gpu():
    if not no_gpu():
        pytest.skip("made-up addresses are only passed through when no GPU is visible")
    assert lh.lib().lh_distill(*distill_args()) == 4
    assert lh.lib().lh_distill(*distill_args(h=A + 128 * MB)) == 4


def fft_ws(B, D, d, T):
    """Workspace of the FFT prefill, from its documented layout: the N-point
    twiddle table, per-mode polar constants, the filter spectrum and the
    spectra of ceil(B/2) row pairs (N D complex64 each), each region rounded
    up to 256 bytes; partial states of the state contraction come on top when
    it splits time into several ranges."""
    up = lambda x: -(-x // 256) * 256  # noqa: E731
    N = 1
    while N < 2 * T - 1:
        N *= 2
    return up(8 * N) + up(16 * D * d) + up(8 * N * D) + up(8 * ((B + 1) // 2) * N * D)


def test_fft_workspace_sizes():
    assert lh.fft_workspace_bytes(3, 8, 4, 0) == 0
    for B, D, d, T in [(3, 10, 4, 100), (1, 1, 1, 1), (2, 7, 3, 2), (4, 33, 8, 256)]:
        assert lh.fft_workspace_bytes(B, D, d, T) == fft_ws(B, D, d, T), (B, D, d, T)
    # two 256-step ranges of the state contraction: partial states [2, B, D, d]
    assert lh.fft_workspace_bytes(4, 33, 8, 257) == fft_ws(4, 33, 8, 257) + 2 * 4 * 33 * 8 * 8
    # the long-prompt workload: 2^17-point transforms, 128 partial states
    assert lh.fft_workspace_bytes(4, 1024, 32, 65536) == (
        fft_ws(4, 1024, 32, 65536) + 128 * 4 * 1024 * 32 * 8)
    L = lh.lib()
    bad = ctypes.c_size_t(-1).value
    max_t = 1 << 19
    assert L.lh_prefill_fft_workspace_bytes(1, 4, 4, max_t) == fft_ws(1, 4, 4, max_t) + (
        # 2048 ranges of 256 steps for 1 x 1 x 1 waves
        2048 * 1 * 4 * 4 * 8)
    for args in [(1, 4, 4, max_t + 1), (0, 4, 4, 8), (1, 0, 4, 8), (1, 4, 0, 8), (1, 4, 1025, 8),
                 (1, 4, 4, -1), (1 << 40, 1 << 20, 64, 1 << 10)]:
        assert L.lh_prefill_fft_workspace_bytes(*args) == bad, args


def fft_args(**kw):
    a = dict(lam=A, R=A + MB, h0=A + 2 * MB, u=A + 3 * MB, B=2, D=8, d=4, T=16, io=lh.LH_F32,
             state=A + 64 * MB, y=A + 128 * MB, ws=A + 256 * MB, ws_bytes=1 << 20, stream=None)
    a.update(kw)
    return [a[k] for k in ("lam", "R", "h0", "u", "B", "D", "d", "T", "io", "state", "y", "ws",
                           "ws_bytes", "stream")]


@pytest.mark.parametrize("kw,status", [
    (dict(lam=None), 1), (dict(R=None), 1), (dict(h0=None), 1), (dict(state=None), 1),
    (dict(u=None), 1), (dict(y=None), 1),
    (dict(B=0), 1), (dict(D=-3), 1), (dict(d=0), 1), (dict(d=1025), 1), (dict(T=-1), 1),
    (dict(T=(1 << 19) + 1), 1),          # longer than the transforms allow
    (dict(io=7), 3),
    (dict(u=A + 3 * MB + 2), 1),         # misaligned float32 input
    (dict(y=A + 3 * MB + 64), 2),        # y overlaps u
    (dict(state=A + MB + 8), 2),         # state overlaps R
    (dict(ws=None), 5),                  # workspace needed
    (dict(ws_bytes=16), 5),              # too small
    (dict(ws=A + 256 * MB + 8), 1),      # misaligned workspace
    (dict(ws=A + 128 * MB), 2),          # workspace overlaps y
])
def test_prefill_fft_rejects_bad_arguments(kw, status):
    L = lh.lib()
    assert L.lh_prefill_fft(*fft_args(**kw)) == status
    assert L.lh_last_error().decode() != ""


def test_prefill_fft_reports_no_device_without_gpu():
    if not no_gpu():
        pytest.skip("made-up addresses are only passed through when no GPU is visible")
    L = lh.lib()
    assert L.lh_prefill_fft(*fft_args()) == 4
    assert L.lh_prefill_fft(*fft_args(io=lh.LH_BF16, B=3, d=7)) == 4
    assert L.lh_prefill_fft(*fft_args(T=0, u=None, y=None, ws=None, ws_bytes=0)) == 4


def comp_coeff_args(**kw):
    a = dict(lam=A, R=A + MB, D=8, d=4, a=A + 64 * MB, beta=A + 65 * MB, stream=None)
    a.update(kw)
    return [a[k] for k in ("lam", "R", "D", "d", "a", "beta", "stream")]


def comp_step_args(**kw):
    a = dict(a=A, beta=A + MB, h0=A + 2 * MB, state=A + 64 * MB, u=A + 3 * MB, y=A + 128 * MB,
             B=2, D=8, d=4, io=lh.LH_F32, stream=None)
    a.update(kw)
    return [a[k] for k in ("a", "beta", "h0", "state", "u", "y", "B", "D", "d", "io", "stream")]


def comp_init_args(**kw):
    a = dict(a=A, u=A + 3 * MB, B=2, D=8, d=4, T=16, io=lh.LH_F32, state=A + 64 * MB,
             ws=A + 256 * MB, ws_bytes=1 << 20, stream=None)
    a.update(kw)
    return [a[k] for k in ("a", "u", "B", "D", "d", "T", "io", "state", "ws", "ws_bytes", "stream")]


@pytest.mark.parametrize("kw,status", [
    (dict(lam=None), 1), (dict(a=None), 1), (dict(beta=None), 1), (dict(D=0), 1), (dict(d=0), 1),
    (dict(d=17), 1),                       # beyond LH_COMPANION_MAX_MODES
    (dict(a=A + MB), 2),                   # a overlaps R
    (dict(beta=A + 64 * MB + 64), 2),      # beta overlaps a
    (dict(a=A + 64 * MB + 4), 1),          # misaligned float64
])
def test_companion_coeffs_rejects_bad_arguments(kw, status):
    L = lh.lib()
    assert L.lh_companion_coeffs(*comp_coeff_args(**kw)) == status
    assert L.lh_last_error().decode() != ""


@pytest.mark.parametrize("kw,status", [
    (dict(a=None), 1), (dict(state=None), 1), (dict(u=None), 1), (dict(y=None), 1),
    (dict(B=0), 1), (dict(d=17), 1), (dict(io=4), 3),
    (dict(state=A + 64 * MB + 8), 1),      # state must be 16-byte aligned
    (dict(beta=A + MB + 8), 1),            # so must the coefficients
    (dict(y=A + 3 * MB), 2),               # y_t aliases u_t
    (dict(state=A + MB), 2),               # state overlaps beta
])
def test_companion_step_rejects_bad_arguments(kw, status):
    L = lh.lib()
    assert L.lh_companion_step(*comp_step_args(**kw)) == status
    assert L.lh_last_error().decode() != ""


@pytest.mark.parametrize("kw,status", [
    (dict(a=None), 1), (dict(state=None), 1), (dict(u=None), 1), (dict(T=-1), 1), (dict(d=17), 1),
    (dict(io=9), 3), (dict(ws=None), 5), (dict(ws_bytes=8), 5),
    (dict(ws=A + 256 * MB + 8), 1),        # misaligned workspace
    (dict(state=A + 3 * MB), 2),           # state overlaps u
    (dict(ws=A + 64 * MB), 2),             # workspace overlaps state
])
def test_companion_init_rejects_bad_arguments(kw, status):
    L = lh.lib()
    assert L.lh_companion_init(*comp_init_args(**kw)) == status
    assert L.lh_last_error().decode() != ""


def test_companion_workspace_and_no_device():
    assert lh.companion_init_workspace_bytes(8, 4, 0) == 0
    assert lh.companion_init_workspace_bytes(8, 4, 16) == 16 * 8 * 8
    assert lh.lib().lh_companion_init_workspace_bytes(8, 17, 16) == ctypes.c_size_t(-1).value
    if not no_gpu():
        pytest.skip("made-up addresses are only passed through when no GPU is visible")
    L = lh.lib()
    assert L.lh_companion_coeffs(*comp_coeff_args()) == 4
    assert L.lh_companion_step(*comp_step_args()) == 4
    assert L.lh_companion_init(*comp_init_args()) == 4
    assert L.lh_companion_init(*comp_init_args(T=0, u=None, ws=None, ws_bytes=0)) == 4


def test_noalloc_rejects_sizes_beyond_its_scratch_before_any_device_work():
    """lh_prefill_noalloc: a plan needing more than LH_NOALLOC_SCRATCH_BYTES of
    scratch is refused on the host (LH_ERR_WORKSPACE), before the device is
    touched; sizes within it reach the device check."""
    L = lh.lib()
    args = auto_args()
    noalloc = args[:11] + [args[-1]]  # no workspace arguments
    big = dict(B=256, D=2048, d=64, T=1024)  # matrix-core tables: 114 MB
    assert lh.workspace_bytes(256, 2048, 64, 1024) > lh.NOALLOC_SCRATCH_BYTES
    a = auto_args(**big)
    assert L.lh_prefill_noalloc(*(a[:11] + [a[-1]])) == 5
    assert "scratch" in L.lh_last_error().decode()
    assert L.lh_prefill_noalloc(*(auto_args(d=0)[:11] + [None])) == 1
    if no_gpu():
        assert L.lh_prefill_noalloc(*noalloc) == 4
    assert header_enum_u64("LH_NOALLOC_SCRATCH_BYTES") == lh.NOALLOC_SCRATCH_BYTES


def header_enum_u64(name):
    text = open(HEADER).read()
    m = re.search(r"#define\s+" + name + r"\s+\(UINT64_C\((\d+)\)\s*<<\s*(\d+)\)", text)
    return int(m.group(1)) << int(m.group(2))


def test_one_hip_runtime_whatever_the_import_order():
    """Loading the library before anything imported torch must still leave
    one HIP runtime in the process (torch's), so that torch's memory and
    streams are the library's too."""
    import subprocess
    import sys

    code = ("import paper_2310_18780_amd as lh; lh.lib(); import torch; "
            "maps = open('/proc/self/maps').read(); "
            "print(len({l.split()[-1] for l in maps.splitlines() if 'libamdhip64' in l}))")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         timeout=120, cwd=ROOT)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip() == "1", out.stdout
