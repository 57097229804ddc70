"""Helpers of the GPU parity tests: run the HIP path through the C ABI on
seeded inputs and compare with the oracle.

Tolerances (derived from float32 arithmetic over the workloads' lengths):

* float32 outputs: per (b, c) row, ``max_t |y_gpu - y_ref| <= 1e-4 * max_t |y_ref|``
  (the relative tolerance 1e-4 applied to the row's infinity norm, since an
  elementwise relative error is undefined where an output crosses zero).  The
  row is the channel's whole output sequence y_0 .. y_{T+K-1} for one batch
  row, prompt outputs and decoded tokens alike (the filter's output y = h * u
  over the sequence): a few decode outputs alone can all be near zero by
  cancellation, where float32 sums of O(1) terms carry errors far above
  1e-4 of their own size;
* states: per (b, c), ``max_n |x_gpu - x_ref| <= 1e-4 * max_n |x_ref|``;
* bfloat16 outputs: elementwise ``|y_gpu - y_ref| <= 2^-8 |y_ref| + 1e-4 * rowmax``,
  i.e. the round-to-nearest error of bfloat16 (half a unit in the last place,
  at most 2^-8 relative) on top of the float32 tolerance.
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np

REL_TOL = 1e-4
BF16_REL = 2.0 ** -8


def to_device(lam, R, h0, up, ud, io: str, device="cuda"):
    import torch

    iot = torch.bfloat16 if io == "bf16" else torch.float32
    t = dict(
        lam=torch.from_numpy(np.ascontiguousarray(lam)).to(device),
        R=torch.from_numpy(np.ascontiguousarray(R)).to(device),
        h0=torch.from_numpy(np.ascontiguousarray(h0)).to(device),
        u=torch.from_numpy(np.ascontiguousarray(up)).to(device).to(iot),
        # decode inputs as [K, B, D] so that step k reads a contiguous [B, D]
        ud=torch.from_numpy(np.ascontiguousarray(ud.transpose(1, 0, 2))).to(device).to(iot),
    )
    return t


def run_gpu(t, plan: int = 0, ws=None):
    """Prefill (lh_prefill, or lh_prefill_with_plan when ``plan`` is not 0)
    then K decode steps; returns device tensors y [B,T,D], x_T, y_dec [K,B,D],
    x_end."""
    import torch

    import paper_2310_18780_amd as lh

    B, T, D = t["u"].shape
    K = t["ud"].shape[0]
    d = t["lam"].shape[1]
    dev = t["u"].device
    y = torch.full((B, T, D), float("nan"), dtype=t["u"].dtype, device=dev)
    state = torch.full((B, D, d), complex(float("nan"), float("nan")), dtype=torch.complex64,
                       device=dev)
    if plan == 0:
        lh.prefill(t["lam"], t["R"], t["h0"], t["u"], state, y, workspace=ws)
    else:
        lh.prefill_with_plan(t["lam"], t["R"], t["h0"], t["u"], state, y, plan, workspace=ws)
    x_T = state.clone()
    y_dec = torch.full((K, B, D), float("nan"), dtype=t["u"].dtype, device=dev)
    for k in range(K):
        lh.step(t["lam"], t["R"], t["h0"], state, t["ud"][k], y_dec[k])
    torch.cuda.synchronize()
    return dict(y_prefill=y, x_T=x_T, y_dec=y_dec, x_end=state)


def _np(x):
    import torch

    if x.dtype == torch.bfloat16:
        x = x.float()
    return x.cpu().numpy()


def seq_rowmax(*parts: np.ndarray) -> np.ndarray:
    """[rows, 1] infinity norms of the rows of the concatenated reference
    output arrays (each [rows, L_i], L_i may be 0)."""
    parts = [np.abs(np.asarray(p, dtype=np.float64)) for p in parts if p.shape[-1] > 0]
    return np.max(np.concatenate(parts, axis=-1), axis=-1, keepdims=True)


def check_y(y_gpu: np.ndarray, y_ref: np.ndarray, io: str, what: str, ref_rounded=False,
            rowmax: Optional[np.ndarray] = None):
    """y_* as [rows, L] arrays (L may be 0).  ``ref_rounded``: the reference is
    itself a bfloat16-rounded result (GPU against GPU), so each side carries
    half a bfloat16 ulp of rounding.  ``rowmax``: [rows, 1] scale of each row
    (default: the infinity norm of the row of ``y_ref``; see ``seq_rowmax``)."""
    if y_ref.shape[-1] == 0:
        return 0.0
    assert np.all(np.isfinite(y_gpu)), f"{what}: non-finite output"
    err = np.abs(y_gpu.astype(np.float64) - y_ref)
    if rowmax is None:
        rowmax = np.max(np.abs(y_ref), axis=-1, keepdims=True)
    if io == "bf16":
        bound = (2 if ref_rounded else 1) * BF16_REL * np.abs(y_ref) + REL_TOL * rowmax
    else:
        bound = REL_TOL * rowmax
    bad = err > bound
    if np.any(bad):
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(
            f"{what}: {int(bad.sum())} outputs out of tolerance; worst at {i}: gpu={y_gpu[i]!r} "
            f"ref={y_ref[i]!r} err={err[i]:.3g} bound={bound[i]:.3g} rowmax={rowmax[i[0]][0]:.3g}")
    return float(np.max(err / np.maximum(rowmax, 1e-300)))


def check_x(x_gpu: np.ndarray, x_ref: np.ndarray, what: str):
    """states as [rows, d] complex arrays."""
    assert np.all(np.isfinite(x_gpu.real)) and np.all(np.isfinite(x_gpu.imag)), f"{what}: non-finite"
    err = np.abs(x_gpu.astype(np.complex128) - x_ref)
    rowmax = np.max(np.abs(x_ref), axis=-1, keepdims=True)
    bad = err > REL_TOL * rowmax
    if np.any(bad):
        i = np.unravel_index(np.argmax(err / np.maximum(rowmax, 1e-300)), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} modes out of tolerance; worst at {i}: "
                             f"gpu={x_gpu[i]!r} ref={x_ref[i]!r} rowmax={rowmax[i[0]][0]:.3g}")
    return float(np.max(err / np.maximum(rowmax, 1e-300))) if err.size else 0.0


def _report(pairs) -> Dict[str, float]:
    """Reported beside the row checks (not asserted): the global relative l2
    error of each result and its worst elementwise error relative to
    max(|ref|, 1e-3 * max |ref|) (an absolute floor at 1e-3 of the scale)."""
    out = {}
    for name, g, r in pairs:
        g = np.asarray(g).astype(np.complex128 if np.iscomplexobj(g) else np.float64)
        r = np.asarray(r)
        if r.size == 0:
            continue
        den = np.linalg.norm(r.ravel())
        out[f"l2_{name}"] = float(np.linalg.norm((g - r).ravel()) / den) if den > 0 else 0.0
        floor = 1e-3 * np.max(np.abs(r))
        out[f"elem_{name}"] = float(np.max(np.abs(g - r) / np.maximum(np.abs(r), max(floor, 1e-300))))
    return out


def compare_full(out, ref, io: str) -> Dict[str, float]:
    """Every output and state of a small case."""
    B, T, D = out["y_prefill"].shape
    yp = _np(out["y_prefill"]).transpose(0, 2, 1).reshape(B * D, T)
    yd = _np(out["y_dec"]).transpose(1, 2, 0).reshape(B * D, -1)
    r_yp = ref["y_prefill"].transpose(0, 2, 1).reshape(B * D, T)
    r_yd = ref["y_dec"].transpose(0, 2, 1).reshape(B * D, -1)
    d = out["x_T"].shape[-1]
    rm = seq_rowmax(r_yp, r_yd)
    xT, xe = _np(out["x_T"]).reshape(-1, d), _np(out["x_end"]).reshape(-1, d)
    res = dict(
        y_prefill=check_y(yp, r_yp, io, "prefill y", rowmax=rm),
        y_dec=check_y(yd, r_yd, io, "decode y", rowmax=rm),
        x_T=check_x(xT, ref["x_T"].reshape(-1, d), "x_T"),
        x_end=check_x(xe, ref["x_end"].reshape(-1, d), "x_end"),
    )
    res.update(_report([("y_prefill", yp, r_yp), ("y_dec", yd, r_yd),
                        ("x_T", xT, ref["x_T"].reshape(-1, d)), ("x_end", xe, ref["x_end"].reshape(-1, d))]))
    return res


def gather_rows(out, rows: Sequence[Tuple[int, int]]):
    """Copy only the selected (b, c) rows of the GPU results to the host."""
    import torch

    bs = torch.tensor([b for b, _ in rows], device=out["y_prefill"].device)
    cs = torch.tensor([c for _, c in rows], device=out["y_prefill"].device)
    return dict(
        y_prefill=_np(out["y_prefill"][bs, :, cs]),  # [rows, T]
        y_dec=_np(out["y_dec"][:, bs, cs].T.contiguous()),  # [rows, K]
        x_T=_np(out["x_T"][bs, cs]),
        x_end=_np(out["x_end"][bs, cs]),
    )


def compare_rows(got, ref, io: str) -> Dict[str, float]:
    rm = seq_rowmax(ref["y_prefill"], ref["y_dec"])
    res = dict(
        y_prefill=check_y(got["y_prefill"], ref["y_prefill"], io, "prefill y", rowmax=rm),
        y_dec=check_y(got["y_dec"], ref["y_dec"], io, "decode y", rowmax=rm),
        x_T=check_x(got["x_T"], ref["x_T"], "x_T"),
        x_end=check_x(got["x_end"], ref["x_end"], "x_end"),
    )
    res.update(_report([(k, got[k], ref[k]) for k in ("y_prefill", "y_dec", "x_T", "x_end")]))
    return res


def sample_rows(B: int, D: int, n: int, seed: int = 123, bn: int = 16,
                cw: int = 16) -> List[Tuple[int, int]]:
    """At least ``n`` (b, c) rows: the first and last row of the first,
    second, middle and last block of ``bn`` batch rows crossed with the first
    and last channel of the first, second, middle and last group of ``cw``
    channels (the tile edges of the matrix-core plans), the four corners, then
    random rows."""
    rng = np.random.default_rng(seed)

    def edges(n_items, size):
        nblk = -(-n_items // size)
        out = set()
        for k in {0, 1, nblk // 2, nblk - 1}:
            if 0 <= k < nblk:
                out.add(k * size)
                out.add(min(k * size + size - 1, n_items - 1))
        return sorted(out)

    rows = {(0, 0), (B - 1, D - 1), (0, D - 1), (B - 1, 0)}
    rows |= {(b, c) for b in edges(B, bn) for c in edges(D, cw)}
    while len(rows) < min(n, B * D):
        rows.add((int(rng.integers(B)), int(rng.integers(D))))
    return sorted(rows)
