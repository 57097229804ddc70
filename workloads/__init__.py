"""Seeded synthetic inputs for the distilled modal recurrence.

This module is shared by the CPU oracle and the HIP path.  It draws random
numbers and lays them out; it performs none of the method's arithmetic (no
powers of the poles, no filter, no convolution, no recurrence).

Shapes follow the deployment setting of the modal recurrence (Sec. 3.4 of the
paper, Proposition "modal realization"): per channel ``c`` a filter with ``d``
complex poles ``lambda[c, n]`` and residues ``R[c, n]`` plus a pass-through
``h0[c]``; an input ``u[b, t, c]`` with the channel index fastest, as in the
language-model activations the filters act on.  The pre-trained filters and the
text corpus the paper distils from are not available, so the parameters are
drawn from the distributions below, which stand in for them:

* ``r ~ U[r_lo, r_hi]``, ``theta ~ U[0, theta_hi]``, ``lambda = r e^{i theta}``
  (polar parametrisation of the poles, App. B.1), formed in float64 and rounded
  once to complex64;
* ``R`` circular complex normal with ``E|R|^2 = r_var`` (real and imaginary parts
  each ``N(0, r_var / 2)``), rounded to complex64;
* ``h0 ~ N(0, 1)`` as float32;
* ``u ~ N(0, 1)`` drawn as float32; for bfloat16 input/output the draw is
  rounded to the nearest bfloat16 (ties to even) and the rounded values are
  what both sides consume.

Random streams: ``numpy.random.default_rng(seed)`` draws, in this order,
``r[D,d]``, ``theta[D,d]``, ``Re R[D,d]``, ``Im R[D,d]``, ``h0[D]``.  The prompt
row of batch element ``b`` comes from ``default_rng([seed, 1, b])`` as a
``[T, D]`` float32 draw and its decode inputs from ``default_rng([seed, 2, b])``
as ``[K, D]``, so any row can be regenerated alone.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Iterator, Tuple

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "workload",
    "make_params",
    "prompt_row",
    "decode_row",
    "make_inputs",
    "bf16_round",
    "bf16_bits",
    "MHWorkload",
    "MH_WORKLOADS",
    "mh_workload",
    "mh_params",
    "mh_row",
    "distill_params",
    "distill_target",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: a bank of ``D`` distilled filters of order ``d``
    applied to ``B`` sequences of ``T`` prompt tokens followed by ``K`` decode
    tokens."""

    name: str
    B: int
    D: int
    d: int
    T: int
    K: int
    io: str  # "f32" or "bf16": dtype of u and y only; the state is complex64
    r_lo: float
    r_hi: float
    theta_hi: float
    r_var: float  # E|R_n|^2
    seed: int = 0

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads.  D = 768 / 2048 are the widths of the 125M / 1.3B
# language models, d = 16 the standard distillation order, d = 32 / 64 the
# larger orders of the state-dimension study, and T = 65536 the long-sequence
# setting of the paper's associative-recall runs.
WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in (
        Workload("tiny_b1_d4_t64", 1, 4, 4, 64, 16, "f32", 0.5, 0.95, math.pi, 1.0),
        Workload("b16_d768_n16_t2048", 16, 768, 16, 2048, 256, "f32", 0.8, 0.999, math.pi, 1.0 / 16),
        Workload("b64_d2048_n16_t4096_bf16", 64, 2048, 16, 4096, 512, "bf16", 0.9, 0.9999, math.pi, 1.0 / 16),
        Workload("b256_d2048_n64_t1024", 256, 2048, 64, 1024, 1024, "f32", 0.9, 0.9999, math.pi, 1.0 / 64),
        Workload("b4_d1024_n32_t65536", 4, 1024, 32, 65536, 128, "f32", 0.999, 0.99999, 0.01 * math.pi, 1.0 / 32),
        # the companion form's workload: an order (2d = 16) and pole radii at which
        # its float64 recurrence keeps the modal path's accuracy
        Workload("cp_b256_d2048_n8_t1024", 256, 2048, 8, 1024, 64, "f32", 0.8, 0.99, math.pi, 1.0 / 8),
    )
}

# Short aliases used on the command line and in tests.
ALIASES = {
    "tiny": "tiny_b1_d4_t64",
    "c1": "tiny_b1_d4_t64",
    "c2": "b16_d768_n16_t2048",
    "c3": "b64_d2048_n16_t4096_bf16",
    "c4": "b256_d2048_n64_t1024",
    "c5": "b4_d1024_n32_t65536",
    "cp": "cp_b256_d2048_n8_t1024",
}


def workload(name: str) -> Workload:
    return WORKLOADS[ALIASES.get(name, name)]


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns
    float32 values that are exactly representable in bfloat16.  NaN stays NaN.
    (For finite inputs and infinities the uint32 sum below cannot wrap.)"""
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32)
    lsb = (bits >> np.uint32(16)) & np.uint32(1)
    rounded = (bits + (np.uint32(0x7FFF) + lsb)) & np.uint32(0xFFFF0000)
    out = rounded.view(np.float32)
    return np.where(np.isnan(x), x, out)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """The upper 16 bits of float32 values that are already bfloat16-exact, as
    uint16 (the bfloat16 encoding)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def make_params(w: Workload) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Return ``(lam, R, h0)``: complex64 ``[D, d]``, complex64 ``[D, d]``,
    float32 ``[D]``."""
    rng = np.random.default_rng(w.seed)
    r = rng.uniform(w.r_lo, w.r_hi, size=(w.D, w.d))
    theta = rng.uniform(0.0, w.theta_hi, size=(w.D, w.d))
    s = math.sqrt(w.r_var / 2.0)
    re_r = rng.standard_normal((w.D, w.d)) * s
    im_r = rng.standard_normal((w.D, w.d)) * s
    h0 = rng.standard_normal(w.D).astype(np.float32)
    lam = (r * np.exp(1j * theta)).astype(np.complex64)
    R = (re_r + 1j * im_r).astype(np.complex64)
    return lam, R, h0


def _round_io(w: Workload, a: np.ndarray) -> np.ndarray:
    return bf16_round(a) if w.io == "bf16" else a


def prompt_row(w: Workload, b: int) -> np.ndarray:
    """Prompt inputs of batch element ``b``: float32 ``[T, D]``."""
    rng = np.random.default_rng([w.seed, 1, b])
    return _round_io(w, rng.standard_normal((w.T, w.D), dtype=np.float32))


def decode_row(w: Workload, b: int) -> np.ndarray:
    """Decode inputs of batch element ``b``: float32 ``[K, D]`` (open loop:
    drawn in advance, no model feeds outputs back)."""
    rng = np.random.default_rng([w.seed, 2, b])
    return _round_io(w, rng.standard_normal((w.K, w.D), dtype=np.float32))


def rows(w: Workload) -> Iterator[Tuple[int, np.ndarray, np.ndarray]]:
    for b in range(w.B):
        yield b, prompt_row(w, b), decode_row(w, b)


def make_inputs(w: Workload):
    """All inputs at once: ``lam, R, h0, u_prompt [B,T,D], u_dec [B,K,D]``
    (float32; bfloat16-exact when ``w.io == "bf16"``)."""
    lam, R, h0 = make_params(w)
    up = np.empty((w.B, w.T, w.D), np.float32)
    ud = np.empty((w.B, w.K, w.D), np.float32)
    for b in range(w.B):
        up[b] = prompt_row(w, b)
        ud[b] = decode_row(w, b)
    return lam, R, h0, up, ud


# ----------------------------------------------------------------------------
# multi-head (head-tied) decode: M heads of N channels (D = M N), one distilled
# filter per head, an N x N grid of entries per head (Sec. 5 of the paper)
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class MHWorkload:
    """``B`` sequences through one multi-head layer of width ``D = M N``: ``T0``
    prompt steps (whose state starts the decode; 0 = an empty prompt) and
    ``K`` decode steps."""

    name: str
    B: int
    M: int
    N: int
    d: int
    T0: int
    K: int
    io: str
    r_lo: float
    r_hi: float
    theta_hi: float
    r_var: float
    seed: int = 0

    @property
    def D(self) -> int:
        return self.M * self.N

    def with_(self, **kw) -> "MHWorkload":
        return dataclasses.replace(self, **kw)


# Eight heads as in the paper's multi-head models, at the 355M width
# (D = 1024, N = 128), d = 16: a 256 MiB state for 16 sequences.
MH_WORKLOADS: Dict[str, MHWorkload] = {
    w.name: w
    for w in (
        MHWorkload("mh_b16_d1024_m8_n16", 16, 8, 128, 16, 0, 64, "f32", 0.9, 0.9999, math.pi, 1.0 / 16),
    )
}


def mh_workload(name: str) -> MHWorkload:
    return MH_WORKLOADS[{"mh": "mh_b16_d1024_m8_n16"}.get(name, name)]


def mh_params(w: MHWorkload) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Per-head filters ``(lam [M,d], R [M,d], h0 [M])``, drawn as in
    ``make_params`` with one filter per head."""
    rng = np.random.default_rng(w.seed)
    r = rng.uniform(w.r_lo, w.r_hi, size=(w.M, w.d))
    theta = rng.uniform(0.0, w.theta_hi, size=(w.M, w.d))
    s = math.sqrt(w.r_var / 2.0)
    re_r = rng.standard_normal((w.M, w.d)) * s
    im_r = rng.standard_normal((w.M, w.d)) * s
    h0 = rng.standard_normal(w.M).astype(np.float32)
    return (r * np.exp(1j * theta)).astype(np.complex64), (re_r + 1j * im_r).astype(np.complex64), h0


def mh_row(w: MHWorkload, b: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """``q, k, v`` of batch element ``b`` for all ``T0 + K`` steps: float32
    ``[T0 + K, M, N]`` each, drawn from ``default_rng([seed, 3, b])`` in the
    order q, k, v (bfloat16-exact when ``w.io == "bf16"``)."""
    rng = np.random.default_rng([w.seed, 3, b])
    L = w.T0 + w.K
    out = []
    for _ in range(3):
        a = rng.standard_normal((L, w.M * w.N), dtype=np.float32)
        out.append((bf16_round(a) if w.io == "bf16" else a).reshape(L, w.M, w.N))
    return out[0], out[1], out[2]


# ----------------------------------------------------------------------------
# distillation objective: modal parameters in polar form and target filters
# ----------------------------------------------------------------------------

def distill_params(w: Workload) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Starting point of a distillation: ``(A [D,d], theta [D,d], R [D,d])``,
    the same draws as ``make_params`` (``A = r``, the pole's modulus, and
    ``theta``) as float32 and complex64."""
    rng = np.random.default_rng(w.seed)
    r = rng.uniform(w.r_lo, w.r_hi, size=(w.D, w.d))
    theta = rng.uniform(0.0, w.theta_hi, size=(w.D, w.d))
    s = math.sqrt(w.r_var / 2.0)
    re_r = rng.standard_normal((w.D, w.d)) * s
    im_r = rng.standard_normal((w.D, w.d)) * s
    return r.astype(np.float32), theta.astype(np.float32), (re_r + 1j * im_r).astype(np.complex64)


def distill_target(w: Workload, L: int, tau: float = 512.0) -> np.ndarray:
    """Synthetic real target filters ``[D, L]`` (``h_1 .. h_L``) standing in for
    pre-trained long-convolution filters: unit normal draws under an
    exponentially decaying envelope ``exp(-t / tau)``, from
    ``default_rng([seed, 4])``."""
    rng = np.random.default_rng([w.seed, 4])
    g = rng.standard_normal((w.D, L), dtype=np.float32)
    env = np.exp(-np.arange(1, L + 1, dtype=np.float64) / tau).astype(np.float32)
    return (g * env[None, :]).astype(np.float32)
