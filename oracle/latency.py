"""Oracle latency model and integer weight normalisation (TEST INFRASTRUCTURE ONLY).

Appendix C: t_MLP = c1 and t_Attn(n) = c2*n + c3, each fitted by least squares
to a profiling sweep over context lengths.

Section 3.4 (integer weight normalisation): the base unit is
Delta = min(t_Attn(n), t_MLP), the integer weights are the rounded ratios
w = round(t / Delta) and the knapsack capacity is K = L*(w_Attn + w_MLP)
(Algorithm 1, initialisation).  The rounding operator has no stated tie rule; it
is read as floor(t/Delta + 1/2) in float64, clamped to at least 1 so that every
sublayer costs something.  A second mode, BINS(c), sets Delta so that the full
model spans c bins, Delta = L*(t_Attn + t_MLP)/c, with the same rounding.

Parity pins: exact recovery of synthetic coefficients by the fit; a worked
example built from the paper's own coefficient table (Appendix C) in
``tests/golden/quantize_appc.txt``.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np


def fit_latency(n_attn, t_attn, t_mlp):
    """Least-squares fit; returns (c1, c2, c3)."""
    n = np.asarray(n_attn, dtype=np.float64)
    A = np.stack([n, np.ones_like(n)], axis=1)
    (c2, c3), *_ = np.linalg.lstsq(A, np.asarray(t_attn, dtype=np.float64), rcond=None)
    c1 = float(np.mean(np.asarray(t_mlp, dtype=np.float64)))
    return c1, float(c2), float(c3)


def latencies(c, n: int):
    """(t_Attn(n), t_MLP) from coefficients c = (c1, c2, c3)."""
    c1, c2, c3 = c
    return c2 * n + c3, c1


def round_half_up(x: float) -> int:
    return int(math.floor(x + 0.5))


@dataclass(frozen=True)
class Weights:
    delta: float
    w_attn: int
    w_mlp: int
    C: int          # capacity L*(w_attn + w_mlp)


def quantize(c, n: int, L: int, mode: str = "paper_min", bins: int = 0) -> Weights:
    t_a, t_m = latencies(c, n)
    if t_a <= 0 or t_m <= 0:
        raise ValueError("latencies must be positive")
    if mode == "paper_min":
        delta = min(t_a, t_m)
    elif mode == "bins":
        if bins < 1:
            raise ValueError("bins must be >= 1")
        delta = L * (t_a + t_m) / bins
    else:
        raise ValueError(mode)
    wa = max(1, round_half_up(t_a / delta))
    wm = max(1, round_half_up(t_m / delta))
    return Weights(delta, wa, wm, L * (wa + wm))
