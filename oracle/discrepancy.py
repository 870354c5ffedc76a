"""Discrepancy measures of threshold sequences (test infrastructure).

Definitions from Appendix A (star discrepancy D*_T) and Appendix B ("Dithers":
local discrepancy LD_W; "Offset near-aliasing": neighbour separation d).
"""
from __future__ import annotations

import numpy as np


def star_discrepancy(u) -> float:
    """D*_T = sup_x |#{t: u_t < x}/T - x| for points in [0, 1).

    For sorted points v_1 <= ... <= v_T the supremum is attained next to a point:
    max_i max(i/T - v_i, v_i - (i-1)/T).
    """
    v = np.sort(np.asarray(u, np.float64))
    T = v.size
    i = np.arange(1, T + 1, dtype=np.float64)
    return float(max(np.max(i / T - v), np.max(v - (i - 1) / T)))


def count_below(u, x) -> int:
    """A_T(x) = #{t: u_t < x} (Appendix A)."""
    return int(np.count_nonzero(np.asarray(u, np.float64) < x))


def weyl_float(alpha: float, offset: float, t0: int, T: int) -> np.ndarray:
    """u_t = {offset + t alpha} for t = t0+1 .. t0+T, phase reduced mod 1 in float64."""
    t = np.arange(t0 + 1, t0 + T + 1, dtype=np.float64)
    phase = np.mod(t * alpha, 1.0)
    return np.mod(offset + phase, 1.0)


def local_discrepancy(sequences) -> float:
    """Mean star discrepancy over a list of windows (LD_W with W = window length)."""
    return float(np.mean([star_discrepancy(s) for s in sequences]))


def dist_to_int(v):
    """||v||: distance to the nearest integer."""
    v = np.asarray(v, np.float64)
    return np.abs(v - np.round(v))


def separation(beta: float, gamma: float, alpha: float, span: int = 2, lags: int = 16) -> float:
    """d = min ||dr beta + dc gamma - l alpha|| over |dr|,|dc| <= span (not both 0), |l| <= lags."""
    best = 1.0
    for dr in range(-span, span + 1):
        for dc in range(-span, span + 1):
            if dr == 0 and dc == 0:
                continue
            for ell in range(-lags, lags + 1):
                best = min(best, float(dist_to_int(dr * beta + dc * gamma - ell * alpha)))
    return best
