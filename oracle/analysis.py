"""Closed forms from the paper's analysis (test infrastructure).

- ``e4m3_positive_values``: the 126 positive finite E4M3 values, built from the
  format equations of Sec. 2.1 (subnormals M/8 * 2^-6, normals
  2^(E-7) (1 + M/8), E=15/M=7 reserved).
- ``dp``: the normalised worst-case quantisation step of Definition 1 in
  Sec. 5.2, with the overflow extension of the remark that follows it for
  S > 448.  Reading: the LSB maximum is taken over [0, S) -- the largest gap
  between consecutive representable values that starts below S -- which is what
  the proof of part (i) of the dp-structure theorem uses (top binade
  [2^(k-1), 2^k)) and what reproduces every value of Appendix A.
- ``delta_k``: E[max of k standard normals] (Sec. 3.2).
- ``collapse_fraction``: Corollary (P-collapse fraction),
  F(Delta, S) = Phi(Delta + delta_k - 10 ln 2 - ln S).
- ``critical_delta``: Delta_c = 10 ln 2 + ln S - delta_k (Sec. 7.2).
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import ndtr

LN2 = math.log(2.0)


def e4m3_positive_values() -> np.ndarray:
    """Sorted positive finite E4M3 values (126 of them), from the format equations."""
    vals = [(m / 8.0) * 2.0 ** -6 for m in range(1, 8)]                  # subnormals
    for E in range(1, 16):
        for M in range(8):
            if E == 15 and M == 7:                                          # NaN code
                continue
            vals.append(2.0 ** (E - 7) * (1.0 + M / 8.0))
    return np.array(sorted(vals), dtype=np.float64)


def dp(S: float) -> float:
    """Normalised worst-case quantisation step dp(S) (Sec. 5.2, Definition 1)."""
    if not S > 0:
        raise ValueError("S must be positive")
    grid = np.concatenate([[0.0], e4m3_positive_values()])
    vmax = grid[-1]
    if S > vmax:
        # overflow extension: largest in-range step 32 (binade [256, 512)) and
        # the one-sided saturation error 1 - 448/S converted to a step
        return max(32.0 / S, 2.0 * (1.0 - vmax / S))
    gaps = np.diff(grid)
    starts = grid[:-1]
    return float(gaps[starts < S].max() / S)


def normal_coverage(S: float) -> float:
    """P-domain threshold below which P*S leaves the E4M3 normal range (2^-6 / S)."""
    return 2.0 ** -6 / S


def phi_cdf(x: float) -> float:
    """Standard normal CDF."""
    return 0.5 * math.erfc(-x / math.sqrt(2.0))


def delta_k(k: int, n: int = 400001, lim: float = 12.0) -> float:
    """E[max of k iid N(0,1)] = integral x k phi(x) Phi(x)^(k-1) dx (trapezoid rule)."""
    if k < 1:
        raise ValueError("k >= 1")
    x = np.linspace(-lim, lim, n)
    pdf = np.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)
    cdf = ndtr(x)
    f = x * k * pdf * cdf ** (k - 1)
    return float(np.sum((f[1:] + f[:-1]) * 0.5 * np.diff(x)))


_DELTA_CACHE: dict[int, float] = {}


def delta(k: int) -> float:
    if k not in _DELTA_CACHE:
        _DELTA_CACHE[k] = delta_k(k)
    return _DELTA_CACHE[k]


def underflow_logit_threshold(S: float) -> float:
    """Prop. 1: p*S < 2^-10  <=>  s - m < -(10 ln 2 + ln S)."""
    return -(10.0 * LN2 + math.log(S))


def collapse_fraction(Delta: float, S: float, k_sink: int = 4) -> float:
    """Corollary (P-collapse fraction): Phi(Delta + delta_k - 10 ln 2 - ln S)."""
    return phi_cdf(Delta + delta(k_sink) - 10.0 * LN2 - math.log(S))


def critical_delta(S: float, k_sink: int = 4) -> float:
    """Delta_c = 10 ln 2 + ln S - delta_k (Sec. 7.2, structural interpretation)."""
    return 10.0 * LN2 + math.log(S) - delta(k_sink)


def reverse_survival_margin(S: float) -> float:
    """Theorem 2: a P value survives when s > m - (10 ln 2 + ln S); 18 ln 2 at S=256."""
    return 10.0 * LN2 + math.log(S)
