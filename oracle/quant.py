"""Scalar quantizer and distortion model of KV-COBRA, written plainly (oracle).

Test infrastructure only: nothing in the product path may import this module.

Passages followed
-----------------
* Distortion model q(b) = 2^(-2b)/12: Eq. (eq:q) in Section 3 and its
  normalised restatement Eq. (eq:q-normalized) in Appendix A.1.
* The quantizer: a uniform b-bit scalar quantizer applied per rotated
  coordinate with one step per head (Appendix A.1, Lemma lem:bennett; the
  step uses the equalised variance sigma_bar^2 = (1/r) sum_{i<=r} lambda_i of
  Section 3.4 / Appendix A.1).
* Readings (the paper is silent or inconsistent here):
  - The clip range [-L sigma, L sigma] split into 2^b cells of width
    2 L sigma / 2^b is a mid-rise partition, so the levels are
    (k - 2^(b-1) + 1/2) * step for k in [0, 2^b) and out-of-range inputs
    saturate.
  - The loading factor L is never given ("absorbed into alpha"). The step is
    sigma_bar * delta_b with delta_b the step that minimises the exact mean
    squared error of the 2^b-level mid-rise quantizer on a unit Gaussian,
    rounded to four significant digits (these are the classical optimum
    uniform-quantizer steps tabulated by J. Max, 1960).
  - The code of a coordinate y is k = clamp(floor(y / step) + 2^(b-1), 0,
    2^b - 1), decided exactly (y is the exact rational projection of the
    fp16 input by the fp16 basis).
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
from scipy.optimize import minimize_scalar

B_MIN_SUPPORTED = 1
B_MAX_SUPPORTED = 8


def q_model(b: float) -> float:
    """Leading-order normalised quantizer distortion q(b) = 2^(-2b) / 12 (Eq. eq:q)."""
    return math.ldexp(1.0, -2 * int(b)) / 12.0 if float(b).is_integer() else 2.0 ** (-2.0 * b) / 12.0


def _std_normal_pdf(x: float) -> float:
    return math.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)


def _std_normal_cdf(x: float) -> float:
    return 0.5 * math.erfc(-x / math.sqrt(2.0))


def gaussian_midrise_mse(step: float, b: int) -> float:
    """Exact MSE of the 2^b-level mid-rise quantizer with the given step on N(0, 1).

    Cell k covers [(k - h) step, (k - h + 1) step) with h = 2^(b-1); the two
    outer cells extend to -inf / +inf (saturation). Level of cell k is
    (k - h + 1/2) step. Uses E[(X - y)^2; lo < X < hi] written with the
    Gaussian moments int x^m phi(x) dx over the cell.
    """
    n_levels = 1 << b
    h = n_levels // 2
    total = 0.0
    for k in range(n_levels):
        lo = -math.inf if k == 0 else (k - h) * step
        hi = math.inf if k == n_levels - 1 else (k - h + 1) * step
        y = (k - h + 0.5) * step

        def m0(a):
            return (1.0 if a > 0 else 0.0) if math.isinf(a) else _std_normal_cdf(a)

        def m1(a):  # antiderivative of x phi(x) is -phi(x)
            return 0.0 if math.isinf(a) else -_std_normal_pdf(a)

        def m2(a):  # antiderivative of x^2 phi(x) is Phi(x) - x phi(x)
            return (1.0 if a > 0 else 0.0) if math.isinf(a) else _std_normal_cdf(a) - a * _std_normal_pdf(a)

        total += (m2(hi) - m2(lo)) - 2.0 * y * (m1(hi) - m1(lo)) + y * y * (m0(hi) - m0(lo))
    return total


def optimal_step(b: int) -> float:
    """Step minimising gaussian_midrise_mse for b bits (unit-variance Gaussian)."""
    res = minimize_scalar(lambda s: gaussian_midrise_mse(s, b), bounds=(1e-4, 3.0),
                          method="bounded", options={"xatol": 1e-13})
    return float(res.x)


def step_table() -> dict[int, float]:
    """delta_b for b = 1..8, the optimum rounded to four significant digits."""
    return {b: float("%.4g" % optimal_step(b)) for b in range(B_MIN_SUPPORTED, B_MAX_SUPPORTED + 1)}


_STEP_CACHE: dict[int, float] | None = None


def delta_b(b: int) -> float:
    global _STEP_CACHE
    if _STEP_CACHE is None:
        _STEP_CACHE = step_table()
    return _STEP_CACHE[b]


def head_step(lambda_retained, b: int) -> np.float32:
    """Per-head step: f32(sigma_bar * delta_b), sigma_bar^2 = (1/r) sum of retained variances.

    The sum runs over the retained directions in importance order, left to
    right, in fp64 (Appendix A.1: after the Hadamard rotation every channel has
    variance equal to the mean retained eigenvalue).
    """
    lam = [float(v) for v in lambda_retained]
    r = len(lam)
    s = 0.0
    for v in lam:
        s = s + v
    sigma2 = s / r
    return np.float32(math.sqrt(sigma2) * delta_b(b))


def code_exact(y: Fraction, step: Fraction, b: int) -> int:
    """k = clamp(floor(y / step) + 2^(b-1), 0, 2^b - 1) with exact rationals."""
    h = 1 << (b - 1)
    k = math.floor(y / step) + h
    return max(0, min((1 << b) - 1, k))


def dequant_level(k, step: float, b: int):
    """Reconstruction level (k - 2^(b-1) + 1/2) * step (mid-rise)."""
    return (np.asarray(k, dtype=np.float64) - float(1 << (b - 1)) + 0.5) * float(step)
