"""Data-free UOS objective (test infrastructure only, like the rest of oracle/).

Sec. 4.1 (Universal Optimal Scaling) defines, for the non-negative E2M1 grid
G+ = {0, .5, 1, 1.5, 2, 3, 4, 6} with round-to-nearest projection Pi and
saturation at 6:

* E(x) = integral over [0, x] of (v - Pi(v))^2 dv  (Eq. uos_local_distortion),
* D(x) = E(x) / x^3, the mean squared projection error on [0, x] over x^2,
* J(q) = integral over (q/2, q] of D(x) g(x) dx (Eq. uos_global_objective),
  where g(x) = H(log2 x) / (x ln 2) is the density of the normalized block
  maximum X_q = M / 2^ceil(log2(M/q)) and H is the period-1 wrapped density of
  log2 M (Eq. uos_wrapped_density; H = 1 is a log-uniform M),
* Delta(q) = E(q) - 8 E(q/2), whose sign is the sign of J'(q) (Eq.
  uos_delta_relation).

E is evaluated exactly (Fraction arithmetic for rational x) by summing the
interval integral of App. "Integrated Quantization Error of the E2M1 Grid"
over the round-to-nearest decision intervals; J by adaptive quadrature with
the decision boundaries as break points.
"""
from __future__ import annotations

import math
from fractions import Fraction
from typing import Callable, Optional

GRID = tuple(Fraction(g) for g in ("0", "1/2", "1", "3/2", "2", "3", "4", "6"))
# Decision boundaries of round-to-nearest between consecutive grid values;
# everything above the last one (5) projects to 6 (saturation).
THRESHOLDS = tuple((a + b) / 2 for a, b in zip(GRID[:-1], GRID[1:]))


def project(v):
    """Pi(v) for v >= 0: nearest grid value (ties are measure-zero here and
    resolved downward), saturating at 6."""
    for t, g in zip(THRESHOLDS, GRID):
        if v <= t:
            return g
    return GRID[-1]


def cumulative_error(x):
    """E(x), exact for Fraction / int arguments, float otherwise."""
    if x < 0:
        raise ValueError("E is defined for x >= 0")
    total = Fraction(0) if isinstance(x, (Fraction, int)) else 0.0
    lo = 0
    edges = list(THRESHOLDS) + [None]
    for r, hi in zip(GRID, edges):
        b = x if hi is None or x < hi else hi
        if b > lo:
            total += ((b - r) ** 3 - (lo - r) ** 3) / 3
        if hi is None or x <= hi:
            break
        lo = hi
    return total


def normalized_error(x):
    """D(x) = E(x) / x^3."""
    return cumulative_error(x) / x ** 3


def delta(q):
    """Delta(q) = E(q) - 8 E(q/2)."""
    return cumulative_error(q) - 8 * cumulative_error(q / 2)


def density(x: float, wrapped: Optional[Callable[[float], float]] = None) -> float:
    """g(x) = H(log2 x) / (x ln 2); H defaults to 1 (log-uniform M)."""
    h = 1.0 if wrapped is None else wrapped(math.log2(x))
    return h / (x * math.log(2.0))


def objective(q: float, wrapped: Optional[Callable[[float], float]] = None) -> float:
    """J(q) = integral over (q/2, q] of D(x) g(x) dx, for q > 0."""
    from scipy.integrate import quad

    a, b = q / 2.0, q
    pts = [float(t) for t in THRESHOLDS if a < t < b]
    f = lambda x: float(normalized_error(x)) * density(x, wrapped)
    val, _ = quad(f, a, b, points=pts or None, epsabs=0.0, epsrel=1e-12, limit=200)
    return val
