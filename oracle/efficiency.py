"""Temporal efficiency of two training runs (Section 4, Eq. 4).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Eq. 4 compares optimizers a and b by the areas under their performance
curves f_a(t), f_b(t) (e.g. accuracy against training time), both taken
over [0, m] with m the minimal shared training time: E(a, b) =
int_0^m f_a dt / int_0^m f_b dt.  E > 1 means a performs better.

Readings of what the equation leaves open:
* a curve is given by samples (t_i, f_i) with t_0 = 0 < t_1 < ... and f is
  the straight line between consecutive samples (the trapezoid rule);
* the minimal shared training time is the smaller of the two last sample
  times; the curve that runs longer is cut there, its value at m taken on
  the line between the samples around m.
"""
from __future__ import annotations

import numpy as np

__all__ = ["curve_area", "temporal_efficiency"]


def _check(t, f):
    t = [float(v) for v in t]
    f = [float(v) for v in f]
    if len(t) != len(f) or len(t) < 2:
        raise ValueError("a curve needs at least two (time, value) samples")
    if t[0] != 0.0:
        raise ValueError("a curve starts at time 0")
    for i in range(1, len(t)):
        if not t[i] > t[i - 1]:
            raise ValueError("sample times must increase")
    if not all(np.isfinite(t)) or not all(np.isfinite(f)):
        raise ValueError("samples must be finite")
    return t, f


def curve_area(t, f, upto: float) -> float:
    """Area under the piecewise-linear curve through (t_i, f_i) over
    [0, upto], 0 < upto <= t_last, summed segment by segment."""
    t, f = _check(t, f)
    if not (0.0 < upto <= t[-1]):
        raise ValueError("upto must lie in (0, last sample time]")
    area = 0.0
    for i in range(1, len(t)):
        t0, t1 = t[i - 1], t[i]
        if t0 >= upto:
            break
        f0, f1 = f[i - 1], f[i]
        if t1 > upto:        # cut the segment at upto, value on its line
            f1 = f0 + (f1 - f0) * (upto - t0) / (t1 - t0)
            t1 = upto
        area += 0.5 * (f0 + f1) * (t1 - t0)
    return area


def temporal_efficiency(ta, fa, tb, fb) -> float:
    """E(a, b) of Eq. 4 over the minimal shared training time."""
    ta, fa = _check(ta, fa)
    tb, fb = _check(tb, fb)
    m = min(ta[-1], tb[-1])
    den = curve_area(tb, fb, m)
    if den == 0.0:
        raise ValueError("the area of curve b is zero")
    return curve_area(ta, fa, m) / den
