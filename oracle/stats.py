"""Timing statistics of the paper's fidelity metric -- TEST INFRASTRUCTURE.

Eq. 1 (Section 6.4): P = p95(r) - 1 with r = t_measured / t_native, reported
as a percentage. The paper does not name a percentile method; the reading
here is linear interpolation between order statistics (position
q (n - 1) in the sorted sample), written out plainly. Section 2.1 names the
median as the summary of a timed loop; Section 6.6 compares single-shot and
median-of-ten timing.
"""
import math


def percentile_linear(values, q):
    xs = sorted(float(v) for v in values)
    if not xs:
        raise ValueError("empty sample")
    h = q * (len(xs) - 1)
    lo = math.floor(h)
    hi = min(lo + 1, len(xs) - 1)
    return xs[lo] + (h - lo) * (xs[hi] - xs[lo])


def median(values):
    return percentile_linear(values, 0.5)


def timing_ratios(measured, native):
    """r_k = t_measured,k / t_native; native is one reference duration or one per sample."""
    if isinstance(native, (int, float)):
        return [float(m) / float(native) for m in measured]
    return [float(m) / float(n) for m, n in zip(measured, native)]


def p95_inflation(measured, native):
    """P = p95(r) - 1, as a fraction (multiply by 100 for the paper's percent)."""
    return percentile_linear(timing_ratios(measured, native), 0.95) - 1.0


def median_of_groups(values, group):
    """Median of each consecutive group of `group` timings (median-of-ten, Section 6.6)."""
    return [median(values[i:i + group]) for i in range(0, len(values) - group + 1, group)]
