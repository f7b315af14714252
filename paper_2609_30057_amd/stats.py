"""Timing statistics of the fidelity measurement.

Section 6.4, Eq. 1: P = p95(r) - 1, r = t_measured / t_native, with the p95
taken by linear interpolation between order statistics (numpy's default).
Section 6.6: single-shot timing and median-of-ten timing.
"""
import numpy as np


def p95_inflation(measured, native):
    """P as a fraction; native is one reference duration or one per sample."""
    r = np.asarray(measured, dtype=np.float64) / np.asarray(native, dtype=np.float64)
    return float(np.percentile(r, 95.0)) - 1.0


def median_ratio(measured, native):
    return float(np.median(np.asarray(measured, dtype=np.float64) / native))


def within(measured, native, frac=0.05):
    r = np.asarray(measured, dtype=np.float64) / native
    return float(np.mean(np.abs(r - 1.0) <= frac))


def medians_of(values, group=10):
    v = np.asarray(values, dtype=np.float64)
    m = (v.size // group) * group
    return np.median(v[:m].reshape(-1, group), axis=1)
