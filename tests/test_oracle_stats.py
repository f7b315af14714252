"""Pins the oracle's timing statistics (Eq. 1 of Section 6.4) on hand-worked
samples, and against numpy's default (linear) percentile."""
import numpy as np

from oracle import stats


def test_p95_hand_worked():
    # 21 ratios 1.00, 1.01, ..., 1.20: p95 position 0.95 * 20 = 19 -> 1.19, P = 0.19
    native = 2.0
    measured = [native * (1 + k / 100) for k in range(21)]
    assert abs(stats.p95_inflation(measured, native) - 0.19) < 1e-12


def test_p95_interpolates():
    # 11 ratios 1.0 .. 1.10 step 0.01 except the largest 2.0: position 9.5
    # between 1.09 and 2.0 -> 1.09 + 0.5 * 0.91 = 1.545
    r = [1 + k / 100 for k in range(10)] + [2.0]
    assert abs(stats.p95_inflation(r, 1.0) - 0.545) < 1e-12


def test_median_and_groups():
    assert stats.median([3.0, 1.0, 2.0]) == 2.0
    assert stats.median([4.0, 1.0, 2.0, 3.0]) == 2.5
    assert stats.median_of_groups(list(range(20)), 10) == [4.5, 14.5]


def test_per_sample_native():
    assert stats.timing_ratios([2.0, 3.0], [1.0, 2.0]) == [2.0, 1.5]


def test_agrees_with_numpy_linear_percentile():
    rng = np.random.default_rng(3)
    for n in (1, 2, 7, 100, 1001):
        x = rng.lognormal(0, 0.1, n)
        for q in (0.5, 0.95, 0.99):
            assert abs(stats.percentile_linear(x, q) - np.percentile(x, 100 * q)) < 1e-12
