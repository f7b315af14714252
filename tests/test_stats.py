"""The benchmark's timing statistics (Eq. 1 of Section 6.4) against the
oracle's plainly written version, on random samples and hand-worked ones."""
import numpy as np

from oracle import stats as ostats
from paper_2609_30057_amd import stats


def test_p95_inflation_matches_oracle():
    rng = np.random.default_rng(0)
    for n in (1, 2, 10, 1000):
        t = rng.lognormal(0.0, 0.05, n)
        native = float(np.median(rng.lognormal(0.0, 0.05, 99)))
        assert abs(stats.p95_inflation(t, native) - ostats.p95_inflation(list(t), native)) < 1e-12


def test_hand_worked():
    measured = [2.0 * (1 + k / 100) for k in range(21)]
    assert abs(stats.p95_inflation(measured, 2.0) - 0.19) < 1e-12
    assert stats.median_ratio([1.0, 2.0, 3.0], 2.0) == 1.0
    assert stats.within([1.0, 1.04, 1.06, 0.9], 1.0) == 0.5


def test_median_of_ten():
    v = list(range(25))
    assert list(stats.medians_of(v, 10)) == ostats.median_of_groups(v, 10)
