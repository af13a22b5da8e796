"""Seeded input generators shared by the tests and the bench."""

import numpy as np

from workload import lengths_skewed


def test_skewed_lengths_keep_the_mean_and_bounds():
    for batch in (4, 16, 64, 256):
        for mean in (1024, 16384):
            flat = lengths_skewed(batch, mean, 0.0, seed=batch)
            assert (flat == mean).all()
            skew = lengths_skewed(batch, mean, 1.0, seed=batch)
            assert abs(skew.mean() - mean) <= 0.01 * mean + 1  # clamp and rounding only
            assert skew.min() >= 16 and skew.max() <= 16 * mean
            assert skew.std() > 0.3 * mean  # sigma = 1 spreads the batch
    a = lengths_skewed(64, 4096, 1.0, seed=3)
    assert (a == lengths_skewed(64, 4096, 1.0, seed=3)).all()
    assert not (a == lengths_skewed(64, 4096, 1.0, seed=4)).all()
