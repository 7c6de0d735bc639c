"""Host logic of the fragility protection (paper Section 3, "Activation-
fragility profiling and protection"), CPU only: the product's score, top-N
selection and rank-stability check against the oracle's independent ones."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2606_12280_amd import fragility


def test_scores_are_mean_kurtosis_over_steps():
    rng = np.random.default_rng(130)
    k = rng.lognormal(1.0, 1.0, (211, 48))
    assert np.allclose(fragility.fragility_scores(k), oracle.fragility_scores(k), rtol=1e-15)


@pytest.mark.parametrize("seed", range(10))
def test_selection_matches_oracle_with_ties(seed):
    rng = np.random.default_rng([131, seed])
    scores = rng.integers(0, 12, 211).astype(float)      # many equal scores
    for n in (0, 1, 8, 17, 211, 300):
        assert fragility.select_protected(scores, n) == oracle.top_n(scores, n)


def test_selection_picks_the_outlier_layers():
    """Down-projection-like layers with heavy-tailed inputs are the top 17."""
    rng = np.random.default_rng(132)
    scores = rng.uniform(2.5, 4.0, 211)
    heavy = rng.choice(211, 17, replace=False)
    scores[heavy] = rng.uniform(20, 400, 17)
    assert sorted(fragility.select_protected(scores, 17)) == sorted(heavy.tolist())


@pytest.mark.parametrize("seed", range(10))
def test_rank_stability_matches_oracle(seed):
    rng = np.random.default_rng([133, seed])
    a = rng.integers(0, 9, 60).astype(float)
    b = a + rng.normal(0, 2, 60)
    assert fragility.rank_stability(a, b) == pytest.approx(oracle.spearman(a, b), abs=1e-12)
    assert fragility.rank_stability(a, a) == pytest.approx(1.0)
