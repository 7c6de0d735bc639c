"""Host logic of the fragility protection (paper Section 3, "Activation-
fragility profiling and protection"), CPU only: the library's host calls
w8a8_fragility_scores, w8a8_select_protected and w8a8_rank_correlation
(through the marshaller in fragility.py and directly through the C ABI)
against the oracle's independent score, top-N and Spearman, and scipy."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest
import scipy.stats

import oracle
import paper_2606_12280_amd as pkg
from paper_2606_12280_amd import fragility

OK, NULL, SHAPE, UNSUP = 0, 1, 2, 5


def _dp(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def test_scores_are_mean_kurtosis_over_steps():
    rng = np.random.default_rng(130)
    k = rng.lognormal(1.0, 1.0, (211, 48))
    assert np.allclose(fragility.fragility_scores(k), oracle.fragility_scores(k), rtol=1e-15)
    # a contiguous range of steps: the early and late halves
    assert np.allclose(fragility.fragility_scores(k, 0, 24), oracle.fragility_scores(k[:, :24]),
                       rtol=1e-15)
    assert np.allclose(fragility.fragility_scores(k, 24, 48), oracle.fragility_scores(k[:, 24:]),
                       rtol=1e-15)


def test_scores_exact_on_small_integers():
    """Sums of small integers are exact, so the mean is one correctly
    rounded division: equal to the oracle's bit for bit."""
    rng = np.random.default_rng(134)
    k = rng.integers(0, 1000, (37, 11)).astype(np.float64)
    assert np.array_equal(fragility.fragility_scores(k), oracle.fragility_scores(k))
    assert list(fragility.fragility_scores([[3, 5], [10, 12], [3, 5], [12, 10]])) == [4, 11, 4, 11]


@pytest.mark.parametrize("seed", range(10))
def test_selection_matches_oracle_with_ties(seed):
    rng = np.random.default_rng([131, seed])
    scores = rng.integers(0, 12, 211).astype(float)      # many equal scores
    for n in (0, 1, 8, 17, 211, 300):
        assert fragility.select_protected(scores, n) == oracle.top_n(scores, n)


def test_selection_of_random_scores_matches_oracle():
    rng = np.random.default_rng(135)
    for _ in range(20):
        s = rng.lognormal(1.0, 1.5, 211)
        assert fragility.select_protected(s, 17) == oracle.top_n(s, 17)


def test_selection_picks_the_outlier_layers():
    """Down-projection-like layers with heavy-tailed inputs are the top 17."""
    rng = np.random.default_rng(132)
    scores = rng.uniform(2.5, 4.0, 211)
    heavy = rng.choice(211, 17, replace=False)
    scores[heavy] = rng.uniform(20, 400, 17)
    assert sorted(fragility.select_protected(scores, 17)) == sorted(heavy.tolist())


def test_profile_table_to_protection_end_to_end():
    """kurtosis table -> scores -> the protected set, against the oracle's
    composition of the same two steps."""
    rng = np.random.default_rng(136)
    k = rng.lognormal(1.2, 0.4, (211, 48))
    k[rng.choice(211, 17, replace=False)] *= 30.0
    got = fragility.select_protected(fragility.fragility_scores(k), 17)
    assert got == oracle.top_n(oracle.fragility_scores(k), 17)


@pytest.mark.parametrize("seed", range(10))
def test_rank_stability_matches_oracle(seed):
    rng = np.random.default_rng([133, seed])
    a = rng.integers(0, 9, 60).astype(float)
    b = a + rng.normal(0, 2, 60)
    assert fragility.rank_stability(a, b) == pytest.approx(oracle.spearman(a, b), abs=1e-12)
    assert fragility.rank_stability(a, b) == pytest.approx(scipy.stats.spearmanr(a, b)[0],
                                                           abs=1e-12)
    assert fragility.rank_stability(a, a) == pytest.approx(1.0)
    assert fragility.rank_stability(a, -a) == pytest.approx(-1.0)


def test_host_calls_validate_arguments():
    lib = pkg.load()
    k = np.ones((4, 6))
    s = np.empty(4)
    idx = np.empty(4, np.int32)
    rho = ctypes.c_double()
    f = lib.w8a8_fragility_scores
    assert f(None, 4, 6, 0, 6, _dp(s)) == NULL
    assert f(_dp(k), 4, 6, 0, 6, None) == NULL
    assert f(_dp(k), 0, 6, 0, 6, _dp(s)) == SHAPE
    assert f(_dp(k), 4, 6, 3, 3, _dp(s)) == SHAPE            # no steps
    assert f(_dp(k), 4, 6, 0, 7, _dp(s)) == SHAPE            # past the table
    assert f(_dp(k), 4, 6, -1, 6, _dp(s)) == SHAPE
    bad = k.copy()
    bad[2, 3] = np.nan
    assert f(_dp(bad), 4, 6, 0, 6, _dp(s)) == UNSUP
    assert f(_dp(k), 4, 6, 0, 6, _dp(s)) == OK
    g = lib.w8a8_select_protected
    assert g(None, 4, 2, _dp(idx)) == NULL
    assert g(_dp(s), 4, 2, None) == NULL
    assert g(_dp(s), 4, 0, None) == OK                        # nothing to write
    assert g(_dp(s), 4, 5, _dp(idx)) == SHAPE
    assert g(_dp(s), 4, -1, _dp(idx)) == SHAPE
    inf = np.array([1.0, np.inf, 0.0, 2.0])
    assert g(_dp(inf), 4, 2, _dp(idx)) == UNSUP
    r = lib.w8a8_rank_correlation
    a, b = np.arange(5.0), np.arange(5.0)[::-1].copy()
    assert r(_dp(a), _dp(b), 5, None) == NULL
    assert r(_dp(a), _dp(b), 1, ctypes.byref(rho)) == SHAPE
    assert r(_dp(np.ones(5)), _dp(b), 5, ctypes.byref(rho)) == UNSUP   # constant: no ranking
    assert r(_dp(a), _dp(b), 5, ctypes.byref(rho)) == OK and rho.value == -1.0
