"""Pins of the oracle's Analyzer statistics (Section IV-C: an operator's
(mean, std) of scores across epochs and Spearman rank correlation with model
metrics; Section V-C: scores in units of the FP64 error's score) against
numpy (mean, var with ddof=1, nan-aware variants), math.fsum and exact
fractions, scipy.stats.spearmanr (average ranks for ties) and closed
forms."""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import oracle


@pytest.mark.parametrize("seed", range(5))
def test_series_stats_against_numpy(seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(int(rng.integers(2, 2000))) * 10.0 ** rng.integers(-8, 8)
    x[rng.random(x.size) < 0.1] = np.nan
    got = oracle.series_stats(x)
    v = x[~np.isnan(x)]
    assert got["count"] == v.size
    assert got["min"] == v.min() and got["max"] == v.max()
    assert abs(got["mean"] - math.fsum(v) / v.size) <= 1e-15 * abs(np.mean(np.abs(v)))
    var = float(np.var(v, ddof=1))
    assert abs(got["var"] - var) <= 1e-12 * var
    assert abs(got["std"] - math.sqrt(var)) <= 1e-12 * math.sqrt(var)


def test_series_stats_exact_small():
    x = [0.1, 0.2, 0.7, 1e-300]
    got = oracle.series_stats(x)
    f = [Fraction(v) for v in x]
    mean = sum(f) / 4
    var = sum((v - mean) ** 2 for v in f) / 3
    assert got["mean"] == float(mean)
    assert abs(got["var"] - float(var)) <= 1e-15 * float(var)


def test_series_stats_degenerate():
    assert oracle.series_stats([])["count"] == 0 and math.isnan(oracle.series_stats([])["mean"])
    one = oracle.series_stats([3.0, np.nan])
    assert one["count"] == 1 and one["mean"] == 3.0 and math.isnan(one["var"]) and one["min"] == one["max"] == 3.0
    const = oracle.series_stats([2.5] * 10)
    assert const["var"] == 0.0 and const["std"] == 0.0


@pytest.mark.parametrize("seed", range(6))
def test_spearman_against_scipy(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(3, 400))
    x = rng.standard_normal(n)
    y = x * rng.random() + rng.standard_normal(n)
    # ties in both series
    x[: n // 5] = np.round(x[: n // 5], 1)
    y[n // 3: n // 2] = 0.5
    want = stats.spearmanr(x, y).statistic
    assert abs(oracle.spearman(x, y) - want) <= 1e-12


def test_spearman_nan_pairs_excluded_and_closed_forms():
    x = np.array([1.0, 2.0, np.nan, 4.0, 5.0, 6.0])
    y = np.array([10.0, 20.0, 30.0, np.nan, 50.0, 60.0])
    assert oracle.spearman(x, y) == pytest.approx(1.0, abs=1e-15)
    assert oracle.spearman([1, 2, 3, 4], [4, 3, 2, 1]) == pytest.approx(-1.0, abs=1e-15)
    # no ties: rho = 1 - 6 sum d^2 / (n (n^2 - 1))
    x = [1, 2, 3, 4, 5]
    y = [2, 1, 4, 3, 5]
    d2 = sum((a - b) ** 2 for a, b in zip(x, y))
    assert oracle.spearman(x, y) == pytest.approx(1 - 6 * d2 / (5 * 24), abs=1e-15)
    assert math.isnan(oracle.spearman([1.0], [2.0]))
    assert math.isnan(oracle.spearman([1.0, 1.0, 1.0], [1.0, 2.0, 3.0]))


def test_normalize():
    s = np.array([1.0, 3.0, 0.0, 5.0, np.inf])
    u = np.array([4.0, 0.0, 0.0, -2.0, 2.0])
    got = oracle.normalize(s, u)
    assert got[0] == 0.25 and got[1] == np.inf and math.isnan(got[2]) and got[3] == -2.5 and got[4] == np.inf


def test_series_stats_infinite_entries_follow_ieee_sum():
    # the mean is the IEEE sum over the count: one +inf makes it +inf, +inf
    # and -inf together make it NaN; the deviations are then undefined (NaN)
    r = oracle.series_stats([1.0, math.inf, 2.0])
    assert r["count"] == 3 and r["mean"] == math.inf and r["max"] == math.inf
    assert math.isnan(r["var"]) and math.isnan(r["std"])
    r = oracle.series_stats([-math.inf, 4.0])
    assert r["mean"] == -math.inf and r["min"] == -math.inf
    r = oracle.series_stats([math.inf, -math.inf, 0.0])
    assert math.isnan(r["mean"])
