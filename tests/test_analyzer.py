"""The library's host Analyzer statistics (peat_series_stats, peat_spearman,
peat_normalize_scores) against the oracle on seeded series: Welford's update
and sort-based ranks on the library side, two-pass variance and quadratic
ranking on the oracle side (Section IV-C, Section V-C).  Host code only: no
GPU is touched."""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
import paper_2609_13544_amd as P

RTOL = 1e-12   # different summation orders of at most a few thousand binary64 terms


def _close(a, b, rtol=RTOL):
    if math.isnan(a) or math.isnan(b):
        return math.isnan(a) and math.isnan(b)
    return abs(a - b) <= rtol * max(abs(a), abs(b), 1e-300)


def _series(seed, n, nan_frac=0.0, ties=False):
    rng = np.random.default_rng(seed)
    x = rng.lognormal(-8.0, 2.0, n)
    if ties:
        x = np.round(rng.integers(0, 7, n).astype(np.float64) * 0.25, 2)
    if nan_frac:
        x[rng.random(n) < nan_frac] = np.nan
    return x


@pytest.mark.parametrize("seed,n,nan_frac,ties", [
    (1, 0, 0, False), (2, 1, 0, False), (3, 2, 0, False), (4, 37, 0, False),
    (5, 1000, 0.1, False), (6, 4096, 0, True), (7, 5, 1.0, False), (8, 300, 0.5, True)])
def test_series_stats_matches_oracle(seed, n, nan_frac, ties):
    x = _series(seed, n, nan_frac, ties)
    got, want = P.series_stats(x), oracle.series_stats(x)
    assert got["count"] == want["count"]
    for k in ("min", "max"):
        assert (got[k] == want[k]) or (math.isnan(got[k]) and math.isnan(want[k])), k
    for k in ("mean", "var", "std"):
        assert _close(got[k], want[k]), (k, got[k], want[k])


def test_series_stats_constant_and_infinite():
    got = P.series_stats([3.5] * 10)
    assert got["mean"] == 3.5 and got["var"] == 0.0 and got["std"] == 0.0
    want = oracle.series_stats([1.0, math.inf, 2.0])
    got = P.series_stats([1.0, math.inf, 2.0])
    assert got["count"] == want["count"] == 3 and got["max"] == math.inf
    assert got["mean"] == want["mean"] == math.inf
    assert math.isnan(got["var"]) and math.isnan(want["var"])


@pytest.mark.parametrize("seed,n,nan_frac,ties", [
    (11, 0, 0, False), (12, 1, 0, False), (13, 2, 0, False), (14, 50, 0, False),
    (15, 777, 0.2, False), (16, 2000, 0, True), (17, 100, 0.9, True), (18, 64, 0, True)])
def test_spearman_matches_oracle(seed, n, nan_frac, ties):
    x = _series(seed, n, nan_frac, ties)
    rng = np.random.default_rng(seed + 100)
    y = (x + rng.normal(0, 1e-3, n)) if not ties else rng.integers(0, 4, n).astype(np.float64)
    if n:
        y[rng.random(n) < nan_frac / 2] = np.nan
    assert _close(P.spearman(x, y), oracle.spearman(x, y))


def test_spearman_monotone_and_constant():
    x = np.arange(20.0)
    assert P.spearman(x, np.exp(x / 3)) == pytest.approx(1.0, abs=1e-15)
    assert P.spearman(x, -x ** 3) == pytest.approx(-1.0, abs=1e-15)
    assert math.isnan(P.spearman(x, np.full(20, 2.0)))


def test_normalize_matches_oracle():
    rng = np.random.default_rng(21)
    s = rng.lognormal(0, 3, 500)
    u = rng.lognormal(-5, 1, 500)
    s[:4] = [0.0, math.inf, math.nan, 1.0]
    u[:4] = [0.0, 2.0, 1.0, 0.0]
    got, want = P.normalize_scores(s, u), oracle.normalize(s, u)
    assert np.array_equal(got, want, equal_nan=True)


def test_analyzer_argument_errors():
    with pytest.raises(ValueError):
        P.spearman([1.0, 2.0], [1.0])
    with pytest.raises(ValueError):
        P.normalize_scores([1.0], [1.0, 2.0])
    L = P.lib()
    assert L.peat_series_stats(None, 3, None) == -1
    assert L.peat_spearman(None, None, -1, None) == -1
