"""Pins of the oracle's top-k error mean (the paper's main score, "mean of the
top 10% errors", Section IV-B.3 / IV-C) against what the definition fixes
independently of the oracle's code: the k largest of the multiset of errors
(heapq / torch.topk on exact, correctly rounded errors), math.fsum sums,
integer ceilings, closed forms for arithmetic progressions and ties, and the
special cases (NaN pairs excluded, infinite errors, no valid pair)."""
from __future__ import annotations

import heapq
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

F32, F16, BF16 = oracle.F32, oracle.F16, oracle.BF16


def exact_errors(g: np.ndarray, t: np.ndarray) -> list[float]:
    """Errors of the valid pairs: |T - G| from exact rationals, rounded once
    to the nearest binary64 (Python's Fraction -> float is correctly rounded);
    equal values give 0; infinities by IEEE rules."""
    out = []
    for G, T in zip(g.astype(np.float64).tolist(), t.astype(np.float64).tolist()):
        if math.isnan(G) or math.isnan(T):
            continue
        if G == T:
            out.append(0.0)
        elif math.isinf(G) or math.isinf(T):
            out.append(math.inf)
        else:
            out.append(float(abs(Fraction(T) - Fraction(G))))
    return out


def ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def expected(errs: list[float], num: int, den: int) -> dict:
    n = len(errs)
    k = ceil_div(n * num, den)
    if k == 0:
        return {"n_valid": n, "k": 0, "count_above": 0, "kth_value": math.nan, "sum_topk": 0.0,
                "mean_topk": math.nan}
    top = heapq.nlargest(k, errs)
    kth = top[-1]
    s = math.inf if math.isinf(top[0]) else math.fsum(top)
    return {"n_valid": n, "k": k, "count_above": sum(1 for x in errs if x > kth), "kth_value": kth,
            "sum_topk": s, "mean_topk": s / k}


def check(got: dict, want: dict, rel: float = 1e-15):
    for key in ("n_valid", "k", "count_above"):
        assert got[key] == want[key], (key, got[key], want[key])
    for key in ("kth_value", "sum_topk", "mean_topk"):
        a, b = got[key], want[key]
        if math.isnan(b):
            assert math.isnan(a), key
        elif math.isinf(b) or key == "kth_value":
            assert a == b, (key, a, b)
        else:
            assert abs(a - b) <= rel * abs(b), (key, a, b)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("frac", [(1, 10), (1, 100), (3, 7), (1, 1), (99, 100)])
def test_random_f32_against_nlargest_and_fsum(seed, frac):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 3000))
    g = rng.standard_normal(n).astype(np.float32)
    t = (g * (1 + rng.standard_normal(n) * 1e-3)).astype(np.float32)
    eq = rng.random(n) < 0.05                         # some zero errors
    t[eq] = g[eq]
    check(oracle.topk(g, t, num=frac[0], den=frac[1]), expected(exact_errors(g, t), *frac))


def test_f16_grid_against_torch_topk():
    # every finite f16 value as test against a few goldens
    bits = np.arange(0, 1 << 16, dtype=np.uint16)
    vals = bits.view(np.float16)
    t = vals[np.isfinite(vals)]
    for gv in (0.0, 1.0, -3.5, 65504.0, 6.1e-5):
        g = np.full_like(t, np.float16(gv))
        errs = exact_errors(g, t)
        for num, den in ((1, 10), (1, 1000)):
            got = oracle.topk(g, t, num=num, den=den)
            k = ceil_div(len(errs), 10 if den == 10 else 1000) if num == 1 else None
            vals_t, _ = torch.topk(torch.tensor(errs, dtype=torch.float64), k)
            assert got["k"] == k
            assert got["kth_value"] == float(vals_t[-1])
            assert abs(got["sum_topk"] - math.fsum(vals_t.tolist())) <= 1e-15 * got["sum_topk"]


def test_arithmetic_progression_closed_form():
    # errors {0, d, 2d, ..., (n-1)d} in a shuffled order: the top k sum is
    # d * k * (2n - k - 1) / 2, the k-th largest is (n - k) d
    d = 2.0 ** -10
    n = 1001
    rng = np.random.default_rng(7)
    perm = rng.permutation(n)
    g = np.full(n, 8.0, dtype=np.float32)
    t = (g + perm.astype(np.float32) * np.float32(d)).astype(np.float32)
    for num, den in ((1, 10), (1, 3), (1, 1), (1, 1000)):
        k = ceil_div(n * num, den)
        got = oracle.topk(g, t, num=num, den=den)
        assert got["k"] == k
        assert got["kth_value"] == (n - k) * d
        assert got["count_above"] == k - 1
        assert got["sum_topk"] == d * k * (2 * n - k - 1) / 2


def test_ceiling_not_floor():
    g = np.zeros(11, dtype=np.float32)
    t = np.arange(11, dtype=np.float32)
    got = oracle.topk(g, t, num=1, den=10)
    assert got["k"] == 2 and got["sum_topk"] == 19.0 and got["kth_value"] == 9.0


def test_ties_count_above_is_strict():
    g = np.zeros(20, dtype=np.float32)
    t = np.array([5.0] * 3 + [2.0] * 10 + [1.0] * 7, dtype=np.float32)
    got = oracle.topk(g, t, num=1, den=2)           # k = 10: three 5s and seven 2s
    assert got["k"] == 10 and got["kth_value"] == 2.0 and got["count_above"] == 3
    assert got["sum_topk"] == 29.0 and got["mean_topk"] == 2.9


def test_all_errors_equal():
    g = np.linspace(-4, 4, 1000).astype(np.float32)
    t = (g + np.float32(0.25)).astype(np.float32)
    errs = exact_errors(g, t)
    check(oracle.topk(g, t, num=1, den=10), expected(errs, 1, 10))


def test_nan_pairs_are_excluded_and_inf_dominates():
    g = np.array([1, 2, np.nan, 4, 5, 6, 7, 8, 9, 10, 11], dtype=np.float32)
    t = np.array([1, 3, 0, np.nan, 5, np.inf, 7, 8, 9, 10, 12], dtype=np.float32)
    got = oracle.topk(g, t, num=1, den=10)          # 9 valid pairs -> k = 1
    assert got["n_valid"] == 9 and got["k"] == 1
    assert got["kth_value"] == math.inf and got["sum_topk"] == math.inf and got["count_above"] == 0
    got = oracle.topk(g, t, num=1, den=3)           # k = 3: inf, 1, 1
    assert got["k"] == 3 and got["kth_value"] == 1.0 and got["count_above"] == 1
    assert got["sum_topk"] == math.inf and got["mean_topk"] == math.inf


def test_no_valid_pair_and_empty():
    g = np.full(5, np.nan, dtype=np.float32)
    got = oracle.topk(g, g, num=1, den=10)
    assert got["n_valid"] == 0 and got["k"] == 0 and got["sum_topk"] == 0.0
    assert math.isnan(got["kth_value"]) and math.isnan(got["mean_topk"])
    e = np.zeros(0, dtype=np.float32)
    got = oracle.topk(e, e, num=1, den=10)
    assert got["k"] == 0 and math.isnan(got["mean_topk"])


def test_bf16_and_dtype_codes():
    rng = np.random.default_rng(3)
    f = rng.standard_normal(4000).astype(np.float32)
    gb = (f.view(np.uint32) >> 16).astype(np.uint16)
    tb = gb ^ rng.integers(0, 2, 4000, dtype=np.uint16)       # last-bit flips
    g = (gb.astype(np.uint32) << 16).view(np.float32)
    t = (tb.astype(np.uint32) << 16).view(np.float32)
    check(oracle.topk(gb, tb, dtype=BF16, num=1, den=10), expected(exact_errors(g, t), 1, 10))


def test_validation_codes():
    assert oracle.topk_rc(4, F32, 0, 10) == oracle.EINVAL
    assert oracle.topk_rc(4, F32, 11, 10) == oracle.EINVAL
    assert oracle.topk_rc(4, 7, 1, 10) == oracle.EDTYPE
    assert oracle.topk_rc(-1, F32, 1, 10) == oracle.EINVAL
