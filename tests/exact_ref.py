"""Independent exact references used to pin the oracle.

Nothing here calls the oracle or the GPU library.  Values are decoded with
numpy/torch conversions (not the oracle's decoder), errors are computed in
exact integer or rational arithmetic, sums are correctly rounded (Python int
-> float conversion, int/int true division and math.fsum are all correctly
rounded), ULP distances come from ranks in the sorted set of representable
values, and closeness comes from torch.isclose.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
import torch

POW2 = np.array([1 << k for k in range(63)], dtype=np.int64)


def floor_log2_int(x: np.ndarray) -> np.ndarray:
    """floor(log2(x)) for positive int64 x, by comparison with exact powers of 2."""
    return np.searchsorted(POW2, x, side="right") - 1


def all_f16() -> np.ndarray:
    """All 65536 binary16 bit patterns as uint16."""
    return np.arange(65536, dtype=np.uint32).astype(np.uint16)


def f16_values(bits: np.ndarray) -> np.ndarray:
    return bits.view(np.float16).astype(np.float64)


def f16_rank_table():
    """Rank of every non-NaN f16 value in the sorted set of distinct values
    (+0 and -0 are one value; +-Inf are the extreme ranks)."""
    vals = f16_values(all_f16())
    distinct = np.unique(vals[~np.isnan(vals)])
    return distinct


def ulp_by_rank(g_vals: np.ndarray, t_vals: np.ndarray, distinct: np.ndarray) -> np.ndarray:
    rg = np.searchsorted(distinct, g_vals)
    rt = np.searchsorted(distinct, t_vals)
    assert np.all(distinct[rg] == g_vals) and np.all(distinct[rt] == t_vals)
    return np.abs(rt - rg)


def exact_f16_signature(g_bits: np.ndarray, t_bits: np.ndarray, bins, thresholds, distinct):
    """Every signature field for f16 pairs, computed exactly.

    Finite f16 values are integer multiples of 2^-24 (|value| * 2^24 < 2^40),
    so differences and products are exact integers in units of 2^-24 / 2^-48.
    """
    lo, hi, nb = bins
    w = (hi - lo) // nb
    G = f16_values(g_bits)
    T = f16_values(t_bits)
    n = G.size
    nan_g, nan_t = np.isnan(G), np.isnan(T)
    inf_g, inf_t = np.isinf(G), np.isinf(T)
    nanpair = nan_g | nan_t
    valid = ~nanpair
    finite = valid & ~inf_g & ~inf_t
    res = {
        "n": n, "n_valid": int(valid.sum()), "n_finite": int(finite.sum()),
        "n_nan_golden": int(nan_g.sum()), "n_nan_test": int(nan_t.sum()),
        "n_inf_golden": int(inf_g.sum()), "n_inf_test": int(inf_t.sum()),
        "n_nan_pairs": int(nanpair.sum()),
        "first_nan_index": int(np.argmax(nanpair)) if nanpair.any() else -1,
    }
    # exact |T - G| in units of 2^-24 for finite pairs; inf handling by cases
    kg = np.zeros(n, dtype=np.int64)
    kt = np.zeros(n, dtype=np.int64)
    kg[finite] = (G[finite] * 2.0 ** 24).astype(np.int64)
    kt[finite] = (T[finite] * 2.0 ** 24).astype(np.int64)
    assert np.all(kg[finite] * 2.0 ** -24 == G[finite])
    a_int = np.abs(kt - kg)
    a_inf = valid & ~finite & ~((inf_g & inf_t) & (G == T))   # one side inf, or opposite infs
    a_zero_inf = valid & ~finite & ~a_inf                     # equal infinities
    a = np.where(finite, a_int.astype(np.float64) * 2.0 ** -24, 0.0)
    a[a_inf] = np.inf
    a[~valid] = np.nan

    # histogram
    zero = valid & (a == 0)
    res["hist_zero"] = int(zero.sum())
    pos = finite & (a_int > 0)
    k = np.full(n, 10 ** 6, dtype=np.int64)
    k[pos] = floor_log2_int(a_int[pos]) - 24
    res["hist_under"] = int((pos & (k < lo)).sum())
    res["hist_over"] = int((pos & (k >= hi)).sum() + a_inf.sum())
    hist = [0] * 64
    inb = pos & (k >= lo) & (k < hi)
    for kk in k[inb]:
        hist[(int(kk) - lo) // w] += 1
    res["hist"] = hist
    assert res["hist_zero"] + res["hist_under"] + sum(hist) + res["hist_over"] == res["n_valid"]

    # mismatches from torch.isclose on float64 (rtol = 0, equal_nan = False)
    tg, tt = torch.from_numpy(G), torch.from_numpy(T)
    res["n_mismatch"] = [int((~torch.isclose(tt, tg, rtol=0.0, atol=float(th), equal_nan=False)).sum())
                         for th in thresholds]

    # ULP by rank
    ulp = np.zeros(n, dtype=np.int64)
    ulp[valid] = ulp_by_rank(G[valid], T[valid], distinct)
    res["sum_ulp"] = int(ulp[valid].sum())
    vidx = np.nonzero(valid)[0]
    if vidx.size:
        j = int(np.argmax(ulp[vidx]))        # first occurrence of the maximum
        res["max_ulp"], res["argmax_ulp"] = int(ulp[vidx][j]), int(vidx[j])
        av = a[vidx]
        j = int(np.argmax(av))
        res["max_abs"], res["argmax_abs"] = float(av[j]), int(vidx[j])
    else:
        res["max_ulp"], res["argmax_ulp"] = 0, -1
        res["max_abs"], res["argmax_abs"] = math.nan, -1

    # fp64 sums, correctly rounded from exact integers
    fi = np.nonzero(finite)[0]
    ai = [int(x) for x in a_int[fi]]
    gi = [int(x) for x in kg[fi]]
    ti = [int(x) for x in kt[fi]]
    res["sum_abs"] = sum(ai) / (1 << 24)
    res["sum_sq"] = math.fsum(float(x * x) * 2.0 ** -48 for x in ai)   # sum of RN(a^2)
    res["sum_g2"] = sum(x * x for x in gi) / (1 << 48)
    res["sum_t2"] = sum(x * x for x in ti) / (1 << 48)
    res["sum_gt"] = sum(x * y for x, y in zip(gi, ti)) / (1 << 48)
    rel = [(x / abs(y), idx) for x, y, idx in zip(ai, gi, fi) if y != 0]  # RN(a/|G|)
    res["n_rel"] = len(rel)
    res["sum_rel"] = math.fsum(r for r, _ in rel)
    if rel:
        best = max(r for r, _ in rel)
        res["max_rel"] = best
        res["argmax_rel"] = int(min(idx for r, idx in rel if r == best))
    else:
        res["max_rel"], res["argmax_rel"] = math.nan, -1
    return res


def fraction_abs_diff(g: float, t: float) -> float:
    """|t - g| correctly rounded to binary64 (exact rational, then one rounding)."""
    return float(abs(Fraction(t) - Fraction(g)))
