"""Pins of the oracle's mixed-precision pairs (Section III-C: an FP32 golden
output against the output of the same operation in FP16 or in FP64) against
what the definitions fix independently of the oracle's code:

  - a wide side holding values of the narrow format, widened exactly, gives
    the same-type signature field for field (values, ULP keys, sums);
  - the ULP distance is the distance of bit-pattern keys in the narrower
    format after rounding the wider value to it, with the rounding done here
    by exact rational arithmetic (round to nearest, ties to even, overflow to
    Inf past the largest finite value) and cross-checked with numpy's casts;
  - the error and its sums from exact rationals and math.fsum, the
    closeness counts from torch.isclose in float64, the top-k mean from a sort;
  - the type rules (binary64 only on the test side, nested formats only).
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

F32, F16, BF16, F64 = oracle.F32, oracle.F16, oracle.BF16, oracle.F64
FMT = {F32: (24, -126, 127), F16: (11, -14, 15), BF16: (8, -126, 127), F64: (53, -1022, 1023)}
WIDTH = {F32: 32, F16: 16, BF16: 16}


def rn_exact(x: float, dt: int) -> float:
    """x rounded to format dt: nearest, ties to even, Inf beyond the largest
    finite value (exact rational arithmetic)."""
    if x == 0 or math.isinf(x) or math.isnan(x):
        return x
    p, emin, emax = FMT[dt]
    a = Fraction(abs(x))
    E = max(math.frexp(abs(x))[1] - 1, emin)
    q = Fraction(2) ** (E - p + 1)
    r = a / q
    n = r.numerator // r.denominator
    rem = r - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    v = n * q
    largest = (2 - Fraction(2) ** (1 - p)) * Fraction(2) ** emax
    if v > largest:
        return math.copysign(math.inf, x)
    return math.copysign(float(v), x)


def key_of(v: float, dt: int) -> int:
    """Signed-magnitude key of the bit pattern of v (v representable in dt)."""
    if dt == F32:
        b = int(np.array([v], dtype=np.float32).view(np.uint32)[0])
    elif dt == F16:
        b = int(np.array([v], dtype=np.float16).view(np.uint16)[0])
    else:
        b32 = int(np.array([v], dtype=np.float32).view(np.uint32)[0])
        assert b32 & 0xFFFF == 0
        b = b32 >> 16
    s = 1 << (WIDTH[dt] - 1)
    return -(b & (s - 1)) if b & s else (b & (s - 1))


def values(arr: np.ndarray, dt: int) -> list[float]:
    """Exact binary64 values of an array of bit patterns (or of floats)."""
    if dt == BF16:
        return (arr.astype(np.uint32) << 16).view(np.float32).astype(np.float64).tolist()
    if arr.dtype == np.uint32:
        arr = arr.view(np.float32)
    elif arr.dtype == np.uint16:
        arr = arr.view(np.float16)
    return arr.astype(np.float64).tolist()


def narrow_of(g: int, t: int) -> int:
    return g if FMT[g][0] <= FMT[t][0] else t


def expected_ulps(gv: list[float], tv: list[float], gdt: int, tdt: int) -> list[int | None]:
    nd = narrow_of(gdt, tdt)
    out = []
    for G, T in zip(gv, tv):
        if math.isnan(G) or math.isnan(T):
            out.append(None)
            continue
        out.append(abs(key_of(rn_exact(T, nd), nd) - key_of(rn_exact(G, nd), nd)))
    return out


def random_bits16(rng, n):
    return rng.integers(0, 1 << 16, n, dtype=np.uint64).astype(np.uint16)


def widen_bits(bits: np.ndarray, dt: int, to: int) -> np.ndarray:
    """Exact widening of narrow bit patterns to the wider type's array."""
    if dt == F16:
        v = bits.view(np.float16)
    elif dt == BF16:
        v = (bits.astype(np.uint32) << 16).view(np.float32)
    else:
        v = bits.view(np.float32)
    return v.astype(np.float32 if to == F32 else np.float64)


NESTED = [(F16, F32), (BF16, F32), (F32, F64), (F16, F64), (BF16, F64)]


@pytest.mark.parametrize("narrow,wide", NESTED)
@pytest.mark.parametrize("golden_narrow", [True, False])
def test_exactly_widened_side_gives_the_same_type_signature(narrow, wide, golden_narrow):
    if not golden_narrow and wide == F64:
        pytest.skip("the golden side is never binary64")
    rng = np.random.default_rng(7 + narrow * 10 + wide)
    n = 3000
    if narrow == F32:
        gb = rng.integers(0, 1 << 32, n, dtype=np.uint64).astype(np.uint32)
        tb = gb ^ rng.integers(0, 1 << 12, n, dtype=np.uint64).astype(np.uint32)
    else:
        gb = random_bits16(rng, n)
        tb = gb ^ random_bits16(rng, n) % 64
    tb[::7] = random_bits16(rng, len(tb[::7])).astype(tb.dtype)   # sign changes, NaN, Inf, zeros
    thr = (1e-6, (1e-3, 1e-2), 0.5)
    same = oracle.signature(gb, tb, dtype=narrow, thresholds=thr)
    if golden_narrow:
        mixed = oracle.signature_mixed(gb, widen_bits(tb, narrow, wide), gdtype=narrow, tdtype=wide,
                                       thresholds=thr)
    else:
        mixed = oracle.signature_mixed(widen_bits(gb, narrow, wide), tb, gdtype=wide, tdtype=narrow,
                                       thresholds=thr)
    for k, v in same.items():
        w = mixed[k]
        if isinstance(v, float) and math.isnan(v):
            assert math.isnan(w), k
        else:
            assert w == v, (k, v, w)


def _pairs_near(rng, n, gdt):
    """Golden values of format gdt and binary64 test values near them: tiny
    perturbations, exact ties of the golden format, values past its range,
    subnormals, sign changes."""
    p, emin, emax = FMT[gdt]
    r = min(20, emax // 2)
    g = rng.standard_normal(n) * np.exp2(rng.integers(-r, r, n))
    g = np.array([rn_exact(x, gdt) for x in g.tolist()])
    t = g * (1 + rng.standard_normal(n) * np.exp2(-rng.integers(5, 60, n)))
    ulp = np.exp2(np.floor(np.log2(np.abs(g))) - (p - 1))
    t[0::11] = g[0::11] + 0.5 * ulp[0::11]                          # exact ties
    t[1::11] = g[1::11] - 0.5 * ulp[1::11]
    t[2::11] = g[2::11] + 0.5 * ulp[2::11] * (1 + 2.0 ** -40)        # just past a tie
    t[3::11] = math.ldexp(1.0, emax + 1) * rng.uniform(0.9, 1.1, len(t[3::11]))   # around overflow
    t[4::11] = math.ldexp(1.0, emin - p + 1) * rng.uniform(-3, 3, len(t[4::11]))  # subnormal range
    t[5::11] = -g[5::11]                                             # sign change
    return g, t


def _to_bits(g: np.ndarray, dt: int) -> np.ndarray:
    if dt == F32:
        return g.astype(np.float32).view(np.uint32)
    if dt == F16:
        return g.astype(np.float16).view(np.uint16)
    return (g.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


@pytest.mark.parametrize("gdt", [F32, F16, BF16])
def test_ulp_of_a_binary64_test_is_counted_in_the_golden_format(gdt):
    rng = np.random.default_rng(100 + gdt)
    g, t = _pairs_near(rng, 4000, gdt)
    gb = _to_bits(g, gdt)
    gv = values(gb, gdt)
    want = expected_ulps(gv, t.tolist(), gdt, F64)
    s = oracle.signature_mixed(gb, t, gdtype=gdt, tdtype=F64, thresholds=())
    valid = [u for u in want if u is not None]
    assert s["sum_ulp"] == sum(valid)
    assert s["max_ulp"] == max(valid)
    assert s["argmax_ulp"] == want.index(max(valid))


@pytest.mark.parametrize("tdt", [F16, BF16])
def test_ulp_of_a_narrow_test_is_counted_in_its_format(tdt):
    rng = np.random.default_rng(200 + tdt)
    t, g = _pairs_near(rng, 4000, tdt)          # test of the narrow format, golden f32 near it
    g = g.astype(np.float32)
    g[np.isinf(g)] = 1.0
    tb = _to_bits(t, tdt)
    want = expected_ulps(g.astype(np.float64).tolist(), values(tb, tdt), F32, tdt)
    s = oracle.signature_mixed(g, tb, gdtype=F32, tdtype=tdt, thresholds=())
    valid = [u for u in want if u is not None]
    assert s["sum_ulp"] == sum(valid)
    assert s["max_ulp"] == max(valid)


def test_exact_rounding_agrees_with_numpy_casts():
    # the test's own rounding against numpy's float64 -> float32 / float16 casts
    rng = np.random.default_rng(5)
    for dt, npt in ((F32, np.float32), (F16, np.float16)):
        g, t = _pairs_near(rng, 3000, dt)
        with np.errstate(over="ignore"):
            cast = t.astype(npt).astype(np.float64)
        mine = np.array([rn_exact(x, dt) for x in t.tolist()])
        assert np.array_equal(cast, mine)


@pytest.mark.parametrize("t,ulp", [
    (1.0 + 2.0 ** -24, 0),                   # a tie rounds to the even 1.0
    (1.0 + 3 * 2.0 ** -24, 2),               # a tie rounds to the even 1 + 2^-22
    (1.0 + 2.0 ** -24 + 2.0 ** -50, 1),      # just past the tie
    (1.0 - 2.0 ** -25, 0),                   # a tie below 1 (ULP 2^-24 there) rounds to 1.0
    (2.0 ** 128, 0x7F800000 - 0x3F800000),   # beyond FP32: Inf
    (-1.0, 2 * 0x3F800000),                  # sign change: through zero
    (2.0 ** -150, 0x3F800000),               # rounds to +0 (a tie with the smallest subnormal)
    (3 * 2.0 ** -151, 0x3F800000 - 1),       # rounds to the smallest subnormal
])
def test_f32_golden_one_against_binary64_closed_forms(t, ulp):
    s = oracle.signature_mixed(np.array([1.0], np.float32), np.array([t]), thresholds=())
    assert s["max_ulp"] == ulp
    assert s["max_abs"] == float(abs(Fraction(t) - 1))


def test_double_rounding_would_be_wrong():
    # 1 + 2^-11 + 2^-40 rounds to 1 + 2^-10 in FP16; through FP32 first it
    # would become the tie 1 + 2^-11 and then 1.0
    s = oracle.signature_mixed(np.array([1.0], np.float16), np.array([1 + 2.0 ** -11 + 2.0 ** -40]),
                               thresholds=())
    assert s["max_ulp"] == 1
    s = oracle.signature_mixed(np.array([0x3F80], np.uint16), np.array([1 + 2.0 ** -8 + 2.0 ** -40]),
                               gdtype=BF16, thresholds=())
    assert s["max_ulp"] == 1


@pytest.mark.parametrize("gdt,tdt", [(F32, F64), (F16, F64), (F32, F16), (F16, F32), (BF16, F64)])
def test_error_sums_counts_and_closeness(gdt, tdt):
    rng = np.random.default_rng(300 + 4 * gdt + tdt)
    n = 2500
    base = rng.standard_normal(n)
    gb = _to_bits(base, gdt)
    gv = np.array(values(gb, gdt))
    tw = gv * (1 + 1e-3 * rng.standard_normal(n))
    tw[::97] = np.nan
    tw[5::131] = np.inf
    tb = tw if tdt == F64 else _to_bits(tw, tdt)
    tv = np.array(tw if tdt == F64 else values(tb, tdt))
    thr = (1e-4, (1e-5, 1e-3), 0.0)
    s = oracle.signature_mixed(gb, tb, gdtype=gdt, tdtype=tdt, thresholds=thr)
    ok = ~(np.isnan(gv) | np.isnan(tv))
    fin = ok & np.isfinite(gv) & np.isfinite(tv)
    err = [float(abs(Fraction(T) - Fraction(G))) for G, T in zip(gv[fin].tolist(), tv[fin].tolist())]
    assert s["n_valid"] == int(ok.sum()) and s["n_finite"] == int(fin.sum())
    assert s["sum_abs"] == pytest.approx(math.fsum(err), rel=1e-15)
    assert s["sum_sq"] == pytest.approx(math.fsum(e * e for e in err), rel=1e-13)
    assert s["sum_gt"] == pytest.approx(math.fsum((gv[fin] * tv[fin]).tolist()), rel=1e-12)
    G, T = torch.from_numpy(gv), torch.from_numpy(tv)
    for j, x in enumerate(thr):
        atol, rtol = (x, 0.0) if not isinstance(x, tuple) else x
        want = int((~torch.isclose(T, G, rtol=rtol, atol=atol, equal_nan=False)).sum())
        assert s["n_mismatch"][j] == want


@pytest.mark.parametrize("gdt,tdt", [(F32, F64), (F32, F16), (BF16, F32)])
def test_topk_mixed_from_a_sort(gdt, tdt):
    rng = np.random.default_rng(400 + gdt + tdt)
    n = 3001
    gb = _to_bits(rng.standard_normal(n), gdt)
    gv = np.array(values(gb, gdt))
    tw = gv + 1e-3 * rng.standard_normal(n)
    tw[::50] = np.nan
    tb = tw if tdt == F64 else _to_bits(tw, tdt)
    tv = np.array(tw if tdt == F64 else values(tb, tdt))
    ok = ~(np.isnan(gv) | np.isnan(tv))
    err = sorted((float(abs(Fraction(T) - Fraction(G))) for G, T in zip(gv[ok].tolist(), tv[ok].tolist())),
                 reverse=True)
    k = -(-len(err) // 10)
    r = oracle.topk_mixed(gb, tb, gdtype=gdt, tdtype=tdt)
    assert r["n_valid"] == len(err) and r["k"] == k
    assert r["kth_value"] == err[k - 1]
    assert r["sum_topk"] == pytest.approx(math.fsum(err[:k]), rel=1e-15)


def test_topk_mixed_with_exactly_widened_test_is_the_same_type_score():
    rng = np.random.default_rng(9)
    g = rng.standard_normal(5000).astype(np.float32)
    t = (g + 1e-4 * rng.standard_normal(5000)).astype(np.float32)
    assert oracle.topk_mixed(g, t.astype(np.float64), tdtype=F64) == oracle.topk(g, t)


@pytest.mark.parametrize("gdt,tdt,ok", [
    (F32, F64, True), (F16, F64, True), (BF16, F64, True), (F32, F16, True), (F16, F32, True),
    (F32, BF16, True), (BF16, F32, True), (F32, F32, True), (F16, F16, True),
    (F64, F32, False), (F64, F64, False), (F16, BF16, False), (BF16, F16, False), (F32, 7, False),
    (-1, F32, False)])
def test_type_rules(gdt, tdt, ok):
    assert oracle.signature_mixed_rc(gdt, tdt) == (oracle.OK if ok else oracle.EDTYPE)


def test_subnormal_binary64_errors_lie_below_every_bin():
    # a zero golden against binary64 subnormals: errors below 2^-1022, which
    # the histogram counts under its lowest bin; the top-k orders them
    g = np.zeros(6, np.float32)
    t = np.array([0.0, 5e-324, 2 * 5e-324, -3 * 5e-324, 2.0 ** -1030, 2.0 ** -1022])
    s = oracle.signature_mixed(g, t, bins=(-1022, 0, 1), thresholds=())
    assert s["hist_zero"] == 1 and s["hist_under"] == 4 and s["hist"][0] == 1
    assert s["max_abs"] == 2.0 ** -1022 and s["argmax_abs"] == 5
    r = oracle.topk_mixed(g, t, num=1, den=2)          # k = 3: 2^-1022, 2^-1030, 3 * 2^-1074
    assert r["k"] == 3 and r["kth_value"] == 3 * 5e-324 and r["count_above"] == 2
    assert r["sum_topk"] == 2.0 ** -1022 + 2.0 ** -1030 + 3 * 5e-324
