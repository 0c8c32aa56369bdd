"""Pins of the CPU oracle against facts it does not compute itself.

Each test fixes a field (or the injector's draw) by something other than the
oracle: exact integer/rational arithmetic, brute force over every binary16 and
bfloat16 value, ranks in the sorted set of representable values, the
Philox4x32-10 known-answer vectors and rocRAND's implementation, torch's
float64 isclose/norm/cosine/var, math.fsum, IEEE-754 closed forms, and the paper's own statement about exponent bit flips
(Section II-B "Error Models", fixture in tests/golden/).
"""
from __future__ import annotations

import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from tests import philox_ref
from tests import exact_ref as X

HERE = os.path.dirname(os.path.abspath(__file__))
M64 = (1 << 64) - 1
M32 = (1 << 32) - 1

SUM_FIELDS = ("sum_abs", "sum_sq", "sum_rel", "sum_g2", "sum_t2", "sum_gt")


def _close_ulps(a: float, b: float, k: int = 2) -> bool:
    if math.isnan(a) or math.isnan(b):
        return math.isnan(a) and math.isnan(b)
    return abs(a - b) <= k * math.ulp(max(abs(a), abs(b)))


def _assert_sig_equal(sig: dict, ref: dict, ctx: str = ""):
    for k, v in ref.items():
        got = sig[k]
        if k in SUM_FIELDS:
            assert _close_ulps(got, v), f"{ctx} {k}: oracle {got!r} exact {v!r}"
        elif isinstance(v, float) and math.isnan(v):
            assert math.isnan(got), f"{ctx} {k}: oracle {got!r} expected NaN"
        else:
            assert got == v, f"{ctx} {k}: oracle {got!r} exact {v!r}"


# ---------------------------------------------------------------------------
# Philox4x32-10 against the published known-answer vectors (Random123, Salmon
# et al., SC'11) and rocRAND's implementation.
# ---------------------------------------------------------------------------
KAT = [  # (counter, key, block)
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((M32, M32, M32, M32), (M32, M32), (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("counter,key,block", KAT)
def test_philox_known_answers(counter, key, block):
    assert oracle.philox4x32_10(counter, key) == list(block)


needs_ref = pytest.mark.skipif(not philox_ref.available(), reason="hipcc (for rocRAND's header) not found")


@needs_ref
def test_philox_matches_rocrand_on_random_counters_and_keys():
    rng = np.random.default_rng(2609)
    ctr = rng.integers(0, 1 << 32, (300, 4), dtype=np.uint64).astype(np.uint32)
    key = rng.integers(0, 1 << 32, (300, 2), dtype=np.uint64).astype(np.uint32)
    ctr[:20] = [[c, 0, s, 0] for c in range(5) for s in range(4)]      # the library's counters
    want = philox_ref.blocks(ctr, key)
    for i in range(ctr.shape[0]):
        assert oracle.philox4x32_10(ctr[i], key[i]) == [int(x) for x in want[i]], i


# ---------------------------------------------------------------------------
# Rate threshold T = floor(rate * 2^64), exactly.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("rate", [1e-8, 1e-7, 1e-9, 0.5, 2.0 ** -56, 3e-300, 0.1,
                                  float(np.nextafter(1.0, 0.0)), 5e-324])
def test_rate_threshold_exact(rate):
    T, all_ = oracle.rate_threshold(rate)
    assert not all_
    assert T == math.floor(Fraction(rate) * (1 << 64))


def test_rate_threshold_edges():
    assert oracle.rate_threshold(0.0) == (0, False)
    assert oracle.rate_threshold(1.0)[1] is True
    assert oracle.rate_threshold(7.5)[1] is True
    assert oracle.rate_threshold(1e-8)[0] == 184467440737


# ---------------------------------------------------------------------------
# Brute force over every binary16 value.
# ---------------------------------------------------------------------------
_F16_GOLDENS = [0x0000, 0x8000, 0x0001, 0x8001, 0x0200, 0x03FF, 0x0400, 0x3C00, 0xBC00,
                0x3E00, 0x3C01, 0x7BFF, 0xFBFF, 0x7C00, 0xFC00, 0x7E00, 0x5640, 0x1234]
_F16_THR = (0.0, 2.0 ** -24, 1e-3, 0.5, 1.0, 65504.0, math.inf)
_BINS_SETS = [(-40, 24, 64), (-26, 18, 22), (-28, 20, 12), (-10, 6, 1)]


@pytest.fixture(scope="module")
def f16_distinct():
    return X.f16_rank_table()


@pytest.mark.parametrize("bins", _BINS_SETS)
def test_f16_bruteforce_test_side(bins, f16_distinct):
    """Golden fixed, test = every f16 bit pattern (NaNs, infinities, zeros,
    subnormals included).  Every field against the exact reference."""
    rng = np.random.default_rng(7)
    goldens = _F16_GOLDENS + [int(x) for x in rng.integers(0, 65536, 6)]
    t_bits = X.all_f16()
    for gb in goldens:
        g_bits = np.full(65536, gb, dtype=np.uint16)
        sig = oracle.signature(g_bits, t_bits, dtype=oracle.F16, bins=bins, thresholds=_F16_THR)
        ref = X.exact_f16_signature(g_bits, t_bits, bins, _F16_THR, f16_distinct)
        _assert_sig_equal(sig, ref, f"golden=0x{gb:04x} bins={bins}")


def test_f16_bruteforce_golden_side(f16_distinct):
    """Test fixed, golden = every f16 bit pattern: exercises the relative
    error (division by every golden value) and the zero-golden exclusion."""
    bins = (-40, 24, 64)
    g_bits = X.all_f16()
    for tb in (0x0000, 0x3C00, 0xC500, 0x0001, 0x7BFF, 0x7C00, 0x7E01, 0x2E66):
        t_bits = np.full(65536, tb, dtype=np.uint16)
        sig = oracle.signature(g_bits, t_bits, dtype=oracle.F16, bins=bins, thresholds=_F16_THR)
        ref = X.exact_f16_signature(g_bits, t_bits, bins, _F16_THR, f16_distinct)
        _assert_sig_equal(sig, ref, f"test=0x{tb:04x}")


def test_f16_random_pairs_with_ties(f16_distinct):
    """Random pairs from a small value pool, so maxima tie many times and the
    lowest-index rule is exercised on every maximum."""
    rng = np.random.default_rng(11)
    pool = np.array([0x3C00, 0x3C01, 0x3BFF, 0x4000, 0x0000, 0x8000, 0x7C00, 0x7E00, 0x0001], np.uint16)
    g_bits = pool[rng.integers(0, pool.size, 50000)]
    t_bits = pool[rng.integers(0, pool.size, 50000)]
    for bins in _BINS_SETS[:2]:
        sig = oracle.signature(g_bits, t_bits, dtype=oracle.F16, bins=bins, thresholds=_F16_THR)
        ref = X.exact_f16_signature(g_bits, t_bits, bins, _F16_THR, f16_distinct)
        _assert_sig_equal(sig, ref, f"bins={bins}")


# ---------------------------------------------------------------------------
# bfloat16: brute force over every bf16 value with exact rational differences.
# ---------------------------------------------------------------------------
def _bf16_values(bits: np.ndarray) -> np.ndarray:
    return torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).double().numpy()


@pytest.mark.parametrize("gb", [0x3F80, 0x0001, 0x8000, 0x7F7F, 0xFF80, 0x3C23])
def test_bf16_bruteforce(gb):
    bins = (-140, 130, 54)   # 5 binades per bin, covers the whole bf16 range
    thr = (0.0, 1e-3, 1.0, 1e30)
    t_bits = X.all_f16()          # all 65536 16-bit patterns, read as bf16
    g_bits = np.full(65536, gb, dtype=np.uint16)
    sig = oracle.signature(g_bits, t_bits, dtype=oracle.BF16, bins=bins, thresholds=thr)
    G, T = _bf16_values(g_bits), _bf16_values(t_bits)
    valid = ~(np.isnan(G) | np.isnan(T))
    finite = valid & np.isfinite(G) & np.isfinite(T)
    a = np.full(G.size, np.nan)
    for i in np.nonzero(valid)[0]:
        if G[i] == T[i]:
            a[i] = 0.0
        elif not (np.isfinite(G[i]) and np.isfinite(T[i])):
            a[i] = math.inf
        else:
            a[i] = X.fraction_abs_diff(G[i], T[i])
    assert sig["n_valid"] == int(valid.sum()) and sig["n_finite"] == int(finite.sum())
    av = a[valid]
    vidx = np.nonzero(valid)[0]
    j = int(np.argmax(av))
    assert sig["max_abs"] == av[j] and sig["argmax_abs"] == int(vidx[j])
    # bins by comparison with exact float64 powers of two
    pw = np.array([2.0 ** k for k in range(-1074, 1024)])
    fin_pos = valid & np.isfinite(a) & (a > 0)
    k = np.searchsorted(pw, a[fin_pos], side="right") - 1 - 1074
    lo, hi, nb = bins
    w = (hi - lo) // nb
    hist = [0] * 64
    for kk in k[(k >= lo) & (k < hi)]:
        hist[(int(kk) - lo) // w] += 1
    assert sig["hist"] == hist
    assert sig["hist_zero"] == int((valid & (a == 0)).sum())
    assert sig["hist_under"] == int((k < lo).sum())
    assert sig["hist_over"] == int((k >= hi).sum() + np.isinf(a[valid]).sum())
    tg, tt = torch.from_numpy(G), torch.from_numpy(T)
    assert sig["n_mismatch"] == [int((~torch.isclose(tt, tg, rtol=0.0, atol=th, equal_nan=False)).sum())
                                 for th in thr]
    distinct = np.unique(_bf16_values(X.all_f16())[~np.isnan(_bf16_values(X.all_f16()))])
    ulp = X.ulp_by_rank(G[valid], T[valid], distinct)
    assert sig["sum_ulp"] == int(ulp.sum())
    j = int(np.argmax(ulp))
    assert sig["max_ulp"] == int(ulp[j]) and sig["argmax_ulp"] == int(vidx[j])
    fi = np.nonzero(finite)[0]
    assert _close_ulps(sig["sum_abs"], math.fsum(a[fi]))
    assert _close_ulps(sig["sum_g2"], float(sum(Fraction(G[i]) ** 2 for i in fi)))
    assert _close_ulps(sig["sum_gt"], float(sum(Fraction(G[i]) * Fraction(T[i]) for i in fi)))


# ---------------------------------------------------------------------------
# binary32: hand-computed signature, closed forms, library routines.
# ---------------------------------------------------------------------------
def test_f32_hand_computed():
    """Worked by hand (see the comment per element).  Bins [2^-2, 2^2) in
    four binades; thresholds 0.5 and 1.0."""
    sub = np.float32(2.0 ** -149)
    G = np.array([1.0, -0.0, 2.0, sub, np.inf, 3.0, 4.0, np.nan, 1.0, -1.0], np.float32)
    T = np.array([1.5, 0.0, 1.0, 2 * sub, np.inf, 2.5, 3.0, 1.0, -1.0, 1.0], np.float32)
    # i  a        ulp                          rel    bin
    # 0  0.5      0x3FC00000-0x3F800000=2^22    0.5    [0.5,1)
    # 1  0        0 (-0 vs +0)                  --     zero (golden 0: no rel)
    # 2  1        0x40000000-0x3F800000=2^23    0.5    [1,2)
    # 3  2^-149   1                             1.0    under
    # 4  0        0 (equal infinities)          --     zero (not finite: no sums)
    # 5  0.5      0x40400000-0x40200000=2^21    1/6    [0.5,1)
    # 6  1        0x40800000-0x40400000=2^22    0.25   [1,2)   (ties max a=1 of i=2)
    # 7  NaN golden: NaN pair, first NaN index 7
    # 8  2        0x3F800000+0x3F800000         2.0    [2,4)
    # 9  2        same                          2.0    [2,4)   (ties i=8)
    sig = oracle.signature(G, T, bins=(-2, 2, 4), thresholds=(0.5, 1.0))
    assert sig["n"] == 10 and sig["n_valid"] == 9 and sig["n_finite"] == 8 and sig["n_rel"] == 7
    assert (sig["n_nan_golden"], sig["n_nan_test"], sig["n_inf_golden"], sig["n_inf_test"]) == (1, 0, 1, 1)
    assert sig["n_nan_pairs"] == 1 and sig["first_nan_index"] == 7
    assert sig["hist_zero"] == 2 and sig["hist_under"] == 1 and sig["hist_over"] == 0
    assert sig["hist"][:4] == [0, 2, 2, 2] and sum(sig["hist"][4:]) == 0
    assert sig["n_mismatch"] == [5, 3]
    assert sig["max_abs"] == 2.0 and sig["argmax_abs"] == 8
    assert sig["max_ulp"] == 0x7F000000 and sig["argmax_ulp"] == 8
    assert sig["sum_ulp"] == 2 ** 22 + 2 ** 23 + 1 + 2 ** 21 + 2 ** 22 + 2 * 0x7F000000
    assert sig["max_rel"] == 2.0 and sig["argmax_rel"] == 8
    assert sig["sum_abs"] == 7.0 and sig["sum_sq"] == 10.5
    assert sig["sum_g2"] == 32.0 and sig["sum_t2"] == 20.5 and sig["sum_gt"] == 21.0
    assert sig["sum_rel"] == math.fsum([0.5, 0.5, 1.0, 1 / 6, 0.25, 2.0, 2.0])


def test_paper_exponent_msb_flip_fixture():
    """Section II-B: flipping the first exponent bit of a value in [1, 2)."""
    rows = []
    with open(os.path.join(HERE, "golden", "exponent_msb_flip_f32.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                v, b0, b1, cls = line.split()
                rows.append((np.float32(float(v)), int(b0, 16), int(b1, 16), cls))
    G = np.array([r[0] for r in rows], np.float32)
    assert [int(x) for x in G.view(np.uint32)] == [r[1] for r in rows]
    T = G.copy()
    n = oracle.inject(T.view(np.uint32), seed=1, rate=1.0, mask=1 << 30)  # every element, bit 30
    assert n == len(rows)
    assert [int(x) for x in T.view(np.uint32)] == [r[2] for r in rows]
    sig = oracle.signature(G, T)
    n_nan = sum(r[3] == "nan" for r in rows)
    assert sig["n_nan_test"] == n_nan and sig["n_inf_test"] == len(rows) - n_nan
    assert sig["first_nan_index"] == [r[3] for r in rows].index("nan")
    assert sig["hist_over"] == len(rows) - n_nan        # the +Inf results: infinite error
    assert sig["n_mismatch"] == [len(rows), len(rows)]


@pytest.mark.parametrize("b", list(range(31)))
def test_f32_single_bit_flip_closed_form(b):
    """Flipping bit b <= 30 of a finite value (result finite) moves it exactly
    2^b representable values; for a fraction bit of g with floor(log2|g|) = E
    the error is exactly 2^(E - 23 + b)."""
    rng = np.random.default_rng(100 + b)
    g = (rng.uniform(0.5, 4.0, 4000) * rng.choice([-1, 1], 4000)).astype(np.float32)
    t = (g.view(np.uint32) ^ np.uint32(1 << b)).view(np.float32)
    keep = np.isfinite(t) & (t != 0)
    g, t = g[keep], t[keep]
    sig = oracle.signature(g, t, bins=(-200, 200, 50), thresholds=())
    assert sig["max_ulp"] == 2 ** b and sig["sum_ulp"] == g.size * 2 ** b
    assert sig["argmax_ulp"] == 0
    if b <= 22:
        E = np.floor(np.log2(np.abs(g.astype(np.float64))))
        a_expected = np.exp2(E - 23 + b)
        assert sig["max_abs"] == a_expected.max()
        assert sig["argmax_abs"] == int(np.argmax(a_expected))
        assert sig["sum_abs"] == math.fsum(a_expected)


def test_f32_ulp_by_nextafter_walks():
    """ULP distance of t = g stepped k times with nextafter (crossing zero
    and the subnormal range included) is k."""
    rng = np.random.default_rng(5)
    starts = np.concatenate([rng.standard_normal(300).astype(np.float32),
                             np.array([0.0, -0.0, 1e-45, -1e-45, 1.1754944e-38, -3e-45], np.float32)])
    for g0 in starts:
        k = int(rng.integers(0, 60))
        direction = np.float32(np.inf if rng.random() < 0.5 else -np.inf)
        t = np.float32(g0)
        for _ in range(k):
            t = np.nextafter(t, direction, dtype=np.float32)
            if t == 0:           # +0 and -0 are one value: step over the other zero
                t = np.float32(0.0)
        sig = oracle.signature(np.array([g0], np.float32), np.array([t], np.float32), thresholds=())
        assert sig["max_ulp"] == k, (g0, t, k)


def test_f32_subnormal_pair():
    g = np.array([2.0 ** -149], np.float32)
    t = np.array([2.0 ** -148], np.float32)
    sig = oracle.signature(g, t)
    assert sig["max_ulp"] == 1 and sig["max_abs"] == 2.0 ** -149 and sig["hist_under"] == 1
    assert sig["max_rel"] == 1.0


def test_f32_identical_tensors():
    rng = np.random.default_rng(3)
    g = rng.standard_normal(100000).astype(np.float32)
    g[[5, 77]] = np.nan
    g[[9]] = np.inf
    sig = oracle.signature(g, g.copy())
    st = oracle.stats(sig)
    assert sig["hist_zero"] == sig["n_valid"] == g.size - 2
    assert sig["max_abs"] == 0.0 and sig["argmax_abs"] == 0
    assert sig["max_ulp"] == 0 and sig["argmax_ulp"] == 0 and sig["sum_ulp"] == 0
    assert sig["max_rel"] == 0.0 and sig["argmax_rel"] == 0
    assert sig["n_mismatch"] == [2, 2] and sig["first_nan_index"] == 5
    assert sig["sum_abs"] == 0.0 and sig["sum_sq"] == 0.0
    assert sig["sum_g2"] == sig["sum_t2"] == sig["sum_gt"]
    assert st["cos"] == 1.0                          # sqrt(RN(S*S)) == S exactly
    assert st["var_abs"] == 0.0 and st["mean_abs"] == 0.0


def test_f32_sums_against_fsum_and_fraction():
    rng = np.random.default_rng(21)
    g = (rng.standard_normal(20000) * rng.choice([1e-3, 1.0, 50.0], 20000)).astype(np.float32)
    t = (g.astype(np.float64) * (1 + 1e-3 * rng.standard_normal(20000))).astype(np.float32)
    sig = oracle.signature(g, t)
    G, T = g.astype(np.float64), t.astype(np.float64)
    a = [X.fraction_abs_diff(x, y) for x, y in zip(G, T)]
    assert _close_ulps(sig["sum_abs"], math.fsum(a))
    assert _close_ulps(sig["sum_sq"], math.fsum(x * x for x in a))
    assert _close_ulps(sig["sum_g2"], float(sum(Fraction(x) ** 2 for x in G)))
    assert _close_ulps(sig["sum_t2"], float(sum(Fraction(x) ** 2 for x in T)))
    assert _close_ulps(sig["sum_gt"], float(sum(Fraction(x) * Fraction(y) for x, y in zip(G, T))))
    rel = [float(Fraction(ai) / abs(Fraction(x))) for ai, x in zip(a, G) if x != 0]
    assert _close_ulps(sig["sum_rel"], math.fsum(rel))
    j = int(np.argmax(rel))
    assert sig["max_rel"] == rel[j]


def test_f32_stats_against_torch_float64():
    rng = np.random.default_rng(8)
    g = rng.standard_normal(50000).astype(np.float32)
    t = (g + 1e-4 * rng.standard_normal(50000)).astype(np.float32)
    sig = oracle.signature(g, t)
    st = oracle.stats(sig)
    G, T = torch.from_numpy(g).double(), torch.from_numpy(t).double()
    A = (T - G).abs()
    rel = lambda x, y: abs(x - y) <= 1e-12 * abs(y)
    assert rel(st["mean_abs"], A.mean().item())
    assert abs(st["var_abs"] - A.var().item()) <= 1e-12 * (A * A).mean().item()
    assert rel(st["l2_err"], torch.linalg.norm(A).item())
    assert rel(st["l2_g"], torch.linalg.norm(G).item())
    assert rel(st["l2_t"], torch.linalg.norm(T).item())
    cs = torch.nn.functional.cosine_similarity(G, T, dim=0, eps=0.0).item()
    assert abs(st["cos"] - cs) <= 1e-13          # torch's own rounding is ~1e-14
    # exact: products of binary32 values are exact rationals; one final rounding
    sg = sum(Fraction(float(x)) ** 2 for x in g)
    stt = sum(Fraction(float(x)) ** 2 for x in t)
    sgt = sum(Fraction(float(x)) * Fraction(float(y)) for x, y in zip(g, t))
    from decimal import Decimal, getcontext
    getcontext().prec = 60
    exact_cos = (Decimal(sgt.numerator) / Decimal(sgt.denominator)) / (
        (Decimal(sg.numerator) / Decimal(sg.denominator)) *
        (Decimal(stt.numerator) / Decimal(stt.denominator))).sqrt()
    assert abs(st["cos"] - float(exact_cos)) <= 4 * 2.0 ** -53
    assert rel(st["mean_rel"], (A / G.abs()).mean().item())


def test_bf16_rounding_workload_properties():
    """t = bf16_RNE(g): the low 16 bits of t are zero, the ULP distance is at
    most 2^15 (exactly 2^15 only at ties) and the relative error is <= 2^-8."""
    rng = np.random.default_rng(2)
    g = rng.standard_normal(200000).astype(np.float32)
    # exact ties: binary32 values in [1, 2) halfway between two bf16 values
    g[:64] = (((np.arange(64, dtype=np.uint32) + 0x3F80) << 16) | 0x8000).view(np.float32)
    t = torch.from_numpy(g).to(torch.bfloat16).float().numpy()
    assert np.all(t.view(np.uint32) & 0xFFFF == 0)
    sig = oracle.signature(g, t)
    assert sig["max_ulp"] <= 32768 and sig["max_rel"] <= 2.0 ** -8
    ties = sig["max_ulp"] == 32768
    assert ties


def test_empty_and_degenerate():
    e = np.zeros(0, np.float32)
    sig = oracle.signature(e, e)
    assert sig["n"] == 0 and sig["argmax_abs"] == -1 and math.isnan(sig["max_abs"])
    assert math.isnan(sig["max_rel"]) and sig["argmax_rel"] == -1 and sig["first_nan_index"] == -1
    assert sig["max_ulp"] == 0 and sig["argmax_ulp"] == -1
    nan = np.full(10, np.nan, np.float32)
    sig = oracle.signature(nan, nan)
    assert sig["n_nan_pairs"] == 10 and sig["n_valid"] == 0 and sig["first_nan_index"] == 0
    assert sig["n_mismatch"] == [10, 10] and sig["argmax_abs"] == -1


def test_signature_argument_validation():
    ok = (-40, 24, 64)
    assert oracle.signature_rc(None, None, 0, oracle.F32, ok, (1e-6,)) == oracle.OK
    assert oracle.signature_rc(None, None, 5, oracle.F32, ok, (1e-6,)) == oracle.EINVAL
    assert oracle.signature_rc(None, None, -1, oracle.F32, ok, (1e-6,)) == oracle.EINVAL
    assert oracle.signature_rc(None, None, 0, 7, ok, (1e-6,)) == oracle.EDTYPE
    for bad in [(-40, 24, 0), (-40, 24, 65), (-40, 24, 7), (10, 10, 1), (-1023, 0, 1), (0, 1025, 1)]:
        assert oracle.signature_rc(None, None, 0, oracle.F32, bad, ()) == oracle.EINVAL, bad
    assert oracle.signature_rc(None, None, 0, oracle.F32, ok, (math.nan,)) == oracle.EINVAL
    assert oracle.signature_rc(None, None, 0, oracle.F32, ok, (-1.0,)) == oracle.EINVAL
    assert oracle.signature_rc(None, None, 0, oracle.F32, ok, (0.0,) * 9) == oracle.EINVAL


# ---------------------------------------------------------------------------
# Injector.
# ---------------------------------------------------------------------------
def _ref_flips(n, seed, rate, mask):
    """Flip set and bits from rocRAND's Philox4x32-10 and the per-element
    uniform's composition: top byte = byte (i mod 16) of block i/16 of stream
    0; low 56 bits = 64-bit word (i mod 2) of block i/2 of stream 1; the bit
    from word 0 of block i of stream 2."""
    i = np.arange(n, dtype=np.uint64)
    A = philox_ref.seeded(seed, np.arange((n + 15) // 16), 0)
    B = philox_ref.seeded(seed, np.arange((n + 1) // 2), 1).astype(np.uint64)
    byte = (i & np.uint64(15)).astype(np.int64)
    word = A[(i >> np.uint64(4)).astype(np.int64), byte >> 2].astype(np.uint64)
    top = (word >> (np.uint64(8) * (byte & 3).astype(np.uint64))) & np.uint64(0xFF)
    h = (i & np.uint64(1)).astype(np.int64)
    rows = B[(i >> np.uint64(1)).astype(np.int64)]
    w64 = rows[np.arange(n), 2 * h] | (rows[np.arange(n), 2 * h + 1] << np.uint64(32))
    U = (top << np.uint64(56)) | (w64 & np.uint64((1 << 56) - 1))
    if rate >= 1:
        flip = np.ones(n, bool)
    else:
        T = math.floor(Fraction(rate) * (1 << 64))
        flip = U < np.uint64(T) if T < (1 << 64) else np.ones(n, bool)
    setbits = [b for b in range(64) if (mask >> b) & 1]
    p = len(setbits)
    idx = np.nonzero(flip)[0]
    C = philox_ref.seeded(seed, idx, 2) if idx.size else np.zeros((0, 4), np.uint32)
    bits = {int(k): setbits[(int(C[r, 0]) * p) >> 32] for r, k in enumerate(idx)}
    return flip, bits


@needs_ref
@pytest.mark.parametrize("rate,n", [(0.01, 20000), (2e-3, 50000), (0.3, 3000), (2.0 ** -56 * 5, 1000),
                                    (1e-3, 33)])
def test_inject_matches_rocrand_philox(rate, n):
    seed = 0xC0FFEE00 + 17 + (5 << 40)
    mask = 0x7F800000
    x = np.random.default_rng(1).standard_normal(n).astype(np.float32).view(np.uint32)
    before = x.copy()
    cnt = oracle.inject(x, seed=seed, rate=rate, mask=mask)
    flip, bits = _ref_flips(n, seed, rate, mask)
    changed = before != x
    assert np.array_equal(changed, flip) and cnt == int(flip.sum())
    for idx, b in bits.items():
        assert int(before[idx] ^ x[idx]) == 1 << b
        assert oracle.inject_decide(idx, oracle.F32, seed, rate, mask) == (True, b)


def test_inject_rate_edges_and_masks():
    x = np.arange(1000, dtype=np.uint32)
    y = x.copy()
    assert oracle.inject(y, seed=3, rate=0.0, mask=0xFFFFFFFF) == 0 and np.array_equal(x, y)
    assert oracle.inject(y, seed=3, rate=1.0, mask=1 << 7) == 1000
    assert np.array_equal(y, x ^ np.uint32(1 << 7))
    z = x.copy()
    cnt = oracle.inject(z, seed=3, rate=float(np.nextafter(1.0, 0.0)), mask=0xF0)
    assert cnt == 1000  # T = 2^64 - 2048: no 64-bit uniform among 1000 reaches it
    assert np.all(((x ^ z) & ~np.uint32(0xF0)) == 0)
    assert np.all(np.array([bin(int(v)).count("1") for v in (x ^ z)]) == 1)


def test_inject_involution_and_dtype_independence():
    n = 100000
    seed, rate, mask = 99, 1e-3, 0x3FF
    a32 = np.random.default_rng(0).standard_normal(n).astype(np.float32).view(np.uint32)
    a16 = np.random.default_rng(1).standard_normal(n).astype(np.float16).view(np.uint16)
    b32, b16 = a32.copy(), a16.copy()
    c1 = oracle.inject(b32, seed=seed, rate=rate, mask=mask)
    c2 = oracle.inject(b16, dtype=oracle.F16, seed=seed, rate=rate, mask=mask)
    assert c1 == c2 > 0
    assert np.array_equal(np.nonzero(a32 != b32)[0], np.nonzero(a16 != b16)[0])
    assert np.array_equal((a32 ^ b32)[a32 != b32], (a16 ^ b16)[a16 != b16].astype(np.uint32))
    oracle.inject(b32, seed=seed, rate=rate, mask=mask)
    assert np.array_equal(a32, b32)


def test_inject_statistics():
    """Count ~ Binomial(n, T/2^64) within 4 sigma; chosen bits uniform over
    the mask (chi-square, 15 degrees of freedom, p ~ 1e-4 cut)."""
    n = 400000
    x = np.zeros(n, np.uint16)
    rate = 0.02
    cnt = oracle.inject(x, dtype=oracle.F16, seed=12345, rate=rate, mask=0xFFFF)
    mu, sd = n * rate, math.sqrt(n * rate * (1 - rate))
    assert abs(cnt - mu) < 4 * sd
    bits = np.log2(x[x != 0].astype(np.float64)).astype(int)
    counts = np.bincount(bits, minlength=16)
    e = cnt / 16
    chi2 = float(((counts - e) ** 2 / e).sum())
    assert chi2 < 44.0, (chi2, counts)


def test_inject_argument_validation():
    assert oracle.inject_rc(10, oracle.F32, 1, 0.5, 0) == oracle.EBITMASK
    assert oracle.inject_rc(10, oracle.F16, 1, 0.5, 0x10000) == oracle.EBITMASK
    assert oracle.inject_rc(10, oracle.F32, 1, 0.5, 1 << 32) == oracle.EBITMASK
    assert oracle.inject_rc(10, oracle.F32, 1, math.nan, 1) == oracle.ERATE
    assert oracle.inject_rc(10, oracle.F32, 1, -1e-9, 1) == oracle.ERATE
    assert oracle.inject_rc(10, 9, 1, 0.5, 1) == oracle.EDTYPE
    assert oracle.inject_rc(0, oracle.F32, 1, 0.5, 1) == 0


# ---------------------------------------------------------------------------
# Closeness with a relative tolerance (torch.isclose with rtol > 0).
# ---------------------------------------------------------------------------
RTOL_SETS = [[(0.0, 1e-3)], [(1e-5, 1e-2), (0.0, 0.5), (1e-3, 0.0)], [(0.0, 2.0 ** -10), (2.0 ** -20, 2.0 ** -11)],
             [(0.0, np.inf), (np.inf, 0.0), (1.0, 1e300)]]


@pytest.mark.parametrize("tset", range(len(RTOL_SETS)))
def test_mismatch_rtol_against_torch_isclose_f16_grid(tset):
    tols = RTOL_SETS[tset]
    t16 = X.all_f16().view(np.float16)             # every binary16 value, NaNs included
    for gv in (0.0, 1.0, -3.5, 1e-4, 65504.0, -np.inf, np.nan):
        G = np.full(t16.shape, gv, dtype=np.float16)
        sig = oracle.signature(G, t16, thresholds=tols)
        tg = torch.from_numpy(G.astype(np.float64))
        tt = torch.from_numpy(t16.astype(np.float64))
        want = [int((~torch.isclose(tt, tg, rtol=r, atol=a, equal_nan=False)).sum()) for a, r in tols]
        assert sig["n_mismatch"] == want, (gv, tols)


def test_mismatch_rtol_random_f32():
    rng = np.random.default_rng(8)
    G = (rng.standard_normal(200000) * 10.0 ** rng.integers(-6, 6, 200000)).astype(np.float32)
    T = (G * (1 + rng.standard_normal(200000) * 10.0 ** rng.integers(-8, 0, 200000))).astype(np.float32)
    T[::997] = -T[::997]
    tols = [(1e-6, 1e-3), (0.0, 1e-5), (1e-9, 1e-7), (1e-3, 0.1)]
    sig = oracle.signature(G, T, thresholds=tols)
    tg = torch.from_numpy(G.astype(np.float64))
    tt = torch.from_numpy(T.astype(np.float64))
    assert sig["n_mismatch"] == [int((~torch.isclose(tt, tg, rtol=r, atol=a, equal_nan=False)).sum())
                                 for a, r in tols]


def test_rtol_validation():
    g = np.zeros(4, np.float32)
    assert oracle.signature_rc(g.ctypes.data, g.ctypes.data, 4, 0, (-40, 24, 64), [(1e-6, -1.0)]) == oracle.EINVAL
    assert oracle.signature_rc(g.ctypes.data, g.ctypes.data, 4, 0, (-40, 24, 64), [(1e-6, float("nan"))]) == oracle.EINVAL
