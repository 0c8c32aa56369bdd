"""GPU parity of mixed-precision pairs (Section III-C: an FP32 golden output
against the same operation run in FP16 or FP64) against the oracle:
peat_signature_mixed, peat_signature_mixed_batched and
peat_topk_mean_mixed_batched for every accepted golden/test combination.
Tolerances as for same-type pairs (tests/parity.py): counts, histograms,
indices, maxima and ULP sums bit-exact, binary64 sums within 1e-12.  Inputs:
test values near the golden ones (the fast path), ties of the narrower
format, values past its range, NaN/Inf/zeros/subnormals, sign changes, equal
pairs; several chunks with ragged tails, unaligned pointers, a 2^24-element
pair, and batches mixing every kind."""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_13544_amd as P
from tests.parity import _SPECIALS, assert_parity, float_to_bits, to_device

pytestmark = pytest.mark.gpu

F32, F16, BF16, F64 = 0, 1, 2, 3
KINDS = [(F32, F64), (F32, F16), (F32, BF16), (F16, F32), (BF16, F32), (F16, F64), (BF16, F64)]
PREC = {F32: 24, F16: 11, BF16: 8, F64: 53}
MAXEXP = {F32: 127, F16: 15, BF16: 127, F64: 1023}
THR = (1e-6, (1e-4, 1e-3), 0.25)


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _device():
    assert torch.cuda.is_available(), "GPU tests need the MI355X"
    P.lib()
    assert oracle.lib()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _values(bits: np.ndarray, code: int) -> np.ndarray:
    if code == F32:
        return bits.view(np.float32).astype(np.float64)
    if code == F16:
        return bits.view(np.float16).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _side(values: np.ndarray, code: int) -> np.ndarray:
    """float64 values as the side's host array (bits, or float64 itself)."""
    return values.copy() if code == F64 else float_to_bits(values, code).copy()


def mixed_pair(n: int, gdt: int, tdt: int, seed: int, rel: float = 1e-3):
    """Seeded golden (bits of gdt) and test (bits of tdt, or float64) arrays."""
    rng = np.random.default_rng(seed)
    r = min(20, MAXEXP[min(gdt, tdt, key=lambda c: MAXEXP[c])] // 2)
    G = rng.standard_normal(n) * np.exp2(rng.integers(-r, r, n)) if n else np.zeros(0)
    gb = float_to_bits(G, gdt).copy()
    Gv = _values(gb, gdt)
    T = Gv * (1.0 + rel * rng.standard_normal(n))
    if n:
        k = max(1, n // 500)
        nar = gdt if PREC[gdt] <= PREC[tdt] else tdt
        with np.errstate(all="ignore"):
            ulp = np.exp2(np.floor(np.log2(np.abs(Gv))) - (PREC[nar] - 1))
            idx = rng.integers(0, n, k)
            T[idx] = Gv[idx] + 0.5 * ulp[idx]                                   # ties of the narrow format
            idx = rng.integers(0, n, k)
            T[idx] = Gv[idx] - 0.5 * ulp[idx] * (1 + 2.0 ** -30)
        idx = rng.integers(0, n, k)
        T[idx] = -Gv[idx]                                                       # sign changes
        idx = rng.integers(0, n, k)
        T[idx] = Gv[idx]                                                        # equal
        if tdt == F64:
            idx = rng.integers(0, n, k)
            T[idx] = math.ldexp(1.0, MAXEXP[gdt] + 1) * rng.uniform(0.5, 1.5, k)  # past the golden range
            idx = rng.integers(0, n, k)
            T[idx] = math.ldexp(1.0, -140) * rng.uniform(-2, 2, k)               # below f32 subnormals
    tb = _side(T, tdt)
    if n:
        sp = _SPECIALS
        for name, val in sp[gdt].items():
            gb[rng.integers(0, n, max(1, n // 2000))] = val
        if tdt == F64:
            for v in (math.nan, math.inf, -math.inf, 0.0, -0.0, 5e-324, 1e200):
                tb[rng.integers(0, n, max(1, n // 2000))] = v
        else:
            for name, val in sp[tdt].items():
                tb[rng.integers(0, n, max(1, n // 2000))] = val
        idx = rng.integers(0, n, max(1, n // 1000))                              # repeated pairs: ties
        src = int(rng.integers(0, n))
        gb[idx] = gb[src]
        tb[idx] = tb[src]
    return gb, tb


def dev(arr: np.ndarray, code: int) -> torch.Tensor:
    if code == F64:
        return torch.from_numpy(arr).cuda()
    return to_device(arr, code)


def ref_sig(gb, tb, gdt, tdt, thr=THR):
    return oracle.signature_mixed(gb, tb, gdtype=gdt, tdtype=tdt, thresholds=thr)


@pytest.mark.parametrize("gdt,tdt", KINDS)
def test_signature_sizes_and_specials(gdt, tdt):
    for i, n in enumerate([0, 1, 5, 2047, 4097, 65536 + 13, 300007, (1 << 20) + 5]):
        log(f"  mixed {gdt}/{tdt} n={n}")
        gb, tb = mixed_pair(n, gdt, tdt, seed=9000 + 31 * i + 7 * gdt + tdt)
        got = P.signature_mixed(dev(gb, gdt), dev(tb, tdt), thresholds=THR)
        assert_parity(got, ref_sig(gb, tb, gdt, tdt), f"{gdt}/{tdt} n={n}")


@pytest.mark.parametrize("gdt,tdt", KINDS)
def test_signature_unaligned_and_wide_noise(gdt, tdt):
    n = 70001
    gb, tb = mixed_pair(n + 1, gdt, tdt, seed=9500 + 7 * gdt + tdt, rel=0.7)   # many rare elements
    g, t = dev(gb, gdt), dev(tb, tdt)
    log(f"  mixed {gdt}/{tdt} unaligned")
    got = P.signature_mixed(g[1:], t[1:], thresholds=THR)                     # 2- or 4-byte offset
    assert_parity(got, ref_sig(gb[1:], tb[1:], gdt, tdt), f"{gdt}/{tdt} unaligned")
    got = P.signature_mixed(g, t, bins=(-160, 136, 37), thresholds=())
    ref = oracle.signature_mixed(gb, tb, gdtype=gdt, tdtype=tdt, bins=(-160, 136, 37), thresholds=())
    assert_parity(got, ref, f"{gdt}/{tdt} wide bins")


def test_signature_large_f32_against_f64():
    n = (1 << 24) + 777
    log(f"  mixed f32/f64 n={n}")
    gb, tb = mixed_pair(n, F32, F64, seed=9901, rel=1e-7)
    got = P.signature_mixed(dev(gb, F32), dev(tb, F64), thresholds=THR)
    assert_parity(got, ref_sig(gb, tb, F32, F64), "f32/f64 large")


def test_same_types_through_the_mixed_entry_point():
    from tests.parity import special_pair
    for code in (F32, F16, BF16):
        gb, tb = special_pair(100003, code, seed=9700 + code)
        g, t = to_device(gb, code), to_device(tb, code)
        a = P.signature_mixed(g, t, thresholds=THR)
        b = P.signature(g, t, thresholds=THR)
        assert all(a[k] == b[k] or (isinstance(a[k], float) and math.isnan(a[k]) and math.isnan(b[k]))
                   for k in a), code


def test_batched_mixes_every_kind_and_matches_single_calls():
    pairs, hosts = [], []
    kinds = KINDS + [(F32, F32), (F16, F16), (BF16, BF16)]
    for i, (gdt, tdt) in enumerate(kinds * 2):
        n = [4096 * 3 + 17, 1000, 0, 250001][i % 4]
        gb, tb = mixed_pair(n, gdt, tdt, seed=9800 + i)
        hosts.append((gb, tb, gdt, tdt))
        pairs.append((dev(gb, gdt), dev(tb, tdt)))
    log(f"  mixed batched {len(pairs)} pairs")
    outs = P.signature_mixed_batched(pairs, thresholds=THR)
    for k, ((g, t), (gb, tb, gdt, tdt)) in enumerate(zip(pairs, hosts)):
        single = P.signature_mixed(g, t, thresholds=THR)
        assert all(outs[k][f] == single[f] or (isinstance(single[f], float) and math.isnan(single[f])
                                               and math.isnan(outs[k][f])) for f in single), k
        assert_parity(outs[k], ref_sig(gb, tb, gdt, tdt), f"batched {k} {gdt}/{tdt}")


def assert_topk(got: dict, ref: dict, ctx: str = ""):
    for key in ("n_valid", "k", "count_above"):
        assert got[key] == ref[key], f"{ctx}: {key} {got[key]} != {ref[key]}"
    for key in ("kth_value", "sum_topk", "mean_topk"):
        a, b = got[key], ref[key]
        if math.isnan(b):
            assert math.isnan(a), f"{ctx}: {key} {a} != NaN"
        elif math.isinf(b) or key == "kth_value":
            assert a == b, f"{ctx}: {key} {a!r} != {b!r}"
        else:
            assert abs(a - b) <= 1e-12 * abs(b), f"{ctx}: {key} {a!r} vs {b!r}"


def test_topk_mixed_every_kind():
    pairs, hosts = [], []
    for i, (gdt, tdt) in enumerate(KINDS):
        for j, n in enumerate([0, 4099, 300001]):
            gb, tb = mixed_pair(n, gdt, tdt, seed=9600 + 10 * i + j)
            hosts.append((gb, tb, gdt, tdt))
            pairs.append((dev(gb, gdt), dev(tb, tdt)))
    sigs = P.signature_mixed_batched(pairs, thresholds=THR)
    for num, den in [(1, 10), (1, 1), (3, 7)]:
        log(f"  mixed top-k {num}/{den} over {len(pairs)} pairs")
        outs = P.topk_mean_mixed_batched(pairs, num, den)
        # given the signatures (one-binade bins): the same records, bit for bit
        fs = P.topk_mean_mixed_from_signature_batched(pairs, sigs, num=num, den=den)
        for k, (gb, tb, gdt, tdt) in enumerate(hosts):
            ref = oracle.topk_mixed(gb, tb, gdtype=gdt, tdtype=tdt, num=num, den=den)
            assert_topk(outs[k], ref, f"{gdt}/{tdt} pair {k} {num}/{den}")
            assert all(fs[k][f] == outs[k][f] or (fs[k][f] != fs[k][f] and outs[k][f] != outs[k][f])
                       for f in outs[k]), f"{gdt}/{tdt} pair {k}: from signature {fs[k]} != {outs[k]}"


def test_topk_and_histogram_of_subnormal_binary64_errors():
    # errors below 2^-1022: the histogram's under slot and a top-k boundary
    # inside binade 0 (the level rounds on subnormal keys), with and without
    # a few normal errors above them
    rng = np.random.default_rng(9990)
    n = 200003
    g = np.zeros(n, np.float32)
    gb = g.view(np.uint32)
    base = rng.integers(0, 1 << 40, n).astype(np.float64) * 5e-324 * rng.choice([-1.0, 1.0], n)
    for variant in ("subnormal only", "with normals"):
        t = base.copy()
        if variant == "with normals":
            t[::1000] = rng.standard_normal(len(t[::1000]))
        pairs = [(dev(gb, F32), dev(t, F64))]
        ref = ref_sig(gb, t, F32, F64)
        assert ref["hist_under"] > n // 2
        assert_parity(P.signature_mixed(*pairs[0], thresholds=THR), ref, variant)
        for num, den in [(1, 10), (1, 2), (1, 1), (1, 1000)]:
            log(f"  {variant} top-k {num}/{den}")
            got = P.topk_mean_mixed_batched(pairs, num, den)[0]
            assert_topk(got, oracle.topk_mixed(gb, t, gdtype=F32, tdtype=F64, num=num, den=den),
                        f"{variant} {num}/{den}")


def test_mixed_index_beyond_2_31():
    """64-bit indexing of a mixed pair: n > 2^31, FP32 golden zeros against a
    binary64 test with planted values at known places (closed forms)."""
    n = (1 << 31) + 4096 + 1000
    base = 1 << 31
    log(f"  mixed f32/f64 n={n}")
    g = torch.zeros(n, dtype=torch.float32, device="cuda")
    t = torch.zeros(n, dtype=torch.float64, device="cuda")
    t[base + 77] = 1.0
    t[base + 500] = -1.0                       # ties |err| = 1 with base + 77
    t[base + 900] = float("nan")
    t[base + 5095] = 0.5 + 2.0 ** -30          # rounds to 0.5 in FP32
    got = P.signature_mixed(g, t, (-40, 24, 64), (1e-6, 1e-3))
    assert got["n"] == n and got["n_nan_pairs"] == 1 and got["first_nan_index"] == base + 900
    assert got["max_abs"] == 1.0 and got["argmax_abs"] == base + 77
    assert got["max_ulp"] == 0x3F800000 and got["argmax_ulp"] == base + 77
    assert got["sum_ulp"] == 2 * 0x3F800000 + 0x3F000000
    assert got["n_rel"] == 0 and math.isnan(got["max_rel"]) and got["argmax_rel"] == -1
    assert got["hist_zero"] == n - 4 and got["hist"][40] == 2 and got["hist"][39] == 1
    assert got["sum_abs"] == 2.5 + 2.0 ** -30 and got["n_mismatch"] == [4, 4]
    tk = P.topk_mean_mixed_batched([(g, t)], 1, 10)[0]
    assert tk["n_valid"] == n - 1 and tk["k"] == -(-(n - 1) // 10)
    assert tk["kth_value"] == 0.0 and tk["count_above"] == 3 and tk["sum_topk"] == 2.5 + 2.0 ** -30
    del g, t
    torch.cuda.empty_cache()


def test_mixed_async_records_match_sync():
    pairs = []
    for i, (gdt, tdt) in enumerate(KINDS):
        gb, tb = mixed_pair(70001 + 13 * i, gdt, tdt, seed=9950 + i)
        pairs.append((dev(gb, gdt), dev(tb, tdt)))
    sync = P.signature_mixed_batched(pairs, thresholds=THR)
    d_out = torch.empty(len(pairs) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    P.signature_mixed_batched_async(pairs, d_out, thresholds=THR, stream=stream)
    stream.synchronize()
    recs = P.decode_records(d_out, len(pairs), nthr=len(THR))
    for a, b in zip(recs, sync):
        assert all(a[k] == b[k] or (isinstance(b[k], float) and math.isnan(b[k]) and math.isnan(a[k])) for k in b)
