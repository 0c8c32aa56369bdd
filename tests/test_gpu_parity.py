"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Every test compares device results element by element with the oracle on the
same seeded inputs: bit-exact for counts, histograms, indices, maxima, ULP
sums and injected bits; 1e-12 for the binary64 sums (see tests/parity.py).
Small cases span several chunks and ragged tails; the workload tests run the
five workloads at full size in the launch configuration the benchmark times
and check sampled tensors (all of a small one, the largest ones) against the
oracle, plus properties that hold at any size.
"""
from __future__ import annotations

import math
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_13544_amd as P
import synth
from tests.parity import (assert_parity, float_to_bits, oracle_sig, records_equal, special_pair, to_device,
                          to_host_bits)

pytestmark = pytest.mark.gpu

BINS_SETS = [synth.BINS, (-30, 20, 25), (-20, 40, 12), (-160, 136, 37)]
THR_SETS = [synth.THRESHOLDS, (), (0.0,), (1e-7, 1e-5, 1e-3, 0.1, 1.0), (0.0, 1e-9, 1e-6, 1e-4, 1e-2, 1.0, 100.0, math.inf),
            # torch.isclose's relative form: (atol, rtol) pairs
            ((1e-6, 1e-3), (0.0, 1e-5)), ((0.0, math.inf), (1e-3, 0.1), (1e-9, 2.0 ** -11), (0.0, 0.0))]


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


def _check_pair(gb, tb, code, bins=synth.BINS, thr=synth.THRESHOLDS, ctx=""):
    g = to_device(gb, code)
    t = to_device(tb, code)
    got = P.signature(g, t, bins, thr)
    ref = oracle_sig(gb, tb, code, bins, thr)
    assert_parity(got, ref, ctx)
    return got


# ---------------------------------------------------------------------------
# signature: sizes, dtypes, specials, bins, thresholds
# ---------------------------------------------------------------------------
SIZES = [0, 1, 3, 4, 7, 9, 255, 4095, 4096, 4097, 8191, 65536 + 13, 300005, (1 << 20) + 3]


@pytest.mark.parametrize("code", [0, 1, 2])
def test_sizes_and_specials(code):
    for i, n in enumerate(SIZES):
        gb, tb = special_pair(n, code, seed=1000 + 17 * i + code)
        log(f"  dtype={code} n={n}")
        _check_pair(gb, tb, code, ctx=f"dtype={code} n={n}")


@pytest.mark.parametrize("code", [0, 1, 2])
def test_bins_and_thresholds(code):
    n = 150001
    for bi, bins in enumerate(BINS_SETS):
        for ti, thr in enumerate(THR_SETS):
            gb, tb = special_pair(n, code, seed=77 + 10 * bi + ti, rel_noise=10.0 ** -(1 + ti))
            log(f"  dtype={code} bins={bins} thr={thr}")
            _check_pair(gb, tb, code, bins, thr, ctx=f"bins={bins} thr={thr}")


@pytest.mark.parametrize("code", [0, 1, 2])
def test_ordinary_data_without_specials(code):
    """The fast path alone (no special values anywhere)."""
    for n in (4096 * 64, 4096 * 300 + 77):
        gb, tb = special_pair(n, code, seed=5 + n, special_frac=0.0, rel_noise=1e-4)
        _check_pair(gb, tb, code, ctx=f"ordinary n={n}")


@pytest.mark.parametrize("code", [0, 1, 2])
def test_unaligned_pointers(code):
    """Views offset by one element are not 16-byte aligned (generic path)."""
    n = 70000
    gb, tb = special_pair(n + 1, code, seed=31 + code)
    g = to_device(gb, code)[1:]
    t = to_device(tb, code)[1:]
    got = P.signature(g, t, synth.BINS, synth.THRESHOLDS)
    assert_parity(got, oracle_sig(gb[1:], tb[1:], code, synth.BINS, synth.THRESHOLDS), "unaligned")
    # golden aligned, test not
    t2 = to_device(np.concatenate([tb[:1], tb[:n]]), code)[1:]
    got = P.signature(to_device(gb[:n], code), t2, synth.BINS, synth.THRESHOLDS)
    assert_parity(got, oracle_sig(gb[:n], tb[:n], code, synth.BINS, synth.THRESHOLDS), "mixed alignment")


def test_degenerate_inputs():
    for code in (0, 1, 2):
        sp = {0: (0x7FC00000, 0x7F800000, 0x3F800000), 1: (0x7E00, 0x7C00, 0x3C00), 2: (0x7FC0, 0x7F80, 0x3F80)}[code]
        dt = np.uint32 if code == 0 else np.uint16
        for n in (1, 5000, 70001):
            for gval, tval in [(sp[0], sp[0]), (sp[2], sp[2]), (0, 0), (sp[1], sp[1]), (sp[1], sp[2]),
                               (sp[2], 0), (0, sp[2])]:
                gb = np.full(n, gval, dt)
                tb = np.full(n, tval, dt)
                _check_pair(gb, tb, code, ctx=f"const {gval:#x}/{tval:#x} n={n}")


def test_workload1_full():
    G, T = synth.config1()
    _check_pair(G.reshape(-1).view(np.uint32), T.reshape(-1).view(np.uint32), 0, ctx="workload 1")


@pytest.mark.parametrize("code", [1, 2])
def test_equal_vectors(code):
    """Test tensors equal to their golden bit for bit over most of the pair
    (the 16-bit kernels' equal-vector branch) with differences planted at a
    low rate (some in a chunk's first vector), special goldens (zero, -0,
    +-Inf, NaN, subnormal, the largest finite) that T repeats, +-0 pairs, and
    bf16 values whose products leave binary32's normal range; each against
    the oracle under absolute and relative thresholds, and single == batched."""
    rng = np.random.default_rng(2609 + code)
    sp = {1: [0x0000, 0x8000, 0x7C00, 0xFC00, 0x7E00, 0x0001, 0x83FF, 0x7BFF],
          2: [0x0000, 0x8000, 0x7F80, 0xFF80, 0x7FC0, 0x0001, 0x807F, 0x7F7F]}[code]
    cases = []
    for n in (4096 * 64 + 4097, (1 << 20) + 3, 300005):
        gb, _ = special_pair(n, code, seed=4400 + n, special_frac=0.0)
        cases.append((f"all equal n={n}", gb, gb.copy()))
        tb = gb.copy()
        idx = rng.integers(0, n, max(1, n // 20000))
        tb[idx] ^= np.asarray(1 << rng.integers(0, 16, idx.size), dtype=np.uint16)
        tb[np.arange(0, n, 4096 * 3)] ^= 1                 # the first element of every third chunk
        cases.append((f"planted flips n={n}", gb, tb))
        g2 = gb.copy()
        for val in sp:
            g2[rng.integers(0, n, 3)] = val
        cases.append((f"special goldens n={n}", g2, g2.copy()))
        t3 = g2.copy()
        z = rng.integers(0, n, 5)
        g2z = g2.copy()
        g2z[z] = 0x0000
        t3[z] = 0x8000                                      # +0 against -0
        cases.append((f"signed zeros n={n}", g2z, t3))
    if code == 2:                                           # bf16 magnitudes near 2^+-120
        n = 70001
        big = float_to_bits(np.exp2(rng.uniform(100, 127, n)) * rng.choice([-1.0, 1.0], n), 2)
        tiny = float_to_bits(np.exp2(rng.uniform(-133, -100, n)), 2)
        cases.append(("bf16 huge", big, big.copy()))
        cases.append(("bf16 tiny", tiny, tiny.copy()))
    thr_rt = ((1e-6, 1e-3), (0.0, 1e-5))
    for ctx, gb, tb in cases:
        log(f"  dtype={code} {ctx}")
        _check_pair(gb, tb, code, ctx=ctx)
        _check_pair(gb, tb, code, thr=thr_rt, ctx=ctx + " rtol")
    dev = [(to_device(gb, code), to_device(tb, code)) for _, gb, tb in cases]
    batched = P.signature_batched(dev, synth.BINS, synth.THRESHOLDS)
    for k, (g, t) in enumerate(dev):
        assert records_equal(batched[k], P.signature(g, t, synth.BINS, synth.THRESHOLDS)), cases[k][0]


def test_batched_equals_single_and_is_deterministic():
    pairs_host = []
    rng = np.random.default_rng(4)
    for k in range(12):
        code = k % 3
        n = int(rng.integers(0, 300000)) if k % 4 else 4096 * 70
        pairs_host.append((code,) + special_pair(n, code, seed=900 + k))
    dev = [(to_device(gb, c), to_device(tb, c)) for c, gb, tb in pairs_host]
    batched = P.signature_batched(dev, synth.BINS, synth.THRESHOLDS)
    again = P.signature_batched(dev, synth.BINS, synth.THRESHOLDS)
    for k, ((c, gb, tb), (g, t)) in enumerate(zip(pairs_host, dev)):
        single = P.signature(g, t, synth.BINS, synth.THRESHOLDS)
        assert single == batched[k] == again[k], f"pair {k}: batched/single/rerun differ"
        assert_parity(batched[k], oracle_sig(gb, tb, c, synth.BINS, synth.THRESHOLDS), f"pair {k}")


def test_batched_mixed_chunk_sizes():
    """A batch whose pairs have chunks of 2^12, 2^13, 2^14, 2^17 and 2^18
    elements, in no order of size, across the three same-type kinds: the
    launch works them largest chunks first, yet every record equals its
    single call bit for bit; the smaller pairs also equal the oracle."""
    spec = [(5000, 0), ((1 << 24) + 7, 0), ((1 << 21) + 3, 1), (1 << 20, 0), ((1 << 22) + 5, 1),
            (600000, 2), (1 << 21, 0), (1 << 23, 1), (3 << 20, 2), ((1 << 24) + 7, 1), (4097, 2)]
    hosts, dev = [], []
    for k, (n, code) in enumerate(spec):
        gb, tb = special_pair(n, code, seed=61000 + k)
        hosts.append((gb, tb, code))
        dev.append((to_device(gb, code), to_device(tb, code)))
    recs = P.signature_batched(dev, synth.BINS, synth.THRESHOLDS)
    for k, ((gb, tb, code), (g, t)) in enumerate(zip(hosts, dev)):
        single = P.signature(g, t, synth.BINS, synth.THRESHOLDS)
        assert records_equal(recs[k], single), f"pair {k} (n={spec[k][0]}): batched and single differ"
        if spec[k][0] <= (1 << 21) + 3:
            assert_parity(recs[k], oracle_sig(gb, tb, code, synth.BINS, synth.THRESHOLDS), f"pair {k}")
    del dev
    torch.cuda.empty_cache()


def test_async_records_match_sync():
    gb, tb = special_pair(123457, 1, seed=3)
    g, t = to_device(gb, 1), to_device(tb, 1)
    d_out = torch.empty(3 * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        P.signature_batched_async([(g, t), (t, g), (g, g)], d_out, synth.BINS, synth.THRESHOLDS, stream=s)
    s.synchronize()
    recs = P.decode_records(d_out, 3, nthr=2)
    sync = P.signature_batched([(g, t), (t, g), (g, g)], synth.BINS, synth.THRESHOLDS)
    assert recs == sync


@pytest.mark.parametrize("code", [0, 1])
def test_block_chunk_sequences(code):
    """A batch with enough chunks (over 16 per resident block) that blocks take
    two consecutive chunks: chunks without a full super-step (short pairs,
    unaligned pairs) alternate with full and ragged chunks, runs of two chunks
    of one pair with runs that cross pairs, with and without special values.
    Every record equals its single call (one chunk per block) and the oracle."""
    sizes = [2048, 3 * 4096, 4096 + 904, 20000, 4095, 9000]
    hosts, dev = [], []
    for k in range(7000):
        n = sizes[k % len(sizes)]
        gb, tb = special_pair(n, code, seed=50000 + k, special_frac=1e-3 if k % 3 == 0 else 0.0)
        g, t = to_device(gb, code), to_device(tb, code)
        if k % 7 == 3:                  # not 16-byte aligned: no super-steps
            g, t = to_device(np.concatenate([gb[:1], gb]), code)[1:], to_device(np.concatenate([tb[:1], tb]), code)[1:]
        hosts.append((gb, tb))
        dev.append((g, t))
    recs = P.signature_batched(dev, synth.BINS, synth.THRESHOLDS)
    for k, ((gb, tb), (g, t)) in enumerate(zip(hosts, dev)):
        single = P.signature(g, t, synth.BINS, synth.THRESHOLDS)
        assert all(recs[k][f] == v or (isinstance(v, float) and math.isnan(v) and math.isnan(recs[k][f]))
                   for f, v in single.items()), f"pair {k}: batched and single differ"
        assert_parity(recs[k], oracle_sig(gb, tb, code, synth.BINS, synth.THRESHOLDS), f"pair {k}")


def test_chunk_size_rule_boundaries():
    """Pairs on both sides of the switch from ~256 to ~64 chunks per pair
    (2^22 elements) and at the 2^18-element chunk cap, against the oracle;
    batched records equal the single calls."""
    pairs, hosts = [], []
    for i, n in enumerate([(1 << 22) - 1, 1 << 22, (1 << 22) + 1, (1 << 24) - 3, (1 << 24) + 4097]):
        log(f"  f32 n={n}")
        gb, tb = special_pair(n, 0, seed=7700 + i)
        g, t = to_device(gb, 0), to_device(tb, 0)
        got = P.signature(g, t, synth.BINS, synth.THRESHOLDS)
        assert_parity(got, oracle_sig(gb, tb, 0, synth.BINS, synth.THRESHOLDS), f"n={n}")
        pairs.append((g, t))
        hosts.append(got)
    outs = P.signature_batched(pairs, synth.BINS, synth.THRESHOLDS)
    for a, b in zip(outs, hosts):
        assert all(a[k] == b[k] or (isinstance(b[k], float) and math.isnan(b[k]) and math.isnan(a[k])) for k in b)


def test_index_beyond_2_31():
    """64-bit indexing: n > 2^31 f16 elements, planted values at known places."""
    n = (1 << 31) + 4096 + 1000
    g = torch.zeros(n, dtype=torch.float16, device="cuda")
    t = torch.zeros(n, dtype=torch.float16, device="cuda")
    base = 1 << 31
    t[base + 77] = 1.0
    t[base + 500] = -1.0          # ties |err| = 1 with base+77; sign differs from +0
    t[base + 900] = float("nan")
    t[base + 4096 + 999] = 0.5
    got = P.signature(g, t, synth.BINS, synth.THRESHOLDS)
    assert got["n"] == n and got["n_nan_pairs"] == 1 and got["first_nan_index"] == base + 900
    assert got["max_abs"] == 1.0 and got["argmax_abs"] == base + 77
    assert got["argmax_ulp"] == base + 77 and got["max_ulp"] == 0x3C00
    assert got["n_rel"] == 0 and math.isnan(got["max_rel"]) and got["argmax_rel"] == -1
    assert got["hist_zero"] == n - 4 and got["hist"][40] == 2 and got["hist"][39] == 1
    assert got["sum_abs"] == 2.5 and got["sum_sq"] == 2.25 and got["sum_ulp"] == 2 * 0x3C00 + 0x3800
    assert got["n_mismatch"] == [4, 4]
    del g, t
    torch.cuda.empty_cache()


@pytest.mark.parametrize("m", [255, 256, 257, 512])
def test_finalize_batch_boundaries(m):
    """Pairs of m chunks of 2^18 f16 elements around the finalize's batches
    of 256 records: values planted in the first, 256th, 257th and last
    chunks, with ties across batches (the lowest index must win)."""
    c = 1 << 18
    n = m * c
    g = torch.zeros(n, dtype=torch.float16, device="cuda")
    t = torch.zeros(n, dtype=torch.float16, device="cuda")
    plant = {3: 0.5, n - 1: -0.5}                # first and last chunk: |err| 0.5
    if m > 255:
        plant[255 * c + 7] = 0.5                 # the 256th chunk, last of the first batch
    if m > 256:
        plant[256 * c + 9] = -0.5                # the 257th, first of the second batch
    for i, v in plant.items():
        t[i] = v
    t[n - 2] = float("nan")
    got = P.signature(g, t, synth.BINS, synth.THRESHOLDS)
    k = len(plant)
    assert got["n"] == n and got["n_valid"] == n - 1 and got["n_nan_pairs"] == 1
    assert got["first_nan_index"] == n - 2 and got["n_nan_test"] == 1
    assert got["max_abs"] == 0.5 and got["argmax_abs"] == 3
    assert got["max_ulp"] == 0x3800 and got["argmax_ulp"] == 3
    assert got["hist_zero"] == n - 1 - k and got["hist"][39] == k
    assert got["sum_abs"] == 0.5 * k and got["sum_sq"] == 0.25 * k and got["sum_ulp"] == k * 0x3800
    assert got["n_mismatch"] == [k + 1, k + 1]
    del g, t
    torch.cuda.empty_cache()


def test_more_than_16384_chunks():
    """A pair of more than 2^32 f16 elements (16385 chunks of 2^18): the
    finalize reads its records in many batches and forms the counts in
    binary64 (beyond 2^31 per wave); planted values near both ends."""
    n = (1 << 32) + (1 << 18) + 123
    g = torch.zeros(n, dtype=torch.float16, device="cuda")
    t = torch.zeros(n, dtype=torch.float16, device="cuda")
    t[5] = 2.0
    t[n - 7] = -2.0               # ties |err| = 2 with index 5
    t[n - 3] = float("inf")
    t[(1 << 32) + 11] = 0.25
    got = P.signature(g, t, synth.BINS, synth.THRESHOLDS)
    assert got["n"] == n and got["n_valid"] == n and got["n_finite"] == n - 1 and got["n_inf_test"] == 1
    assert got["n_nan_pairs"] == 0 and got["first_nan_index"] == -1
    assert got["max_abs"] == math.inf and got["argmax_abs"] == n - 3
    assert got["argmax_ulp"] == n - 3 and got["max_ulp"] == 0x7C00
    assert got["n_rel"] == 0 and math.isnan(got["max_rel"]) and got["argmax_rel"] == -1
    assert got["hist_zero"] == n - 4 and got["hist_over"] == 1
    assert got["hist"][41] == 2 and got["hist"][38] == 1
    assert got["sum_abs"] == 4.25 and got["sum_sq"] == 8.0625
    assert got["sum_ulp"] == 2 * 0x4000 + 0x3400 + 0x7C00
    assert got["n_mismatch"] == [4, 4]
    del g, t
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# injector
# ---------------------------------------------------------------------------
INJ_RATES = [0.0, 1e-7, 1e-3, 0.01, 0.3, 1.0, float(np.nextafter(1.0, 0.0))]


@pytest.mark.parametrize("code", [0, 1, 2])
def test_inject_parity(code):
    masks = {0: [0x7F800000, 0xFFFFFFFF, 1 << 31, 0x5], 1: [0xFFFF, 0x7C00, 1], 2: [0xFFFF, 0x7F80, 0x8000]}[code]
    for n in (1, 33, 4097, (1 << 20) + 7, 3 * (1 << 20)):
        for ri, rate in enumerate(INJ_RATES):
            mask = masks[(n + ri) % len(masks)]
            seed = synth.inject_seed(9, 31 * ri + n % 1000)
            gb, _ = special_pair(n, code, seed=n + ri)
            x = to_device(gb, code)
            log(f"  dtype={code} n={n} rate={rate} mask={mask:#x}")
            cnt = P.inject(x, seed=seed, rate=rate, bitmask=mask)
            host = gb.copy()
            cnt_ref = oracle.inject(host, dtype=code, seed=seed, rate=rate, mask=mask)
            assert cnt == cnt_ref, (n, rate, cnt, cnt_ref)
            assert np.array_equal(to_host_bits(x), host), f"bits differ n={n} rate={rate}"


def test_inject_batched_involution_and_async():
    items_host = []
    for k in range(7):
        code = k % 3
        n = [5, 4096, 100003, 1 << 20, (1 << 21) + 9, 0, 77][k]
        gb, _ = special_pair(n, code, seed=40 + k)
        items_host.append((code, gb, synth.inject_seed(9, 500 + k), [1e-3, 2e-2, 1e-7, 1.0, 5e-4, 0.5, 0.0][k],
                           {0: 0x7F800000, 1: 0xFFFF, 2: 0x7FFF}[code]))
    xs = [to_device(gb, c) for c, gb, *_ in items_host]
    counts = P.inject_batched([(x, s, r, m) for x, (_, _, s, r, m) in zip(xs, items_host)])
    for k, ((c, gb, s, r, m), x) in enumerate(zip(items_host, xs)):
        host = gb.copy()
        assert counts[k] == oracle.inject(host, dtype=c, seed=s, rate=r, mask=m)
        assert np.array_equal(to_host_bits(x), host)
    # async, same seeds again: restores the inputs
    d_counts = torch.empty(len(xs), dtype=torch.int64, device="cuda")
    P.inject_batched_async([(x, s, r, m) for x, (_, _, s, r, m) in zip(xs, items_host)], d_counts)
    torch.cuda.synchronize()
    assert d_counts.cpu().tolist() == counts
    for (c, gb, *_), x in zip(items_host, xs):
        assert np.array_equal(to_host_bits(x), gb)


# ---------------------------------------------------------------------------
# the five workloads
# ---------------------------------------------------------------------------
def test_workload2_full_sampled():
    """32 pairs of f32 [8, 512, 4096], bf16 rounding: one batched call; three
    pairs checked in full against the oracle, bf16 properties on every pair."""
    pairs = synth.config2_all("cuda")
    log("  workload 2 generated")
    recs = P.signature_batched(pairs, synth.BINS, synth.THRESHOLDS)
    for k in (0, 13, 31):
        G, T = pairs[k]
        ref = oracle_sig(to_host_bits(G), to_host_bits(T), 0, synth.BINS, synth.THRESHOLDS)
        assert_parity(recs[k], ref, f"workload 2 pair {k}")
    for r in recs:
        assert r["max_ulp"] <= 32768 and r["max_rel"] <= 2.0 ** -8 and r["n_valid"] == r["n"]
    del pairs
    torch.cuda.empty_cache()


def test_workload3_full_sampled():
    tensors = synth.config3_all("cuda")
    log("  workload 3 generated")
    recs = P.signature_batched([(G, T) for _, G, T in tensors], synth.BINS, synth.THRESHOLDS)
    sample = [0, 1, 2, 3, 4, 5, 9, 100, 289, 290, 291]
    for k in sample:
        name, G, T = tensors[k]
        ref = oracle_sig(to_host_bits(G), to_host_bits(T), 0, synth.BINS, synth.THRESHOLDS)
        assert_parity(recs[k], ref, f"workload 3 {name}")
    total_nan = sum(r["n_nan_test"] for r in recs)
    assert total_nan == sum(int(torch.isnan(T).sum()) for _, _, T in tensors)
    del tensors
    torch.cuda.empty_cache()


def _pool_map(fn, items, what: str):
    """fn over items on a thread pool (the oracle's C calls release the GIL),
    sized to the host share of one GPU; logs progress."""
    from concurrent.futures import ThreadPoolExecutor
    out = []
    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        for j, r in enumerate(ex.map(fn, items)):
            out.append(r)
            if (j + 1) % 20 == 0 or j + 1 == len(items):
                log(f"    {what}: {j + 1}/{len(items)}")
    return out


def test_workload4_replay():
    """The replay workload in full: 1000 replayed f16 [4096, 4096] calls of
    one golden output (33.5 GB of test tensors), every 10th injected at rate
    1e-7 over all 16 bits by one batched injection, then one batched
    signature over all 1000 calls (the workload's small-launch batched path).
    Every injected call (100) is checked against the oracle: flip count,
    flipped positions and bits, record.  The 900 others are untouched and
    give the closed form of identical tensors.  Single async calls on one
    stream give the same records (30 calls)."""
    G = synth.config4_golden("cuda")
    gb = to_host_bits(G).reshape(-1)
    calls = synth.CONFIG4_CALLS
    tests = [G.clone() for _ in range(calls)]
    inj = [c for c in range(calls) if synth.config4_injected(c)]
    assert len(inj) == 100
    counts = P.inject_batched([(tests[c], synth.inject_seed(4, c), synth.CONFIG4_RATE, synth.CONFIG4_MASK)
                               for c in inj])
    recs = P.signature_batched([(G, T) for T in tests], synth.BINS, synth.THRESHOLDS)
    log(f"  workload 4: {sum(counts)} flips in {len(inj)} injected calls")
    G16 = G.view(torch.int16).view(-1)
    diffs = {}
    for c in inj:                                  # flipped positions and bits on the device
        t16 = tests[c].view(torch.int16).view(-1)
        idx = torch.nonzero(t16 != G16).flatten()
        diffs[c] = (idx.cpu().numpy(), t16[idx].cpu().numpy().view(np.uint16))

    def ref(c):
        tb = gb.copy()
        n = oracle.inject(tb, dtype=1, seed=synth.inject_seed(4, c), rate=synth.CONFIG4_RATE,
                          mask=synth.CONFIG4_MASK)
        pos = np.nonzero(tb != gb)[0]
        return n, pos, tb[pos], oracle_sig(gb, tb, 1, synth.BINS, synth.THRESHOLDS)

    for j, (c, (n, pos, bits, sig)) in enumerate(zip(inj, _pool_map(ref, inj, "oracle calls"))):
        assert n == counts[j], (c, n, counts[j])
        assert np.array_equal(diffs[c][0], pos) and np.array_equal(diffs[c][1], bits), f"call {c}: flipped bits"
        assert_parity(recs[c], sig, f"call {c}")
    plain = [c for c in range(calls) if not synth.config4_injected(c)]
    for c in plain:
        r = recs[c]
        assert records_equal(r, recs[plain[0]]), f"call {c}"
    r = recs[plain[0]]
    n = G.numel()
    assert r["n"] == n and r["hist_zero"] == r["n_valid"] == n - r["n_nan_pairs"]
    assert r["max_ulp"] == 0 and r["sum_ulp"] == 0 and r["max_abs"] == 0.0 and r["sum_abs"] == 0.0
    assert r["n_mismatch"][:2] == [r["n_nan_pairs"]] * 2
    # single async calls on one stream give the same records
    sub = list(range(30))
    d_out = torch.empty(len(sub) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    prepared = [P.PreparedPairs([(G, tests[c])]) for c in sub]
    for j in range(len(sub)):
        P.signature_batched_async(prepared[j], d_out[j * P.SIG_BYTES:], synth.BINS, synth.THRESHOLDS)
    torch.cuda.synchronize()
    single = P.decode_records(d_out, len(sub), nthr=2)
    assert all(records_equal(single[j], recs[c]) for j, c in enumerate(sub))
    del tests, G, prepared
    torch.cuda.empty_cache()


def test_workload5_full_sampled():
    """The Llama-7B-shaped pair (873 f32 tensors, 161.7 GB on device) in the
    benchmark's own launch: one fused injection + signature call over all 873
    pairs (rate 1e-8, exponent bits; about 77k chunks, so every block takes
    two chunks).  Every record equals peat_signature_batched's over the
    flipped tensors afterwards; sampled tensors (all three states of the
    smallest and largest shapes) match the oracle's injection and signature;
    the injection kernel with the same seeds returns the same count for every
    tensor and restores the sampled tensors' original bits."""
    from tests.parity import TWO_CHUNK_MIN, chunk_count
    tensors = synth.config5_all("cuda")
    log(f"  workload 5 generated: {torch.cuda.memory_allocated() / 1e9:.1f} GB")
    pairs = [(G, T) for _, _, G, T in tensors]
    assert sum(chunk_count(G.numel()) for G, _ in pairs) >= TWO_CHUNK_MIN
    names = [name for name, *_ in tensors]
    sample = [k for k, nm in enumerate(names) if nm in ("l0.in_norm", "norm", "l0.q", "l31.down", "embed")]
    pre = {k: (to_host_bits(tensors[k][2]), to_host_bits(tensors[k][3])) for k in sample}
    seeds = [synth.inject_seed(5, k) for k in range(len(pairs))]
    d_out = torch.empty(len(pairs) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    d_counts = torch.empty(len(pairs), dtype=torch.int64, device="cuda")
    P.profile_enable(True)
    P.profile_read(P.K_SIG_INJECT)
    P.inject_signature_batched_async(P.PreparedPairs(pairs), seeds, synth.CONFIG5_RATE, synth.CONFIG5_MASK,
                                     d_out, d_counts, synth.BINS, synth.THRESHOLDS)
    torch.cuda.synchronize()
    assert P.profile_read(P.K_SIG_INJECT)[1] == 1, "expected the fused pass"
    P.profile_enable(False)
    recs = P.decode_records(d_out, len(pairs), nthr=len(synth.THRESHOLDS))
    counts = d_counts.cpu().tolist()
    log(f"  workload 5: {sum(counts)} flips")
    again = P.signature_batched(pairs, synth.BINS, synth.THRESHOLDS)
    bad = [k for k in range(len(pairs)) if not records_equal(recs[k], again[k])]
    assert not bad, f"fused records differ from the signature of the flipped tensors: {bad[:10]}"
    flipped = {k: to_host_bits(tensors[k][3]) for k in sample}

    def ref(k):
        gbits, tbits = pre[k]
        tb = tbits.copy()
        n = oracle.inject(tb, dtype=0, seed=seeds[k], rate=synth.CONFIG5_RATE, mask=synth.CONFIG5_MASK)
        return n, tb, oracle_sig(gbits, tb, 0, synth.BINS, synth.THRESHOLDS)

    for k, (n, tb, sig) in zip(sample, _pool_map(ref, sample, "oracle tensors")):
        name, state = tensors[k][0], tensors[k][1]
        assert n == counts[k], (name, state, n, counts[k])
        assert np.array_equal(flipped[k], tb), f"{name}/{state}: injected bits differ"
        assert_parity(recs[k], sig, f"{name}/{state}")
    # the injection kernel with the same seeds: same decisions, flips undone
    undo = P.inject_batched([(T, s, synth.CONFIG5_RATE, synth.CONFIG5_MASK) for (_, T), s in zip(pairs, seeds)])
    assert undo == counts
    for k in sample:
        assert np.array_equal(to_host_bits(tensors[k][3]), pre[k][1]), f"{names[k]}: not restored"
    for r in recs:
        assert r["n_nan_pairs"] == 0 or r["n_nan_test"] > 0
        assert r["hist_zero"] + r["hist_under"] + sum(r["hist"]) + r["hist_over"] == r["n_valid"]
    del tensors, pairs
    torch.cuda.empty_cache()


def test_threads_on_their_own_streams():
    """Calls from several host threads, each on its own stream (the stream is
    per thread), give the same records as the same calls made one by one."""
    import threading
    cases = []
    for i in range(6):
        gb, tb = special_pair(300007 + 1000 * i, i % 3, seed=8800 + i)
        cases.append((to_device(gb, i % 3), to_device(tb, i % 3)))
    want = [P.signature(g, t, synth.BINS, synth.THRESHOLDS) for g, t in cases]
    got = [None] * len(cases)
    errors = []

    def work(k):
        try:
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                for _ in range(3):
                    got[k] = P.signature(cases[k][0], cases[k][1], synth.BINS, synth.THRESHOLDS)
        except Exception as e:  # reported below
            errors.append(e)

    torch.cuda.synchronize()
    threads = [threading.Thread(target=work, args=(k,)) for k in range(len(cases))]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors, errors
    for a, b in zip(got, want):
        assert all(a[k] == b[k] or (isinstance(b[k], float) and math.isnan(b[k]) and math.isnan(a[k])) for k in b)
