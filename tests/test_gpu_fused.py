"""GPU parity of the fused injection + signature pass
(peat_inject_signature_batched_async): its records, flip counts and flipped
test tensors against the CPU oracle's injection followed by the oracle's
signature, and bit for bit against the library's separate calls
(peat_inject_batched then peat_signature_batched)."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_13544_amd as P
import synth
from tests.parity import (NP_BITS, TORCH_INT, TWO_CHUNK_MIN, _SPECIALS, assert_parity, chunk_count, float_to_bits,
                          oracle_sig, special_pair, to_device, to_host_bits)


pytestmark = pytest.mark.gpu

MASKS = {0: [0x7F800000, 0xFFFFFFFF, 1 << 31], 1: [0xFFFF, 0x7C00, 1], 2: [0xFFFF, 0x7F80, 0x8000]}


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


def _same(a: dict, b: dict) -> bool:
    return all(a[k] == v or (isinstance(v, float) and v != v and a[k] != a[k]) for k, v in b.items())


def _fused(dev_pairs, seeds, rate, mask):
    d_out = torch.empty(len(dev_pairs) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    d_counts = torch.full((len(dev_pairs),), -1, dtype=torch.int64, device="cuda")
    P.inject_signature_batched_async(dev_pairs, seeds, rate, mask, d_out, d_counts, synth.BINS, synth.THRESHOLDS)
    torch.cuda.synchronize()
    return P.decode_records(d_out, len(dev_pairs), nthr=len(synth.THRESHOLDS)), d_counts.cpu().tolist()


@pytest.mark.parametrize("code", [0, 1, 2])
def test_fused_against_oracle(code):
    """Sizes spanning one and several chunks with ragged tails, every
    injection regime (top-byte filter, general threshold, every element,
    none), masks of one and many bits, special values in the data."""
    cases = [(1, 1e-3), (33, 0.3), (4097, 2e-2), (70001, 1e-3), ((1 << 20) + 7, 5e-4), (3 * (1 << 20), 1e-5),
             (5000, 1.0), (12345, 0.0)]
    for ci, (n, rate) in enumerate(cases):
        mask = MASKS[code][ci % len(MASKS[code])]
        gb, tb = special_pair(n, code, seed=700 + ci)
        seed = synth.inject_seed(11, 13 * ci + code)
        g, t = to_device(gb, code), to_device(tb, code)
        log(f"  dtype={code} n={n} rate={rate} mask={mask:#x}")
        recs, counts = _fused([(g, t)], [seed], rate, mask)
        host = tb.copy()
        cnt_ref = oracle.inject(host, dtype=code, seed=seed, rate=rate, mask=mask)
        assert counts[0] == cnt_ref, (n, rate, counts[0], cnt_ref)
        assert np.array_equal(to_host_bits(t), host), f"flipped bits differ n={n} rate={rate}"
        assert np.array_equal(to_host_bits(g), gb), "golden modified"
        assert_parity(recs[0], oracle_sig(gb, host, code, synth.BINS, synth.THRESHOLDS), f"n={n} rate={rate}")


def _profile_counts(fn):
    """Run fn with the library's kernel timing on; return the launches of the
    fused chunk pass and of the injection kernel it made."""
    P.profile_enable(True)
    for k in (P.K_SIG_INJECT, P.K_INJECT):
        P.profile_read(k)
    try:
        out = fn()
    finally:
        torch.cuda.synchronize()
        fused = P.profile_read(P.K_SIG_INJECT)[1]
        inj = P.profile_read(P.K_INJECT)[1]
        P.profile_enable(False)
    return out, fused, inj


def test_fused_equals_separate_calls_many_pairs():
    """A batch of 4500 pairs of three types (about 2,200 chunks per type, so
    one chunk per block), unaligned golden tensors (the generic path inside
    the fused pass) and special values: the fused call runs the fused pass and
    matches inject_batched + signature_batched bit for bit."""
    sizes = [2048, 3 * 4096, 4096 + 904, 20000, 4095, 9000, 1 << 16]
    hosts, fused_pairs, sep_pairs, seeds, codes = [], [], [], [], []
    for k in range(4500):
        code = (k // 3) % 3
        n = sizes[k % len(sizes)]
        gb, tb = special_pair(n, code, seed=90000 + k, special_frac=1e-3 if k % 5 == 0 else 0.0)
        if k % 11 == 4:                          # golden not 16-byte aligned
            g = to_device(np.concatenate([gb[:1], gb]), code)[1:]
        else:
            g = to_device(gb, code)
        hosts.append((gb, tb))
        fused_pairs.append((g, to_device(tb, code)))
        sep_pairs.append((g, to_device(tb, code)))
        seeds.append(synth.inject_seed(12, k))
        codes.append(code)
    rate, mask_of = 3e-3, {0: 0x7F800000, 1: 0x7C00, 2: 0x7F80}
    # one call per dtype group (a batched call takes one bitmask)
    for code in range(3):
        idx = [k for k in range(len(codes)) if codes[k] == code]
        log(f"  dtype={code}: {len(idx)} pairs, {sum(chunk_count(hosts[k][0].size) for k in idx)} chunks")
        (recs, counts), nfused, ninj = _profile_counts(
            lambda: _fused([fused_pairs[k] for k in idx], [seeds[k] for k in idx], rate, mask_of[code]))
        assert (nfused, ninj) == (1, 0), "expected the fused pass"
        sep_counts = P.inject_batched([(sep_pairs[k][1], seeds[k], rate, mask_of[code]) for k in idx])
        sep_recs = P.signature_batched([sep_pairs[k] for k in idx], synth.BINS, synth.THRESHOLDS)
        assert counts == sep_counts
        for j, k in enumerate(idx):
            assert _same(recs[j], sep_recs[j]), f"pair {k}: fused and separate records differ"
            assert np.array_equal(to_host_bits(fused_pairs[k][1]), to_host_bits(sep_pairs[k][1])), \
                f"pair {k}: flipped tensors differ"
        for j in range(0, len(idx), 97):                        # a sample against the oracle
            k = idx[j]
            host = hosts[k][1].copy()
            assert oracle.inject(host, dtype=code, seed=seeds[k], rate=rate, mask=mask_of[code]) == counts[j]
            assert_parity(recs[j], oracle_sig(hosts[k][0], host, code, synth.BINS, synth.THRESHOLDS), f"pair {k}")


def _bits_to_f64(bits: np.ndarray, code: int) -> np.ndarray:
    if code == 0:
        return bits.view(np.float32).astype(np.float64)
    if code == 1:
        return bits.view(np.float16).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _packed(code: int, sizes, seed: int, align: int, gap: int, offsets=None, specials: int = 0,
            equal: bool = False):
    """Seeded pairs packed into one golden and one test allocation (torch
    allocations start on 512-byte boundaries).  Pair k starts at the first
    multiple of `align` bytes at least `gap` bytes after the end of pair
    k - 1, plus offsets[k] bytes; `specials` special values (NaN, Inf, zero,
    subnormal, ...) are planted at distinct positions of the test buffer;
    with equal the test buffer starts as a copy of the golden one.  Returns the pairs' host bits (golden, test), the device pairs (views) and
    the flat device test buffer."""
    es = 4 if code == 0 else 2
    starts, pos = [], 0
    for k, n in enumerate(sizes):
        pos = -(-(pos + gap) // align) * align + (offsets[k] if offsets else 0)
        assert pos % es == 0
        starts.append(pos // es)
        pos += n * es
    total = pos // es + 1
    rng = np.random.default_rng(seed)
    gflat = float_to_bits(rng.standard_normal(total), code).copy()
    tflat = float_to_bits(_bits_to_f64(gflat, code) * (1 + 1e-3 * rng.standard_normal(total)), code).copy()
    if equal:
        tflat = gflat.copy()
    if specials:
        sp = np.array(list(_SPECIALS[code].values()), dtype=NP_BITS[code])
        tflat[rng.choice(total, specials, replace=False)] = sp[rng.integers(0, sp.size, specials)]
    gdev, tdev = to_device(gflat, code), to_device(tflat, code)
    pairs = [(gdev[s0:s0 + n], tdev[s0:s0 + n]) for n, s0 in zip(sizes, starts)]
    hosts = [(gflat[s0:s0 + n].copy(), tflat[s0:s0 + n].copy()) for n, s0 in zip(sizes, starts)]
    return hosts, pairs, tdev


def _fused_vs_separate(code, pairs, pairs2, tflat, tflat2, seeds, rate, mask, sample, path):
    """One fused call on pairs and the two separate calls on pairs2 (an equal
    copy): counts, flipped buffers and records equal; the sampled pairs'
    flips and records against the oracle.  path: the expected kernels."""
    gold = {k: to_host_bits(pairs[k][0]) for k in sample}
    want = {k: to_host_bits(pairs[k][1]) for k in sample}
    (recs, counts), nfused, ninj = _profile_counts(lambda: _fused(pairs, seeds, rate, mask))
    assert (nfused, ninj) == ((1, 0) if path == "fused" else (0, 1)), (path, nfused, ninj)
    sep_counts = P.inject_batched([(t, s, rate, mask) for (_, t), s in zip(pairs2, seeds)])
    sep_recs = P.signature_batched(pairs2, synth.BINS, synth.THRESHOLDS)
    assert counts == sep_counts
    assert torch.equal(tflat.view(TORCH_INT[code]), tflat2.view(TORCH_INT[code])), "flipped tensors differ"
    bad = [k for k in range(len(pairs)) if not _same(recs[k], sep_recs[k])]
    assert not bad, f"fused and separate records differ for pairs {bad[:10]}"
    for k in sample:
        n = oracle.inject(want[k], dtype=code, seed=seeds[k], rate=rate, mask=mask)
        assert n == counts[k], (k, n, counts[k])
        assert np.array_equal(to_host_bits(pairs[k][1]), want[k]), f"pair {k}: flipped bits"
        assert_parity(recs[k], oracle_sig(gold[k], want[k], code, synth.BINS, synth.THRESHOLDS),
                      f"rate={rate} pair {k}")
    return counts


@pytest.mark.parametrize("code", [0, 1, 2])
def test_fused_two_chunk_blocks(code):
    """The launch shape the benchmark times: at least 12288 chunks in one
    fused launch, so every block injects two consecutive chunks before it
    reads either (see TWO_CHUNK_MIN).  About 920 pairs of 2^12..2^18
    elements (15.4k chunks, 62 M elements) packed at line-private offsets
    (so the fused pass runs), unaligned goldens for every 13th pair (the
    generic path), special values;
    two calls, in the top-byte filter regime (rate 3e-3) and in the general
    one (0.3), every bit of the type in the mask.  Flipped tensors and records
    equal peat_inject_batched followed by peat_signature_batched bit for bit;
    sampled pairs match the oracle's injection followed by its signature."""
    cycle = [1 << 16, (1 << 14) + 904, 3 * 4096 + 17, 40000, (1 << 16) - 5, 1 << 18, 4096, 70001]
    sizes = []
    while sum(chunk_count(n) for n in sizes) < 1.25 * TWO_CHUNK_MIN:
        sizes.append(cycle[len(sizes) % len(cycle)])
    nchunks = sum(chunk_count(n) for n in sizes)
    assert nchunks >= TWO_CHUNK_MIN
    hosts, pairs, tflat = _packed(code, sizes, seed=5100 + code, align=256, gap=256, specials=20000)
    _, pairs2, tflat2 = _packed(code, sizes, seed=5100 + code, align=256, gap=256, specials=20000)
    assert torch.equal(tflat.view(TORCH_INT[code]), tflat2.view(TORCH_INT[code]))
    for k in range(0, len(sizes), 13):            # golden not 16-byte aligned
        g = to_device(np.concatenate([hosts[k][0][:1], hosts[k][0]]), code)[1:]
        pairs[k] = (g, pairs[k][1])
        pairs2[k] = (g, pairs2[k][1])
    seeds = [synth.inject_seed(15, 10 * k + code) for k in range(len(sizes))]
    mask = {0: 0xFFFFFFFF, 1: 0xFFFF, 2: 0xFFFF}[code]
    sample = sorted({0, 1, 5, len(sizes) - 1, *range(13, len(sizes), 151)})
    log(f"  dtype={code}: {len(sizes)} pairs, {nchunks} chunks (two-chunk blocks from {TWO_CHUNK_MIN})")
    for rate in (3e-3, 0.3):
        counts = _fused_vs_separate(code, pairs, pairs2, tflat, tflat2, seeds, rate, mask, sample, "fused")
        log(f"    rate={rate}: {sum(counts)} flips, {len(sample)} pairs against the oracle")


@pytest.mark.parametrize("code", [1, 2])
def test_fused_replay_like(code):
    """Replayed outputs: every test tensor starts bit-identical to its golden
    and the fused pass injects at low rates, so almost every lane vector of
    the 16-bit kernels takes the equal-vector branch and the flipped ones the
    full path, in blocks of two chunks (the same 15.4k-chunk batch as
    test_fused_two_chunk_blocks, special values in the goldens, which the
    test tensors repeat).  Records, counts and flipped tensors equal the
    separate calls bit for bit; sampled pairs match the oracle."""
    cycle = [1 << 16, (1 << 14) + 904, 3 * 4096 + 17, 40000, (1 << 16) - 5, 1 << 18, 4096, 70001]
    sizes = []
    while sum(chunk_count(n) for n in sizes) < 1.25 * TWO_CHUNK_MIN:
        sizes.append(cycle[len(sizes) % len(cycle)])
    _, pairs, tflat = _packed(code, sizes, seed=5300 + code, align=256, gap=256, equal=True)
    _, pairs2, tflat2 = _packed(code, sizes, seed=5300 + code, align=256, gap=256, equal=True)
    sp = np.array(list(_SPECIALS[code].values()), dtype=NP_BITS[code])
    rng = np.random.default_rng(77 + code)
    for k in range(0, len(sizes), 7):             # specials in the golden, repeated by the test
        pos = rng.integers(0, sizes[k], 4)
        val = sp[rng.integers(0, sp.size, 4)]
        for (g, t) in (pairs[k], pairs2[k]):
            g.view(TORCH_INT[code])[torch.from_numpy(pos).cuda()] = torch.from_numpy(val.view(np.int16)).cuda()
            t.view(TORCH_INT[code])[torch.from_numpy(pos).cuda()] = torch.from_numpy(val.view(np.int16)).cuda()
    seeds = [synth.inject_seed(16, 10 * k + code) for k in range(len(sizes))]
    sample = sorted({0, 7, 14, len(sizes) - 1, *range(21, len(sizes), 173)})
    log(f"  dtype={code}: {len(sizes)} pairs of test == golden")
    for rate in (1e-5, 3e-3):
        counts = _fused_vs_separate(code, pairs, pairs2, tflat, tflat2, seeds, rate, 0xFFFF, sample, "fused")
        log(f"    rate={rate}: {sum(counts)} flips, {len(sample)} pairs against the oracle")


@pytest.mark.parametrize("code", [0, 1, 2])
def test_fused_packed_offsets(code):
    """Pairs packed in one allocation at 4/16/64/100-byte offsets (2 bytes
    instead of 4 for f16/bf16) from their neighbours, so test tensors share
    cache lines with other tensors: such a batch takes the two launches
    (injection kernel, then the signature).  The same sizes at line-private
    offsets (128-byte starts, a 128-byte gap) take the fused pass.  Both at
    rate 1 (every element flips, every chunk edge included) and 0.3, against
    separate calls and the oracle."""
    es = 4 if code == 0 else 2
    sizes = [4096 * 3 + 5, 4096, 70001, 1 << 14, 33, 4096 * 9 - 1, 100000, 8191]
    mask = {0: 1 << 30, 1: 1 << 14, 2: 1 << 14}[code]
    for layout in ("shared", "private"):
        if layout == "shared":
            kw = dict(align=es, gap=0, offsets=[[es, 16, 64, 100][k % 4] for k in range(len(sizes))])
        else:
            kw = dict(align=128, gap=128)
        _, pairs, tflat = _packed(code, sizes, seed=6200 + code, specials=300, **kw)
        _, pairs2, tflat2 = _packed(code, sizes, seed=6200 + code, specials=300, **kw)
        assert torch.equal(tflat.view(TORCH_INT[code]), tflat2.view(TORCH_INT[code]))
        seeds = [synth.inject_seed(16, 10 * k + code) for k in range(len(sizes))]
        for rate in (1.0, 0.3):
            path = "fused" if layout == "private" else "two launches"
            counts = _fused_vs_separate(code, pairs, pairs2, tflat, tflat2, seeds, rate, mask,
                                        list(range(len(sizes))), path)
            log(f"  dtype={code} {layout}: rate={rate} {sum(counts)} flips ok")


def test_fused_llama_tensors_full_size():
    """The largest tensors of the Llama-7B-shaped workload at their real shapes
    (embedding, MLP, attention), with the benchmark's rate and mask: fused
    equals separate calls, and sampled outputs match the oracle."""
    shapes = [(32000, 4096), (11008, 4096), (4096, 4096)]
    rate, mask = synth.CONFIG5_RATE, synth.CONFIG5_MASK
    pairs_a, pairs_b, seeds = [], [], []
    for k, shp in enumerate(shapes):
        g = torch.randn(shp, device="cuda") * 0.02
        t = g * (1 + 1e-7 * torch.randn(shp, device="cuda"))
        pairs_a.append((g, t.clone()))
        pairs_b.append((g, t))
        seeds.append(synth.inject_seed(5, 1000 + k))
    # the attention-shaped pair before injection, for the oracle
    gb, tb = to_host_bits(pairs_a[2][0]), to_host_bits(pairs_a[2][1])
    recs, counts = _fused(pairs_a, seeds, rate, mask)
    sep_counts = P.inject_batched([(t, s, rate, mask) for (_, t), s in zip(pairs_b, seeds)])
    sep = P.signature_batched(pairs_b, synth.BINS, synth.THRESHOLDS)
    log(f"  counts {counts}")
    assert counts == sep_counts
    for k in range(len(shapes)):
        assert _same(recs[k], sep[k]), f"tensor {k}"
        assert np.array_equal(to_host_bits(pairs_a[k][1]), to_host_bits(pairs_b[k][1]))
    host = tb.copy()
    assert oracle.inject(host, dtype=0, seed=seeds[2], rate=rate, mask=mask) == counts[2]
    assert np.array_equal(to_host_bits(pairs_a[2][1]), host)
    assert_parity(recs[2], oracle_sig(gb, host, 0, synth.BINS, synth.THRESHOLDS), "attention-shaped tensor")


THR_SETS = [(), (0.0,), (1e-7, 1e-5, 1e-3, 0.1), (0.0, 1e-9, 1e-6, 1e-4, 1e-2, 1.0, 100.0, float("inf")),
            ((1e-6, 1e-3), (0.0, 1e-5)), ((0.0, float("inf")), (1e-3, 0.1), (1e-9, 2.0 ** -11), (0.0, 0.0))]


@pytest.mark.parametrize("code", [0, 1, 2])
def test_fused_threshold_and_bin_variants(code):
    """Every instantiation of the fused pass (2, 4 or 8 compared thresholds,
    absolute or torch.isclose-style relative tolerances) and other bin
    layouts, against the oracle's injection followed by its signature."""
    bins_sets = [synth.BINS, (-30, 20, 25), (-160, 136, 37)]
    for i, thr in enumerate(THR_SETS):
        bins = bins_sets[i % len(bins_sets)]
        n = [70001, 4096 * 3 + 17, 250000][i % 3]
        gb, tb = special_pair(n, code, seed=4400 + 10 * i + code)
        seed = synth.inject_seed(13, 7 * i + code)
        rate, mask = [1e-3, 2e-2][i % 2], MASKS[code][i % len(MASKS[code])]
        g, t = to_device(gb, code), to_device(tb, code)
        log(f"  dtype={code} n={n} thresholds={thr} bins={bins}")
        d_out = torch.empty(P.SIG_BYTES, dtype=torch.uint8, device="cuda")
        d_counts = torch.empty(1, dtype=torch.int64, device="cuda")
        P.inject_signature_batched_async([(g, t)], [seed], rate, mask, d_out, d_counts, bins, thr)
        torch.cuda.synchronize()
        nthr = len(thr)
        rec = P.decode_records(d_out, 1, nthr=nthr)[0]
        host = tb.copy()
        assert int(d_counts.item()) == oracle.inject(host, dtype=code, seed=seed, rate=rate, mask=mask)
        assert np.array_equal(to_host_bits(t), host)
        assert_parity(rec, oracle_sig(gb, host, code, bins, thr), f"thresholds={thr}")


def test_fused_empty_pairs_shared_golden_and_repeat():
    """Empty pairs in the batch (zero records, zero counts), two pairs sharing
    one golden tensor (allowed: only test tensors are written), and the same
    call twice with the same seeds (the flips undo themselves: the tensors
    come back to their first state, and the second records are those of the
    original tests)."""
    code = 0
    gb, tb = special_pair(40000, code, seed=31)
    _, tb2 = special_pair(40000, code, seed=32)
    g = to_device(gb, code)
    t1, t2 = to_device(tb, code), to_device(tb2, code)
    empty = torch.empty(0, dtype=torch.float32, device="cuda")
    pairs = [(g, t1), (empty, torch.empty(0, dtype=torch.float32, device="cuda")), (g, t2)]
    seeds = [synth.inject_seed(14, 1), synth.inject_seed(14, 2), synth.inject_seed(14, 3)]
    rate, mask = 2e-3, 0xFFFFFFFF
    recs, counts = _fused(pairs, seeds, rate, mask)
    h1, h2 = tb.copy(), tb2.copy()
    assert counts[0] == oracle.inject(h1, dtype=code, seed=seeds[0], rate=rate, mask=mask)
    assert counts[2] == oracle.inject(h2, dtype=code, seed=seeds[2], rate=rate, mask=mask)
    assert counts[1] == 0 and recs[1]["n"] == 0 and recs[1]["n_valid"] == 0
    assert_parity(recs[0], oracle_sig(gb, h1, code, synth.BINS, synth.THRESHOLDS), "pair 0")
    assert_parity(recs[2], oracle_sig(gb, h2, code, synth.BINS, synth.THRESHOLDS), "pair 2")
    assert np.array_equal(to_host_bits(g), gb)
    recs2, counts2 = _fused(pairs, seeds, rate, mask)
    assert counts2 == counts
    assert np.array_equal(to_host_bits(t1), tb) and np.array_equal(to_host_bits(t2), tb2)
    assert_parity(recs2[0], oracle_sig(gb, tb, code, synth.BINS, synth.THRESHOLDS), "pair 0, second call")
