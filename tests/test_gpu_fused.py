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
from tests.parity import assert_parity, oracle_sig, special_pair, to_device, to_host_bits

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


def test_fused_equals_separate_calls_many_pairs():
    """A batch large enough for two-chunk blocks (injection of both chunks
    before either is read), mixed types and sizes, unaligned pairs: the fused
    call matches inject_batched + signature_batched bit for bit."""
    sizes = [2048, 3 * 4096, 4096 + 904, 20000, 4095, 9000, 1 << 16]
    hosts, fused_pairs, sep_pairs, seeds, codes = [], [], [], [], []
    for k in range(4500):
        code = (k // 3) % 3
        n = sizes[k % len(sizes)]
        gb, tb = special_pair(n, code, seed=90000 + k, special_frac=1e-3 if k % 5 == 0 else 0.0)
        g = to_device(gb, code)
        if k % 11 == 4:                          # test not 16-byte aligned
            t1 = to_device(np.concatenate([tb[:1], tb]), code)[1:]
            t2 = to_device(np.concatenate([tb[:1], tb]), code)[1:]
        else:
            t1, t2 = to_device(tb, code), to_device(tb, code)
        hosts.append((gb, tb))
        fused_pairs.append((g, t1))
        sep_pairs.append((g, t2))
        seeds.append(synth.inject_seed(12, k))
        codes.append(code)
    rate, mask_of = 3e-3, {0: 0x7F800000, 1: 0x7C00, 2: 0x7F80}
    # one call per dtype group (a batched call takes one bitmask)
    for code in range(3):
        idx = [k for k in range(len(codes)) if codes[k] == code]
        log(f"  dtype={code}: {len(idx)} pairs")
        recs, counts = _fused([fused_pairs[k] for k in idx], [seeds[k] for k in idx], rate, mask_of[code])
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
