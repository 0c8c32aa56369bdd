"""GPU test of peat_signature_batched_noalloc, the entry point for callers
that cannot allocate: through the C ABI, its records equal those of
peat_signature_batched_async (the entry point it mirrors) bit for bit, on two
calls in a row -- a large batch, then a smaller one that must not see what
the first left in the shared scratch array -- and sampled records match the
oracle."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_13544_amd as P
import synth
from tests.parity import assert_parity, chunk_count, oracle_sig, records_equal, special_pair, to_device

pytestmark = pytest.mark.gpu


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def _batch(seed: int, count: int, sizes):
    pairs, hosts = [], []
    for k in range(count):
        code = k % 3
        n = sizes[k % len(sizes)]
        gb, tb = special_pair(n, code, seed=seed + k, special_frac=1e-3 if k % 4 == 0 else 0.0)
        g = to_device(gb, code)
        if k % 7 == 3:                                    # unaligned test tensor
            t = to_device(np.concatenate([tb[:1], tb]), code)[1:]
        else:
            t = to_device(tb, code)
        pairs.append((g, t))
        hosts.append((gb, tb, code))
    return pairs, hosts


def _records(fn, pairs, bins, thr):
    d_out = torch.full((len(pairs) * P.SIG_BYTES,), 0xA5, dtype=torch.uint8, device="cuda")
    fn(pairs, d_out, bins, thr)
    torch.cuda.synchronize()
    return P.decode_records(d_out, len(pairs), nthr=len(thr))


def test_noalloc_matches_async_twice():
    assert torch.cuda.is_available()
    P.lib().peat_init()
    # call 1: many pairs of mixed types and sizes (thousands of chunks, some
    # pairs of 2^22+ elements), call 2: fewer and smaller pairs, other bins
    big, big_h = _batch(1000, 300, [1, 4095, 4096 * 3 + 7, 70001, 1 << 20, (1 << 22) + 5, 0, 250000])
    small, small_h = _batch(2000, 17, [33, 5000, 4096, 100003])
    for name, pairs, hosts, bins, thr in (
            ("first (large)", big, big_h, synth.BINS, synth.THRESHOLDS),
            ("second (smaller)", small, small_h, (-30, 20, 25), (0.0, 1e-5, 1e-2))):
        chunks = sum(chunk_count(g.numel()) for g, _ in pairs)
        log(f"  {name}: {len(pairs)} pairs, {chunks} chunks")
        got = _records(P.signature_batched_noalloc, pairs, bins, thr)
        want = _records(P.signature_batched_async, pairs, bins, thr)
        bad = [k for k in range(len(pairs)) if not records_equal(got[k], want[k])]
        assert not bad, f"{name}: noalloc and async records differ for pairs {bad[:10]}"
        for k in range(0, len(pairs), max(1, len(pairs) // 12)):
            gb, tb, code = hosts[k]
            assert_parity(got[k], oracle_sig(gb, tb, code, bins, thr), f"{name} pair {k}")
    # a repeated small call on another stream after the large one: same records
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        again = _records(lambda p, o, b, t: P.signature_batched_noalloc(p, o, b, t, stream=s), small,
                         (-30, 20, 25), (0.0, 1e-5, 1e-2))
    first = _records(P.signature_batched_async, small, (-30, 20, 25), (0.0, 1e-5, 1e-2))
    assert all(records_equal(a, b) for a, b in zip(again, first))


def test_noalloc_rejects_batches_beyond_the_scratch():
    """A batch whose records would not fit the static array is refused with
    PEAT_EINVAL and a message, before any work is enqueued."""
    x = torch.zeros(1 << 20, dtype=torch.float32, device="cuda")
    # 2^20-element pairs take 256 chunks each: 612 B x 256 = 153 KiB per pair
    pairs = [(x, x)] * (P.NOALLOC_SCRATCH_BYTES // (612 * 256) + 1)
    d_out = torch.empty(len(pairs) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    with pytest.raises(P.PeatError) as e:
        P.signature_batched_noalloc(pairs, d_out)
    assert e.value.code == -1 and "scratch" in str(e.value)
