"""GPU parity of the chunk pass when a block streams a long group of small
chunks: about 200 pairs of 2^20 elements make 51200 chunks of 2^12, enough
for eight-chunk blocks.  Batched records (and the fused injection's records,
flip counts and flipped tensors) bit for bit against single calls, whose
launches give every chunk a block of its own, and sampled pairs against the
oracle."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import paper_2609_13544_amd as P
import synth
from tests.parity import (assert_parity, chunk_count, group_size, oracle_sig, records_equal, special_pair,
                          to_device)

pytestmark = pytest.mark.gpu

NPAIRS = 200


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def _pairs(code: int):
    rng = np.random.default_rng(7100 + code)
    sizes = [(1 << 20) - int(rng.integers(0, 4096)) for _ in range(NPAIRS)]
    host = []
    for k, n in enumerate(sizes):
        if k < 3:
            host.append(special_pair(n, code, seed=7200 + k))
        else:
            host.append(special_pair(n, code, seed=7200 + k, special_frac=1e-5))
    nch = sum(chunk_count(n) for n in sizes)
    k = group_size(nch, sum(sizes))
    log(f"  dtype={code}: {len(sizes)} pairs, {nch} chunks, {k} chunks per block")
    assert k >= 6
    return host


@pytest.mark.parametrize("code", [0, 1])
def test_long_groups_equal_single_calls(code):
    host = _pairs(code)
    dev = [(to_device(g, code), to_device(t, code)) for g, t in host]
    d_out = torch.empty(len(dev) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    P.signature_batched_async(dev, d_out, synth.BINS, synth.THRESHOLDS)
    torch.cuda.synchronize()
    batched = P.decode_records(d_out, len(dev), nthr=len(synth.THRESHOLDS))
    for k, (g, t) in enumerate(dev):
        single = P.signature(g, t, synth.BINS, synth.THRESHOLDS)
        assert records_equal(batched[k], single), f"pair {k}"
    for k in (0, 1, 2, 57, NPAIRS - 1):
        gb, tb = host[k]
        assert_parity(batched[k], oracle_sig(gb, tb, code, synth.BINS, synth.THRESHOLDS), f"pair {k}")


@pytest.mark.parametrize("code", [0, 1])
def test_long_groups_fused_equal_separate(code):
    host = _pairs(code)
    dev = [(to_device(g, code), to_device(t, code)) for g, t in host]
    dev2 = [(g, t.clone()) for g, t in dev]
    seeds = [9000 + k for k in range(len(dev))]
    mask = 0x7F800000 if code == 0 else 0x7C00
    rate = 2e-4
    d_out = torch.empty(len(dev) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    d_cnt = torch.full((len(dev),), -1, dtype=torch.int64, device="cuda")
    P.inject_signature_batched_async(dev, seeds, rate, mask, d_out, d_cnt, synth.BINS, synth.THRESHOLDS)
    torch.cuda.synchronize()
    fused = P.decode_records(d_out, len(dev), nthr=len(synth.THRESHOLDS))
    counts = d_cnt.cpu().tolist()
    items = [(t, seeds[k], rate, mask) for k, (_, t) in enumerate(dev2)]
    sep_counts = P.inject_batched(items)
    sep = P.signature_batched(dev2, synth.BINS, synth.THRESHOLDS)
    assert counts == list(sep_counts)
    assert sum(counts) > 0
    for k in range(len(dev)):
        assert records_equal(fused[k], sep[k]), f"pair {k}"
        assert torch.equal(dev[k][1].view(torch.int16 if code else torch.int32),
                           dev2[k][1].view(torch.int16 if code else torch.int32)), f"flipped tensor {k}"
