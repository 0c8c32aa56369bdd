"""Randomised GPU parity sweep against the oracle: seeded draws of the
golden/test type combination (same-type and mixed-precision), the element
count (empty, tiny, ragged, several chunks, both sides of the chunk-size
switch), an element offset (unaligned pointers), the value distribution
(scale, relative noise, specials), the histogram bins and the thresholds
(absolute and relative).  Each case checks the signature and the top-k mean
(with a random fraction) field by field with the parity tolerances of
tests/parity.py."""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_13544_amd as P
from tests.parity import assert_parity
from tests.test_gpu_mixed import F16, F32, F64, BF16, KINDS, assert_topk, dev, mixed_pair

pytestmark = pytest.mark.gpu

ALL_KINDS = [(F32, F32), (F16, F16), (BF16, BF16)] + KINDS
SIZES = [0, 1, 3, 17, 255, 4095, 4097, 9999, 65537, 262145, 1000003, (1 << 22) - 5, (1 << 22) + 7]
BINS = [(-40, 24, 64), (-30, 20, 25), (-160, 136, 37), (-24, 16, 8), (-1022, 1018, 40)]


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def _case(rng):
    gdt, tdt = ALL_KINDS[rng.integers(len(ALL_KINDS))]
    n = int(SIZES[rng.integers(len(SIZES))])
    off = int(rng.integers(0, 3))
    rel = float(10.0 ** rng.uniform(-8, 0))
    bins = BINS[rng.integers(len(BINS))]
    nthr = int(rng.integers(0, 9))
    thr = []
    for _ in range(nthr):
        atol = float(10.0 ** rng.uniform(-9, 1)) if rng.random() < 0.8 else 0.0
        thr.append((atol, float(10.0 ** rng.uniform(-6, -1))) if rng.random() < 0.4 else atol)
    num = int(rng.integers(1, 8))
    den = int(rng.integers(num, 40))
    return gdt, tdt, n, off, rel, bins, tuple(thr), num, den


@pytest.mark.parametrize("seed", range(64))
def test_random_case(seed):
    rng = np.random.default_rng(31000 + seed)
    gdt, tdt, n, off, rel, bins, thr, num, den = _case(rng)
    log(f"  seed={seed} kind={gdt}/{tdt} n={n} off={off} rel={rel:.2e} bins={bins} nthr={len(thr)} k={num}/{den}")
    gb, tb = mixed_pair(n + off, gdt, tdt, seed=32000 + seed, rel=rel)
    gb, tb = gb[off:], tb[off:]
    g, t = dev(np.ascontiguousarray(gb), gdt), dev(np.ascontiguousarray(tb), tdt)
    if off:
        # an element offset inside one allocation: pointers not 16-byte aligned
        g2, t2 = dev(np.concatenate([gb[:1], gb]), gdt), dev(np.concatenate([tb[:1], tb]), tdt)
        g, t = g2[1:], t2[1:]
    got = P.signature_mixed(g, t, bins, thr)
    ref = oracle.signature_mixed(gb, tb, gdtype=gdt, tdtype=tdt, bins=bins, thresholds=thr)
    assert_parity(got, ref, f"seed {seed}")
    tk = P.topk_mean_mixed_batched([(g, t)], num, den)[0]
    assert_topk(tk, oracle.topk_mixed(gb, tb, gdtype=gdt, tdtype=tdt, num=num, den=den), f"seed {seed}")
