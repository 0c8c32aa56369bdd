"""GPU parity of the other error models against the oracle, bit for bit:
the rate-mode zero / NaN / bit-flip / random-value (the tensor's own value
at a random index, read from the tensor as it was before the call) /
uniformly random bit pattern models (peat_inject_model and batched items),
the num_pos position mode with the same models (peat_corrupt_positions),
and the FP16 / BF16 cast error (peat_cast_round), over the three element
types, ragged sizes, unaligned tensors and the workloads' rates."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_13544_amd as P
from tests.parity import special_pair, to_device, to_host_bits

pytestmark = pytest.mark.gpu

MASKS = {0: 0x7F800000, 1: 0xFFFF, 2: 0x7F80}


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("code", [0, 1, 2])
def test_rate_models(code):
    for n in (0, 1, 5000, (1 << 20) + 7):
        gb, _ = special_pair(n, code, seed=300 + n % 97 + code)
        for rate in (0.0, 1e-4, 1e-2, 1.0):
            for model in (P.MODEL_ZERO, P.MODEL_NAN, P.MODEL_BITFLIP, P.MODEL_VALUE, P.MODEL_UNIFORM):
                log(f"  dtype={code} n={n} rate={rate} model={model}")
                x = to_device(gb, code)
                cnt = P.inject_model(x, 1234 + n, rate, model, MASKS[code])
                ref = gb.copy()
                cnt_ref = oracle.inject_model(ref, dtype=code, seed=1234 + n, rate=rate, model=model,
                                              mask=MASKS[code])
                assert cnt == cnt_ref
                assert np.array_equal(to_host_bits(x), ref)


@pytest.mark.parametrize("code", [0, 1, 2])
def test_rate_value_models_distinct_values(code):
    """Random value at a rate over tensors of distinct values spanning
    several injector segments (2^20 elements each): a chosen element must
    get the value its source held before the call, even when the source is
    itself chosen (rate 1 and 0.5 make that common); also the uniformly
    random bit pattern model."""
    for n in (3 * (1 << 20) + 11, 40000):
        rng = np.random.default_rng(n + code)
        if code == 0:
            gb = rng.permutation(np.arange(0x3F800000, 0x3F800000 + n, dtype=np.uint32))
        else:
            gb = rng.integers(1, 0x7C00, n, dtype=np.uint16)
        for rate in (1.0, 0.5, 1e-3):
            for model in (P.MODEL_VALUE, P.MODEL_UNIFORM):
                log(f"  dtype={code} n={n} rate={rate} model={model}")
                x = to_device(gb, code)
                cnt = P.inject_model(x, 4321 + n, rate, model)
                ref = gb.copy()
                assert cnt == oracle.inject_model(ref, dtype=code, seed=4321 + n, rate=rate, model=model)
                assert np.array_equal(to_host_bits(x), ref)


def test_rate_models_batched():
    items, refs, expect = [], [], []
    for k, (n, code, model) in enumerate([(70001, 0, P.MODEL_NAN), (4096, 1, P.MODEL_ZERO),
                                          (200000, 2, P.MODEL_BITFLIP), (0, 0, P.MODEL_NAN),
                                          (300001, 0, P.MODEL_VALUE), (5000, 1, P.MODEL_UNIFORM),
                                          (70000, 2, P.MODEL_VALUE), (1 << 20, 1, P.MODEL_VALUE)]):
        gb, _ = special_pair(n, code, seed=50 + k)
        x = to_device(gb, code)
        items.append((x, 77 + k, 3e-3, MASKS[code], model))
        ref = gb.copy()
        expect.append(oracle.inject_model(ref, dtype=code, seed=77 + k, rate=3e-3, model=model, mask=MASKS[code]))
        refs.append(ref)
    counts = P.inject_batched(items)
    assert counts == expect
    for (x, *_), ref in zip(items, refs):
        assert np.array_equal(to_host_bits(x), ref)


@pytest.mark.parametrize("code", [0, 1, 2])
def test_positions(code):
    for n, num_pos in ((1, 1), (10, 10), (1000, 5), (5000, 4096), ((1 << 20) + 3, 4096), (3, 0)):
        gb, _ = special_pair(n, code, seed=900 + n % 89 + code)
        for model in (P.MODEL_VALUE, P.MODEL_ZERO, P.MODEL_NAN, P.MODEL_BITFLIP, P.MODEL_UNIFORM):
            for seed in (0, 2 ** 63 + 11):
                log(f"  dtype={code} n={n} num_pos={num_pos} model={model} seed={seed}")
                x = to_device(gb, code)
                pos = P.corrupt_positions(x, seed, model, num_pos, MASKS[code])
                ref = gb.copy()
                rc, pos_ref = oracle.corrupt_positions(ref, dtype=code, seed=seed, model=model, num_pos=num_pos,
                                                       mask=MASKS[code])
                assert rc == num_pos and pos == pos_ref
                assert np.array_equal(to_host_bits(x), ref)


def _cast_inputs(n, seed):
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 2 ** 32, n, dtype=np.uint32)
    # ties for both narrower types, boundaries, NaN payloads, subnormals
    x[: n // 8] = (x[: n // 8] & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    x[n // 8: n // 4] = (x[n // 8: n // 4] & np.uint32(0xFFFFE000)) | np.uint32(0x1000)
    special = np.array([0x7FC00000, 0xFFC00001, 0x7F800001, 0x7F800000, 0xFF800000, 0, 0x80000000, 1,
                        0x807FFFFF, 0x477FF000, 0x477FEFFF, 0x477FE000, 0x7F7FFFFF, 0x7F7F8000, 0x33800000,
                        0x33000000, 0x33000001, 0xB3400000], np.uint32)
    x[: len(special)] = special[: min(len(special), n)] if n >= len(special) else special[:n]
    return x


@pytest.mark.parametrize("to", [1, 2])
def test_cast_round(to):
    for n in (1, 7, 4096, (1 << 20) + 5):
        xb = _cast_inputs(n, 40 + n % 13)
        log(f"  to={to} n={n}")
        d = to_device(xb, 0)
        P.cast_round(d, to)
        ref = xb.copy()
        assert oracle.cast_round(ref, to) == 0
        assert np.array_equal(to_host_bits(d), ref)
    # an unaligned view (scalar path)
    xb = _cast_inputs(10001, 5)
    d = to_device(xb, 0)[1:]
    P.cast_round(d, to)
    ref = xb[1:].copy()
    oracle.cast_round(ref, to)
    assert np.array_equal(to_host_bits(d), ref)
    torch.cuda.synchronize()
