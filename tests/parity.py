"""Shared helpers of the GPU parity tests: seeded host inputs with special
values, host<->device transfer of raw bit patterns, and the parity check of a
device signature against the oracle's.

Tolerance (derived from the arithmetic): every count, histogram bin, index,
maximum and the ULP sum must match exactly; the binary64 sums of non-negative
terms (sum_abs, sum_sq, sum_rel, sum_g2, sum_t2) within 1e-12 relative, and
sum_gt within 1e-12 * sqrt(sum_g2 * sum_t2), which keeps the cosine within
1e-12 absolute.  The device sums each lane's <= 1024 terms sequentially and
then a fixed tree of depth <= 30, a relative error below 1.2e-13 for
non-negative terms; the oracle's compensated sum is within ~1 ulp.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle

NP_BITS = {0: np.uint32, 1: np.uint16, 2: np.uint16}
TORCH_DT = {0: torch.float32, 1: torch.float16, 2: torch.bfloat16}
TORCH_INT = {0: torch.int32, 1: torch.int16, 2: torch.int16}
NONNEG_SUMS = ("sum_abs", "sum_sq", "sum_rel", "sum_g2", "sum_t2")
REL_TOL = 1e-12


def to_device(bits: np.ndarray, code: int, device="cuda") -> torch.Tensor:
    """Raw bit patterns (uint32/uint16) -> device tensor of the float type."""
    signed = bits.view(np.int32 if code == 0 else np.int16)
    return torch.from_numpy(signed.copy()).to(device).view(TORCH_DT[code])


def to_host_bits(t: torch.Tensor) -> np.ndarray:
    code = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}[t.dtype]
    ints = t.detach().contiguous().view(TORCH_INT[code]).cpu().numpy()
    return ints.view(NP_BITS[code])


def float_to_bits(x: np.ndarray, code: int) -> np.ndarray:
    """float64 values -> bit patterns of the element type (round to nearest even)."""
    if code == 0:
        return x.astype(np.float32).view(np.uint32)
    if code == 1:
        return x.astype(np.float16).view(np.uint16)
    t = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


_SPECIALS = {
    0: {"nan": 0x7FC00000, "nan2": 0xFFA00001, "inf": 0x7F800000, "ninf": 0xFF800000,
        "zero": 0x00000000, "nzero": 0x80000000, "sub": 0x00000001, "sub2": 0x807FFFFF,
        "big": 0x7F7FFFFF},
    1: {"nan": 0x7E00, "nan2": 0xFE01, "inf": 0x7C00, "ninf": 0xFC00, "zero": 0x0000,
        "nzero": 0x8000, "sub": 0x0001, "sub2": 0x83FF, "big": 0x7BFF},
    2: {"nan": 0x7FC0, "nan2": 0xFFA1, "inf": 0x7F80, "ninf": 0xFF80, "zero": 0x0000,
        "nzero": 0x8000, "sub": 0x0001, "sub2": 0x807F, "big": 0x7F7F},
}


def special_pair(n: int, code: int, seed: int, special_frac: float = 1e-3, rel_noise: float = 1e-3,
                 scale: float = 1.0):
    """Seeded golden/test bit patterns: Gaussian golden, relative-noise test,
    plus NaN/Inf/zero/subnormal/max values, sign flips and bit-equal pairs at
    random positions, and repeated values (ties of the maxima)."""
    rng = np.random.default_rng(seed)
    G = rng.standard_normal(n) * scale
    T = G * (1.0 + rel_noise * rng.standard_normal(n))
    gb = float_to_bits(G, code).copy()
    tb = float_to_bits(T, code).copy()
    if n == 0:
        return gb, tb
    sp = _SPECIALS[code]
    k = max(1, int(n * special_frac)) if special_frac > 0 else 0
    for name, val in sp.items():
        for arr in (gb, tb):
            idx = rng.integers(0, n, k)
            arr[idx] = val
    if k:
        idx = rng.integers(0, n, k)                       # sign flips
        tb[idx] = gb[idx] ^ (1 << (8 * gb.itemsize - 1))
        idx = rng.integers(0, n, k)                       # bit-equal pairs
        tb[idx] = gb[idx]
        idx = rng.integers(0, n, k)                       # duplicated pairs: ties
        src = rng.integers(0, n, 1)
        gb[idx] = gb[src]
        tb[idx] = tb[src]
    return gb, tb


def assert_parity(got: dict, ref: dict, ctx: str = "") -> None:
    for k, v in ref.items():
        g = got[k]
        if isinstance(v, float) and math.isinf(v):
            assert g == v, f"{ctx} {k}: gpu {g!r} oracle {v!r}"
        elif k in NONNEG_SUMS:
            assert abs(g - v) <= REL_TOL * abs(v), f"{ctx} {k}: gpu {g!r} oracle {v!r}"
        elif k == "sum_gt":
            scale = math.sqrt(ref["sum_g2"] * ref["sum_t2"])
            assert abs(g - v) <= REL_TOL * scale, f"{ctx} {k}: gpu {g!r} oracle {v!r}"
        elif isinstance(v, float) and math.isnan(v):
            assert isinstance(g, float) and math.isnan(g), f"{ctx} {k}: gpu {g!r} expected NaN"
        else:
            assert g == v, f"{ctx} {k}: gpu {g!r} oracle {v!r}"


def oracle_sig(gb: np.ndarray, tb: np.ndarray, code: int, bins, thresholds) -> dict:
    return oracle.signature(gb, tb, dtype=code, bins=bins, thresholds=thresholds)


def chunk_count(n: int) -> int:
    """Chunks of an n-element pair under the library's chunk rule: the next
    power of two >= n/256 elements below 2^22 elements (>= n/64 from 2^22 on),
    clamped to [2^12, 2^18]."""
    if n == 0:
        return 0
    target = 64 if n >= (1 << 22) else 256
    per = -(-n // target)
    log2 = max(12, min(18, (per - 1).bit_length()))
    return -(-n // (1 << log2))


# Launch-shape bound of the chunk pass: a block takes two consecutive chunks
# once a launch has at least 2 x 8 x (resident blocks) chunks.  Resident
# blocks are at most 3 per compute unit (a block holds ~52 KB of the 160 KB
# of LDS) on 256 compute units, so 12288 chunks per launch force two-chunk
# blocks.
TWO_CHUNK_MIN = 2 * 8 * 3 * 256


def group_size(nchunks: int, nelems: int, resident: int = 3 * 256) -> int:
    """Chunks per block of a chunk-pass launch: nchunks // (8 x resident),
    clamped to [1, kmax] with kmax = 2^19 // (average chunk size) in [2, 8]."""
    if nchunks == 0:
        return 1
    kmax = max(2, min(8, (1 << 19) // max(1, nelems // nchunks)))
    return max(1, min(kmax, nchunks // (8 * resident)))


def records_equal(a: dict, b: dict) -> bool:
    """Bit-level equality of two decoded records (NaN equals NaN)."""
    return a.keys() == b.keys() and all(
        a[k] == v or (isinstance(v, float) and math.isnan(v) and isinstance(a[k], float) and math.isnan(a[k]))
        for k, v in b.items())
