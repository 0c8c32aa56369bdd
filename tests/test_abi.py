"""CPU tests of the C-ABI library: it loads, exports every entry point that
include/peat.h declares, its struct layouts match the header, and argument
validation returns the documented codes before any device access."""
from __future__ import annotations

import ctypes
import math
import os
import re

import pytest

import paper_2609_13544_amd as P
from paper_2609_13544_amd import _binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "peat.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(peat_[a-z_0-9]+)\s*\(", text)
    return sorted(set(names))


def test_header_declares_expected_entry_points():
    names = _declared_functions()
    for must in ("peat_signature", "peat_signature_batched", "peat_signature_batched_async",
                 "peat_inject", "peat_inject_batched", "peat_inject_batched_async",
                 "peat_finalize_stats", "peat_strerror", "peat_last_error"):
        assert must in names


def test_library_exports_every_declared_symbol():
    L = P.lib()
    for name in _declared_functions():
        assert hasattr(L, name), f"libpeat.so does not export {name}"
    assert set(_declared_functions()) == set(B._PROTOS), "binding prototypes out of sync with header"


def test_struct_layouts():
    assert ctypes.sizeof(B.Signature) == 784
    assert ctypes.sizeof(B.Pair) == 32
    assert ctypes.sizeof(B.InjectItem) == 48
    assert ctypes.sizeof(B.Bins) == 16
    assert ctypes.sizeof(B.Thresholds) == 136
    assert B.Signature.max_abs.offset == 8 * (10 + 8 + 3 + 64)
    assert B.Signature.sum_gt.offset == 784 - 8
    assert ctypes.sizeof(B.TopK) == 48
    assert ctypes.sizeof(B.MixedPair) == 32


def test_abi_version_and_strerror():
    L = P.lib()
    assert L.peat_abi_version() == 6
    for code in range(0, -8, -1):
        assert L.peat_strerror(code)
    assert L.peat_strerror(-99) == b"unknown error code"


def _sig_rc(n=0, dtype=0, bins=(-40, 24, 64), thr=(1e-6,), g=None, t=None, bins_reserved=0):
    b = B.Bins(bins[0], bins[1], bins[2], bins_reserved)
    th = B.Thresholds()
    th.count = len(thr)
    for j, v in enumerate(thr[:8]):
        th.abs_tol[j] = v
    out = B.Signature()
    return P.lib().peat_signature(g, t, n, dtype, ctypes.byref(b), ctypes.byref(th), ctypes.byref(out))


def test_signature_validation_codes():
    assert _sig_rc(n=5) == B.EINVAL                      # NULL tensors with n > 0
    assert _sig_rc(n=-1) == B.EINVAL
    assert _sig_rc(dtype=7) == B.EDTYPE
    for bad in [(-40, 24, 0), (-40, 24, 65), (-40, 24, 7), (3, 3, 1), (-1023, 0, 1), (0, 1025, 1)]:
        assert _sig_rc(bins=bad) == B.EINVAL, bad
    assert _sig_rc(bins_reserved=1) == B.EINVAL
    assert _sig_rc(thr=(math.nan,)) == B.EINVAL
    assert _sig_rc(thr=(-1e-9,)) == B.EINVAL
    for bad in (math.nan, -1.0):                           # relative tolerances
        th = B.Thresholds()
        th.count = 1
        th.rel_tol[0] = bad
        b = B.Bins(-40, 24, 64, 0)
        assert P.lib().peat_signature(None, None, 0, 0, ctypes.byref(b), ctypes.byref(th),
                                      ctypes.byref(B.Signature())) == B.EINVAL
    th = B.Thresholds()
    th.count = 9
    b = B.Bins(-40, 24, 64, 0)
    assert P.lib().peat_signature(None, None, 0, 0, ctypes.byref(b), ctypes.byref(th),
                                  ctypes.byref(B.Signature())) == B.EINVAL
    assert P.lib().peat_signature(None, None, 0, 0, None, ctypes.byref(th),
                                  ctypes.byref(B.Signature())) == B.EINVAL
    assert b"threshold" in P.lib().peat_last_error() or P.lib().peat_last_error()


def test_batched_empty_is_ok_and_validation():
    b = B.Bins(-40, 24, 64, 0)
    th = B.Thresholds()
    L = P.lib()
    assert L.peat_signature_batched(None, 0, ctypes.byref(b), ctypes.byref(th), None) == B.OK
    assert L.peat_signature_batched(None, -1, ctypes.byref(b), ctypes.byref(th), None) == B.EINVAL
    pairs = (B.Pair * 2)(B.Pair(None, None, 0, 0, 0), B.Pair(None, None, 0, 5, 0))
    outs = (B.Signature * 2)()
    assert L.peat_signature_batched(pairs, 2, ctypes.byref(b), ctypes.byref(th), outs) == B.EDTYPE
    assert L.peat_signature_batched_async(pairs, 2, ctypes.byref(b), ctypes.byref(th), None, None) == B.EDTYPE


def test_inject_validation_codes():
    L = P.lib()
    assert L.peat_inject(None, 10, 0, 1, 0.5, 0) == B.EBITMASK
    assert L.peat_inject(None, 10, 1, 1, 0.5, 0x10000) == B.EBITMASK
    assert L.peat_inject(None, 10, 0, 1, 0.5, 1 << 32) == B.EBITMASK
    assert L.peat_inject(None, 10, 0, 1, math.nan, 1) == B.ERATE
    assert L.peat_inject(None, 10, 0, 1, -1.0, 1) == B.ERATE
    assert L.peat_inject(None, 10, 9, 1, 0.5, 1) == B.EDTYPE
    assert L.peat_inject(None, 10, 0, 1, 0.5, 1) == B.EINVAL       # NULL tensor
    assert L.peat_inject_batched(None, 0, None) == B.OK
    counts = (ctypes.c_int64 * 1)()
    items = (B.InjectItem * 1)(B.InjectItem(None, 4, 0, 2, 0, 0.5, 1))   # random value, NULL tensor
    assert L.peat_inject_batched(items, 1, counts) == B.EINVAL
    items = (B.InjectItem * 1)(B.InjectItem(None, 4, 0, 5, 0, 0.5, 1))   # past the last model
    assert L.peat_inject_batched(items, 1, counts) == B.EINVAL
    items = (B.InjectItem * 1)(B.InjectItem(None, 4, 0, 9, 0, 0.5, 1))   # unknown model
    assert L.peat_inject_batched(items, 1, counts) == B.EINVAL
    # zero / NaN models ignore the mask; a NULL tensor is still an error
    assert L.peat_inject_model(None, 10, 0, 1, 0.5, 1, 0) == B.EINVAL
    assert L.peat_inject_model(None, 10, 0, 1, 0.5, 0, 0) == B.EBITMASK
    assert L.peat_inject_model(None, 10, 0, 1, 0.5, 2, 1) == B.EINVAL      # NULL tensor
    assert L.peat_inject_model(None, 10, 0, 1, 0.5, 5, 1) == B.EINVAL      # unknown model


def test_error_model_validation_codes():
    L = P.lib()
    pos = (ctypes.c_int64 * 4)()
    assert L.peat_corrupt_positions(None, 10, 0, 1, 1, 0, 0, pos) == 0          # nothing to corrupt
    assert L.peat_corrupt_positions(None, 10, 0, 1, 1, 3, 0, pos) == B.EINVAL   # NULL tensor
    assert L.peat_corrupt_positions(None, 10, 0, 1, 1, 11, 0, pos) == B.EINVAL  # num_pos > n
    assert L.peat_corrupt_positions(None, 10 ** 6, 0, 1, 1, 4097, 0, pos) == B.EINVAL
    assert L.peat_corrupt_positions(None, 10, 0, 1, 7, 1, 0, pos) == B.EINVAL   # unknown model
    assert L.peat_corrupt_positions(None, 10, 0, 1, 5, 1, 0, pos) == B.EINVAL
    assert L.peat_corrupt_positions(None, 10, 0, 1, 0, 1, 0, pos) == B.EBITMASK
    assert L.peat_corrupt_positions(None, 10, 5, 1, 1, 1, 0, pos) == B.EDTYPE
    assert L.peat_cast_round(None, 0, 1) == B.OK
    assert L.peat_cast_round(None, 4, 1) == B.EINVAL
    assert L.peat_cast_round(None, 4, 0) == B.EDTYPE
    # tensors must be aligned to their element size
    assert L.peat_inject(18, 4, 0, 1, 0.5, 1) == B.EINVAL
    assert L.peat_inject_model(17, 4, 1, 1, 0.5, 1, 0) == B.EINVAL
    assert L.peat_corrupt_positions(18, 10, 0, 1, 1, 1, 0, pos) == B.EINVAL
    assert L.peat_cast_round(18, 4, 1) == B.EINVAL


def test_stream_read_validation_codes():
    L = P.lib()
    assert L.peat_stream_read(None, 0, None, None) == B.OK          # nothing to read
    assert L.peat_stream_read(None, -16, None, None) == B.EINVAL
    assert L.peat_stream_read(None, 16, None, None) == B.EINVAL     # NULL buffer
    assert L.peat_stream_read(16, 15, 64, None) == B.EINVAL         # size not a multiple of 16
    assert L.peat_stream_read(8, 16, 64, None) == B.EINVAL          # misaligned buffer
    assert L.peat_stream_read(16, 16, 2, None) == B.EINVAL          # misaligned sink


def test_topk_validation_codes():
    L = P.lib()
    out = B.TopK()
    outs = (B.TopK * 1)()
    assert L.peat_topk_mean(None, None, 4, 0, 1, 10, ctypes.byref(out)) == B.EINVAL      # NULL tensors
    assert L.peat_topk_mean(None, None, 0, 0, 0, 10, ctypes.byref(out)) == B.EINVAL      # num < 1
    assert L.peat_topk_mean(None, None, 0, 0, 11, 10, ctypes.byref(out)) == B.EINVAL     # num > den
    assert L.peat_topk_mean(None, None, 0, 0, 1, (1 << 20) + 1, ctypes.byref(out)) == B.EINVAL
    assert L.peat_topk_mean(None, None, 0, 7, 1, 10, ctypes.byref(out)) == B.EDTYPE
    assert L.peat_topk_mean(None, None, 0, 0, 1, 10, None) == B.EINVAL
    assert L.peat_topk_mean_batched(None, 0, 1, 10, outs) == B.OK                        # nothing to do
    assert L.peat_topk_mean_batched(None, -1, 1, 10, outs) == B.EINVAL
    pairs = (B.Pair * 1)(B.Pair(None, None, 4, 0, 0))
    assert L.peat_topk_mean_batched(pairs, 1, 1, 10, outs) == B.EINVAL                    # NULL tensors


def test_mixed_pair_validation_codes():
    L = P.lib()
    b = B.Bins(-40, 24, 64, 0)
    th = B.Thresholds()
    out = B.Signature()
    F32, F16, BF16, F64 = B.F32, B.F16, B.BF16, B.F64
    # the golden side is never binary64; the formats must nest
    for g, t in [(F64, F32), (F64, F64), (F16, BF16), (BF16, F16), (F32, 9), (-1, F32)]:
        assert L.peat_signature_mixed(None, g, None, t, 0, ctypes.byref(b), ctypes.byref(th),
                                      ctypes.byref(out)) == B.EDTYPE, (g, t)
    assert L.peat_signature_mixed(None, F32, None, F64, 4, ctypes.byref(b), ctypes.byref(th),
                                  ctypes.byref(out)) == B.EINVAL          # NULL tensors
    assert L.peat_signature_mixed(None, F32, None, F64, -1, ctypes.byref(b), ctypes.byref(th),
                                  ctypes.byref(out)) == B.EINVAL
    assert L.peat_signature_mixed(None, F32, None, F64, 0, ctypes.byref(b), ctypes.byref(th), None) == B.EINVAL
    assert L.peat_signature_mixed(16, F32, 20, F64, 4, ctypes.byref(b), ctypes.byref(th),
                                  ctypes.byref(out)) == B.EINVAL          # test not 8-byte aligned
    # binary64 is not a same-type pair type
    assert _sig_rc(dtype=F64) == B.EDTYPE
    outs = (B.Signature * 2)()
    pairs = (B.MixedPair * 2)(B.MixedPair(None, None, 0, F32, F64), B.MixedPair(None, None, 0, F16, BF16))
    assert L.peat_signature_mixed_batched(pairs, 2, ctypes.byref(b), ctypes.byref(th), outs) == B.EDTYPE
    assert L.peat_signature_mixed_batched(None, 0, ctypes.byref(b), ctypes.byref(th), None) == B.OK
    assert L.peat_signature_mixed_batched(None, -1, ctypes.byref(b), ctypes.byref(th), None) == B.EINVAL
    assert L.peat_signature_mixed_batched_async(pairs, 2, ctypes.byref(b), ctypes.byref(th), None, None) == B.EDTYPE
    assert L.peat_signature_mixed_batched_async(None, 0, ctypes.byref(b), ctypes.byref(th), None, None) == B.OK
    touts = (B.TopK * 2)()
    assert L.peat_topk_mean_mixed_batched(pairs, 2, 1, 10, touts) == B.EDTYPE
    assert L.peat_topk_mean_mixed_batched(pairs, 1, 0, 10, touts) == B.EINVAL          # num < 1
    assert L.peat_topk_mean_mixed_batched(None, 0, 1, 10, touts) == B.OK


def test_finalize_stats_host():
    s = B.Signature()
    s.n_finite = 4
    s.n_valid = 4
    s.n_rel = 2
    s.sum_abs = 2.0
    s.sum_sq = 2.0
    s.sum_g2 = 4.0
    s.sum_t2 = 9.0
    s.sum_gt = 6.0
    s.sum_rel = 1.0
    s.sum_ulp = 10
    st = B.Stats()
    assert P.lib().peat_finalize_stats(ctypes.byref(s), ctypes.byref(st)) == B.OK
    assert st.mean_abs == 0.5 and st.var_abs == (2.0 - 2.0 * 0.5) / 3.0
    assert st.cos == 1.0 and st.l2_g == 2.0 and st.l2_t == 3.0
    assert st.mean_rel == 0.5 and st.mean_ulp == 2.5


@pytest.mark.skipif(__import__("torch").cuda.is_available(), reason="checks the no-GPU error path")
def test_no_device_is_an_error_not_a_crash():
    rc = _sig_rc(n=0)
    assert rc in (B.EHIP, B.ENODEV)
    assert P.lib().peat_init() in (B.EHIP, B.ENODEV)


def test_inject_signature_validation_codes():
    """The fused injection + signature call: rate, bitmask and seeds are
    checked, and test tensors may not overlap another tensor of the batch;
    all before any device access (the pointers below are never touched)."""
    L = P.lib()
    b = B.Bins(-40, 24, 64, 0)
    th = B.Thresholds()
    th.count = 1
    th.abs_tol[0] = 1e-6
    seeds = (ctypes.c_uint64 * 3)(1, 2, 3)

    def rc(pairs, rate=1e-6, mask=0x7F800000, sd=seeds, outs=None):
        arr = (B.Pair * max(1, len(pairs)))(*[B.Pair(g, t, n, dt, 0) for g, t, n, dt in pairs])
        return L.peat_inject_signature_batched_async(arr, len(pairs), sd, rate, mask, ctypes.byref(b),
                                                     ctypes.byref(th), outs, outs, None)

    A = 1 << 40                                  # fake, aligned device addresses
    assert L.peat_inject_signature_batched_async(None, 0, None, 1e-6, 1, ctypes.byref(b), ctypes.byref(th),
                                                 None, None, None) == B.OK
    ok_pairs = [(A, A + 4096, 1000, 0), (A, A + 8192, 1000, 0)]      # shared golden, distinct tests
    assert rc(ok_pairs) == B.EINVAL and b"d_outs" in L.peat_last_error()
    assert rc(ok_pairs, rate=math.nan) == B.ERATE
    assert rc(ok_pairs, rate=-1.0) == B.ERATE
    assert rc(ok_pairs, mask=0) == B.EBITMASK
    assert rc([(A, A + 4096, 1000, 1)], mask=1 << 16) == B.EBITMASK    # beyond binary16
    assert rc(ok_pairs, sd=None) == B.EINVAL and b"seeds" in L.peat_last_error()
    assert rc([(A, A, 1000, 0)]) == B.EINVAL and b"overlaps" in L.peat_last_error()
    assert rc([(A, A + 4096, 1000, 0), (A + 16384, A + 4096 + 3996, 10, 0)]) == B.EINVAL   # two tests
    assert rc([(A, A + 4096, 1000, 0), (A + 4100, A + 65536, 10, 0)]) == B.EINVAL          # golden in a test
    assert rc([(A, A + 3996, 1000, 0)]) == B.EINVAL and b"overlaps" in L.peat_last_error()  # own golden
    # adjacent tensors and empty pairs do not overlap
    assert rc([(A, A + 4000, 1000, 0), (A + 8192, A + 4000, 0, 0)]) == B.EINVAL and b"d_outs" in L.peat_last_error()


def test_topk_from_signature_validation_codes():
    """Top-k from signatures: the records are checked against the pairs and
    the bins before any device access (the pointers below are never touched)."""
    L = P.lib()
    A = 1 << 40
    arr = (B.Pair * 1)(B.Pair(A, A + 4096, 1000, 0, 0))
    outs = (B.TopK * 1)()
    b = B.Bins(-40, 24, 64, 0)
    sig = B.Signature()
    sig.n, sig.n_valid, sig.hist_zero = 1000, 1000, 1000
    recs = (B.Signature * 1)(sig)
    call = L.peat_topk_mean_from_signature_batched
    assert call(None, 0, 1, 10, None, None, None) == B.OK
    assert call(arr, 1, 1, 10, None, ctypes.byref(b), outs) == B.EINVAL and b"sigs" in L.peat_last_error()
    assert call(arr, 1, 1, 10, recs, None, outs) == B.EINVAL and b"bins" in L.peat_last_error()
    assert call(arr, 1, 1, 10, recs, ctypes.byref(B.Bins(-40, 24, 7, 0)), outs) == B.EINVAL   # 7 does not divide 64
    assert call(arr, 1, 0, 10, recs, ctypes.byref(b), outs) == B.EINVAL                       # num < 1
    bad = B.Signature()
    bad.n, bad.n_valid, bad.hist_zero = 999, 999, 999                  # another pair's record
    assert call(arr, 1, 1, 10, (B.Signature * 1)(bad), ctypes.byref(b), outs) == B.EINVAL
    assert b"does not match" in L.peat_last_error()
    bad2 = B.Signature()
    bad2.n, bad2.n_valid, bad2.hist_zero = 1000, 1000, 990             # histogram total below n_valid
    assert call(arr, 1, 1, 10, (B.Signature * 1)(bad2), ctypes.byref(b), outs) == B.EINVAL


def test_signature_dict_round_trip():
    """dict_to_sig is the inverse of sig_to_dict (the records the top-k call
    takes back from Python)."""
    s = B.Signature()
    for i, (name, typ) in enumerate(B._SIG_FIELDS):
        if name in ("n_mismatch", "hist"):
            arr = getattr(s, name)
            for j in range(len(arr)):
                arr[j] = 1000 * i + j
        elif typ is ctypes.c_double:
            setattr(s, name, 0.5 + i)
        else:
            setattr(s, name, 7 * i + 1)
    d = B.sig_to_dict(s)
    assert B.sig_to_dict(B.dict_to_sig(d)) == d
    assert bytes(B.dict_to_sig(d)) == bytes(s)


def test_sig_to_dict_matches_field_by_field_reading():
    """The one-step unpacking of a record equals reading the struct field by
    field (random bit patterns: NaN and infinite doubles, negative and
    unsigned 64-bit integers), for every number of thresholds."""
    import random
    rng = random.Random(11)
    for _ in range(200):
        raw = bytes(rng.getrandbits(8) for _ in range(ctypes.sizeof(B.Signature)))
        s = B.Signature.from_buffer_copy(raw)
        for nthr in (None, 0, 1, 2, 8):
            d = B.sig_to_dict(s, nthr=nthr)
            assert list(d) == [name for name, _ in B._SIG_FIELDS]
            for name, typ in B._SIG_FIELDS:
                want = getattr(s, name)
                got = d[name]
                if name in ("n_mismatch", "hist"):
                    want = list(want)[: (B.MAX_THRESHOLDS if nthr is None else nthr)] if name == "n_mismatch" \
                        else list(want)
                    assert got == want and all(type(x) is int for x in got), name
                elif typ is ctypes.c_double:
                    assert type(got) is float and (got == want or (math.isnan(got) and math.isnan(want))), name
                else:
                    assert type(got) is int and got == want, name


def test_batched_record_decoding_matches_single():
    """Records decoded in one pass over a buffer (batched calls, device
    records) and one by one from numpy records equal sig_to_dict's."""
    import numpy as np
    rng = np.random.default_rng(12)
    raw = rng.integers(0, 256, size=(64, ctypes.sizeof(B.Signature)), dtype=np.uint8)
    arr = (B.Signature * 64).from_buffer_copy(raw.tobytes())
    recs = raw.view(B.SIG_NP_DTYPE).reshape(-1)

    def same(a, b):
        assert list(a) == list(b)
        for k in a:
            if isinstance(a[k], float) and math.isnan(a[k]):
                assert math.isnan(b[k])
            else:
                assert a[k] == b[k] and type(a[k]) is type(b[k]), k

    for nthr in (None, 2):
        batch = B._records_to_dicts(raw, 64, nthr)
        assert len(batch) == 64
        for i in range(64):
            ref = B.sig_to_dict(arr[i], nthr=nthr)
            same(ref, batch[i])
            same(ref, B.record_to_dict(recs[i], nthr))
