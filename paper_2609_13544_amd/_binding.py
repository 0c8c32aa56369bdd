"""ctypes binding of libpeat (include/peat.h): argument marshalling only.

Every step of the signature and the injector runs in the HIP kernels of
libpeat.so; this module converts torch tensors to device pointers and streams,
packs the C structs and unpacks the results.  If the library is missing the
calls raise -- there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os
import struct
import threading

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libpeat.so")

F32, F16, BF16, F64 = 0, 1, 2, 3
MODEL_BITFLIP, MODEL_ZERO, MODEL_VALUE, MODEL_NAN, MODEL_UNIFORM = 0, 1, 2, 3, 4
MAX_POSITIONS = 4096
OK, EINVAL, EDTYPE, EBITMASK, ERATE, EHIP, ENOMEM, ENODEV = 0, -1, -2, -3, -4, -5, -6, -7
MAX_THRESHOLDS, MAX_BINS = 8, 64

# kernel classes of peat_profile_read
K_SIG_CHUNK, K_SIG_FINALIZE, K_INJECT, K_INJECT_SUM, K_STREAM_READ, K_TOPK_A, K_TOPK_B = 0, 1, 2, 3, 4, 5, 6
K_SIG_INJECT = 7   # chunk pass with the injection


class PeatError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str):
        super().__init__(f"{where} failed with {code}: {detail}")
        self.code = code


class Bins(ctypes.Structure):
    _fields_ = [("lo_log2", ctypes.c_int32), ("hi_log2", ctypes.c_int32),
                ("nbins", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class Thresholds(ctypes.Structure):
    _fields_ = [("count", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("abs_tol", ctypes.c_double * MAX_THRESHOLDS), ("rel_tol", ctypes.c_double * MAX_THRESHOLDS)]


_SIG_FIELDS = [
    ("n", ctypes.c_int64), ("n_valid", ctypes.c_int64), ("n_finite", ctypes.c_int64),
    ("n_rel", ctypes.c_int64), ("n_nan_golden", ctypes.c_int64), ("n_nan_test", ctypes.c_int64),
    ("n_inf_golden", ctypes.c_int64), ("n_inf_test", ctypes.c_int64),
    ("n_nan_pairs", ctypes.c_int64), ("first_nan_index", ctypes.c_int64),
    ("n_mismatch", ctypes.c_int64 * MAX_THRESHOLDS),
    ("hist_zero", ctypes.c_int64), ("hist_under", ctypes.c_int64), ("hist_over", ctypes.c_int64),
    ("hist", ctypes.c_int64 * MAX_BINS),
    ("max_abs", ctypes.c_double), ("argmax_abs", ctypes.c_int64),
    ("max_ulp", ctypes.c_int64), ("argmax_ulp", ctypes.c_int64), ("sum_ulp", ctypes.c_uint64),
    ("max_rel", ctypes.c_double), ("argmax_rel", ctypes.c_int64),
    ("sum_abs", ctypes.c_double), ("sum_sq", ctypes.c_double), ("sum_rel", ctypes.c_double),
    ("sum_g2", ctypes.c_double), ("sum_t2", ctypes.c_double), ("sum_gt", ctypes.c_double),
]


class Signature(ctypes.Structure):
    _fields_ = _SIG_FIELDS


class Stats(ctypes.Structure):
    _fields_ = [(k, ctypes.c_double) for k in
                ("mean_abs", "var_abs", "l2_err", "l2_g", "l2_t", "cos", "mean_rel", "mean_ulp")]


class TopK(ctypes.Structure):
    _fields_ = [("n_valid", ctypes.c_int64), ("k", ctypes.c_int64), ("count_above", ctypes.c_int64),
                ("kth_value", ctypes.c_double), ("sum_topk", ctypes.c_double), ("mean_topk", ctypes.c_double)]


class Series(ctypes.Structure):
    _fields_ = [("count", ctypes.c_int64)] + [(k, ctypes.c_double) for k in ("mean", "var", "std", "min", "max")]


class Pair(ctypes.Structure):
    _fields_ = [("golden", ctypes.c_void_p), ("test", ctypes.c_void_p), ("n", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class MixedPair(ctypes.Structure):
    _fields_ = [("golden", ctypes.c_void_p), ("test", ctypes.c_void_p), ("n", ctypes.c_int64),
                ("golden_dtype", ctypes.c_int32), ("test_dtype", ctypes.c_int32)]


class InjectItem(ctypes.Structure):
    _fields_ = [("tensor", ctypes.c_void_p), ("n", ctypes.c_int64), ("dtype", ctypes.c_int32),
                ("model", ctypes.c_int32), ("seed", ctypes.c_uint64), ("rate", ctypes.c_double),
                ("bitmask", ctypes.c_uint64)]


def _np_sig_dtype():
    fields = []
    for name, ct in _SIG_FIELDS:
        if name in ("n_mismatch", "hist"):
            fields.append((name, np.int64, (ct._length_,)))
        elif ct is ctypes.c_double:
            fields.append((name, np.float64))
        elif ct is ctypes.c_uint64:
            fields.append((name, np.uint64))
        else:
            fields.append((name, np.int64))
    dt = np.dtype(fields)
    assert dt.itemsize == ctypes.sizeof(Signature)
    return dt


SIG_NP_DTYPE = _np_sig_dtype()
SIG_BYTES = ctypes.sizeof(Signature)

_lib = None
_lock = threading.Lock()

# name -> (restype, argtypes) of every entry point in include/peat.h
_PROTOS = {
    "peat_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "peat_last_error": (ctypes.c_char_p, []),
    "peat_abi_version": (ctypes.c_int, []),
    "peat_init": (ctypes.c_int, []),
    "peat_set_stream": (ctypes.c_int, [ctypes.c_void_p]),
    "peat_signature": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                      ctypes.POINTER(Bins), ctypes.POINTER(Thresholds),
                                      ctypes.POINTER(Signature)]),
    "peat_signature_batched": (ctypes.c_int, [ctypes.POINTER(Pair), ctypes.c_int32, ctypes.POINTER(Bins),
                                              ctypes.POINTER(Thresholds), ctypes.POINTER(Signature)]),
    "peat_signature_batched_async": (ctypes.c_int, [ctypes.POINTER(Pair), ctypes.c_int32,
                                                    ctypes.POINTER(Bins), ctypes.POINTER(Thresholds),
                                                    ctypes.c_void_p, ctypes.c_void_p]),
    "peat_signature_batched_noalloc": (ctypes.c_int, [ctypes.POINTER(Pair), ctypes.c_int32,
                                                      ctypes.POINTER(Bins), ctypes.POINTER(Thresholds),
                                                      ctypes.c_void_p, ctypes.c_void_p]),
    "peat_inject_signature_batched_async": (ctypes.c_int, [ctypes.POINTER(Pair), ctypes.c_int32,
                                                           ctypes.POINTER(ctypes.c_uint64), ctypes.c_double,
                                                           ctypes.c_uint64, ctypes.POINTER(Bins),
                                                           ctypes.POINTER(Thresholds), ctypes.c_void_p,
                                                           ctypes.c_void_p, ctypes.c_void_p]),
    "peat_inject": (ctypes.c_int64, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_uint64,
                                     ctypes.c_double, ctypes.c_uint64]),
    "peat_inject_model": (ctypes.c_int64, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_uint64,
                                           ctypes.c_double, ctypes.c_int32, ctypes.c_uint64]),
    "peat_corrupt_positions": (ctypes.c_int64, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_uint64,
                                                ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64,
                                                ctypes.POINTER(ctypes.c_int64)]),
    "peat_cast_round": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int]),
    "peat_inject_batched": (ctypes.c_int, [ctypes.POINTER(InjectItem), ctypes.c_int32,
                                           ctypes.POINTER(ctypes.c_int64)]),
    "peat_inject_batched_async": (ctypes.c_int, [ctypes.POINTER(InjectItem), ctypes.c_int32,
                                                 ctypes.c_void_p, ctypes.c_void_p]),
    "peat_topk_mean": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                      ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(TopK)]),
    "peat_topk_mean_batched": (ctypes.c_int, [ctypes.POINTER(Pair), ctypes.c_int32, ctypes.c_int32,
                                              ctypes.c_int32, ctypes.POINTER(TopK)]),
    "peat_signature_mixed": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                            ctypes.c_int64, ctypes.POINTER(Bins), ctypes.POINTER(Thresholds),
                                            ctypes.POINTER(Signature)]),
    "peat_signature_mixed_batched": (ctypes.c_int, [ctypes.POINTER(MixedPair), ctypes.c_int32,
                                                    ctypes.POINTER(Bins), ctypes.POINTER(Thresholds),
                                                    ctypes.POINTER(Signature)]),
    "peat_signature_mixed_batched_async": (ctypes.c_int, [ctypes.POINTER(MixedPair), ctypes.c_int32,
                                                          ctypes.POINTER(Bins), ctypes.POINTER(Thresholds),
                                                          ctypes.c_void_p, ctypes.c_void_p]),
    "peat_topk_mean_mixed_batched": (ctypes.c_int, [ctypes.POINTER(MixedPair), ctypes.c_int32, ctypes.c_int32,
                                                    ctypes.c_int32, ctypes.POINTER(TopK)]),
    "peat_topk_mean_from_signature_batched": (ctypes.c_int, [ctypes.POINTER(Pair), ctypes.c_int32, ctypes.c_int32,
                                                             ctypes.c_int32, ctypes.POINTER(Signature),
                                                             ctypes.POINTER(Bins), ctypes.POINTER(TopK)]),
    "peat_topk_mean_mixed_from_signature_batched": (ctypes.c_int, [ctypes.POINTER(MixedPair), ctypes.c_int32,
                                                                   ctypes.c_int32, ctypes.c_int32,
                                                                   ctypes.POINTER(Signature), ctypes.POINTER(Bins),
                                                                   ctypes.POINTER(TopK)]),
    "peat_topk_mean_batched_async": (ctypes.c_int, [ctypes.POINTER(Pair), ctypes.c_int32, ctypes.c_int32,
                                                    ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "peat_topk_mean_mixed_batched_async": (ctypes.c_int, [ctypes.POINTER(MixedPair), ctypes.c_int32,
                                                          ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                                          ctypes.c_void_p]),
    "peat_topk_mean_from_signature_batched_async": (ctypes.c_int, [ctypes.POINTER(Pair), ctypes.c_int32,
                                                                   ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                                                   ctypes.POINTER(Bins), ctypes.c_void_p,
                                                                   ctypes.c_void_p]),
    "peat_topk_mean_mixed_from_signature_batched_async": (ctypes.c_int, [ctypes.POINTER(MixedPair),
                                                                         ctypes.c_int32, ctypes.c_int32,
                                                                         ctypes.c_int32, ctypes.c_void_p,
                                                                         ctypes.POINTER(Bins), ctypes.c_void_p,
                                                                         ctypes.c_void_p]),
    "peat_topk_set_entry_capacity": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int64]),
    "peat_stream_read": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]),
    "peat_finalize_stats": (ctypes.c_int, [ctypes.POINTER(Signature), ctypes.POINTER(Stats)]),
    "peat_series_stats": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(Series)]),
    "peat_spearman": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                     ctypes.POINTER(ctypes.c_double)]),
    "peat_normalize_scores": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]),
    "peat_profile_enable": (ctypes.c_int, [ctypes.c_int]),
    "peat_profile_read": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_int64)]),
}


def lib():
    """The loaded libpeat.so; raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                    "(there is no CPU fallback)")
            L = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in _PROTOS.items():
                fn = getattr(L, name)
                fn.restype = res
                fn.argtypes = args
            _lib = L
    return _lib


def _check(rc: int, where: str) -> int:
    if rc < 0:
        L = lib()
        detail = L.peat_last_error().decode() or L.peat_strerror(rc).decode()
        raise PeatError(rc, where, detail)
    return rc


def strerror(code: int) -> str:
    return lib().peat_strerror(code).decode()


# ---------------------------------------------------------------------------
# marshalling helpers
# ---------------------------------------------------------------------------
def _torch():
    import torch
    return torch


_DTYPE_CODES: dict = {}


def dtype_code(t) -> int:
    if not _DTYPE_CODES:
        torch = _torch()
        _DTYPE_CODES.update({torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16, torch.float64: F64})
    code = _DTYPE_CODES.get(t.dtype)
    if code is None:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return code


def _dev_tensor(t, name: str):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def make_bins(bins) -> Bins:
    return Bins(int(bins[0]), int(bins[1]), int(bins[2]), 0)


def make_thresholds(thresholds) -> Thresholds:
    """Absolute tolerances, or (abs_tol, rel_tol) pairs (torch.isclose's atol
    and rtol)."""
    th = Thresholds()
    th.count = len(thresholds)
    th.reserved = 0
    for j, v in enumerate(list(thresholds)[:MAX_THRESHOLDS]):
        if isinstance(v, (tuple, list)):
            th.abs_tol[j], th.rel_tol[j] = float(v[0]), float(v[1])
        else:
            th.abs_tol[j] = float(v)
    return th


def _stream_ptr(stream) -> int | None:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _sig_layout():
    """One struct format for the whole record and, per field, its slice of
    the unpacked values (None for a scalar)."""
    codes = {ctypes.c_int64: "q", ctypes.c_uint64: "Q", ctypes.c_double: "d"}
    fmt, layout, pos = "<", [], 0
    for name, typ in _SIG_FIELDS:
        if hasattr(typ, "_length_"):
            fmt += codes[typ._type_] * typ._length_
            layout.append((name, pos, typ._length_))
            pos += typ._length_
        else:
            fmt += codes[typ]
            layout.append((name, pos, None))
            pos += 1
    return struct.Struct(fmt), layout


_SIG_STRUCT, _SIG_LAYOUT = _sig_layout()
assert _SIG_STRUCT.size == ctypes.sizeof(Signature)


def _vals_to_dict(vals, nthr: int | None) -> dict:
    """A record's unpacked values by field name (ints, floats, lists for the
    two arrays; n_mismatch cut to the thresholds used)."""
    d = {}
    for name, pos, length in _SIG_LAYOUT:
        if length is None:
            d[name] = vals[pos]
        elif name == "n_mismatch":
            d[name] = list(vals[pos:pos + (MAX_THRESHOLDS if nthr is None else nthr)])
        else:
            d[name] = list(vals[pos:pos + length])
    return d


def sig_to_dict(s: Signature, nbins: int | None = None, nthr: int | None = None) -> dict:
    """The record's fields by name, unpacked in one step."""
    return _vals_to_dict(_SIG_STRUCT.unpack(ctypes.string_at(ctypes.addressof(s), _SIG_STRUCT.size)), nthr)


def _records_to_dicts(buf, count: int, nthr: int | None) -> list[dict]:
    """count consecutive records held in a bytes-like buffer, decoded."""
    raw = bytes(memoryview(buf).cast("B")[: count * _SIG_STRUCT.size])
    return [_vals_to_dict(v, nthr) for v in _SIG_STRUCT.iter_unpack(raw)]


def dict_to_sig(d: dict) -> Signature:
    """A Signature struct holding the fields of a record dict (lists padded with 0)."""
    s = Signature()
    for name, typ in _SIG_FIELDS:
        v = d[name]
        if name in ("n_mismatch", "hist"):
            arr = getattr(s, name)
            for i, x in enumerate(v):
                arr[i] = int(x)
        else:
            setattr(s, name, float(v) if typ is ctypes.c_double else int(v))
    return s


def record_to_dict(rec, nthr: int | None = None) -> dict:
    """Convert one element of a SIG_NP_DTYPE array to a dict."""
    return _vals_to_dict(_SIG_STRUCT.unpack(rec.tobytes()), nthr)


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------
def set_stream(stream=None) -> None:
    _check(lib().peat_set_stream(_stream_ptr(stream)), "peat_set_stream")


def signature(golden, test, bins=(-40, 24, 64), thresholds=(1e-6, 1e-3), *, dtype: int | None = None,
              n: int | None = None) -> dict:
    """peat_signature on two device tensors (same dtype and element count)."""
    _dev_tensor(golden, "golden")
    _dev_tensor(test, "test")
    code = dtype_code(golden) if dtype is None else dtype
    if n is None:
        if golden.numel() != test.numel() or golden.dtype != test.dtype:
            raise ValueError("golden and test differ in size or dtype")
        n = golden.numel()
    out = Signature()
    b, th = make_bins(bins), make_thresholds(thresholds)
    set_stream()
    _check(lib().peat_signature(golden.data_ptr() if n else None, test.data_ptr() if n else None,
                                n, code, ctypes.byref(b), ctypes.byref(th), ctypes.byref(out)),
           "peat_signature")
    return sig_to_dict(out, nthr=len(thresholds))


def _pairs_array(pairs):
    arr = (Pair * max(1, len(pairs)))()
    for k, p in enumerate(pairs):
        if isinstance(p, Pair):
            arr[k] = p
            continue
        g, t = p[0], p[1]
        _dev_tensor(g, f"pairs[{k}].golden")
        _dev_tensor(t, f"pairs[{k}].test")
        if g.numel() != t.numel() or g.dtype != t.dtype:
            raise ValueError(f"pair {k}: golden and test differ in size or dtype")
        arr[k] = Pair(g.data_ptr(), t.data_ptr(), g.numel(), dtype_code(g), 0)
    return arr


def signature_batched(pairs, bins=(-40, 24, 64), thresholds=(1e-6, 1e-3)) -> list[dict]:
    """peat_signature_batched over a list of (golden, test) device tensor pairs."""
    arr = _pairs_array(pairs)
    outs = (Signature * max(1, len(pairs)))()
    b, th = make_bins(bins), make_thresholds(thresholds)
    set_stream()
    _check(lib().peat_signature_batched(arr, len(pairs), ctypes.byref(b), ctypes.byref(th), outs),
           "peat_signature_batched")
    return _records_to_dicts(outs, len(pairs), len(thresholds))


def signature_mixed(golden, test, bins=(-40, 24, 64), thresholds=(1e-6, 1e-3)) -> dict:
    """peat_signature_mixed on two device tensors of the same element count
    whose types may differ (e.g. a float32 golden and a float64 or float16 test)."""
    _dev_tensor(golden, "golden")
    _dev_tensor(test, "test")
    if golden.numel() != test.numel():
        raise ValueError("golden and test differ in size")
    n = golden.numel()
    out = Signature()
    b, th = make_bins(bins), make_thresholds(thresholds)
    set_stream()
    _check(lib().peat_signature_mixed(golden.data_ptr() if n else None, dtype_code(golden),
                                      test.data_ptr() if n else None, dtype_code(test), n,
                                      ctypes.byref(b), ctypes.byref(th), ctypes.byref(out)),
           "peat_signature_mixed")
    return sig_to_dict(out, nthr=len(thresholds))


def _mixed_pairs_array(pairs):
    arr = (MixedPair * max(1, len(pairs)))()
    for k, p in enumerate(pairs):
        if isinstance(p, MixedPair):
            arr[k] = p
            continue
        g, t = p[0], p[1]
        _dev_tensor(g, f"pairs[{k}].golden")
        _dev_tensor(t, f"pairs[{k}].test")
        if g.numel() != t.numel():
            raise ValueError(f"pair {k}: golden and test differ in size")
        arr[k] = MixedPair(g.data_ptr(), t.data_ptr(), g.numel(), dtype_code(g), dtype_code(t))
    return arr


def signature_mixed_batched(pairs, bins=(-40, 24, 64), thresholds=(1e-6, 1e-3)) -> list[dict]:
    """peat_signature_mixed_batched over (golden, test) device tensor pairs of
    any accepted type combination."""
    arr = _mixed_pairs_array(pairs)
    outs = (Signature * max(1, len(pairs)))()
    b, th = make_bins(bins), make_thresholds(thresholds)
    set_stream()
    _check(lib().peat_signature_mixed_batched(arr, len(pairs), ctypes.byref(b), ctypes.byref(th), outs),
           "peat_signature_mixed_batched")
    return _records_to_dicts(outs, len(pairs), len(thresholds))


def signature_mixed_batched_async(pairs, d_out, bins=(-40, 24, 64), thresholds=(1e-6, 1e-3),
                                  stream=None) -> None:
    """peat_signature_mixed_batched_async: records land in d_out, a device uint8
    tensor of at least len(pairs) * SIG_BYTES bytes, when the stream gets there."""
    arr = _mixed_pairs_array(pairs)
    _dev_tensor(d_out, "d_out")
    if d_out.numel() * d_out.element_size() < len(pairs) * SIG_BYTES:
        raise ValueError("d_out too small")
    b, th = make_bins(bins), make_thresholds(thresholds)
    _check(lib().peat_signature_mixed_batched_async(arr, len(pairs), ctypes.byref(b), ctypes.byref(th),
                                                    d_out.data_ptr(), _stream_ptr(stream)),
           "peat_signature_mixed_batched_async")


def topk_mean_mixed_batched(pairs, num: int = 1, den: int = 10) -> list[dict]:
    """peat_topk_mean_mixed_batched over (golden, test) device tensor pairs of
    any accepted type combination."""
    arr = _mixed_pairs_array(pairs)
    outs = (TopK * max(1, len(pairs)))()
    set_stream()
    _check(lib().peat_topk_mean_mixed_batched(arr, len(pairs), num, den, outs), "peat_topk_mean_mixed_batched")
    return [topk_to_dict(outs[k]) for k in range(len(pairs))]


def topk_to_dict(t: TopK) -> dict:
    return {name: (float(getattr(t, name)) if typ is ctypes.c_double else int(getattr(t, name)))
            for name, typ in TopK._fields_}


def topk_mean(golden, test, num: int = 1, den: int = 10, *, dtype: int | None = None,
              n: int | None = None) -> dict:
    """peat_topk_mean: mean of the ceil(n_valid num/den) largest errors of
    two device tensors (default: the top 10%)."""
    _dev_tensor(golden, "golden")
    _dev_tensor(test, "test")
    code = dtype_code(golden) if dtype is None else dtype
    if n is None:
        if golden.numel() != test.numel() or golden.dtype != test.dtype:
            raise ValueError("golden and test differ in size or dtype")
        n = golden.numel()
    out = TopK()
    set_stream()
    _check(lib().peat_topk_mean(golden.data_ptr() if n else None, test.data_ptr() if n else None, n, code,
                                num, den, ctypes.byref(out)), "peat_topk_mean")
    return topk_to_dict(out)


def topk_mean_batched(pairs, num: int = 1, den: int = 10) -> list[dict]:
    """peat_topk_mean_batched over a list of (golden, test) device tensor pairs
    (or a PreparedPairs)."""
    if isinstance(pairs, PreparedPairs):
        arr, count = pairs.arr, pairs.count
    else:
        arr, count = _pairs_array(pairs), len(pairs)
    outs = (TopK * max(1, count))()
    set_stream()
    _check(lib().peat_topk_mean_batched(arr, count, num, den, outs), "peat_topk_mean_batched")
    return [topk_to_dict(outs[k]) for k in range(count)]


def topk_mean_from_signature_batched(pairs, sigs, bins=(-40, 24, 64), num: int = 1, den: int = 10) -> list[dict]:
    """peat_topk_mean_from_signature_batched: peat_topk_mean_batched given the
    pairs' signatures (record dicts of signature_batched with these bins),
    whose one-binade histograms let the first streaming pass skip the pairs."""
    if isinstance(pairs, PreparedPairs):
        arr, count = pairs.arr, pairs.count
    else:
        arr, count = _pairs_array(pairs), len(pairs)
    if len(sigs) != count:
        raise ValueError("one signature per pair")
    recs = (Signature * max(1, count))()
    for k, d in enumerate(sigs):
        recs[k] = d if isinstance(d, Signature) else dict_to_sig(d)
    b = make_bins(bins)
    outs = (TopK * max(1, count))()
    set_stream()
    _check(lib().peat_topk_mean_from_signature_batched(arr, count, num, den, recs, ctypes.byref(b), outs),
           "peat_topk_mean_from_signature_batched")
    return [topk_to_dict(outs[k]) for k in range(count)]


def topk_mean_mixed_from_signature_batched(pairs, sigs, bins=(-40, 24, 64), num: int = 1,
                                           den: int = 10) -> list[dict]:
    """peat_topk_mean_mixed_from_signature_batched: topk_mean_mixed_batched
    given the pairs' signatures (record dicts of signature_mixed_batched)."""
    arr = _mixed_pairs_array(pairs)
    if len(sigs) != len(pairs):
        raise ValueError("one signature per pair")
    recs = (Signature * max(1, len(pairs)))()
    for k, d in enumerate(sigs):
        recs[k] = d if isinstance(d, Signature) else dict_to_sig(d)
    b = make_bins(bins)
    outs = (TopK * max(1, len(pairs)))()
    set_stream()
    _check(lib().peat_topk_mean_mixed_from_signature_batched(arr, len(pairs), num, den, recs, ctypes.byref(b), outs),
           "peat_topk_mean_mixed_from_signature_batched")
    return [topk_to_dict(outs[k]) for k in range(len(pairs))]


TOPK_BYTES = ctypes.sizeof(TopK)


def _pairs_arg(pairs):
    if isinstance(pairs, PreparedPairs):
        return pairs.arr, pairs.count
    return _pairs_array(pairs), len(pairs)


def _topk_out(d_out, count: int) -> None:
    _dev_tensor(d_out, "d_out")
    if d_out.numel() * d_out.element_size() < count * TOPK_BYTES:
        raise ValueError("d_out too small")


def _sig_in(d_sigs, count: int) -> None:
    _dev_tensor(d_sigs, "d_sigs")
    if d_sigs.numel() * d_sigs.element_size() < count * SIG_BYTES:
        raise ValueError("d_sigs too small")


def topk_mean_batched_async(pairs, d_out, num: int = 1, den: int = 10, stream=None) -> None:
    """peat_topk_mean_batched_async: records land in d_out, a device uint8
    tensor of at least len(pairs) * TOPK_BYTES bytes, when the stream gets
    there (decode_topk reads them)."""
    arr, count = _pairs_arg(pairs)
    _topk_out(d_out, count)
    _check(lib().peat_topk_mean_batched_async(arr, count, num, den, d_out.data_ptr(), _stream_ptr(stream)),
           "peat_topk_mean_batched_async")


def topk_mean_mixed_batched_async(pairs, d_out, num: int = 1, den: int = 10, stream=None) -> None:
    """peat_topk_mean_mixed_batched_async over (golden, test) device tensor
    pairs of any accepted type combination."""
    arr = _mixed_pairs_array(pairs)
    _topk_out(d_out, len(pairs))
    _check(lib().peat_topk_mean_mixed_batched_async(arr, len(pairs), num, den, d_out.data_ptr(),
                                                    _stream_ptr(stream)),
           "peat_topk_mean_mixed_batched_async")


def topk_mean_from_signature_batched_async(pairs, d_sigs, d_out, bins=(-40, 24, 64), num: int = 1,
                                           den: int = 10, stream=None) -> None:
    """peat_topk_mean_from_signature_batched_async: d_sigs holds the pairs'
    device records (as signature_batched_async leaves them, with these bins)."""
    arr, count = _pairs_arg(pairs)
    _sig_in(d_sigs, count)
    _topk_out(d_out, count)
    b = make_bins(bins)
    _check(lib().peat_topk_mean_from_signature_batched_async(arr, count, num, den, d_sigs.data_ptr(),
                                                             ctypes.byref(b), d_out.data_ptr(),
                                                             _stream_ptr(stream)),
           "peat_topk_mean_from_signature_batched_async")


def topk_mean_mixed_from_signature_batched_async(pairs, d_sigs, d_out, bins=(-40, 24, 64), num: int = 1,
                                                 den: int = 10, stream=None) -> None:
    """peat_topk_mean_mixed_from_signature_batched_async: mixed-precision
    pairs with the device records of signature_mixed_batched_async."""
    arr = _mixed_pairs_array(pairs)
    _sig_in(d_sigs, len(pairs))
    _topk_out(d_out, len(pairs))
    b = make_bins(bins)
    _check(lib().peat_topk_mean_mixed_from_signature_batched_async(arr, len(pairs), num, den, d_sigs.data_ptr(),
                                                                   ctypes.byref(b), d_out.data_ptr(),
                                                                   _stream_ptr(stream)),
           "peat_topk_mean_mixed_from_signature_batched_async")


def decode_topk(d_out, count: int) -> list[dict]:
    """Copy device top-k records to the host and decode them."""
    host = d_out.detach().view(-1)[: count * TOPK_BYTES].cpu().numpy().view(np.uint8)
    buf = (TopK * max(1, count)).from_buffer_copy(host.tobytes() if count else bytes(TOPK_BYTES))
    return [topk_to_dict(buf[k]) for k in range(count)]


def topk_set_entry_capacity(binade_entries: int = -1, bin_entries: int = -1) -> None:
    """peat_topk_set_entry_capacity (-1: sized per call)."""
    _check(lib().peat_topk_set_entry_capacity(binade_entries, bin_entries), "peat_topk_set_entry_capacity")


class PreparedPairs:
    """Pair descriptors built once, for repeated asynchronous calls.  The
    descriptors hold raw device addresses, so the object keeps the golden and
    test tensors alive for as long as it exists (a freed tensor's memory could
    otherwise be handed to another tensor and then read or, by the injecting
    calls, written)."""

    def __init__(self, pairs):
        self.count = len(pairs)
        self.arr = _pairs_array(pairs)
        self.tensors = [x for p in pairs if not isinstance(p, Pair) for x in (p[0], p[1])]


def signature_batched_async(pairs, d_out, bins=(-40, 24, 64), thresholds=(1e-6, 1e-3), stream=None) -> None:
    """peat_signature_batched_async: records land in d_out, a device uint8
    tensor of at least len(pairs) * SIG_BYTES bytes, when the stream gets there."""
    prep = pairs if isinstance(pairs, PreparedPairs) else PreparedPairs(pairs)
    _dev_tensor(d_out, "d_out")
    if d_out.numel() * d_out.element_size() < prep.count * SIG_BYTES:
        raise ValueError("d_out too small")
    b, th = make_bins(bins), make_thresholds(thresholds)
    _check(lib().peat_signature_batched_async(prep.arr, prep.count, ctypes.byref(b), ctypes.byref(th),
                                              d_out.data_ptr(), _stream_ptr(stream)),
           "peat_signature_batched_async")


NOALLOC_SCRATCH_BYTES = 64 << 20


def signature_batched_noalloc(pairs, d_out, bins=(-40, 24, 64), thresholds=(1e-6, 1e-3), stream=None) -> None:
    """peat_signature_batched_noalloc: as signature_batched_async, with every
    intermediate buffer in the library's static device scratch array (no
    allocation by the call).  Calls on one GPU that may overlap race."""
    prep = pairs if isinstance(pairs, PreparedPairs) else PreparedPairs(pairs)
    _dev_tensor(d_out, "d_out")
    if d_out.numel() * d_out.element_size() < prep.count * SIG_BYTES:
        raise ValueError("d_out too small")
    b, th = make_bins(bins), make_thresholds(thresholds)
    _check(lib().peat_signature_batched_noalloc(prep.arr, prep.count, ctypes.byref(b), ctypes.byref(th),
                                                d_out.data_ptr(), _stream_ptr(stream)),
           "peat_signature_batched_noalloc")


def inject_signature_batched_async(pairs, seeds, rate: float, bitmask: int, d_out, d_counts,
                                   bins=(-40, 24, 64), thresholds=(1e-6, 1e-3), stream=None) -> None:
    """peat_inject_signature_batched_async: the bit flips of peat_inject
    (seeds[k], rate, bitmask) go into each pair's test tensor and the
    signatures of the flipped pairs land in d_out (device uint8, at least
    len(pairs) * SIG_BYTES bytes); d_counts (device int64, len(pairs)) gets
    the flip counts, when the stream gets there."""
    prep = pairs if isinstance(pairs, PreparedPairs) else PreparedPairs(pairs)
    _dev_tensor(d_out, "d_out")
    _dev_tensor(d_counts, "d_counts")
    if d_out.numel() * d_out.element_size() < prep.count * SIG_BYTES:
        raise ValueError("d_out too small")
    if d_counts.dtype != _torch().int64 or d_counts.numel() < prep.count:
        raise ValueError("d_counts must be an int64 device tensor of len(pairs) entries")
    if len(seeds) != prep.count:
        raise ValueError("one seed per pair")
    sd = (ctypes.c_uint64 * max(1, prep.count))(*[int(x) & (2 ** 64 - 1) for x in seeds])
    b, th = make_bins(bins), make_thresholds(thresholds)
    _check(lib().peat_inject_signature_batched_async(prep.arr, prep.count, sd, float(rate), bitmask & (2 ** 64 - 1),
                                                     ctypes.byref(b), ctypes.byref(th), d_out.data_ptr(),
                                                     d_counts.data_ptr(), _stream_ptr(stream)),
           "peat_inject_signature_batched_async")


def decode_records(d_out, count: int, nthr: int | None = None) -> list[dict]:
    """Copy device records to the host and decode them."""
    host = d_out.detach().view(-1)[: count * SIG_BYTES].cpu().numpy().view(np.uint8)
    return _records_to_dicts(host, count, nthr)


def inject(tensor, seed: int, rate: float, bitmask: int, *, dtype: int | None = None, n: int | None = None) -> int:
    """peat_inject in place on a device tensor; returns the flip count."""
    _dev_tensor(tensor, "tensor")
    code = dtype_code(tensor) if dtype is None else dtype
    n = tensor.numel() if n is None else n
    set_stream()
    rc = lib().peat_inject(tensor.data_ptr() if n else None, n, code, seed & (2 ** 64 - 1), float(rate),
                           bitmask & (2 ** 64 - 1))
    return _check(rc, "peat_inject")


def inject_model(tensor, seed: int, rate: float, model: int, bitmask: int = 0) -> int:
    """peat_inject_model in place: the elements peat_inject would flip are set
    to zero (MODEL_ZERO), NaN (MODEL_NAN), bit-flipped (MODEL_BITFLIP), to the
    tensor's value before the call at a random index (MODEL_VALUE) or to a
    uniformly random bit pattern (MODEL_UNIFORM)."""
    _dev_tensor(tensor, "tensor")
    n = tensor.numel()
    set_stream()
    rc = lib().peat_inject_model(tensor.data_ptr() if n else None, n, dtype_code(tensor), seed & (2 ** 64 - 1),
                                 float(rate), int(model), bitmask & (2 ** 64 - 1))
    return _check(rc, "peat_inject_model")


def corrupt_positions(tensor, seed: int, model: int, num_pos: int, bitmask: int = 0) -> list[int]:
    """peat_corrupt_positions in place (the paper's num_pos corruption);
    returns the positions in order."""
    _dev_tensor(tensor, "tensor")
    n = tensor.numel()
    pos = (ctypes.c_int64 * max(1, int(num_pos)))()
    set_stream()
    rc = lib().peat_corrupt_positions(tensor.data_ptr() if n else None, n, dtype_code(tensor),
                                      seed & (2 ** 64 - 1), int(model), int(num_pos), bitmask & (2 ** 64 - 1), pos)
    _check(rc, "peat_corrupt_positions")
    return [int(pos[k]) for k in range(rc)]


def cast_round(tensor, to_dtype: int) -> None:
    """peat_cast_round: the FP16 (to_dtype=F16) or BF16 error of an f32 device
    tensor, in place (enqueued on the current stream)."""
    _dev_tensor(tensor, "tensor")
    if dtype_code(tensor) != F32:
        raise ValueError("cast_round needs an f32 tensor")
    n = tensor.numel()
    set_stream()
    _check(lib().peat_cast_round(tensor.data_ptr() if n else None, n, int(to_dtype)), "peat_cast_round")


def _items_array(items):
    arr = (InjectItem * max(1, len(items)))()
    for k, it in enumerate(items):
        if isinstance(it, InjectItem):
            arr[k] = it
            continue
        t, seed, rate, mask = it[:4]
        model = it[4] if len(it) > 4 else MODEL_BITFLIP
        _dev_tensor(t, f"items[{k}].tensor")
        arr[k] = InjectItem(t.data_ptr(), t.numel(), dtype_code(t), model, seed & (2 ** 64 - 1), float(rate),
                            mask & (2 ** 64 - 1))
    return arr


class PreparedItems:
    """Injection descriptors built once, for repeated asynchronous calls; keeps
    the items' tensors alive for its lifetime (the descriptors hold raw device
    addresses that the calls write)."""

    def __init__(self, items):
        self.count = len(items)
        self.arr = _items_array(items)
        self.tensors = [it[0] for it in items if not isinstance(it, InjectItem)]


def inject_batched(items) -> list[int]:
    """peat_inject_batched over (tensor, seed, rate, bitmask) tuples."""
    arr = _items_array(items)
    counts = (ctypes.c_int64 * max(1, len(items)))()
    set_stream()
    _check(lib().peat_inject_batched(arr, len(items), counts), "peat_inject_batched")
    return [int(counts[k]) for k in range(len(items))]


def inject_batched_async(items, d_counts, stream=None) -> None:
    prep = items if isinstance(items, PreparedItems) else PreparedItems(items)
    _dev_tensor(d_counts, "d_counts")
    _check(lib().peat_inject_batched_async(prep.arr, prep.count, d_counts.data_ptr(), _stream_ptr(stream)),
           "peat_inject_batched_async")


def finalize_stats(sig: dict) -> dict:
    s = Signature()
    for name, _ in _SIG_FIELDS:
        v = sig[name]
        if name in ("n_mismatch", "hist"):
            arr = getattr(s, name)
            for j, x in enumerate(v):
                arr[j] = x
        else:
            setattr(s, name, v)
    st = Stats()
    _check(lib().peat_finalize_stats(ctypes.byref(s), ctypes.byref(st)), "peat_finalize_stats")
    return {k: float(getattr(st, k)) for k, _ in Stats._fields_}


STREAM_SPAN = 1 << 21     # bytes per block of peat_stream_read


def stream_read(buf, d_sink, stream=None) -> None:
    """peat_stream_read over the bytes of the contiguous device tensor buf;
    d_sink is a device int32/uint32 tensor of at least ceil(bytes / 2 MiB)
    elements (one XOR checksum per 2 MiB span)."""
    _dev_tensor(buf, "buf")
    _dev_tensor(d_sink, "d_sink")
    nbytes = buf.numel() * buf.element_size()
    if d_sink.element_size() != 4 or d_sink.numel() < (nbytes + STREAM_SPAN - 1) // STREAM_SPAN:
        raise ValueError("d_sink needs one 32-bit word per 2 MiB span")
    _check(lib().peat_stream_read(buf.data_ptr(), nbytes, d_sink.data_ptr(), _stream_ptr(stream)),
           "peat_stream_read")


def series_stats(x) -> dict:
    """peat_series_stats over a sequence of scores (host)."""
    a = np.ascontiguousarray(x, dtype=np.float64)
    out = Series()
    _check(lib().peat_series_stats(a.ctypes.data if a.size else None, a.size, ctypes.byref(out)),
           "peat_series_stats")
    return {k: (int(getattr(out, k)) if k == "count" else float(getattr(out, k))) for k, _ in Series._fields_}


def spearman(x, y) -> float:
    """peat_spearman of two equal-length sequences (host)."""
    a = np.ascontiguousarray(x, dtype=np.float64)
    b = np.ascontiguousarray(y, dtype=np.float64)
    if a.size != b.size:
        raise ValueError("x and y differ in length")
    rho = ctypes.c_double()
    _check(lib().peat_spearman(a.ctypes.data if a.size else None, b.ctypes.data if b.size else None, a.size,
                               ctypes.byref(rho)), "peat_spearman")
    return float(rho.value)


def normalize_scores(scores, units) -> np.ndarray:
    """peat_normalize_scores: scores in units of the FP64 error's score."""
    a = np.ascontiguousarray(scores, dtype=np.float64)
    b = np.ascontiguousarray(units, dtype=np.float64)
    if a.size != b.size:
        raise ValueError("scores and units differ in length")
    out = np.empty_like(a)
    _check(lib().peat_normalize_scores(a.ctypes.data if a.size else None, b.ctypes.data if b.size else None,
                                       a.size, out.ctypes.data if a.size else None), "peat_normalize_scores")
    return out


def profile_enable(on: bool = True) -> None:
    _check(lib().peat_profile_enable(1 if on else 0), "peat_profile_enable")


def profile_read(kernel_class: int):
    ms = ctypes.c_double(0)
    cnt = ctypes.c_int64(0)
    _check(lib().peat_profile_read(kernel_class, ctypes.byref(ms), ctypes.byref(cnt)), "peat_profile_read")
    return float(ms.value), int(cnt.value)
