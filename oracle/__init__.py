"""CPU oracle for the PEAT error signature and bit-flip injector.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg are the only callers.  The GPU library never
imports, links or executes anything in this directory.

The arithmetic lives in ``peat_oracle.c`` (plain scalar C, IEEE binary64,
no contraction, no fast-math), built with gcc into ``liboracle.so`` next to
it.  This module only marshals numpy arrays into that library and returns
plain Python dicts.

Passages followed (the paper is "PEAT: Pseudo-Error Assessment for GPU Kernel
Validation in DNN Training"):
  * Section IV-B.3 "FI Assessment Scores": error = absolute difference of the
    golden and fault-injected outputs; max, mean and variance of it.
  * Section III-A and Fig. "Motivating_isclose": closeness with
    torch.isclose(rtol, atol) -> absolute-threshold mismatch counts.
  * Section V-D, Fig. "tiny_error_gemm_resnet34": error value histograms.
  * Section II-B "Error Models": random bit flip at a bit error rate.
  * Section II-B and Section III-C/V-A: random zero, random NaN, random
    value (num_pos positions) and the FP16/BF16 cast error.
  * Section IV-B.3 "Mean of Top 10% Errors" (the Analyzer's main score,
    Section IV-C): mean of the k largest errors, k = ceil(n_valid num/den).
  * Algorithms 1 and 2: Inject() followed by Err(golden set, FI set).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "peat_oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")

F32, F16, BF16, F64 = 0, 1, 2, 3
_DTYPE_CODE = {np.dtype(np.float32): F32, np.dtype(np.float16): F16}

OK, EINVAL, EDTYPE, EBITMASK, ERATE, ENOMEM = 0, -1, -2, -3, -4, -6
MODEL_BITFLIP, MODEL_ZERO, MODEL_VALUE, MODEL_NAN, MODEL_UNIFORM = 0, 1, 2, 3, 4
MAX_POSITIONS = 4096


class _Sig(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int64), ("n_valid", ctypes.c_int64),
        ("n_finite", ctypes.c_int64), ("n_rel", ctypes.c_int64),
        ("n_nan_golden", ctypes.c_int64), ("n_nan_test", ctypes.c_int64),
        ("n_inf_golden", ctypes.c_int64), ("n_inf_test", ctypes.c_int64),
        ("n_nan_pairs", ctypes.c_int64), ("first_nan_index", ctypes.c_int64),
        ("n_mismatch", ctypes.c_int64 * 8),
        ("hist_zero", ctypes.c_int64), ("hist_under", ctypes.c_int64),
        ("hist_over", ctypes.c_int64),
        ("hist", ctypes.c_int64 * 64),
        ("max_abs", ctypes.c_double), ("argmax_abs", ctypes.c_int64),
        ("max_ulp", ctypes.c_int64), ("argmax_ulp", ctypes.c_int64),
        ("sum_ulp", ctypes.c_uint64),
        ("max_rel", ctypes.c_double), ("argmax_rel", ctypes.c_int64),
        ("sum_abs", ctypes.c_double), ("sum_sq", ctypes.c_double),
        ("sum_rel", ctypes.c_double), ("sum_g2", ctypes.c_double),
        ("sum_t2", ctypes.c_double), ("sum_gt", ctypes.c_double),
    ]


class _TopK(ctypes.Structure):
    _fields_ = [("n_valid", ctypes.c_int64), ("k", ctypes.c_int64), ("count_above", ctypes.c_int64),
                ("kth_value", ctypes.c_double), ("sum_topk", ctypes.c_double),
                ("mean_topk", ctypes.c_double)]


class _Series(ctypes.Structure):
    _fields_ = [("count", ctypes.c_int64)] + [(k, ctypes.c_double) for k in ("mean", "var", "std", "min", "max")]


class _Stats(ctypes.Structure):
    _fields_ = [(k, ctypes.c_double) for k in
                ("mean_abs", "var_abs", "l2_err", "l2_g", "l2_t", "cos",
                 "mean_rel", "mean_ulp")]


_lib = None
_lock = threading.Lock()


def build(force: bool = False) -> str:
    """Compile peat_oracle.c with gcc (no contraction, no fast-math)."""
    if force or not os.path.exists(LIB_PATH) or \
            os.path.getmtime(LIB_PATH) < os.path.getmtime(_SRC):
        tmp = LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call([
            "gcc", "-O2", "-std=c11", "-fPIC", "-shared",
            "-ffp-contract=off", "-fno-fast-math", "-fno-strict-aliasing",
            "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib():
    """Load (building first if absent) the oracle library."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                build()
            L = ctypes.CDLL(LIB_PATH)
            L.oracle_signature.restype = ctypes.c_int
            L.oracle_signature.argtypes = [
                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_Sig)]
            L.oracle_signature_rtol.restype = ctypes.c_int
            L.oracle_signature_rtol.argtypes = [
                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_Sig)]
            L.oracle_signature_mixed.restype = ctypes.c_int
            L.oracle_signature_mixed.argtypes = [
                ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_Sig)]
            L.oracle_topk_mixed.restype = ctypes.c_int
            L.oracle_topk_mixed.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                                            ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.POINTER(_TopK)]
            L.oracle_stats.restype = ctypes.c_int
            L.oracle_stats.argtypes = [ctypes.POINTER(_Sig), ctypes.POINTER(_Stats)]
            L.oracle_philox4x32_10.restype = None
            L.oracle_philox4x32_10.argtypes = [
                ctypes.POINTER(ctypes.c_uint32), ctypes.POINTER(ctypes.c_uint32),
                ctypes.POINTER(ctypes.c_uint32)]
            L.oracle_rate_threshold.restype = ctypes.c_uint64
            L.oracle_rate_threshold.argtypes = [ctypes.c_double, ctypes.POINTER(ctypes.c_int)]
            L.oracle_inject_decide.restype = ctypes.c_int
            L.oracle_inject_decide.argtypes = [
                ctypes.c_int64, ctypes.c_int, ctypes.c_uint64, ctypes.c_double,
                ctypes.c_uint64, ctypes.POINTER(ctypes.c_int)]
            L.oracle_inject.restype = ctypes.c_int64
            L.oracle_inject.argtypes = [
                ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_uint64,
                ctypes.c_double, ctypes.c_uint64]
            L.oracle_topk.restype = ctypes.c_int
            L.oracle_topk.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                      ctypes.c_int, ctypes.c_int, ctypes.POINTER(_TopK)]
            L.oracle_inject_model.restype = ctypes.c_int64
            L.oracle_inject_model.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_uint64,
                                              ctypes.c_double, ctypes.c_int, ctypes.c_uint64]
            L.oracle_corrupt_positions.restype = ctypes.c_int64
            L.oracle_corrupt_positions.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                                   ctypes.c_uint64, ctypes.c_int, ctypes.c_int64,
                                                   ctypes.c_uint64, ctypes.POINTER(ctypes.c_int64)]
            L.oracle_cast_round.restype = ctypes.c_int
            L.oracle_cast_round.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int]
            L.oracle_series_stats.restype = ctypes.c_int
            L.oracle_series_stats.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(_Series)]
            L.oracle_spearman.restype = ctypes.c_int
            L.oracle_spearman.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                          ctypes.POINTER(ctypes.c_double)]
            L.oracle_normalize.restype = ctypes.c_int
            L.oracle_normalize.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
            L.oracle_sizeof_sig.restype = ctypes.c_int
            assert L.oracle_sizeof_sig() == ctypes.sizeof(_Sig)
            L.oracle_sizeof_topk.restype = ctypes.c_int
            assert L.oracle_sizeof_topk() == ctypes.sizeof(_TopK)
            _lib = L
    return _lib


def _code(arr: np.ndarray, dtype_code: int | None) -> int:
    if dtype_code is not None:
        return dtype_code
    if arr.dtype == np.uint16:
        raise ValueError("uint16 arrays need an explicit dtype code (F16 or BF16)")
    if arr.dtype == np.uint32:
        return F32
    return _DTYPE_CODE[arr.dtype]


def _sig_to_dict(s: _Sig, nthr: int) -> dict:
    d = {}
    for name, _ in _Sig._fields_:
        v = getattr(s, name)
        if name == "n_mismatch":
            v = [int(v[j]) for j in range(nthr)]
        elif name == "hist":
            v = [int(x) for x in v]
        elif isinstance(v, float):
            v = float(v)
        else:
            v = int(v)
        d[name] = v
    return d


def split_thresholds(thresholds):
    """([atol], [rtol]) from absolute tolerances or (atol, rtol) pairs."""
    atol, rtol = [], []
    for x in thresholds:
        if isinstance(x, (tuple, list)):
            atol.append(float(x[0]))
            rtol.append(float(x[1]))
        else:
            atol.append(float(x))
            rtol.append(0.0)
    return atol, rtol


def signature(golden: np.ndarray, test: np.ndarray, *, dtype: int | None = None,
              bins=(-40, 24, 64), thresholds=(1e-6, 1e-3), raw: bool = False):
    """Error signature of (golden, test): dict of every field.

    ``golden``/``test`` are contiguous numpy arrays of float32/float16 or raw
    bit patterns (uint32 for f32; uint16 with ``dtype=F16``/``BF16``).
    ``thresholds`` holds absolute tolerances or (atol, rtol) pairs.
    """
    g = np.ascontiguousarray(golden).reshape(-1)
    t = np.ascontiguousarray(test).reshape(-1)
    if g.shape != t.shape or g.dtype != t.dtype:
        raise ValueError("golden and test must have the same shape and dtype")
    code = _code(g, dtype)
    atol, rtol = split_thresholds(thresholds)
    thr = (ctypes.c_double * 8)(*atol)
    rthr = (ctypes.c_double * 8)(*rtol)
    out = _Sig()
    rc = lib().oracle_signature_rtol(
        g.ctypes.data if g.size else None, t.ctypes.data if t.size else None,
        g.size, code, int(bins[0]), int(bins[1]), int(bins[2]), len(thresholds),
        thr, rthr, ctypes.byref(out))
    if rc != OK:
        raise ValueError(f"oracle_signature failed: {rc}")
    if raw:
        return out
    return _sig_to_dict(out, len(thresholds))


def _mixed_code(arr: np.ndarray, dtype_code: int | None) -> int:
    if dtype_code is None and arr.dtype == np.float64:
        return F64
    return _code(arr, dtype_code)


def signature_mixed(golden: np.ndarray, test: np.ndarray, *, gdtype: int | None = None,
                    tdtype: int | None = None, bins=(-40, 24, 64), thresholds=(1e-6, 1e-3)) -> dict:
    """Signature of a pair whose golden and test types may differ (float64 is
    the test side's binary64; uint16 bit patterns need an explicit code)."""
    g = np.ascontiguousarray(golden).reshape(-1)
    t = np.ascontiguousarray(test).reshape(-1)
    if g.shape != t.shape:
        raise ValueError("golden and test must have the same shape")
    gc, tc = _mixed_code(g, gdtype), _mixed_code(t, tdtype)
    atol, rtol = split_thresholds(thresholds)
    thr = (ctypes.c_double * 8)(*atol)
    rthr = (ctypes.c_double * 8)(*rtol)
    out = _Sig()
    rc = lib().oracle_signature_mixed(
        g.ctypes.data if g.size else None, gc, t.ctypes.data if t.size else None, tc,
        g.size, int(bins[0]), int(bins[1]), int(bins[2]), len(thresholds), thr, rthr, ctypes.byref(out))
    if rc != OK:
        raise ValueError(f"oracle_signature_mixed failed: {rc}")
    return _sig_to_dict(out, len(thresholds))


def signature_mixed_rc(gcode: int, tcode: int, n: int = 4) -> int:
    """Return code of oracle_signature_mixed on zero-filled buffers."""
    buf = np.zeros(max(int(n), 1) * 8, dtype=np.uint8)
    thr = (ctypes.c_double * 8)()
    out = _Sig()
    return int(lib().oracle_signature_mixed(buf.ctypes.data, gcode, buf.ctypes.data, tcode, int(n),
                                            -40, 24, 64, 0, thr, None, ctypes.byref(out)))


def topk_mixed(golden: np.ndarray, test: np.ndarray, *, gdtype: int | None = None,
               tdtype: int | None = None, num: int = 1, den: int = 10) -> dict:
    g = np.ascontiguousarray(golden).reshape(-1)
    t = np.ascontiguousarray(test).reshape(-1)
    if g.shape != t.shape:
        raise ValueError("golden and test must have the same shape")
    out = _TopK()
    rc = lib().oracle_topk_mixed(g.ctypes.data if g.size else None, _mixed_code(g, gdtype),
                                 t.ctypes.data if t.size else None, _mixed_code(t, tdtype),
                                 g.size, int(num), int(den), ctypes.byref(out))
    if rc != OK:
        raise ValueError(f"oracle_topk_mixed failed: {rc}")
    return {k: (float(getattr(out, k)) if k in ("kth_value", "sum_topk", "mean_topk") else int(getattr(out, k)))
            for k, _ in _TopK._fields_}


def signature_rc(golden_ptr, test_ptr, n, code, bins, thresholds) -> int:
    """Return code of oracle_signature for argument-validation tests."""
    atol, rtol = split_thresholds(thresholds)
    thr = (ctypes.c_double * max(8, len(thresholds)))(*atol)
    rthr = (ctypes.c_double * max(8, len(thresholds)))(*rtol)
    out = _Sig()
    return lib().oracle_signature_rtol(golden_ptr, test_ptr, n, code, bins[0], bins[1],
                                       bins[2], len(thresholds), thr, rthr, ctypes.byref(out))


def stats(sig: dict) -> dict:
    s = _Sig()
    for name, _ in _Sig._fields_:
        v = sig[name]
        if name == "n_mismatch":
            for j, x in enumerate(v):
                s.n_mismatch[j] = x
        elif name == "hist":
            for j, x in enumerate(v):
                s.hist[j] = x
        else:
            setattr(s, name, v)
    st = _Stats()
    lib().oracle_stats(ctypes.byref(s), ctypes.byref(st))
    return {k: float(getattr(st, k)) for k, _ in _Stats._fields_}


def philox4x32_10(counter, key):
    """One Philox4x32-10 block: four 32-bit counter words, two key words."""
    c = (ctypes.c_uint32 * 4)(*[int(x) & 0xFFFFFFFF for x in counter])
    k = (ctypes.c_uint32 * 2)(*[int(x) & 0xFFFFFFFF for x in key])
    o = (ctypes.c_uint32 * 4)()
    lib().oracle_philox4x32_10(c, k, o)
    return [int(x) for x in o]


def rate_threshold(rate: float):
    """(T, all) with T = floor(rate * 2^64)."""
    a = ctypes.c_int(0)
    T = lib().oracle_rate_threshold(float(rate), ctypes.byref(a))
    return int(T), bool(a.value)


def inject_decide(i: int, dtype: int, seed: int, rate: float, mask: int):
    """(flips, bit) for element i alone."""
    b = ctypes.c_int(-1)
    rc = lib().oracle_inject_decide(int(i), dtype, seed & (2**64 - 1), float(rate),
                                    mask & (2**64 - 1), ctypes.byref(b))
    if rc < 0:
        raise ValueError(f"oracle_inject_decide failed: {rc}")
    return bool(rc), (b.value if rc else None)


def inject(x: np.ndarray, *, dtype: int | None = None, seed: int, rate: float,
           mask: int) -> int:
    """Flip bits of ``x`` in place (x must be C-contiguous); returns the count."""
    if not x.flags.c_contiguous or not x.flags.writeable:
        raise ValueError("inject needs a writeable C-contiguous array")
    code = _code(x, dtype)
    rc = lib().oracle_inject(x.ctypes.data if x.size else None, x.size, code,
                             seed & (2**64 - 1), float(rate), mask & (2**64 - 1))
    if rc < 0:
        raise ValueError(f"oracle_inject failed: {rc}")
    return int(rc)


def inject_rc(n, code, seed, rate, mask) -> int:
    """Return code of oracle_inject on a scratch buffer (validation tests)."""
    buf = np.zeros(max(int(n), 1) * 4, dtype=np.uint8)
    return int(lib().oracle_inject(buf.ctypes.data, int(n), code, seed, float(rate), mask))


def topk(golden: np.ndarray, test: np.ndarray, *, dtype: int | None = None, num: int = 1,
         den: int = 10) -> dict:
    """Mean of the k largest errors over the valid pairs, k = ceil(n_valid num/den):
    dict with n_valid, k, count_above, kth_value, sum_topk, mean_topk."""
    g = np.ascontiguousarray(golden).reshape(-1)
    t = np.ascontiguousarray(test).reshape(-1)
    if g.shape != t.shape or g.dtype != t.dtype:
        raise ValueError("golden and test must have the same shape and dtype")
    code = _code(g, dtype)
    out = _TopK()
    rc = lib().oracle_topk(g.ctypes.data if g.size else None, t.ctypes.data if t.size else None,
                           g.size, code, int(num), int(den), ctypes.byref(out))
    if rc != OK:
        raise ValueError(f"oracle_topk failed: {rc}")
    return {name: (float(getattr(out, name)) if typ is ctypes.c_double else int(getattr(out, name)))
            for name, typ in _TopK._fields_}


def topk_rc(n, code, num, den) -> int:
    """Return code of oracle_topk on zero-filled buffers (validation tests)."""
    buf = np.zeros(max(int(n), 1) * 4, dtype=np.uint8)
    out = _TopK()
    return int(lib().oracle_topk(buf.ctypes.data, buf.ctypes.data, int(n), code, int(num), int(den),
                                 ctypes.byref(out)))


def inject_model(x: np.ndarray, *, dtype: int | None = None, seed: int, rate: float, model: int,
                 mask: int = 0) -> int:
    """Rate-mode error model in place (0 bit flip, 1 zero, 2 a value of the
    uncorrupted tensor at a random index, 3 NaN, 4 a uniformly random bit
    pattern); returns the number of chosen elements (or a negative code)."""
    if not x.flags.c_contiguous or not x.flags.writeable:
        raise ValueError("inject_model needs a writeable C-contiguous array")
    code = _code(x, dtype)
    return int(lib().oracle_inject_model(x.ctypes.data if x.size else None, x.size, code, seed & (2**64 - 1),
                                         float(rate), int(model), mask & (2**64 - 1)))


def corrupt_positions(x: np.ndarray, *, dtype: int | None = None, seed: int, model: int, num_pos: int,
                      mask: int = 0):
    """Position-mode error model in place; returns (rc, positions list)."""
    if not x.flags.c_contiguous or not x.flags.writeable:
        raise ValueError("corrupt_positions needs a writeable C-contiguous array")
    code = _code(x, dtype)
    pos = (ctypes.c_int64 * max(1, int(num_pos)))()
    rc = int(lib().oracle_corrupt_positions(x.ctypes.data if x.size else None, x.size, code,
                                            seed & (2**64 - 1), int(model), int(num_pos), mask & (2**64 - 1),
                                            pos))
    return rc, ([int(pos[k]) for k in range(rc)] if rc > 0 else [])


def cast_round(x: np.ndarray, to_dtype: int) -> int:
    """FP16 (1) / BF16 (2) round-to-nearest-even cast of an f32 array in place."""
    if x.dtype not in (np.float32, np.uint32) or not x.flags.c_contiguous or not x.flags.writeable:
        raise ValueError("cast_round needs a writeable C-contiguous f32 array")
    return int(lib().oracle_cast_round(x.ctypes.data if x.size else None, x.size, int(to_dtype)))


def series_stats(x) -> dict:
    """count, mean, sample var, std, min, max of the non-NaN entries."""
    a = np.ascontiguousarray(x, dtype=np.float64)
    out = _Series()
    rc = lib().oracle_series_stats(a.ctypes.data if a.size else None, a.size, ctypes.byref(out))
    if rc != OK:
        raise ValueError(f"oracle_series_stats failed: {rc}")
    return {k: (int(getattr(out, k)) if k == "count" else float(getattr(out, k))) for k, _ in _Series._fields_}


def spearman(x, y) -> float:
    a = np.ascontiguousarray(x, dtype=np.float64)
    b = np.ascontiguousarray(y, dtype=np.float64)
    rho = ctypes.c_double()
    rc = lib().oracle_spearman(a.ctypes.data if a.size else None, b.ctypes.data if b.size else None, a.size,
                               ctypes.byref(rho))
    if rc != OK:
        raise ValueError(f"oracle_spearman failed: {rc}")
    return float(rho.value)


def normalize(scores, units) -> np.ndarray:
    a = np.ascontiguousarray(scores, dtype=np.float64)
    b = np.ascontiguousarray(units, dtype=np.float64)
    out = np.empty_like(a)
    rc = lib().oracle_normalize(a.ctypes.data if a.size else None, b.ctypes.data if b.size else None, a.size,
                                out.ctypes.data if a.size else None)
    if rc != OK:
        raise ValueError(f"oracle_normalize failed: {rc}")
    return out
