"""rocRAND's Philox4x32-10 (host build of its header) as a reference for the
oracle's generator pins.  Built once per session into tests/_build/."""
from __future__ import annotations

import ctypes
import os
import shutil
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None


def available() -> bool:
    return shutil.which("hipcc") is not None or os.path.exists("/opt/rocm/bin/hipcc")


def lib():
    global _LIB
    if _LIB is None:
        out_dir = os.path.join(HERE, "_build")
        os.makedirs(out_dir, exist_ok=True)
        so = os.path.join(out_dir, "libphilox_ref.so")
        src = os.path.join(HERE, "philox_ref.cpp")
        if not os.path.exists(so) or os.path.getmtime(so) < os.path.getmtime(src):
            hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
            tmp = so + f".tmp{os.getpid()}"
            subprocess.run([hipcc, "-x", "hip", "--offload-arch=gfx950", "-O2", "-shared", "-fPIC",
                            src, "-o", tmp], check=True, capture_output=True)
            os.replace(tmp, so)
        L = ctypes.CDLL(so)
        L.ref_philox4x32_10.restype = None
        L.ref_philox4x32_10.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        _LIB = L
    return _LIB


def blocks(counters: np.ndarray, keys: np.ndarray) -> np.ndarray:
    """counters [m, 4] and keys [m, 2] (uint32) -> blocks [m, 4] (uint32)."""
    c = np.ascontiguousarray(counters, dtype=np.uint32).reshape(-1, 4)
    k = np.ascontiguousarray(np.broadcast_to(keys, (c.shape[0], 2)), dtype=np.uint32)
    out = np.empty_like(c)
    if c.shape[0]:
        lib().ref_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data, c.shape[0])
    return out


def seeded(seed: int, numbers, stream: int) -> np.ndarray:
    """Blocks number c (array) of a stream under a 64-bit seed: key (lo32, hi32)
    of the seed, counter (lo32(c), hi32(c), stream, 0)."""
    c = np.asarray(numbers, dtype=np.uint64).reshape(-1)
    ctr = np.zeros((c.size, 4), np.uint32)
    ctr[:, 0] = (c & np.uint64(0xFFFFFFFF)).astype(np.uint32)
    ctr[:, 1] = (c >> np.uint64(32)).astype(np.uint32)
    ctr[:, 2] = stream
    key = np.array([seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF], np.uint32)
    return blocks(ctr, key)
