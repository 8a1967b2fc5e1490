"""Stored-weight mapping for long float64 oracle runs.  TEST INFRASTRUCTURE ONLY.

`StoredWeights` gives the oracle (`DecoderOracle`) the weights of a full-size model
in their storage form: bf16 bit patterns (uint16) or float32 values, never the
product's device layout.  It provides three things:
- ``w[name]``: the exact float64 values of a tensor, widened on access (as for any
  weights mapping);
- ``w.rows(name, idx)``: only the rows asked for, widened (the embedding gather);
- ``w.project(name, u)``: the product u @ W^T in float64.  For a few rows of u
  (a decode step) it calls the plain C dot products of ``matvec.c``, which read
  the stored weights directly.  For more rows (a prefill) it widens the matrix
  a block of rows at a time and uses numpy's float64 matrix multiply.

Both routes compute the same float64 products and sums.  Only the order of the
additions differs, so results agree to rounding (pinned in
tests/test_oracle_pins.py).  The C library is compiled with gcc on first use
when it has not been built yet.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "matvec.c")
LIB = os.path.join(HERE, "_lib", "liboracle_matvec.so")
# at most this many rows of u take the C dot products; more rows go to the
# widened matrix multiply (compute-bound work that BLAS does better)
C_MAX_ROWS = 16
# the widened multiply takes the weights this many elements at a time (whole
# rows): small temporaries are reused by the allocator, where widening a whole
# matrix at once spends most of its time faulting in fresh pages
WIDEN_BLOCK = 1 << 21

_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile matvec.c into _lib/liboracle_matvec.so with gcc (OpenMP, no fused
    multiply-add contraction, so every product and sum rounds on its own)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        os.makedirs(os.path.dirname(LIB), exist_ok=True)
        tmp = LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-shared", "-fPIC",
                        SRC, "-o", tmp], check=True, capture_output=True, text=True)
        os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            lib = ctypes.CDLL(build())
            for fn, wt in (("oracle_matvec_bf16", ctypes.c_void_p),
                           ("oracle_matvec_f32", ctypes.c_void_p)):
                f = getattr(lib, fn)
                f.argtypes = [wt, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                              ctypes.c_int64, ctypes.c_void_p]
                f.restype = ctypes.c_int
            _lib = lib
    return _lib


def matvec(w: np.ndarray, u: np.ndarray) -> np.ndarray:
    """u @ W^T in float64 through the C dot products.  w: [N, K] uint16 (bf16 bit
    patterns) or float32, C-contiguous; u: [T, K] or [K] float64."""
    lib = _load()
    w = np.ascontiguousarray(w)
    one = u.ndim == 1
    u2 = np.ascontiguousarray(np.atleast_2d(u), dtype=np.float64)
    N, K = w.shape
    T = u2.shape[0]
    if u2.shape[1] != K:
        raise ValueError(f"shape mismatch: W {w.shape}, u {u2.shape}")
    y = np.empty((T, N), np.float64)
    if w.dtype == np.uint16:
        fn = lib.oracle_matvec_bf16
    elif w.dtype == np.float32:
        fn = lib.oracle_matvec_f32
    else:
        raise TypeError(f"stored weights must be uint16 (bf16) or float32, not {w.dtype}")
    st = fn(w.ctypes.data, N, K, u2.ctypes.data, T, y.ctypes.data)
    if st != 0:
        raise ValueError("matvec: bad size")
    return y[0] if one else y


def widen(a: np.ndarray) -> np.ndarray:
    """Exact float64 values of stored weights (bf16 bit patterns or float32)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


class StoredWeights:
    """Read-only mapping name -> float64 weights over stored tensors (see the
    module docstring), with ``rows`` and ``project`` for the oracle's fast paths."""

    def __init__(self, stored: dict):
        self._w = stored

    def __getitem__(self, name: str) -> np.ndarray:
        return widen(self._w[name])

    def __contains__(self, name: str) -> bool:
        return name in self._w

    def keys(self):
        return self._w.keys()

    def rows(self, name: str, idx) -> np.ndarray:
        return widen(self._w[name][np.asarray(idx)])

    def project(self, name: str, u: np.ndarray) -> np.ndarray:
        w = self._w[name]
        if u.ndim == 2 and u.shape[0] > C_MAX_ROWS:
            N, K = w.shape
            y = np.empty((u.shape[0], N))
            step = max(1, WIDEN_BLOCK // max(K, 1))
            for r in range(0, N, step):
                y[:, r:r + step] = u @ widen(w[r:r + step]).T
            return y
        return matvec(w, u)
