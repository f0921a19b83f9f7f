"""Plain CPU oracle for batched HDC inference (ScalableHD, Alg. 1, Eq. 1 and 7-9).

TEST INFRASTRUCTURE ONLY: only ``tests/``, the smoke check and the bench's
CPU-baseline leg may import this package. It shares no code with the GPU
library and never imports it.

The arithmetic lives in ``hd_oracle.c`` (plain loops, float64 accumulation);
this module only converts numpy arrays to float64 and calls it through ctypes.
Inputs must be float arrays holding the exact values the GPU sees (fp32, or
bf16 values stored in float32); widening them to float64 is exact.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_HERE = os.path.dirname(os.path.abspath(__file__))

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int32)
_lp = ctypes.POINTER(ctypes.c_int64)
_i64 = ctypes.c_int64

ACTS = {"hardsign": 0, "identity": 1}


def _f64(a):
    return np.ascontiguousarray(np.asarray(a), dtype=np.float64)


def _ptr(a, t=_dp):
    return None if a is None else a.ctypes.data_as(t)


class Oracle:
    """ctypes wrapper around one build of ``hd_oracle.c``."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        lib.oracle_encode.argtypes = [_dp, _dp, _i64, _i64, _i64, ctypes.c_int, _dp, _dp, _dp,
                                      ctypes.c_int]
        lib.oracle_encode.restype = ctypes.c_int
        lib.oracle_similarity.argtypes = [_dp, _dp, _i64, _i64, _i64, _dp, _ip, ctypes.c_int]
        lib.oracle_similarity.restype = ctypes.c_int
        lib.oracle_infer.argtypes = [_dp, _dp, _dp, _i64, _i64, _i64, _i64, ctypes.c_int, _lp,
                                     _i64, _ip, _dp, _dp, _dp, ctypes.c_int]
        lib.oracle_infer.restype = ctypes.c_int
        lib.oracle_bundle.argtypes = [_dp, _dp, _ip, _i64, _i64, _i64, _i64, _lp, _dp,
                                      ctypes.c_int]
        lib.oracle_bundle.restype = ctypes.c_int
        lib.oracle_threads.argtypes = [ctypes.c_int]
        lib.oracle_threads.restype = ctypes.c_int
        self.lib = lib
        self.path = path

    def threads(self, nthreads: int = 0) -> int:
        """Threads the oracle's parallel loops use for a request (0 = default)."""
        return int(self.lib.oracle_threads(int(nthreads)))

    def infer(self, X, B, C, act: str = "hardsign", rows=None, want_va: bool = False,
              nthreads: int = 0):
        """Alg. 1 on the listed rows of X (all rows when ``rows`` is None).

        Returns a dict with ``y`` (int32 labels), ``S`` (float64 scores) and,
        when ``want_va``, ``V`` (pre-activation encodings, Eq. 7) and ``A``
        (sum_f |x_f||b_fd|, the scale that bounds summation error of V).
        """
        X, B, C = _f64(X), _f64(B), _f64(C)
        N, F = X.shape
        F2, D = B.shape
        K, D2 = C.shape
        if F2 != F or D2 != D:
            raise ValueError("shape mismatch")
        ridx = None
        if rows is not None:
            ridx = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
            R = ridx.shape[0]
        else:
            R = N
        y = np.zeros(R, dtype=np.int32)
        S = np.zeros((R, K), dtype=np.float64)
        V = np.zeros((R, D), dtype=np.float64) if want_va else None
        A = np.zeros((R, D), dtype=np.float64) if want_va else None
        rc = self.lib.oracle_infer(_ptr(X), _ptr(B), _ptr(C), N, F, D, K, ACTS[act],
                                   _ptr(ridx, _lp), R, _ptr(y, _ip), _ptr(S), _ptr(V), _ptr(A),
                                   int(nthreads))
        if rc != 0:
            raise RuntimeError("oracle_infer failed")
        out = {"y": y, "S": S}
        if want_va:
            out["V"] = V
            out["A"] = A
        return out

    def encode(self, X, B, act: str = "hardsign", want_va: bool = False, nthreads: int = 0):
        """Stage I alone (Eq. 7 then Eq. 1): dict with ``H`` (and V, A)."""
        X, B = _f64(X), _f64(B)
        N, F = X.shape
        F2, D = B.shape
        if F2 != F:
            raise ValueError("shape mismatch")
        H = np.zeros((N, D), dtype=np.float64)
        V = np.zeros((N, D), dtype=np.float64) if want_va else None
        A = np.zeros((N, D), dtype=np.float64) if want_va else None
        rc = self.lib.oracle_encode(_ptr(X), _ptr(B), N, F, D, ACTS[act], _ptr(V), _ptr(A),
                                    _ptr(H), int(nthreads))
        if rc != 0:
            raise RuntimeError("oracle_encode failed")
        out = {"H": H}
        if want_va:
            out["V"] = V
            out["A"] = A
        return out

    def bundle(self, X, B, y, K: int, nthreads: int = 0):
        """Single-pass training (Sec. II-C): dict with ``counts`` (int64 [K, D],
        the per-class sums of the encoded bipolar hypervectors) and ``M``
        (float64 [K, D], HardSign of the counts)."""
        X, B = _f64(X), _f64(B)
        N, F = X.shape
        F2, D = B.shape
        if F2 != F:
            raise ValueError("shape mismatch")
        yy = np.ascontiguousarray(np.asarray(y), dtype=np.int32)
        if yy.shape != (N,):
            raise ValueError("labels must be [N]")
        counts = np.zeros((K, D), dtype=np.int64)
        M = np.zeros((K, D), dtype=np.float64)
        rc = self.lib.oracle_bundle(_ptr(X), _ptr(B), _ptr(yy, _ip), N, F, D, int(K),
                                    _ptr(counts, _lp), _ptr(M), int(nthreads))
        if rc != 0:
            raise RuntimeError("oracle_bundle failed")
        return {"counts": counts, "M": M}

    def similarity(self, H, C, nthreads: int = 0):
        """Stage II alone (Eq. 8 then Eq. 9) on a real matrix H: dict with y, S."""
        H, C = _f64(H), _f64(C)
        N, D = H.shape
        K, D2 = C.shape
        if D2 != D:
            raise ValueError("shape mismatch")
        y = np.zeros(N, dtype=np.int32)
        S = np.zeros((N, K), dtype=np.float64)
        rc = self.lib.oracle_similarity(_ptr(H), _ptr(C), N, D, K, _ptr(S), _ptr(y, _ip),
                                        int(nthreads))
        if rc != 0:
            raise RuntimeError("oracle_similarity failed")
        return {"y": y, "S": S}


_default = None


def default() -> Oracle:
    """The oracle built from ``hd_oracle.c`` (compiled on first use)."""
    global _default
    if _default is None:
        path = _build.LIB
        if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_build.SRC):
            _build.build()
        _default = Oracle(path)
    return _default


def threads(nthreads: int = 0) -> int:
    return default().threads(nthreads)


def infer(X, B, C, act: str = "hardsign", rows=None, want_va: bool = False, nthreads: int = 0):
    return default().infer(X, B, C, act=act, rows=rows, want_va=want_va, nthreads=nthreads)


def encode(X, B, act: str = "hardsign", want_va: bool = False, nthreads: int = 0):
    return default().encode(X, B, act=act, want_va=want_va, nthreads=nthreads)


def similarity(H, C, nthreads: int = 0):
    return default().similarity(H, C, nthreads=nthreads)


def bundle(X, B, y, K: int, nthreads: int = 0):
    return default().bundle(X, B, y, K, nthreads=nthreads)
