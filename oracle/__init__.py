"""fp64 CPU oracle of exact k-means (Lloyd iteration).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library.

``kmeans_oracle.c`` holds the arithmetic (assignment by direct squared
distances with a lowest-index arg-min, per-cluster means with empty clusters
kept, the objective, and the k nearest rows of a KNN search).  This module only marshals numpy arrays into it.  Points
are passed as stored: float32 arrays, or uint16 arrays of bf16/fp16 bits.
``oracle/exact.py`` has an exact-rational version for tiny inputs.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

from . import build as _build

_DT = {"f32": 0, "bf16": 1, "f16": 2}
_lib = None


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load ``liboracle.so`` (compiling it first only if it does not exist)."""
    global _lib
    if path is None and _lib is not None:
        return _lib
    p = path or _build.LIB
    if path is None and not os.path.exists(p):
        _build.build()
    lib = ctypes.CDLL(p)
    i64, i32, vp, dp = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p
    lib.oracle_widen.argtypes = [vp, i32, i64, dp]
    lib.oracle_assign.argtypes = [vp, i32, dp, i64, i64, i64, i64, vp, dp, dp]
    lib.oracle_update.argtypes = [vp, i32, vp, dp, i64, i64, i64, i64, dp, vp]
    lib.oracle_lloyd.argtypes = [vp, i32, dp, i64, i64, i64, i64, i32, dp, vp, dp, vp, dp]
    lib.oracle_knn.argtypes = [vp, vp, i32, i64, i64, i64, i64, i64, vp, dp, dp]
    for f in (lib.oracle_widen, lib.oracle_assign, lib.oracle_update, lib.oracle_lloyd,
              lib.oracle_knn):
        f.restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


class Oracle:
    """Array-level wrapper over one compiled oracle library."""

    def __init__(self, path: Optional[str] = None):
        self.lib = load(path)

    @staticmethod
    def _points(X: np.ndarray, dtype: str):
        X = np.ascontiguousarray(X)
        want = np.float32 if dtype == "f32" else np.uint16
        if X.dtype != want:
            raise TypeError(f"{dtype} points must be a {np.dtype(want)} array, got {X.dtype}")
        if X.ndim == 2:
            X = X[None]
        if X.ndim != 3:
            raise ValueError("points must be [N, D] or [B, N, D]")
        return X

    @staticmethod
    def _ptr(a: np.ndarray):
        return a.ctypes.data_as(ctypes.c_void_p)

    def widen(self, X: np.ndarray, dtype: str) -> np.ndarray:
        X = np.ascontiguousarray(X)
        out = np.empty(X.shape, np.float64)
        rc = self.lib.oracle_widen(self._ptr(X), _DT[dtype], X.size, self._ptr(out))
        if rc:
            raise ValueError(f"oracle_widen failed ({rc})")
        return out

    def assign(self, X: np.ndarray, dtype: str, C: np.ndarray):
        """Returns idx [B,N] int32, min_dist [B,N] fp64, gap [B,N] fp64."""
        X = self._points(X, dtype)
        B, N, D = X.shape
        C = np.ascontiguousarray(C, dtype=np.float64).reshape(B, -1, D)
        K = C.shape[1]
        idx = np.empty((B, N), np.int32)
        md = np.empty((B, N), np.float64)
        gap = np.empty((B, N), np.float64)
        rc = self.lib.oracle_assign(self._ptr(X), _DT[dtype], self._ptr(C), B, N, D, K,
                                    self._ptr(idx), self._ptr(md), self._ptr(gap))
        if rc:
            raise ValueError(f"oracle_assign failed ({rc})")
        return idx, md, gap

    def update(self, X: np.ndarray, dtype: str, idx: np.ndarray, C_prev: np.ndarray):
        """Returns C' [B,K,D] fp64 and counts [B,K] int64."""
        X = self._points(X, dtype)
        B, N, D = X.shape
        C_prev = np.ascontiguousarray(C_prev, dtype=np.float64).reshape(B, -1, D)
        K = C_prev.shape[1]
        idx = np.ascontiguousarray(idx, dtype=np.int32).reshape(B, N)
        C_out = np.empty((B, K, D), np.float64)
        counts = np.empty((B, K), np.int64)
        rc = self.lib.oracle_update(self._ptr(X), _DT[dtype], self._ptr(idx), self._ptr(C_prev),
                                    B, N, D, K, self._ptr(C_out), self._ptr(counts))
        if rc:
            raise ValueError(f"oracle_update failed ({rc})")
        return C_out, counts

    def lloyd(self, X: np.ndarray, dtype: str, C0: np.ndarray, iters: int):
        """Returns C_T, idx, min_dist, counts (last iteration) and objective [B, iters]."""
        X = self._points(X, dtype)
        B, N, D = X.shape
        C0 = np.ascontiguousarray(C0, dtype=np.float64).reshape(B, -1, D)
        K = C0.shape[1]
        C_out = np.empty((B, K, D), np.float64)
        idx = np.empty((B, N), np.int32)
        md = np.empty((B, N), np.float64)
        counts = np.empty((B, K), np.int64)
        obj = np.empty((B, iters), np.float64)
        rc = self.lib.oracle_lloyd(self._ptr(X), _DT[dtype], self._ptr(C0), B, N, D, K, iters,
                                   self._ptr(C_out), self._ptr(idx), self._ptr(md),
                                   self._ptr(counts), self._ptr(obj))
        if rc:
            raise ValueError(f"oracle_lloyd failed ({rc})")
        return C_out, idx, md, counts, obj

    def knn(self, Q: np.ndarray, R: np.ndarray, dtype: str, k: int):
        """KNN search: returns idx [B,M,k] int32, dist [B,M,k] fp64 (increasing,
        ties to the lowest index) and next_dist [B,M] (the (k+1)-th distance)."""
        Q = self._points(Q, dtype)
        R = self._points(R, dtype)
        B, M, D = Q.shape
        if R.shape[0] != B or R.shape[2] != D:
            raise ValueError("queries and database must share B and D")
        N = R.shape[1]
        idx = np.empty((B, M, k), np.int32)
        dist = np.empty((B, M, k), np.float64)
        nxt = np.empty((B, M), np.float64)
        rc = self.lib.oracle_knn(self._ptr(Q), self._ptr(R), _DT[dtype], B, M, N, D, k,
                                 self._ptr(idx), self._ptr(dist), self._ptr(nxt))
        if rc:
            raise ValueError(f"oracle_knn failed ({rc})")
        return idx, dist, nxt


_default: Optional[Oracle] = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
