"""ctypes binding of ``libflashkmeans.so`` (the C ABI in ``include/flashkmeans.h``).

Argument marshalling only: every step of the Lloyd iteration runs in the HIP
kernels of the library.  Tensors must be CUDA (HIP) tensors on the current
device; work is enqueued on torch's current stream.  Importing this module
raises if the library has not been built -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libflashkmeans.so")

F32, BF16, F16 = 0, 1, 2
_DTYPE = {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16}
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_SCRATCH = 0, -1, -2, -3, -4, -5
SCRATCH_BYTES = 64 << 20  # KMEANS_SCRATCH_BYTES


class KMeansError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_string(status)} ({status})")
        self.status = status


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2608_12629_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    i64, i32, vp, sz = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t
    lib.kmeans_workspace_bytes.argtypes = [i64, i64, i64, i64, i32]
    lib.kmeans_workspace_bytes.restype = sz
    lib.kmeans_assign.argtypes = [vp, i32, vp, i64, i64, i64, i64, vp, vp, vp, sz, vp]
    lib.kmeans_update.argtypes = [vp, i32, vp, vp, i64, i64, i64, i64, vp, vp, vp, sz, vp]
    lib.kmeans_lloyd.argtypes = [vp, i32, vp, i64, i64, i64, i64, i32, vp, vp, vp, vp, vp, sz, vp]
    lib.kmeans_lloyd_noalloc.argtypes = [vp, i32, vp, i64, i64, i64, i64, i32, vp, vp, vp, vp, vp]
    lib.kmeans_knn_workspace_bytes.argtypes = [i64, i64, i64, i64, i32, i32]
    lib.kmeans_knn_workspace_bytes.restype = sz
    lib.kmeans_knn.argtypes = [vp, vp, i32, i64, i64, i64, i64, i32, vp, vp, vp, sz, vp]
    for f in (lib.kmeans_assign, lib.kmeans_update, lib.kmeans_lloyd, lib.kmeans_lloyd_noalloc,
              lib.kmeans_knn):
        f.restype = ctypes.c_int
    lib.kmeans_status_string.argtypes = [ctypes.c_int]
    lib.kmeans_status_string.restype = ctypes.c_char_p
    return lib


lib = _load()


def status_string(status: int) -> str:
    return lib.kmeans_status_string(int(status)).decode()


def _check(rc: int, where: str) -> None:
    if rc != OK:
        raise KMeansError(rc, where)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _shapes(X: torch.Tensor, C: torch.Tensor) -> Tuple[int, int, int, int]:
    if X.dim() == 2:
        X = X.unsqueeze(0)
    if C.dim() == 2:
        C = C.unsqueeze(0)
    if X.dim() != 3 or C.dim() != 3 or X.shape[0] != C.shape[0] or X.shape[2] != C.shape[2]:
        raise ValueError(f"shapes X{tuple(X.shape)} C{tuple(C.shape)}: want [B,N,D] and [B,K,D]")
    return X.shape[0], X.shape[1], X.shape[2], C.shape[1]


def _dt(X: torch.Tensor) -> int:
    try:
        return _DTYPE[X.dtype]
    except KeyError:
        raise TypeError(f"points must be float32, bfloat16 or float16, got {X.dtype}") from None


def _need(t: torch.Tensor, name: str, dtype=None, numel: Optional[int] = None) -> None:
    """A contiguous tensor on the current GPU (the library works on the current
    device); `numel`: the number of elements the kernels read or write there
    (any shape with that many, so [N] serves for one instance as well as
    [1, N]).  The C ABI sees pointers only, so these checks are what keeps a
    kernel inside the tensors it is given."""
    if not t.is_cuda or t.device.index != torch.cuda.current_device():
        raise ValueError(f"{name} must be a tensor on the current GPU (cuda:"
                         f"{torch.cuda.current_device()}), got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements (shape {tuple(t.shape)}), want {numel}")


def workspace_bytes(B: int, N: int, D: int, K: int, dtype: torch.dtype) -> int:
    return int(lib.kmeans_workspace_bytes(B, N, D, K, _DTYPE[dtype]))


class Workspace:
    """A device buffer of ``kmeans_workspace_bytes`` bytes, reused across calls."""

    def __init__(self, B: int, N: int, D: int, K: int, dtype: torch.dtype, device=None):
        n = workspace_bytes(B, N, D, K, dtype)
        if n == 0:
            raise KMeansError(ERR_UNSUPPORTED, "kmeans_workspace_bytes")
        self.nbytes = n
        self.buf = torch.empty(n, dtype=torch.uint8, device=device or "cuda")


def _ws(ws: Optional[Workspace], B, N, D, K, dtype, device) -> Workspace:
    if ws is None or ws.nbytes < workspace_bytes(B, N, D, K, dtype):
        ws = Workspace(B, N, D, K, dtype, device)
    _need(ws.buf, "workspace", torch.uint8, ws.nbytes)
    return ws


def kmeans_assign(X: torch.Tensor, C: torch.Tensor, idx: Optional[torch.Tensor] = None,
                  min_dist: Optional[torch.Tensor] = None, ws: Optional[Workspace] = None):
    """idx, min_dist of the nearest centroid of every point (see ``kmeans_assign`` in the header)."""
    B, N, D, K = _shapes(X, C)
    _need(X, "X")
    _need(C, "C", torch.float32)
    idx = torch.empty((B, N), dtype=torch.int32, device=X.device) if idx is None else idx
    min_dist = torch.empty((B, N), dtype=torch.float32, device=X.device) if min_dist is None else min_dist
    _need(idx, "idx", torch.int32, B * N)
    _need(min_dist, "min_dist", torch.float32, B * N)
    ws = _ws(ws, B, N, D, K, X.dtype, X.device)
    _check(lib.kmeans_assign(_ptr(X), _dt(X), _ptr(C), B, N, D, K, _ptr(idx), _ptr(min_dist),
                             _ptr(ws.buf), ws.nbytes, _stream()), "kmeans_assign")
    return idx, min_dist


def kmeans_update(X: torch.Tensor, idx: torch.Tensor, C_prev: torch.Tensor,
                  C_out: Optional[torch.Tensor] = None, counts: Optional[torch.Tensor] = None,
                  ws: Optional[Workspace] = None):
    """C_out, counts of the centroid update (see ``kmeans_update`` in the header)."""
    B, N, D, K = _shapes(X, C_prev)
    _need(X, "X")
    _need(idx, "idx", torch.int32, B * N)
    _need(C_prev, "C_prev", torch.float32)
    C_out = torch.empty((B, K, D), dtype=torch.float32, device=X.device) if C_out is None else C_out
    counts = torch.empty((B, K), dtype=torch.int32, device=X.device) if counts is None else counts
    _need(C_out, "C_out", torch.float32, B * K * D)
    _need(counts, "counts", torch.int32, B * K)
    ws = _ws(ws, B, N, D, K, X.dtype, X.device)
    _check(lib.kmeans_update(_ptr(X), _dt(X), _ptr(idx), _ptr(C_prev), B, N, D, K, _ptr(C_out),
                             _ptr(counts), _ptr(ws.buf), ws.nbytes, _stream()), "kmeans_update")
    return C_out, counts


def kmeans_lloyd(X: torch.Tensor, C: torch.Tensor, iters: int, *,
                 idx: Optional[torch.Tensor] = None, min_dist: Optional[torch.Tensor] = None,
                 counts: Optional[torch.Tensor] = None, objective=True,
                 ws: Optional[Workspace] = None):
    """Run ``iters`` Lloyd iterations, updating C in place.

    ``objective``: True (a new [B, iters] fp64 tensor), False (none), or a
    [B, iters] fp64 device tensor to write into (nothing is allocated when
    every output and ``ws`` are given, so the call can be captured in a graph).
    Returns (C, idx, min_dist, counts, objective[B, iters] fp64 or None).
    """
    B, N, D, K = _shapes(X, C)
    _need(X, "X")
    _need(C, "C", torch.float32)
    dev = X.device
    idx = torch.empty((B, N), dtype=torch.int32, device=dev) if idx is None else idx
    min_dist = torch.empty((B, N), dtype=torch.float32, device=dev) if min_dist is None else min_dist
    counts = torch.empty((B, K), dtype=torch.int32, device=dev) if counts is None else counts
    if isinstance(objective, torch.Tensor):
        obj = objective
        _need(obj, "objective", torch.float64)
        if tuple(obj.shape) != (B, iters):
            raise ValueError(f"objective has shape {tuple(obj.shape)}, want {(B, iters)}")
    else:
        obj = torch.empty((B, iters), dtype=torch.float64, device=dev) if objective else None
    for t, name, dt, n in ((idx, "idx", torch.int32, B * N), (min_dist, "min_dist", torch.float32, B * N),
                           (counts, "counts", torch.int32, B * K)):
        _need(t, name, dt, n)
    ws = _ws(ws, B, N, D, K, X.dtype, dev)
    _check(lib.kmeans_lloyd(_ptr(X), _dt(X), _ptr(C), B, N, D, K, int(iters), _ptr(idx),
                            _ptr(min_dist), _ptr(counts), _ptr(obj), _ptr(ws.buf), ws.nbytes,
                            _stream()), "kmeans_lloyd")
    return C, idx, min_dist, counts, obj


def kmeans_lloyd_noalloc(X: torch.Tensor, C: torch.Tensor, iters: int, idx: torch.Tensor,
                         min_dist: torch.Tensor, counts: torch.Tensor,
                         objective: Optional[torch.Tensor] = None):
    """``kmeans_lloyd`` on the library's static scratch array: every output is
    passed in, nothing is allocated (see ``kmeans_lloyd_noalloc`` in the header).
    Returns (C, idx, min_dist, counts, objective)."""
    B, N, D, K = _shapes(X, C)
    _need(X, "X")
    _need(C, "C", torch.float32)
    for t, name, dt, shape in ((idx, "idx", torch.int32, (B, N)),
                               (min_dist, "min_dist", torch.float32, (B, N)),
                               (counts, "counts", torch.int32, (B, K))):
        _need(t, name, dt)
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} has shape {tuple(t.shape)}, want {shape}")
    if objective is not None:
        _need(objective, "objective", torch.float64)
        if tuple(objective.shape) != (B, iters):
            raise ValueError(f"objective has shape {tuple(objective.shape)}, want {(B, iters)}")
    _check(lib.kmeans_lloyd_noalloc(_ptr(X), _dt(X), _ptr(C), B, N, D, K, int(iters), _ptr(idx),
                                    _ptr(min_dist), _ptr(counts), _ptr(objective), _stream()),
           "kmeans_lloyd_noalloc")
    return C, idx, min_dist, counts, objective


def knn_workspace_bytes(B: int, M: int, N: int, D: int, k: int, dtype: torch.dtype) -> int:
    return int(lib.kmeans_knn_workspace_bytes(B, M, N, D, k, _DTYPE[dtype]))


def kmeans_knn(Q: torch.Tensor, R: torch.Tensor, k: int, nbr_idx: Optional[torch.Tensor] = None,
               nbr_dist: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """KNN search: nbr_idx [B,M,k] int32 and nbr_dist [B,M,k] fp32 of the k nearest
    database rows of every query (see ``kmeans_knn`` in the header)."""
    if Q.dim() == 2:
        Q = Q.unsqueeze(0)
    if R.dim() == 2:
        R = R.unsqueeze(0)
    if Q.dim() != 3 or R.dim() != 3 or Q.shape[0] != R.shape[0] or Q.shape[2] != R.shape[2]:
        raise ValueError(f"shapes Q{tuple(Q.shape)} R{tuple(R.shape)}: want [B,M,D] and [B,N,D]")
    if Q.dtype != R.dtype:
        raise TypeError("queries and database must share a dtype")
    B, M, D = Q.shape
    N = R.shape[1]
    _need(Q, "Q")
    _need(R, "R")
    dev = Q.device
    nbr_idx = torch.empty((B, M, k), dtype=torch.int32, device=dev) if nbr_idx is None else nbr_idx
    nbr_dist = torch.empty((B, M, k), dtype=torch.float32, device=dev) if nbr_dist is None else nbr_dist
    _need(nbr_idx, "nbr_idx", torch.int32, B * M * k)
    _need(nbr_dist, "nbr_dist", torch.float32, B * M * k)
    need = knn_workspace_bytes(B, M, N, D, k, Q.dtype)
    if ws is None or ws.numel() < need:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _need(ws, "ws", torch.uint8)
    _check(lib.kmeans_knn(_ptr(Q), _ptr(R), _dt(Q), B, M, N, D, int(k), _ptr(nbr_idx),
                          _ptr(nbr_dist), _ptr(ws), ws.numel(), _stream()), "kmeans_knn")
    return nbr_idx, nbr_dist
