"""Comparison of GPU outputs with the fp64 oracle, to the tolerances of the contract.

* assignments: identical, except points whose oracle gap (second-smallest minus
  smallest squared distance) is below 1e-3 * |x|^2; disagreements on those
  points are counted and reported, never hidden, and the centroid chosen
  there must itself lie within that window: d(x, c_gpu) - d_min <= 1e-3 * |x|^2.
* min_dist: |gpu - d(x, c_gpu_idx)| <= tol * (|x|^2 + |c_gpu_idx|^2).
* centroids: per centroid, |c_gpu - c_oracle| <= tol * |c_oracle| (norm-wise).
* counts: identical.  objective: relative difference <= tol (with an absolute
  floor of 1e-3 * tol * sum_i (|x_i|^2 + |c_i|^2) for objectives near zero).
tol = 1e-3 for bf16/fp16 points and 1e-5 for fp32 points.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch

GAP_REL = 1e-3


def tol_for(dtype: str) -> float:
    return 1e-5 if dtype == "f32" else 1e-3


def raw(X: torch.Tensor) -> np.ndarray:
    """Stored bits of a (CPU or GPU) point tensor as the oracle takes them."""
    X = X.detach().cpu().contiguous()
    if X.dtype in (torch.bfloat16, torch.float16):
        return X.view(torch.int16).numpy().view(np.uint16)
    return X.numpy()


@dataclasses.dataclass
class AssignReport:
    n: int
    mismatches: int          # all disagreements (every one of them exempt if ok)
    exempt_points: int       # points whose oracle gap is below the exemption threshold
    worst_md_err: float      # max of |md - d| / (|x|^2 + |c|^2)
    J_gpu: float
    J_oracle: float


def check_assign(o, X_raw, dtype, C64, idx_gpu, md_gpu) -> AssignReport:
    """X_raw [B,N,D] raw points, C64 [B,K,D] fp64 (the centroids the GPU was given)."""
    B, N, D = X_raw.shape
    tol = tol_for(dtype)
    idx_o, md_o, gap_o = o.assign(X_raw, dtype, C64)
    x64 = o.widen(X_raw, dtype)
    xn = (x64 * x64).sum(-1)
    exempt = gap_o < GAP_REL * xn
    idx_gpu = np.asarray(idx_gpu).reshape(B, N)
    md_gpu = np.asarray(md_gpu, np.float64).reshape(B, N)
    assert idx_gpu.min() >= 0 and idx_gpu.max() < C64.shape[1], "index out of range"
    bad = idx_gpu != idx_o
    hard = bad & ~exempt
    assert not hard.any(), (f"{int(hard.sum())} non-exempt assignment mismatches, e.g. at "
                            f"{np.argwhere(hard)[:5].tolist()}")
    # distance to the centroid the GPU chose, in fp64
    d_choice = md_o.copy()
    if bad.any():
        bi, ni = np.nonzero(bad)
        c = C64[bi, idx_gpu[bi, ni]]
        d_choice[bi, ni] = ((x64[bi, ni] - c) ** 2).sum(-1)
        # an exempt disagreement must still pick a centroid inside the window
        excess = d_choice[bi, ni] - md_o[bi, ni]
        lim = GAP_REL * xn[bi, ni]
        far = excess > lim
        assert not far.any(), (f"{int(far.sum())} exempt mismatches chose a centroid outside the "
                               f"1e-3*|x|^2 window, e.g. point {(bi[far][0], ni[far][0])}: "
                               f"excess {excess[far][0]:.3e} > {lim[far][0]:.3e}")
    cn = (C64 ** 2).sum(-1)
    scale = xn + np.take_along_axis(cn, idx_gpu, axis=1)
    err = np.abs(md_gpu - d_choice) / np.maximum(scale, 1e-300)
    assert err.max() <= tol, f"min_dist error {err.max():.3e} > {tol}"
    J_g, J_o = md_gpu.sum(), md_o.sum()
    # relative, with a floor for (near-)zero objectives: 1e-3 of the summed
    # per-point min_dist tolerances
    floor = 1e-3 * tol * scale.sum()
    assert abs(J_g - J_o) <= max(tol * abs(J_o), floor), f"objective {J_g} vs {J_o}"
    return AssignReport(B * N, int(bad.sum()), int(exempt.sum()), float(err.max()), J_g, J_o)


def check_update(o, X_raw, dtype, idx_gpu, Cprev64, C_gpu, counts_gpu) -> float:
    """Teacher-forced update: the oracle consumes the GPU's own assignment."""
    B, N, D = X_raw.shape
    tol = tol_for(dtype)
    C_o, n_o = o.update(X_raw, dtype, np.asarray(idx_gpu).reshape(B, N), Cprev64)
    counts_gpu = np.asarray(counts_gpu).reshape(n_o.shape)
    assert np.array_equal(counts_gpu, n_o), "counts differ"
    C_gpu = np.asarray(C_gpu, np.float64).reshape(C_o.shape)
    num = np.linalg.norm(C_gpu - C_o, axis=-1)
    den = np.linalg.norm(C_o, axis=-1)
    rel = num / np.maximum(den, 1e-30)
    assert rel.max() <= tol, f"centroid error {rel.max():.3e} > {tol}"
    empty = n_o == 0
    if empty.any():
        assert np.array_equal(C_gpu[empty], np.asarray(Cprev64, np.float32).astype(np.float64)[empty]), \
            "empty cluster did not keep its centroid"
    return float(rel.max())
