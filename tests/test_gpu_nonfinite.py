"""GPU parity with NaN and infinite inputs, per kernel family, against the
oracle's reading of non-finite values: a point with a NaN or infinite
coordinate is unassigned (idx -1, min_dist NaN, no objective term, no count
or sum); a centroid with one is never chosen; a point with no finite centroid
is unassigned.  The paper fixes nothing here; the reading and its pins are
with the oracle.

Each case plants non-finite coordinates in about 2% of the points (NaN, +inf
and -inf, one coordinate each) and in a few centroids, then checks:

* kmeans_assign: the unassigned points are exactly the oracle's; the others
  agree with the oracle to the contract (exempt near-ties only, inside the
  window; min_dist to tolerance); min_dist is NaN exactly where idx is -1;
* kmeans_lloyd, one iteration per call for a few iterations: every finite
  centroid stays finite, the counts equal the oracle's update of the GPU's own
  assignment, the centroids and J_t (assigned points only) agree to the
  tolerance; one call of all the iterations gives the same bits;
* kmeans_update with idx -1 on the planted points: the same as leaving them
  out.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from parity import GAP_REL, raw, tol_for
from paper_2608_12629_amd.synth import make_multiscale, make_workload

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def km():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    from paper_2608_12629_amd import kmeans
    return kmeans


# name: (workload factory, the kernel family it reaches)
CASES = {
    "f32_d64_k100": lambda: make_workload(1, N=8192, K=100, D=64),          # fp32 kernel
    "bf16_d128_k1000": lambda: make_workload(2, N=16384, K=1000),          # streaming kernel
    "f16_d128_k512": lambda: make_workload(4, B=2, N=8192, D=128, K=512),  # streaming, fp16
    "bf16_multiscale_d128": lambda: make_multiscale(1, 8192, 128, 300, "bf16", ratio=1e4),  # wide fallback
    "bf16_d1024_k300": lambda: make_workload(5, N=4096, K=300),            # tiled kernel
    "f16_d64_k64": lambda: make_workload(4, B=4, N=4096),                  # small-K sums / fused step
    "bf16_d8_k40": lambda: make_workload(2, N=4096, K=40, D=8),            # narrow rows, widened to fp32
}


def plant(w, seed):
    """About 2% of the points get one NaN, +inf or -inf coordinate; centroids
    1, 5 (and 9 when K > 9) get one too."""
    rng = np.random.default_rng(seed)
    X = w.X.clone()
    C = w.C0.clone()
    B, N, D = X.shape
    for b in range(B):
        pts = rng.choice(N, size=max(2, N // 50), replace=False)
        for j, p in enumerate(pts):
            X[b, p, rng.integers(D)] = (float("nan"), float("inf"), float("-inf"))[j % 3]
        for j, k in enumerate((1, 5, 9)):
            if k < w.K:
                C[b, k, rng.integers(D)] = (float("nan"), float("inf"), float("-inf"))[j % 3]
    return X, C


def check_assignment(oracle, Xr, dtype, C64, idx_g, md_g):
    idx_o, md_o, gap_o = oracle.assign(Xr, dtype, C64)
    un_o, un_g = idx_o < 0, idx_g < 0
    assert np.array_equal(un_g, un_o), (f"unassigned points differ: GPU {int(un_g.sum())}, "
                                       f"oracle {int(un_o.sum())}")
    assert np.isnan(md_g[un_g]).all() and np.isfinite(md_g[~un_g]).all()
    x64 = oracle.widen(Xr, dtype)
    with np.errstate(invalid="ignore", over="ignore"):
        xn = (x64 * x64).sum(-1)
    ok = ~un_o
    mism = ok & (idx_g != idx_o)
    hard = mism & ~(gap_o < GAP_REL * xn)
    assert not hard.any(), f"{int(hard.sum())} non-exempt mismatches"
    d_choice = md_o.copy()
    if mism.any():
        bi, ni = np.nonzero(mism)
        d_choice[bi, ni] = ((x64[bi, ni] - C64[bi, idx_g[bi, ni]]) ** 2).sum(-1)
        assert np.all(d_choice[bi, ni] - md_o[bi, ni] <= GAP_REL * xn[bi, ni])
    cn = np.nan_to_num((C64 ** 2).sum(-1), nan=0.0, posinf=0.0)
    scale = xn[ok] + np.take_along_axis(cn, np.where(ok, idx_g, 0), axis=1)[ok]
    err = np.abs(md_g[ok] - d_choice[ok]) / np.maximum(scale, 1e-300)
    assert err.max() <= tol_for(dtype), f"min_dist error {err.max():.3e}"
    return int(un_o.sum()), int(mism.sum())


@pytest.mark.parametrize("name", list(CASES))
def test_nonfinite(km, oracle, name):
    w = CASES[name]()
    X, C = plant(w, seed=len(name))
    tol = tol_for(w.dtype)
    say(f"[nonfinite {name}] {w.name} B={w.B} N={w.N} D={w.D} K={w.K} {w.dtype}")
    Xd, Xr = X.cuda(), raw(X)
    C64 = C.double().numpy()
    ws = km.Workspace(w.B, w.N, w.D, w.K, X.dtype)

    idx, md = km.kmeans_assign(Xd, C.cuda(), ws=ws)
    torch.cuda.synchronize()
    n_un, n_flip = check_assignment(oracle, Xr, w.dtype, C64, idx.cpu().numpy(),
                                    md.cpu().numpy().astype(np.float64))
    say(f"  assign: {n_un} unassigned (as the oracle), {n_flip} exempt flips")

    # the update leaves idx -1 out: equal to dropping those points
    Cd = C.cuda()
    C1, n1 = km.kmeans_update(Xd, idx, Cd, ws=ws)
    keep = (idx >= 0).cpu()
    torch.cuda.synchronize()
    C_o, n_o = oracle.update(Xr, w.dtype, idx.cpu().numpy(), C64)
    assert np.array_equal(n1.cpu().numpy(), n_o)
    assert int(n_o.sum()) == int(keep.sum())
    fin = np.isfinite(C_o).all(-1)
    c1 = C1.cpu().double().numpy()
    rel = np.linalg.norm(c1[fin] - C_o[fin], axis=-1) / np.maximum(np.linalg.norm(C_o[fin], axis=-1), 1e-30)
    assert rel.max() <= tol, f"update: centroid error {rel.max():.3e}"

    # Lloyd, one iteration per call; the oracle's update of the GPU's assignment
    T = 3
    Cg = C.cuda()
    for t in range(T):
        Cn, idx_t, md_t, n_t, J = km.kmeans_lloyd(Xd, Cg.clone(), 1, ws=ws)
        torch.cuda.synchronize()
        ig, mg = idx_t.cpu().numpy(), md_t.cpu().numpy().astype(np.float64)
        Cprev = Cg.cpu().double().numpy()
        check_assignment(oracle, Xr, w.dtype, Cprev, ig, mg)
        C_o, n_o = oracle.update(Xr, w.dtype, ig, Cprev)
        assert np.array_equal(n_t.cpu().numpy(), n_o), f"t={t}: counts differ"
        cn = Cn.cpu().double().numpy()
        fin = np.isfinite(Cprev).all(-1)
        assert np.isfinite(cn[fin]).all(), f"t={t}: a finite centroid became non-finite"
        rel = (np.linalg.norm(cn[fin] - C_o[fin], axis=-1) /
               np.maximum(np.linalg.norm(C_o[fin], axis=-1), 1e-30))
        assert rel.max() <= tol, f"t={t}: centroid error {rel.max():.3e}"
        J_ref = np.where(ig >= 0, mg, 0.0).sum(-1)
        Jg = J.cpu().numpy()[:, 0]
        assert np.all(np.abs(Jg - J_ref) <= 1e-6 * np.abs(J_ref)), f"t={t}: J {Jg} vs {J_ref}"
        Cg = Cn
    CT, _, _, _, _ = km.kmeans_lloyd(Xd, C.cuda(), T, ws=ws)
    torch.cuda.synchronize()
    # bit patterns: the planted centroids stay NaN on both sides
    assert torch.equal(CT.view(torch.int32), Cg.view(torch.int32)), \
        "T single iterations differ from one T-iteration call"
