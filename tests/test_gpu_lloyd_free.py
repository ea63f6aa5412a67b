"""GPU parity, free-running: the HIP Lloyd iteration against the oracle's own
Lloyd run from the same C_0, for each workload's configured number of
iterations (paper Section 5: the Lloyd iteration is an assignment then a
centroid update; the contract compares assignments, centroids and objective).

Each side runs on its own state: the GPU advances its fp32 centroids with
kmeans_lloyd, one iteration per call (checked at the end to equal, bit for
bit, one call of all the iterations), and the oracle advances its fp64
centroids with its own assignment and update.  Per iteration:

* every disagreement in the assignment must be exempt (oracle top-2 gap
  below 1e-3 |x|^2) and the centroid the GPU chose there must lie within that
  window of the nearest; such points are near-ties, where either choice is a
  nearest centroid under the contract, and the oracle's run takes the GPU's
  choice for them (only there: its centroids are never taken from the GPU),
  so that one near-tie does not part two otherwise equal runs;
* J_t (the objective of the assignment under C_t), the counts and the new
  centroids (norm-wise) agree within the contract's tolerance;
* the number of exempt disagreements is reported per iteration.

Sizes: the fp32 workload and the batched fp16 workload (which runs the
single-pass small-K step) in full; the 1M-point bf16 workload in full; the
8M-point and the 2M x 1024 workloads on fewer points and clusters, which the
oracle finishes in seconds.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from parity import GAP_REL, raw, tol_for
from paper_2608_12629_amd.synth import make_workload

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


FREE = {
    "blobs_f32_full": dict(wl=1),
    "blobs_1m_bf16_full": dict(wl=2),
    "zipf_bf16_scaled": dict(wl=3, N=262144, K=1024),
    "batched_f16_full": dict(wl=4),
    "subspace_bf16_scaled": dict(wl=5, N=32768, K=1024),
}


@pytest.mark.parametrize("name", list(FREE))
def test_free_running_lloyd(km, oracle, name):
    kw = dict(FREE[name])
    w = make_workload(kw.pop("wl"), **kw)
    T = w.iters
    tol = tol_for(w.dtype)
    say(f"[free {name}] {w.name} B={w.B} N={w.N} D={w.D} K={w.K} {w.dtype} T={T}")
    Xd = w.X.cuda()
    Xr = raw(w.X)
    x64 = oracle.widen(Xr, w.dtype)
    xn = (x64 * x64).sum(-1)
    ws = km.Workspace(w.B, w.N, w.D, w.K, w.X.dtype)

    Cg = w.C0.cuda().clone()                 # GPU state (fp32)
    Co = w.C0.double().numpy().copy()        # oracle state (fp64)
    flips = []
    for t in range(T):
        Cg_next, idx_g, md_g, n_g, J_g = km.kmeans_lloyd(Xd, Cg.clone(), 1, ws=ws)
        torch.cuda.synchronize()
        idx_o, md_o, gap_o = oracle.assign(Xr, w.dtype, Co)
        ig = idx_g.cpu().numpy()
        mism = ig != idx_o
        exempt = gap_o < GAP_REL * xn
        hard = mism & ~exempt
        assert not hard.any(), (f"t={t}: {int(hard.sum())} non-exempt assignment mismatches, "
                                f"e.g. {np.argwhere(hard)[:5].tolist()}")
        md_f = md_o.copy()                   # the oracle's distances under the followed choice
        if mism.any():
            bi, ni = np.nonzero(mism)
            d_g = ((x64[bi, ni] - Co[bi, ig[bi, ni]]) ** 2).sum(-1)
            assert np.all(d_g - md_o[bi, ni] <= GAP_REL * xn[bi, ni]), \
                f"t={t}: an exempt disagreement chose a centroid outside the near-tie window"
            md_f[bi, ni] = d_g
        idx_f = np.where(mism, ig, idx_o).astype(np.int32)
        Co_next, n_o = oracle.update(Xr, w.dtype, idx_f, Co)
        J_o = md_f.sum(-1)
        J_gn = J_g.cpu().numpy()[:, 0]
        rel_J = np.abs(J_gn - J_o) / np.abs(J_o)
        Cgn = Cg_next.cpu().double().numpy()
        rel_C = (np.linalg.norm(Cgn - Co_next, axis=-1) /
                 np.maximum(np.linalg.norm(Co_next, axis=-1), 1e-30))
        flips.append(int(mism.sum()))
        say(f"  t={t} J_gpu={J_gn.sum():.9e} J_oracle={J_o.sum():.9e} rel={rel_J.max():.2e} "
            f"C_err={rel_C.max():.2e} exempt flips={int(mism.sum())} "
            f"(exempt points {int(exempt.sum())})")
        assert rel_J.max() <= tol, f"t={t}: objective off by {rel_J.max():.3e} > {tol}"
        assert np.array_equal(n_g.cpu().numpy(), n_o), f"t={t}: counts differ"
        assert rel_C.max() <= tol, f"t={t}: centroid error {rel_C.max():.3e} > {tol}"
        Cg, Co = Cg_next, Co_next

    # the per-iteration calls are the real free-running run: one call of T
    # iterations gives the same bits
    CT, _, _, _, obj = km.kmeans_lloyd(Xd, w.C0.cuda().clone(), T, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(CT, Cg), "T single-iteration calls differ from one T-iteration call"
    o = obj.cpu().numpy()
    assert np.all(np.diff(o, axis=-1) <= tol * o[:, :-1]), "objective increased"
    rel_C = (np.linalg.norm(CT.cpu().double().numpy() - Co, axis=-1) /
             np.maximum(np.linalg.norm(Co, axis=-1), 1e-30))
    say(f"  final C_T: max norm-wise error {rel_C.max():.2e}; exempt flips per iteration {flips}")
    assert rel_C.max() <= tol
