"""Checks that pin the fp64 oracle to facts other than itself.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises AssertionError if
the oracle disagrees with something the mathematics or an independent library
fixes: exact rational arithmetic, a hand-worked example, library routines
(scipy's vector quantiser, scikit-learn's Lloyd, torch's cdist, numpy's float16
and torch's bfloat16 conversions), closed forms, invariants and brute-force
enumeration.  ``test_oracle_pins.py`` runs them against the real oracle;
``test_oracle_mutants.py`` runs them against copies with planted mistakes and
requires every mistake to be caught.  ``KNN_PINS`` do the same for the KNN
search (exact sorting, scipy's k-d tree, scikit-learn's brute-force
neighbours, torch's cdist, the assignment step as k = 1).
"""
from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np
import torch

from oracle import exact

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------- helpers
def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def _bits(a, dtype: str) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    t = t.to(torch.bfloat16 if dtype == "bf16" else torch.float16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _dyadic(rng, shape, den=8, span=16):
    return rng.integers(-span, span + 1, size=shape) / den


# ------------------------------------------------------------------ widening
def pin_widen_bf16(o):
    """Every bf16 bit pattern widens as torch's bfloat16 -> float64 conversion."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = o.widen(bits, "bf16")
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


def pin_widen_f16(o):
    """Every fp16 bit pattern widens as numpy's float16 -> float64 conversion."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = o.widen(bits, "f16")
    ref = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


# ------------------------------------------------------------- exact rational
def pin_exact_dyadic(o, seed=1):
    """Dyadic inputs: every fp64 step is exact, so the oracle must equal Fractions bit for bit."""
    rng = np.random.default_rng(seed)
    for trial in range(12):
        N = int(rng.integers(1, 13))
        K = int(rng.integers(1, 5))
        D = int(rng.integers(1, 4))
        X = _dyadic(rng, (N, D))
        C = _dyadic(rng, (K, D))
        if trial % 3 == 1:                      # force duplicate centroids / exact ties
            C[-1] = C[0]
        dtype = ("f32", "bf16", "f16")[trial % 3]
        Xs = _f32(X) if dtype == "f32" else _bits(X, dtype)
        Xq, Cq = exact.to_frac(X), exact.to_frac(C)
        e_idx, e_md, e_gap = exact.assign(Xq, Cq)
        idx, md, gap = o.assign(Xs, dtype, C)
        assert idx[0].tolist() == e_idx, (trial, idx, e_idx)
        assert [Fraction(v) for v in md[0]] == e_md
        for g, eg in zip(gap[0], e_gap):
            assert (eg is None and np.isinf(g)) or Fraction(g) == eg
        e_C, e_n = exact.update(Xq, e_idx, Cq)
        C1, n = o.update(Xs, dtype, idx, C)
        assert n[0].tolist() == e_n
        # one rounding (the division) separates the fp64 mean from the exact one
        assert np.array_equal(C1[0], np.array([[float(v) for v in r] for r in e_C]))
        # one Lloyd iteration is exact end to end
        e_C1, e_idx1, e_md1, e_n1, e_obj1 = exact.lloyd(Xq, Cq, 1)
        CT, idxT, mdT, nT, obj = o.lloyd(Xs, dtype, C, 1)
        assert idxT[0].tolist() == e_idx1 and nT[0].tolist() == e_n1
        assert Fraction(obj[0, 0]) == e_obj1[0]
        assert np.array_equal(CT[0], np.array([[float(v) for v in r] for r in e_C1]))
        # later iterations, teacher-forced: exact steps from the oracle's own fp64 state
        iters = 4
        CT, idxT, mdT, nT, obj = o.lloyd(Xs, dtype, C, iters)
        Ct = C
        for t in range(iters):
            e_i, e_m, e_g = exact.assign(Xq, exact.to_frac(np.reshape(Ct, (K, D))))
            i_t, m_t, _ = o.assign(Xs, dtype, Ct)
            for i in range(N):
                if e_g[i] is None or e_g[i] > Fraction(1, 1 << 40):
                    assert i_t[0, i] == e_i[i]
            assert abs(Fraction(obj[0, t]) - sum(e_m, Fraction(0))) <= \
                sum(e_m, Fraction(0)) * Fraction(1, 1 << 48) + Fraction(1, 1 << 60)
            Ct, _ = o.update(Xs, dtype, i_t, Ct)
        assert np.array_equal(Ct, CT)


def pin_exact_general(o, seed=2):
    """Arbitrary fp32 inputs: idx equal unless the exact gap is tiny; values to fp64 rounding."""
    rng = np.random.default_rng(seed)
    for trial in range(6):
        N, K, D = int(rng.integers(4, 13)), int(rng.integers(2, 5)), int(rng.integers(1, 6))
        X = _f32(rng.standard_normal((N, D)))
        C = _f32(rng.standard_normal((K, D))).astype(np.float64)
        Xq, Cq = exact.to_frac(X), exact.to_frac(C)
        e_idx, e_md, e_gap = exact.assign(Xq, Cq)
        idx, md, gap = o.assign(X, "f32", C)
        for i in range(N):
            if e_gap[i] > Fraction(1, 10 ** 9):
                assert idx[0, i] == e_idx[i]
            assert abs(Fraction(md[0, i]) - e_md[i]) <= e_md[i] * Fraction(1, 10 ** 13) + \
                Fraction(1, 10 ** 300)
            assert abs(Fraction(gap[0, i]) - e_gap[i]) <= Fraction(1, 10 ** 12)
        e_C, e_n = exact.update(Xq, idx[0].tolist(), Cq)
        C1, n = o.update(X, "f32", idx, C)
        assert n[0].tolist() == e_n
        ref = np.array([[float(v) for v in r] for r in e_C])
        assert np.allclose(C1[0], ref, rtol=1e-14, atol=1e-15)


def pin_golden_worked(o):
    """The hand-worked 1-D example in tests/golden/lloyd_1d_worked.json."""
    with open(os.path.join(GOLDEN, "lloyd_1d_worked.json")) as f:
        g = json.load(f)
    X = _f32(g["X"])
    C = np.asarray(g["C0"], np.float64)
    for t in range(g["iters"]):
        idx, md, _ = o.assign(X, "f32", C)
        assert idx[0].tolist() == g["idx_per_iter"][t]
        num, den = g["objective_num_den"][t]
        J = md[0].sum()
        assert abs(J - num / den) <= 1e-12 * abs(num / den)
        C, n = o.update(X, "f32", idx, C)
        want = [[float(Fraction(p, q)) for p, q in row] for row in g["C_per_iter_num_den"][t]]
        assert C[0].tolist() == want
    assert n[0].tolist() == g["counts_last"]
    CT, _, _, nT, obj = o.lloyd(X, "f32", np.asarray(g["C0"], np.float64), g["iters"])
    assert nT[0].tolist() == g["counts_last"]
    for t, (num, den) in enumerate(g["objective_num_den"]):
        assert abs(obj[0, t] - num / den) <= 1e-12 * (num / den)


# ----------------------------------------------------------- library routines
def pin_scipy_vq(o, seed=3):
    """scipy.cluster.vq.vq: nearest code and its Euclidean distance."""
    from scipy.cluster.vq import vq
    rng = np.random.default_rng(seed)
    X = _f32(rng.standard_normal((600, 7)))
    C = rng.standard_normal((23, 7))
    code, dist = vq(X.astype(np.float64), C)
    idx, md, gap = o.assign(X, "f32", C)
    clear = gap[0] > 1e-9
    assert np.array_equal(idx[0][clear], code[clear])
    assert np.allclose(md[0], dist ** 2, rtol=1e-12, atol=1e-12)


def pin_torch_cdist(o, seed=4):
    """torch.cdist + argmin in fp64 (argmin returns the first minimum)."""
    rng = np.random.default_rng(seed)
    X = _f32(rng.uniform(-1, 1, (500, 16)))
    C = rng.uniform(-1, 1, (40, 16))
    d = torch.cdist(torch.from_numpy(X.astype(np.float64)), torch.from_numpy(C),
                    compute_mode="donot_use_mm_for_euclid_dist") ** 2
    ref = torch.argmin(d, dim=1).numpy()
    idx, md, gap = o.assign(X, "f32", C)
    clear = gap[0] > 1e-9
    assert np.array_equal(idx[0][clear], ref[clear])
    assert np.allclose(md[0], d.min(dim=1).values.numpy(), rtol=1e-12, atol=1e-12)


def pin_sklearn_lloyd(o, seed=5):
    """scikit-learn's Lloyd k-means from the same initial centroids, no empty clusters."""
    from sklearn.cluster import KMeans
    rng = np.random.default_rng(seed)
    K, D, per = 12, 5, 60
    centres = rng.uniform(-4, 4, (K, D))
    X = _f32(np.repeat(centres, per, axis=0) + 0.6 * rng.standard_normal((K * per, D)))
    X = X[rng.permutation(len(X))]
    C0 = X[:K].astype(np.float64)
    for iters in (1, 2, 4, 7):
        km = KMeans(n_clusters=K, init=C0, n_init=1, max_iter=iters, tol=0.0,
                    algorithm="lloyd").fit(X.astype(np.float64))
        CT, idx, md, n, obj = o.lloyd(X, "f32", C0, iters)
        assert n.min() > 0
        assert np.allclose(CT[0], km.cluster_centers_, rtol=1e-10, atol=1e-12)
        lab, dmin, gap = o.assign(X, "f32", CT)
        clear = gap[0] > 1e-9
        assert np.array_equal(lab[0][clear], km.labels_[clear])
        assert abs(dmin[0].sum() - km.inertia_) <= 1e-9 * km.inertia_


# --------------------------------------------------------------- closed forms
def pin_single_cluster(o, seed=6):
    """K = 1: every index is 0 and the new centroid is the mean of all points."""
    rng = np.random.default_rng(seed)
    X = _f32(rng.standard_normal((257, 9)))
    C = rng.standard_normal((1, 9))
    idx, md, gap = o.assign(X, "f32", C)
    assert not idx.any()
    assert np.all(np.isinf(gap))
    assert np.allclose(md[0], ((X.astype(np.float64) - C) ** 2).sum(1), rtol=1e-13)
    C1, n = o.update(X, "f32", idx, C)
    assert n[0].tolist() == [257]
    assert np.allclose(C1[0, 0], X.astype(np.float64).mean(0), rtol=1e-13, atol=1e-15)


def pin_points_as_centroids(o, seed=7):
    """C = X with distinct points: each point is its own centroid at distance 0."""
    rng = np.random.default_rng(seed)
    X = _f32(rng.standard_normal((64, 5)))
    idx, md, _ = o.assign(X, "f32", X.astype(np.float64))
    assert idx[0].tolist() == list(range(64))
    assert not md.any()
    C1, n = o.update(X, "f32", idx, X.astype(np.float64))
    assert np.array_equal(C1[0], X.astype(np.float64)) and (n == 1).all()


def pin_duplicate_centroids(o, seed=8):
    """A centroid duplicated at a higher index never wins; its cluster is empty and kept."""
    rng = np.random.default_rng(seed)
    X = _f32(rng.standard_normal((300, 4)))
    C = rng.standard_normal((6, 4))
    C[4] = C[1]
    idx, _, _ = o.assign(X, "f32", C)
    assert (idx[0] == 1).any() and not (idx[0] == 4).any()
    C1, n = o.update(X, "f32", idx, C)
    assert n[0, 4] == 0 and np.array_equal(C1[0, 4], C[4])


def pin_1d_midpoints(o, seed=9):
    """D = 1 with sorted centres: the cells are bounded by midpoints (numpy.searchsorted)."""
    rng = np.random.default_rng(seed)
    c = np.sort(rng.choice(np.arange(-64, 64), size=9, replace=False)).astype(np.float64) / 4
    mids = (c[1:] + c[:-1]) / 2
    x = _f32(np.concatenate([rng.uniform(-20, 20, 400), mids]))  # include exact midpoints
    ref = np.searchsorted(mids, x.astype(np.float64), side="left")  # a midpoint goes low
    idx, _, _ = o.assign(x[:, None], "f32", c[:, None])
    assert np.array_equal(idx[0], ref)


def pin_empty_cluster_kept(o, seed=10):
    """A centroid far from every point receives none and keeps its coordinates."""
    rng = np.random.default_rng(seed)
    X = _f32(rng.standard_normal((200, 3)))
    C = np.vstack([rng.standard_normal((3, 3)), [[1e3, 1e3, 1e3]]])
    CT, idx, md, n, _ = o.lloyd(X, "f32", C, 3)
    assert n[0, 3] == 0 and np.array_equal(CT[0, 3], C[3])


def pin_batched_independent(o, seed=11):
    """B instances in one call equal B separate calls."""
    rng = np.random.default_rng(seed)
    X = _f32(rng.standard_normal((3, 100, 6)))
    C0 = rng.standard_normal((3, 5, 6))
    CT, idx, md, n, obj = o.lloyd(X, "f32", C0, 4)
    for b in range(3):
        cb, ib, mb, nb, ob = o.lloyd(X[b], "f32", C0[b], 4)
        assert np.array_equal(cb[0], CT[b]) and np.array_equal(ib[0], idx[b])
        assert np.array_equal(nb[0], n[b]) and np.array_equal(ob[0], obj[b])


# ------------------------------------------------------------------ invariants
def pin_mass_conservation(o, seed=12):
    """sum_k n_k c'_k = sum_i x_i and sum_k n_k = N."""
    rng = np.random.default_rng(seed)
    X = _f32(rng.standard_normal((2, 1000, 8)))
    C = rng.standard_normal((2, 17, 8))
    idx, _, _ = o.assign(X, "f32", C)
    C1, n = o.update(X, "f32", idx, C)
    for b in range(2):
        assert n[b].sum() == 1000
        lhs = (n[b][:, None] * C1[b]).sum(0)
        rhs = X[b].astype(np.float64).sum(0)
        assert np.allclose(lhs, rhs, rtol=1e-12, atol=1e-10)


def pin_monotone(o, workloads):
    """J_t never increases along a Lloyd run (each step can only lower the objective)."""
    for w, X, dtype in workloads:
        _, _, _, _, obj = o.lloyd(X, dtype, w.C0.numpy(), w.iters)
        for b in range(obj.shape[0]):
            assert np.all(np.diff(obj[b]) <= 1e-12 * np.abs(obj[b][:-1])), (w.name, obj[b])


def pin_fixed_point(o, seed=13):
    """Once the assignment stops changing, a further step leaves C bit-identical."""
    rng = np.random.default_rng(seed)
    X = _f32(np.repeat(rng.uniform(-3, 3, (6, 4)), 40, axis=0) + 0.4 * rng.standard_normal((240, 4)))
    C = X[rng.choice(240, 6, replace=False)].astype(np.float64)
    prev = None
    for _ in range(100):
        idx, _, _ = o.assign(X, "f32", C)
        C_next, _ = o.update(X, "f32", idx, C)
        if prev is not None and np.array_equal(prev, idx):
            assert np.array_equal(C_next, C)
            idx2, _, _ = o.assign(X, "f32", C_next)
            assert np.array_equal(idx2, idx)
            return
        prev, C = idx, C_next
    raise AssertionError("Lloyd did not reach a fixed point in 100 steps")


def pin_blob_recovery(o, seed=14):
    """Well-separated blobs, one initial point per blob: labels and means recovered exactly."""
    rng = np.random.default_rng(seed)
    K, D, per = 16, 8, 50
    grid = np.stack(np.meshgrid(*[np.arange(2)] * 4, indexing="ij"), -1).reshape(-1, 4)
    centres = np.hstack([grid, grid]) * 40.0
    truth = np.repeat(np.arange(K), per)
    perm = rng.permutation(K * per)
    truth = truth[perm]
    X = _f32(centres[truth] + 0.05 * rng.standard_normal((K * per, D)))
    first = np.array([np.flatnonzero(truth == k)[0] for k in range(K)])
    C0 = X[first].astype(np.float64)
    CT, idx, _, n, _ = o.lloyd(X, "f32", C0, 2)
    assert np.array_equal(idx[0], truth)
    means = np.stack([X[truth == k].astype(np.float64).mean(0) for k in range(K)])
    assert np.allclose(CT[0], means, rtol=1e-13, atol=1e-12)


def pin_global_minimum(o, seed=15):
    """Tiny sets: a converged Lloyd run is a fixed point with J >= the enumerated optimum."""
    rng = np.random.default_rng(seed)
    for trial in range(4):
        N, K = 7, 2 + trial % 2
        X = _dyadic(rng, (N, 2), den=4, span=12)
        Xq = exact.to_frac(X)
        jstar = exact.global_minimum(Xq, K)
        best = None
        for start in range(4):
            C0 = X[rng.choice(N, K, replace=False)]
            CT, idx, md, n, obj = o.lloyd(_f32(X), "f32", C0, 12)
            # fixed point: assignment under C_T equals the last one, C_T = cluster means
            idx2, md2, _ = o.assign(_f32(X), "f32", CT)
            assert np.array_equal(idx2, idx)
            J = Fraction(md2[0].sum())
            assert J >= jstar * (1 - Fraction(1, 10 ** 12))
            best = J if best is None else min(best, J)
        # with four starts on seven points, at least one start reaches the optimum
        assert abs(best - jstar) <= jstar * Fraction(1, 10 ** 12) + Fraction(1, 10 ** 12)


# ------------------------------------------------------------------ non-finite values
def pin_nonfinite_assign(o):
    """Hand-worked: a point with a NaN or infinite coordinate is unassigned
    (idx -1, min_dist and gap NaN); a centroid with one is never chosen, and a
    finite point with no finite centroid left is unassigned too."""
    X = _f32([[[0, 0], [np.nan, 1], [np.inf, 0], [3, 0], [-np.inf, 2]]])
    C = np.array([[[0, 0], [np.nan, 0], [4, 0], [1, np.inf]]])
    idx, md, gap = o.assign(X, "f32", C)
    assert idx.tolist() == [[0, -1, -1, 2, -1]]
    assert md[0, 0] == 0 and md[0, 3] == 1 and np.isnan(md[0, [1, 2, 4]]).all()
    assert gap[0, 0] == 16 and gap[0, 3] == 8 and np.isnan(gap[0, [1, 2, 4]]).all()
    # one usable centroid: its distance, and no runner-up (+inf)
    idx, md, gap = o.assign(_f32([[[1, 1]]]), "f32", np.array([[[np.nan, 0], [0, 0]]]))
    assert idx.tolist() == [[1]] and md[0, 0] == 2 and gap[0, 0] == np.inf
    # no usable centroid
    idx, md, gap = o.assign(_f32([[[1, 1], [2, 2]]]), "f32", np.array([[[np.inf, 0], [0, np.nan]]]))
    assert idx.tolist() == [[-1, -1]] and np.isnan(md).all()
    # 16-bit storage: a bf16 NaN and an fp16 infinity read as such
    for dt, bits in (("bf16", 0x7FC0), ("f16", 0x7C00)):
        Xb = np.array([[[0, 0], [bits, 0]]], np.uint16)
        idx, md, _ = o.assign(Xb, dt, np.array([[[0.0, 0.0]]]))
        assert idx.tolist() == [[0, -1]] and md[0, 0] == 0 and np.isnan(md[0, 1])


def pin_nonfinite_update_lloyd(o):
    """Hand-worked: the update ignores entries outside [0, K); a Lloyd run on
    points with NaNs leaves them unassigned, keeps every centroid finite and
    counts only the assigned points in J_t."""
    X = _f32([[[0, 0], [2, 0], [np.nan, 0], [10, 0], [12, 0]]])
    C_prev = np.array([[[0.0, 0.0], [10.0, 0.0], [5.0, 5.0]]])
    C1, n = o.update(X, "f32", np.array([[0, 0, -1, 1, 7]], np.int32), C_prev)
    assert n.tolist() == [[2, 1, 0]]
    assert C1[0].tolist() == [[1, 0], [10, 0], [5, 5]]
    CT, idx, md, n, obj = o.lloyd(X, "f32", C_prev, 2)
    assert idx.tolist() == [[0, 0, -1, 1, 1]] and n.tolist() == [[2, 2, 0]]
    assert CT[0].tolist() == [[1, 0], [11, 0], [5, 5]]
    # J_0 = 0 + 4 + 0 + 4 under C_prev; J_1 = 1 + 1 + 1 + 1 under the means
    assert obj.tolist() == [[8.0, 4.0]]


FAST_PINS = [pin_widen_bf16, pin_widen_f16, pin_exact_dyadic, pin_exact_general, pin_golden_worked,
             pin_scipy_vq, pin_torch_cdist, pin_single_cluster, pin_points_as_centroids,
             pin_duplicate_centroids, pin_1d_midpoints, pin_empty_cluster_kept,
             pin_batched_independent, pin_mass_conservation, pin_fixed_point, pin_blob_recovery,
             pin_global_minimum, pin_nonfinite_assign, pin_nonfinite_update_lloyd]


# ------------------------------------------------------------------ KNN search
def pin_knn_exact_dyadic(o, seed=21):
    """Dyadic inputs on a coarse grid (many equal distances): the oracle's k nearest
    rows, their order, distances and the next distance equal exact sorting."""
    rng = np.random.default_rng(seed)
    for trial in range(12):
        M = int(rng.integers(1, 7))
        N = int(rng.integers(1, 12))
        D = int(rng.integers(1, 4))
        k = int(rng.integers(1, N + 1))
        Q = _dyadic(rng, (M, D), den=2, span=3)
        R = _dyadic(rng, (N, D), den=2, span=3)
        idx, dist, nxt = o.knn(_f32(Q), _f32(R), "f32", k)
        ei, ed, en = exact.knn(exact.to_frac(Q), exact.to_frac(R), k)
        for i in range(M):
            assert idx[0, i].tolist() == ei[i]
            assert [Fraction(v) for v in dist[0, i]] == ed[i]
            assert (np.isinf(nxt[0, i]) if en[i] is None else Fraction(nxt[0, i]) == en[i])


def pin_knn_ckdtree(o, seed=22):
    """scipy's k-d tree (exact search) on continuous data: same rows, same order."""
    from scipy.spatial import cKDTree
    rng = np.random.default_rng(seed)
    R = _f32(rng.standard_normal((700, 6)))
    Q = _f32(rng.standard_normal((90, 6)))
    dd, ii = cKDTree(R.astype(np.float64)).query(Q.astype(np.float64), k=9)
    idx, dist, nxt = o.knn(Q, R, "f32", 9)
    assert np.array_equal(idx[0], ii)
    assert np.allclose(dist[0], dd ** 2, rtol=1e-12, atol=1e-12)
    d10, _ = cKDTree(R.astype(np.float64)).query(Q.astype(np.float64), k=10)
    assert np.allclose(nxt[0], d10[:, 9] ** 2, rtol=1e-12, atol=1e-12)


def pin_knn_sklearn_bf16(o, seed=23):
    """bf16 storage: scikit-learn's brute-force neighbours on the widened values."""
    from sklearn.neighbors import NearestNeighbors
    rng = np.random.default_rng(seed)
    Rb = _bits(rng.uniform(-1, 1, (400, 12)), "bf16")
    Qb = _bits(rng.uniform(-1, 1, (60, 12)), "bf16")
    R64 = torch.from_numpy(Rb.view(np.int16)).view(torch.bfloat16).double().numpy()
    Q64 = torch.from_numpy(Qb.view(np.int16)).view(torch.bfloat16).double().numpy()
    nn = NearestNeighbors(n_neighbors=5, algorithm="brute").fit(R64)
    dd, ii = nn.kneighbors(Q64)
    idx, dist, _ = o.knn(Qb, Rb, "bf16", 5)
    # rows within a distance tie may come in another order from the library
    clear = np.all(np.diff(dd ** 2, axis=1) > 1e-12, axis=1)
    assert np.array_equal(idx[0][clear], ii[clear])
    assert np.allclose(dist[0], dd ** 2, rtol=1e-9, atol=1e-12)


def pin_knn_self_and_full_order(o, seed=24):
    """Queries equal to database rows find themselves at distance 0; k = N lists
    every row, by torch.cdist distance (fp64, direct form), stably."""
    rng = np.random.default_rng(seed)
    R = _f32(rng.standard_normal((50, 5)))
    idx, dist, nxt = o.knn(R, R, "f32", 3)
    assert np.array_equal(idx[0, :, 0], np.arange(50))
    assert np.all(dist[0, :, 0] == 0.0)
    Q = _f32(rng.standard_normal((7, 5)))
    idx, dist, nxt = o.knn(Q, R, "f32", 50)
    d = torch.cdist(torch.from_numpy(Q.astype(np.float64)), torch.from_numpy(R.astype(np.float64)),
                    compute_mode="donot_use_mm_for_euclid_dist").numpy() ** 2
    ref = np.argsort(d, axis=1, kind="stable")
    assert np.array_equal(idx[0], ref)
    assert np.all(np.isinf(nxt[0]))


def pin_knn_k1_is_assignment(o, seed=25):
    """k = 1 is the assignment step with the database as the centroids."""
    rng = np.random.default_rng(seed)
    R = _dyadic(rng, (30, 3), den=2, span=2)       # coarse: ties occur
    Q = _dyadic(rng, (200, 3), den=2, span=2)
    idx, dist, nxt = o.knn(_f32(Q), _f32(R), "f32", 1)
    a_idx, a_md, a_gap = o.assign(_f32(Q), "f32", R.astype(np.float64))
    assert np.array_equal(idx[0, :, 0], a_idx[0])
    assert np.array_equal(dist[0, :, 0], a_md[0])
    assert np.array_equal(nxt[0] - dist[0, :, 0], a_gap[0])


def pin_knn_batched(o, seed=26):
    """B instances are independent: stacked results equal per-instance results."""
    rng = np.random.default_rng(seed)
    Q = _f32(rng.standard_normal((3, 20, 4)))
    R = _f32(rng.standard_normal((3, 35, 4)))
    idx, dist, nxt = o.knn(Q, R, "f32", 4)
    for b in range(3):
        i1, d1, n1 = o.knn(Q[b], R[b], "f32", 4)
        assert np.array_equal(idx[b], i1[0]) and np.array_equal(dist[b], d1[0])
        assert np.array_equal(nxt[b], n1[0])


KNN_PINS = [pin_knn_exact_dyadic, pin_knn_ckdtree, pin_knn_sklearn_bf16, pin_knn_self_and_full_order,
            pin_knn_k1_is_assignment, pin_knn_batched]
