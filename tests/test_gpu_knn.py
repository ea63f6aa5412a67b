"""GPU parity of the KNN search (kmeans_knn through the C ABI) against the fp64
oracle's exact k nearest rows.

Unique things are compared exactly and the rest checked for validity: the
returned rows must be distinct, each within the oracle's k nearest up to the
tolerance, every row clearly inside the oracle's k nearest (by more than the
tolerance) must be returned (recall 1.0), the order must follow the oracle's
distances up to the tolerance, and the reported distance must match the
oracle's distance of that row.  The tolerance is 1e-3 |q|^2 for bf16/fp16
rows, as for the assignment's exemption of near-ties.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from parity import raw

pytestmark = pytest.mark.gpu

TOL = 1e-3


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def km():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    from paper_2608_12629_amd import kmeans
    return kmeans


def _data(B, M, N, D, dtype, seed):
    g = torch.Generator().manual_seed(seed)
    centres = torch.rand((B, max(N // 20, 1), D), generator=g) * 2 - 1
    lab = torch.randint(0, centres.shape[1], (B, N), generator=g)
    R = torch.gather(centres, 1, lab[..., None].expand(B, N, D)) + 0.1 * torch.randn((B, N, D), generator=g)
    # half the queries near database rows, half anywhere
    pick = torch.randint(0, N, (B, M), generator=g)
    Q = torch.gather(R, 1, pick[..., None].expand(B, M, D)) + 0.05 * torch.randn((B, M, D), generator=g)
    Q[:, M // 2:] = torch.rand((B, M - M // 2, D), generator=g) * 2 - 1
    t = {"bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    return Q.to(t), R.to(t)


def check_knn(o, Q, R, dtype, k, gi, gd):
    """Returns the number of positions that differ from the oracle's list."""
    B, M, D = Q.shape
    N = R.shape[1]
    oi, od, _ = o.knn(raw(Q), raw(R), dtype, N)          # every row, nearest first
    qn = (o.widen(raw(Q), dtype) ** 2).sum(-1)
    rn = (o.widen(raw(R), dtype) ** 2).sum(-1)
    differ = 0
    for b in range(B):
        for m in range(M):
            rank = np.empty(N, np.int64)
            rank[oi[b, m]] = np.arange(N)
            dist = od[b, m]
            S = gi[b, m]
            tq = TOL * qn[b, m]
            assert len(set(S.tolist())) == k and S.min() >= 0 and S.max() < N, (b, m, S)
            Do = dist[rank[S]]
            dk = dist[k - 1]
            dn = dist[k] if k < N else np.inf
            assert np.all(Do <= dk + tq), (b, m, "a returned row is not among the nearest")
            must = oi[b, m, :k][dist[:k] < dn - tq]
            assert set(must.tolist()) <= set(S.tolist()), (b, m, "recall")
            assert np.all(Do[:-1] <= Do[1:] + tq), (b, m, "order")
            err = np.abs(gd[b, m] - Do)
            assert np.all(err <= TOL * (qn[b, m] + rn[b, S])), (b, m, err.max())
            differ += int(np.sum(S != oi[b, m, :k]))
    return differ


SHAPES = [
    # (B, M, N, D, k, dtype)
    (1, 600, 4000, 64, 10, "bf16"),
    (2, 333, 2049, 128, 32, "f16"),       # ragged stages, the largest k
    (1, 400, 3000, 48, 1, "bf16"),        # k = 1; padded LDS rows
    (1, 257, 129, 256, 8, "bf16"),        # one and a bit stages, widest rows
    (1, 100, 7, 16, 7, "f16"),            # k = N, a database smaller than a tile
    (3, 64, 1000, 96, 16, "bf16"),        # batched
    (1, 500, 5000, 160, 12, "f16"),       # the 16-entry lists in fp16
    (1, 300, 2000, 40, 5, "bf16"),        # D = 40: zero-padded copies to 48
    (2, 200, 1500, 100, 20, "f16"),       # D = 100 -> 112, batched
    (1, 700, 3000, 128, 9, "f16"),        # the 10-entry lists, two query tiles per wave, fp16
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_knn_parity(km, oracle, shape):
    B, M, N, D, k, dt = shape
    Q, R = _data(B, M, N, D, dt, seed=M + N + k)
    say(f"[knn] B={B} M={M} N={N} D={D} k={k} {dt}")
    Qd, Rd = Q.cuda(), R.cuda()
    gi, gd = km.kmeans_knn(Qd, Rd, k)
    gi2, gd2 = km.kmeans_knn(Qd, Rd, k)
    torch.cuda.synchronize()
    assert torch.equal(gi, gi2) and torch.equal(gd, gd2), "two identical calls differ"
    differ = check_knn(oracle, Q, R, dt, k, gi.cpu().numpy(), gd.cpu().numpy().astype(np.float64))
    say(f"  positions differing from the oracle's order (near-ties): {differ} of {B * M * k}")


def test_knn_k1_matches_assignment(km):
    """k = 1 is the assignment with the database rows as centroids (same rows:
    the rows are already in the storage type, so rounding them changes nothing)."""
    Q, R = _data(1, 2000, 500, 128, "bf16", seed=3)
    Qd, Rd = Q.cuda(), R.cuda()
    gi, gd = km.kmeans_knn(Qd, Rd, 1)
    idx, md = km.kmeans_assign(Qd, Rd.float())
    torch.cuda.synchronize()
    same = (gi[..., 0] == idx).float().mean().item()
    assert same > 0.999, same
    scale = (Qd.float() ** 2).sum(-1)
    assert ((gd[..., 0] - md).abs() <= 1e-3 * scale).all()


def test_knn_self_query(km):
    """Queries equal to database rows find themselves first, at distance ~0."""
    _, R = _data(1, 10, 1500, 64, "bf16", seed=4)
    Rd = R.cuda()
    gi, gd = km.kmeans_knn(Rd, Rd, 4)
    torch.cuda.synchronize()
    scale = (Rd.float() ** 2).sum(-1)
    # duplicates in the database are possible after rounding: then the lowest index wins
    first = gi[0, :, 0].cpu()
    own = torch.arange(1500)
    dup_ok = (Rd[0][first.cuda()] == Rd[0]).all(-1).cpu()
    assert bool(((first == own) | dup_ok).all())
    assert (gd[..., 0] <= 1e-3 * scale).all()


def test_knn_full_size_sampled(km, oracle):
    """The bench's search (262,144 queries against 1,048,576 rows, D = 128, k = 10,
    bf16, the same seeded blob recipe) in its launch configuration; 24 sampled
    queries checked against the oracle's 26 nearest rows with the tolerance of
    the small cases, distances of returned rows recomputed exactly."""
    M, N, D, k = 262144, 1 << 20, 128, 10
    g = torch.Generator().manual_seed(7)
    centres = torch.rand((N // 64, D), generator=g) * 2 - 1
    R = (centres[torch.randint(0, N // 64, (N,), generator=g)] + 0.1 * torch.randn((N, D), generator=g))
    Q = (centres[torch.randint(0, N // 64, (M,), generator=g)] + 0.1 * torch.randn((M, D), generator=g))
    R, Q = R.to(torch.bfloat16), Q.to(torch.bfloat16)
    say(f"[knn full] M={M} N={N} D={D} k={k}")
    gi, gd = km.kmeans_knn(Q.cuda(), R.cuda(), k)
    torch.cuda.synchronize()
    rows = np.random.default_rng(11).choice(M, 24, replace=False)
    Qs = Q[None, rows]
    oi, od, _ = oracle.knn(raw(Qs), raw(R[None]), "bf16", k + 16)
    q64 = oracle.widen(raw(Qs), "bf16")[0]
    r64 = oracle.widen(raw(R[None]), "bf16")[0]
    gi_s, gd_s = gi[0].cpu().numpy()[rows], gd[0].cpu().numpy()[rows].astype(np.float64)
    for m in range(len(rows)):
        S = gi_s[m]
        assert len(set(S.tolist())) == k and S.min() >= 0 and S.max() < N
        d_ret = ((r64[S] - q64[m]) ** 2).sum(-1)            # exact distances of the returned rows
        tq = TOL * (q64[m] ** 2).sum()
        dist = od[0, m]
        assert np.all(d_ret <= dist[k - 1] + tq), (m, "a returned row is not among the nearest")
        must = oi[0, m, :k][dist[:k] < dist[k] - tq]
        assert set(must.tolist()) <= set(S.tolist()), (m, "recall")
        assert np.all(d_ret[:-1] <= d_ret[1:] + tq), (m, "order")
        err = np.abs(gd_s[m] - d_ret)
        assert np.all(err <= TOL * ((q64[m] ** 2).sum() + (r64[S] ** 2).sum(-1))), (m, err.max())
