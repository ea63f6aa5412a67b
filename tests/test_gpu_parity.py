"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Teacher-forced steps (the oracle consumes the GPU's own C_t for the assignment
and the GPU's own idx_t for the update) on the same seeded inputs, at sizes the
oracle finishes in seconds; the full-size workloads are checked on sampled rows
for the assignment and in full for the update.  Also: edge cases, determinism,
and that kmeans_lloyd equals the composition of its two steps.
"""
from __future__ import annotations

import os
import sys

import numpy as np
import pytest
import torch

from parity import check_assign, check_update, raw, tol_for
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


def teacher_forced(km, o, X, C0, dtype, iters, rows=None):
    """Run `iters` assign/update steps on the GPU and check each against the oracle
    (given the fp32 centroids the GPU was given)."""
    Xd = X.cuda()
    C = C0.cuda().clone()
    Xr = raw(X)
    Xs = np.ascontiguousarray(Xr[:, rows]) if rows is not None else Xr
    reports = []
    ws = km.Workspace(X.shape[0], X.shape[1], X.shape[2], C.shape[1], X.dtype)
    for t in range(iters):
        idx, md = km.kmeans_assign(Xd, C, ws=ws)
        C1, n = km.kmeans_update(Xd, idx, C, ws=ws)
        torch.cuda.synchronize()
        C64 = C.cpu().double().numpy()
        ig, mg = idx.cpu().numpy(), md.cpu().numpy()
        if rows is not None:
            ig_s, mg_s = ig[:, rows], mg[:, rows]
        else:
            ig_s, mg_s = ig, mg
        rep = check_assign(o, Xs, dtype, C64, ig_s, mg_s)
        err = check_update(o, Xr, dtype, ig, C64, C1.cpu().numpy(), n.cpu().numpy())
        say(f"  t={t} mismatches={rep.mismatches} (exempt pts {rep.exempt_points}) "
            f"md_err={rep.worst_md_err:.2e} J={rep.J_gpu:.6e}/{rep.J_oracle:.6e} C_err={err:.2e}")
        reports.append(rep)
        C = C1
    return reports


# ----------------------------------------------------------------- workloads
SMALL = {
    "blobs_f32_full": dict(wl=1),
    "blobs_bf16_small": dict(wl=2, N=65536, K=256),
    "zipf_bf16_small": dict(wl=3, N=65536, K=512),
    "batched_f16_small": dict(wl=4, B=8, N=4096),
    "subspace_bf16_small": dict(wl=5, N=20000, K=700),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_teacher_forced_small(km, oracle, name):
    kw = dict(SMALL[name])
    w = make_workload(kw.pop("wl"), **kw)
    say(f"[{name}] {w.name} B={w.B} N={w.N} D={w.D} K={w.K} {w.dtype}")
    teacher_forced(km, oracle, w.X, w.C0, w.dtype, min(w.iters, 4))


def test_batched_f16_full_teacher_forced(km, oracle):
    w = make_workload(4)
    say(f"[batched full] {w.name}")
    teacher_forced(km, oracle, w.X, w.C0, w.dtype, 3)


@pytest.mark.parametrize("wl", [2, 3, 5], ids=["blobs_1m_bf16", "zipf_8m_bf16", "subspace_2m_d1024_bf16"])
def test_full_size_sampled(km, oracle, wl):
    """Full-size workload: assignment checked on 4096 sampled rows, update in full."""
    w = make_workload(wl)
    rows = np.sort(np.random.default_rng(wl).choice(w.N, 4096, replace=False))
    say(f"[full] {w.name}")
    teacher_forced(km, oracle, w.X, w.C0, w.dtype, 2, rows=rows)


def test_unpacked_sort_full(km, oracle):
    """N = 2^23 + 4,096 points with K = 65,536: the second radix digit (8 bits)
    and a point id (24 bits) do not fit one int, so the update sorts separate
    key and value arrays and finds the cluster bounds by binary search (every
    smaller problem takes the packed passes).  Assignment on sampled rows,
    update in full."""
    w = make_workload(3, N=(1 << 23) + 4096, K=65536, D=16)
    rows = np.sort(np.random.default_rng(7).choice(w.N, 2048, replace=False))
    say(f"[unpacked sort] {w.name}")
    teacher_forced(km, oracle, w.X, w.C0, w.dtype, 1, rows=rows)


# --------------------------------------------------------------- edge cases
def _blobs(B, N, D, K, dtype, seed, spread=1.0):
    g = torch.Generator().manual_seed(seed)
    centres = torch.rand((B, K, D), generator=g) * 2 - 1
    lab = torch.randint(0, K, (B, N), generator=g)
    X = torch.gather(centres, 1, lab[..., None].expand(B, N, D)) + spread * 0.1 * torch.randn(
        (B, N, D), generator=g)
    X = X.to(dtype)
    C0 = X[:, :K].float().clone()
    return X, C0


DT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
SHAPES = [
    # (B, N, D, K, dtype)
    (1, 1, 64, 1, "bf16"),            # single point, single centroid
    (1, 1000, 64, 1, "f16"),          # K = 1
    (1, 777, 128, 100, "bf16"),       # ragged N and K
    (1, 5000, 32, 7, "f32"),          # fp32 D = 32
    (1, 4097, 64, 300, "f32"),        # ragged sort chunk
    (1, 2049, 128, 64, "f32"),        # fp32 D = 128
    (1, 3000, 256, 50, "bf16"),       # D = 256
    (1, 3000, 256, 33, "f16"),
    (1, 3000, 32, 65, "bf16"),        # D = 32
    (3, 2500, 64, 40, "f16"),         # batched, ragged
    (1, 300, 64, 300, "bf16"),        # K = N
    (2, 6000, 128, 128, "bf16"),      # per-chunk update at K * D = 16384, ragged chunk
    (1, 10000, 32, 512, "f32"),       # per-chunk update, fp32, 9-bit cluster ids
    (1, 3000, 16, 10, "bf16"),        # D = 16: 16-bit rows of <= 16 run as fp32
    (1, 4000, 32, 250, "bf16"),       # one-hot sums with 8 cluster tiles
    (1, 3000, 80, 60, "f16"),         # one-hot sums, odd chunk count (a padded dimension tile)
    (1, 3000, 48, 37, "f16"),         # D = 48: padded LDS rows, masked row lanes
    (2, 1500, 96, 50, "bf16"),        # D = 96
    (1, 2000, 160, 70, "bf16"),       # D = 160: one column tile per wave, padded rows
    (1, 2000, 208, 33, "f16"),        # D = 208
    (1, 3000, 48, 20, "f32"),         # fp32 D = 48: padded LDS rows
    (1, 3000, 112, 40, "f32"),        # fp32 D = 112
    (1, 3000, 80, 300, "f32"),        # fp32 D = 80, sorted update with masked row lanes
    (1, 3000, 144, 30, "f32"),        # fp32 D = 144: two column tiles per wave
    (1, 2000, 256, 50, "f32"),        # fp32 D = 256
    (1, 1500, 384, 300, "bf16"),      # tiled kernel, D = 384
    (1, 1200, 288, 90, "f16"),        # tiled, D = 288: 9 stages + 3 padding stages per block
    (2, 900, 416, 257, "bf16"),       # tiled, D = 416: 13 + 3
    (4, 20000, 128, 1024, "bf16"),    # batched two-pass sort (packed words), ragged chunks
    (1, 700, 992, 40, "bf16"),        # tiled, D = 992: 31 + 1
    (1, 1000, 512, 130, "bf16"),      # tiled kernel: ragged N and K
    (2, 700, 1024, 33, "f16"),        # tiled kernel, batched
    (1, 300, 2048, 260, "bf16"),      # tiled kernel, widest rows
    # widths the kernels do not take run on zero-padded copies of the rows
    (1, 1000, 1, 5, "bf16"),          # D = 1: 16-bit rows below 16 run as fp32 rows of 16
    (1, 3000, 1, 12, "f16"),          # D = 1, fp16
    (1, 3000, 3, 8, "bf16"),          # D = 3, bf16
    (2, 2000, 7, 30, "f16"),          # D = 7, batched
    (1, 2500, 15, 300, "bf16"),       # D = 15, sorted update
    (1, 3000, 3, 8, "f32"),           # D = 3 -> 16
    (1, 3000, 40, 30, "bf16"),        # D = 40 -> 48
    (2, 1500, 100, 70, "f16"),        # D = 100 -> 112, batched
    (1, 2000, 17, 300, "f32"),        # fp32 D = 17 -> 32, sorted update
    (1, 900, 300, 100, "bf16"),       # D = 300 -> 320, tiled kernel
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_edge_shapes(km, oracle, shape):
    B, N, D, K, dt = shape
    X, C0 = _blobs(B, N, D, K, DT[dt], seed=N * 7 + K)
    say(f"[edge] B={B} N={N} D={D} K={K} {dt}")
    teacher_forced(km, oracle, X, C0, dt, 2)


# Points whose squared norms differ by up to 10^4 in every workgroup: the
# shift that keeps the packed scores negative must not widen the tie window or
# the min_dist rounding past the smallest points' own tolerance.  Shapes cover
# the streaming kernel (D = 64, 128; per-workgroup fallback to per-point
# shifts), rows of 16 (always per point), the small-K single-pass kernel
# (per point), the wide-row tiled kernel (per point) and fp32 rows.
MULTISCALE = [
    # (B, N, D, K, dtype)
    (1, 20000, 64, 256, "bf16"),
    (1, 20000, 128, 512, "bf16"),
    (1, 20000, 128, 300, "f16"),
    (1, 20000, 16, 200, "bf16"),
    (2, 8192, 64, 64, "f16"),
    (1, 6000, 1024, 300, "bf16"),
    (1, 20000, 64, 256, "f32"),
]


@pytest.mark.parametrize("shape", MULTISCALE, ids=lambda s: "x".join(map(str, s)))
def test_multiscale_norms(km, oracle, shape):
    from paper_2608_12629_amd.synth import make_multiscale
    B, N, D, K, dt = shape
    w = make_multiscale(B, N, D, K, dt)
    xn = (w.X.double() ** 2).sum(-1)
    blk = xn[0, : (N // 256) * 256].reshape(-1, 256)
    say(f"[multiscale] {w.name}: |x|^2 spread per 256 rows "
        f"{float((blk.max(1).values / blk.min(1).values).min()):.0f}x or more")
    assert float((blk.max(1).values / blk.min(1).values).min()) > 1e3
    teacher_forced(km, oracle, w.X, w.C0, dt, 2)


def test_duplicates_and_empty_clusters(km, oracle):
    """Duplicate centroids (lower index wins), duplicate points, an empty far cluster."""
    X, C0 = _blobs(1, 3000, 64, 16, torch.bfloat16, seed=5)
    X[0, 100:200] = X[0, 50]                 # 101 identical points
    C0[0, 9] = C0[0, 3]                      # duplicate centroid: 9 must never win
    C0[0, 12] = 1e3                          # far away: empty cluster
    Xd, C = X.cuda(), C0.cuda()
    idx, md = km.kmeans_assign(Xd, C)
    C1, n = km.kmeans_update(Xd, idx, C)
    torch.cuda.synchronize()
    ig = idx.cpu().numpy()
    assert not (ig == 9).any() and not (ig == 12).any()
    assert n[0, 9].item() == 0 and n[0, 12].item() == 0
    assert torch.equal(C1[0, 12].cpu(), C0[0, 12]) and torch.equal(C1[0, 9].cpu(), C0[0, 9])
    assert len(set(ig[0, 100:200].tolist() + [ig[0, 50]])) == 1
    teacher_forced(km, oracle, X, C0, "bf16", 2)


def test_all_points_one_cluster(km, oracle):
    """Maximal skew: every point in one cluster (one sorted run spans every chunk)."""
    g = torch.Generator().manual_seed(3)
    X = (0.05 * torch.randn((1, 20000, 128), generator=g)).to(torch.bfloat16)
    C0 = torch.zeros((1, 4, 128))
    C0[0, 1:] = 50.0
    Xd = X.cuda()
    idx, md = km.kmeans_assign(Xd, C0.cuda())
    C1, n = km.kmeans_update(Xd, idx, C0.cuda())
    torch.cuda.synchronize()
    assert n[0].tolist() == [20000, 0, 0, 0]
    mean = X[0].double().mean(0)
    rel = (C1[0, 0].cpu().double() - mean).norm() / mean.norm()
    assert rel < 1e-3
    teacher_forced(km, oracle, X, C0, "bf16", 1)


def test_points_as_centroids(km):
    """C = X: every point is its own nearest centroid at distance 0."""
    g = torch.Generator().manual_seed(11)
    X = torch.randn((1, 256, 64), generator=g).to(torch.bfloat16)
    idx, md = km.kmeans_assign(X.cuda(), X.float().cuda())
    torch.cuda.synchronize()
    assert idx.cpu()[0].tolist() == list(range(256))
    assert md.abs().max().item() <= 1e-3 * float((X.float() ** 2).sum(-1).max())


# ------------------------------------------------------- composition, determinism
@pytest.mark.parametrize("wl,kw", [(1, {}), (3, dict(N=65536, K=512)), (4, dict(B=8, N=4096))],
                         ids=["blobs_f32", "zipf_bf16_small", "batched_f16_small"])
def test_lloyd_equals_steps_and_is_deterministic(km, oracle, wl, kw):
    w = make_workload(wl, **kw)
    Xd = w.X.cuda()
    iters = 3
    C_a, idx_a, md_a, n_a, obj_a = km.kmeans_lloyd(Xd, w.C0.cuda().clone(), iters)
    C_b, idx_b, md_b, n_b, obj_b = km.kmeans_lloyd(Xd, w.C0.cuda().clone(), iters)
    torch.cuda.synchronize()
    for a, b in ((C_a, C_b), (idx_a, idx_b), (md_a, md_b), (n_a, n_b), (obj_a, obj_b)):
        assert torch.equal(a, b), "two identical runs differ"
    C = w.C0.cuda().clone()
    objs = []
    for t in range(iters):
        idx, md = km.kmeans_assign(Xd, C)
        objs.append(md.double().sum(-1))
        C, n = km.kmeans_update(Xd, idx, C)
    torch.cuda.synchronize()
    assert torch.equal(C, C_a) and torch.equal(idx, idx_a) and torch.equal(md, md_a)
    assert torch.equal(n, n_a)
    J = torch.stack(objs, -1)
    assert torch.allclose(J, obj_a, rtol=1e-12, atol=0)
    # the objective never increases (up to the contract's relative tolerance)
    o = obj_a.cpu().numpy()
    assert np.all(np.diff(o, axis=-1) <= tol_for(w.dtype) * o[:, :-1])


@pytest.mark.parametrize("D,Dk,dt", [(40, 48, torch.bfloat16), (3, 16, torch.float32),
                                      (300, 320, torch.float16)])
def test_padded_rows_equal_explicit_padding(km, D, Dk, dt):
    """A width the kernels do not take gives, bit for bit, the results of the
    same rows padded with zeros by the caller (idx, min_dist, counts, the
    objective, and C_T's first D columns; its padding columns stay zero)."""
    X, C0 = _blobs(2, 3000, D, 37, dt, seed=D)
    Xp = torch.nn.functional.pad(X, (0, Dk - D))
    Cp = torch.nn.functional.pad(C0, (0, Dk - D))
    say(f"[padded] D={D} -> {Dk} {dt}")
    a = km.kmeans_lloyd(X.cuda(), C0.cuda(), 3)
    b = km.kmeans_lloyd(Xp.cuda(), Cp.cuda(), 3)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0][..., :D]) and not b[0][..., D:].any()
    for u, v in zip(a[1:], b[1:]):
        assert torch.equal(u, v)
    idx, md = km.kmeans_assign(X.cuda(), C0.cuda())
    idx_p, md_p = km.kmeans_assign(Xp.cuda(), Cp.cuda())
    C1, n1 = km.kmeans_update(X.cuda(), idx, C0.cuda())
    C1p, n1p = km.kmeans_update(Xp.cuda(), idx, Cp.cuda())
    torch.cuda.synchronize()
    assert torch.equal(idx, idx_p) and torch.equal(md, md_p)
    assert torch.equal(C1, C1p[..., :D]) and torch.equal(n1, n1p)


@pytest.mark.parametrize("shape", [(1, 5000, 32, 250, "bf16"), (2, 3000, 128, 64, "f16"),
                                   (1, 3000, 80, 60, "bf16"), (3, 2000, 48, 33, "f16"),
                                   (2, 4500, 32, 100, "bf16"), (1, 2100, 64, 64, "f16")],
                         ids=lambda s: "x".join(map(str, s)))
def test_fused_lloyd_equals_steps(km, shape):
    """Small-K shapes (one-hot sums; the last three assign and sum in one
    kernel): bit-identical to kmeans_assign followed by kmeans_update, and
    repeatable.  N = 2,100 leaves a 52-point last chunk."""
    B, N, D, K, dt = shape
    X, C0 = _blobs(B, N, D, K, DT[dt], seed=N + K)
    Xd = X.cuda()
    say(f"[fused] B={B} N={N} D={D} K={K} {dt}")
    a = km.kmeans_lloyd(Xd, C0.cuda(), 3)
    b = km.kmeans_lloyd(Xd, C0.cuda(), 3)
    C = C0.cuda()
    for t in range(3):
        idx, md = km.kmeans_assign(Xd, C)
        C, n = km.kmeans_update(Xd, idx, C)
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v), "two identical runs differ"
    assert torch.equal(a[0], C) and torch.equal(a[1], idx) and torch.equal(a[2], md)
    assert torch.equal(a[3], n)


def test_mass_conservation_full_zipf_8m(km):
    """sum_k n_k c'_k = sum_i x_i at the full 8M-point workload (no oracle needed)."""
    w = make_workload(3)
    Xd = w.X.cuda()
    idx, md = km.kmeans_assign(Xd, w.C0.cuda())
    C1, n = km.kmeans_update(Xd, idx, w.C0.cuda())
    torch.cuda.synchronize()
    assert int(n.sum()) == w.N
    lhs = (n.double()[0, :, None] * C1.double()[0]).sum(0)
    rhs = Xd.double()[0].sum(0)
    scale = Xd.double()[0].abs().sum(0)
    assert ((lhs - rhs).abs() <= 1e-5 * scale).all()
    assert (md >= 0).all() and int(idx.min()) >= 0 and int(idx.max()) < w.K
