"""GPU: kmeans_lloyd and kmeans_knn captured in a HIP graph (torch.cuda.CUDAGraph)
and replayed.

The library enqueues only kernel launches on the caller's stream (no memsets,
no host synchronisation, no allocation when the workspace and every output are
given), so a whole Lloyd run can be captured once and replayed, which removes
the host launch cost that dominates the small workloads.  Each case replays the
graph several times with the program's own eager work (other calls on the same
workspace) and synchronisations in between, and checks every replay bit for bit
against an eager run from the same starting centroids.
"""
from __future__ import annotations

import sys

import pytest
import torch

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


def _blobs(B, N, D, K, dtype, seed):
    g = torch.Generator().manual_seed(seed)
    centres = torch.rand((B, K, D), generator=g) * 2 - 1
    lab = torch.randint(0, K, (B, N), generator=g)
    X = torch.gather(centres, 1, lab[..., None].expand(B, N, D)) + 0.1 * torch.randn(
        (B, N, D), generator=g)
    X = X.to(dtype)
    return X, X[:, :K].float().clone()


CASES = [
    # (name, maker): one case per assignment / update path
    ("fp32 65,536 x 64, K = 256 (resident fp32, small-K sums)",
     lambda: (lambda w: (w.X, w.C0))(make_workload(1))),
    ("f16 64 x 16,384 x 64, K = 64 (fused small-K kernel)",
     lambda: (lambda w: (w.X, w.C0))(make_workload(4))),
    ("bf16 65,536 x 128, K = 1,024 (pipe, sorted update)",
     lambda: (lambda w: (w.X, w.C0))(make_workload(2, N=65536))),
    ("bf16 5,000 x 100, K = 300 (padded rows)",
     lambda: _blobs(1, 5000, 100, 300, torch.bfloat16, 11)),
    ("bf16 2 x 4,096 x 512, K = 256 (tiled)",
     lambda: _blobs(2, 4096, 512, 256, torch.bfloat16, 12)),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0].split(" (")[0] for c in CASES])
def test_lloyd_graph_replays_equal_eager(km, case):
    name, make = case
    X, C0 = make()
    B, N, D = X.shape
    K = C0.shape[1]
    iters = 3
    say(f"[graph] {name}: B={B} N={N} D={D} K={K}")
    Xd, C0d = X.cuda(), C0.cuda()
    ws = km.Workspace(B, N, D, K, X.dtype)

    def outputs():
        return (torch.empty((B, N), dtype=torch.int32, device="cuda"),
                torch.empty((B, N), dtype=torch.float32, device="cuda"),
                torch.empty((B, K), dtype=torch.int32, device="cuda"),
                torch.empty((B, iters), dtype=torch.float64, device="cuda"))

    # eager reference
    C_e = C0d.clone()
    idx_e, md_e, cnt_e, obj_e = outputs()
    km.kmeans_lloyd(Xd, C_e, iters, idx=idx_e, min_dist=md_e, counts=cnt_e, objective=obj_e, ws=ws)
    torch.cuda.synchronize()

    # capture (after a warm-up on a side stream, as torch recommends)
    C_g = C0d.clone()
    idx_g, md_g, cnt_g, obj_g = outputs()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        km.kmeans_lloyd(Xd, C_g, iters, idx=idx_g, min_dist=md_g, counts=cnt_g, objective=obj_g,
                        ws=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    C_g.copy_(C0d)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        km.kmeans_lloyd(Xd, C_g, iters, idx=idx_g, min_dist=md_g, counts=cnt_g, objective=obj_g,
                        ws=ws)
    torch.cuda.synchronize()

    for r in range(3):
        # the program's own eager work between replays: other calls on the
        # same workspace and outputs, then fresh starting centroids
        km.kmeans_assign(Xd, C0d * 0.5, idx=idx_g, min_dist=md_g, ws=ws)
        km.kmeans_update(Xd, idx_g, C0d, C_out=C_g, counts=cnt_g, ws=ws)
        obj_g.fill_(-1.0)
        torch.cuda.synchronize()
        C_g.copy_(C0d)
        graph.replay()
        torch.cuda.synchronize()
        say(f"[graph]   replay {r}")
        assert torch.equal(C_g, C_e), f"replay {r}: centroids differ from the eager run"
        assert torch.equal(idx_g, idx_e), f"replay {r}: assignments differ"
        assert torch.equal(md_g, md_e), f"replay {r}: min_dist differs"
        assert torch.equal(cnt_g, cnt_e), f"replay {r}: counts differ"
        assert torch.equal(obj_g, obj_e), f"replay {r}: objective differs"


@pytest.mark.parametrize("k", [10, 32])
def test_knn_graph_replays_equal_eager(km, k):
    """kmeans_knn captured in a graph (workspace and outputs preallocated):
    every replay, with other eager searches on the same workspace between
    them, equals the eager result bit for bit."""
    g = torch.Generator().manual_seed(100 + k)
    B, M, N, D = 2, 3000, 20000, 128
    Q = torch.randn((B, M, D), generator=g).to(torch.bfloat16).cuda()
    R = torch.randn((B, N, D), generator=g).to(torch.bfloat16).cuda()
    say(f"[graph knn] B={B} M={M} N={N} D={D} k={k}")
    need = km.knn_workspace_bytes(B, M, N, D, k, torch.bfloat16)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    i_e = torch.empty((B, M, k), dtype=torch.int32, device="cuda")
    d_e = torch.empty((B, M, k), dtype=torch.float32, device="cuda")
    km.kmeans_knn(Q, R, k, nbr_idx=i_e, nbr_dist=d_e, ws=ws)
    torch.cuda.synchronize()
    i_g, d_g = torch.empty_like(i_e), torch.empty_like(d_e)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        km.kmeans_knn(Q, R, k, nbr_idx=i_g, nbr_dist=d_g, ws=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        km.kmeans_knn(Q, R, k, nbr_idx=i_g, nbr_dist=d_g, ws=ws)
    torch.cuda.synchronize()
    for r in range(3):
        km.kmeans_knn(R[:, :M].contiguous(), Q, k, ws=ws)  # other work on the same workspace
        i_g.fill_(-1)
        d_g.fill_(-1.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        say(f"[graph knn]   replay {r}")
        assert torch.equal(i_g, i_e), f"replay {r}: neighbours differ from the eager run"
        assert torch.equal(d_g, d_e), f"replay {r}: distances differ"
