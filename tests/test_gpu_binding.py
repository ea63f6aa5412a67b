"""The binding's argument checks: the C ABI receives pointers only, so a
caller's output tensor of the wrong size, a host tensor or a host workspace
must be refused before any kernel is launched (each case below raises in
Python; no GPU work is enqueued for it)."""
from __future__ import annotations

import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def km():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    from paper_2608_12629_amd import kmeans
    return kmeans


def _data(B=2, N=512, D=64, K=16):
    g = torch.Generator().manual_seed(3)
    X = torch.randn((B, N, D), generator=g).to(torch.bfloat16).cuda()
    C = X[:, :K].float().contiguous()
    return X, C


def test_outputs_of_the_wrong_size_are_refused(km):
    X, C = _data()
    B, N, K, D = 2, 512, 16, 64
    with pytest.raises(ValueError, match="idx has"):
        km.kmeans_assign(X, C, idx=torch.empty(B * N - 1, dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError, match="min_dist has"):
        km.kmeans_assign(X, C, min_dist=torch.empty((B, N + 1), device="cuda"))
    idx = torch.zeros((B, N), dtype=torch.int32, device="cuda")
    with pytest.raises(ValueError, match="idx has"):
        km.kmeans_update(X, idx[:, :-1].contiguous(), C)
    with pytest.raises(ValueError, match="C_out has"):
        km.kmeans_update(X, idx, C, C_out=torch.empty((B, K, D - 1), device="cuda"))
    with pytest.raises(ValueError, match="counts has"):
        km.kmeans_update(X, idx, C, counts=torch.empty((B, K + 1), dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError, match="counts has"):
        km.kmeans_lloyd(X, C.clone(), 1, counts=torch.empty((B, K - 1), dtype=torch.int32, device="cuda"))
    with pytest.raises(ValueError, match="nbr_idx has"):
        km.kmeans_knn(X, X, 4, nbr_idx=torch.empty((B, N, 3), dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()


def test_one_instance_outputs_may_drop_the_batch_axis(km):
    X, C = _data(B=1)
    idx = torch.empty(512, dtype=torch.int32, device="cuda")
    md = torch.empty(512, device="cuda")
    i2, m2 = km.kmeans_assign(X[0], C[0], idx=idx, min_dist=md)
    ref_i, ref_m = km.kmeans_assign(X, C)
    torch.cuda.synchronize()
    assert i2 is idx and torch.equal(idx, ref_i[0]) and torch.equal(md, ref_m[0])


def test_host_tensors_and_host_workspaces_are_refused(km):
    X, C = _data()
    with pytest.raises(ValueError, match="current GPU"):
        km.kmeans_assign(X.cpu(), C)
    with pytest.raises(ValueError, match="current GPU"):
        km.kmeans_assign(X, C, idx=torch.empty((2, 512), dtype=torch.int32))
    ws = km.Workspace(2, 512, 64, 16, X.dtype, device="cpu")
    with pytest.raises(ValueError, match="workspace must be a tensor on the current GPU"):
        km.kmeans_assign(X, C, ws=ws)
    with pytest.raises(ValueError, match="ws must be a tensor on the current GPU"):
        km.kmeans_knn(X, X, 4, ws=torch.empty(1 << 26, dtype=torch.uint8))
    with pytest.raises(ValueError, match="contiguous"):
        km.kmeans_assign(X.transpose(1, 2).contiguous().transpose(1, 2), C)
    torch.cuda.synchronize()
