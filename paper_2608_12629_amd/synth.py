"""Seeded synthetic k-means workloads (inputs only).

This module makes the point sets X and the initial centroids C0 that both the
HIP path and the fp64 oracle consume.  It holds none of the k-means arithmetic
(no distances, no arg-min, no means): it draws Gaussian-mixture points, casts
them once to the storage dtype with round-to-nearest-even, and picks initial
centroids.  The paper motivates Flash-KMeans with token embeddings from a video
diffusion model (Section 5, "Flash-KMeans clean-start workload"); those are not
available, so these mixtures stand in for them with the same shapes.

Recipe (one line per workload, base seeds fixed below):

* ``blobs``: ``n_blobs`` centres uniform in ``[-box, box]^D``; labels drawn iid
  from the blob weights (uniform, or Zipf ``p_r ~ r^-s`` for blob ``r-1``);
  ``x = centre[label] + sigma * N(0, I)`` in fp32, then one RNE cast.
* ``subspace``: ``x = P z + noise * n`` with ``P`` an orthonormal ``D x rank``
  basis (QR of a Gaussian matrix), ``z ~ N(0, I_rank)``, ``n ~ N(0, I_D)``;
  ``x /= ||x||_2`` in fp32, then one RNE cast.
* initial centroids: the first K points (``init="first"``) or a seeded sample
  of K distinct points in draw order (``init="sample"``), widened exactly to
  fp32.
* ``make_multiscale`` (a test input, not a benchmark workload): blob points
  as above, each multiplied by its own scale drawn log-uniformly from
  ``[1, ratio]``, so that points whose squared norms differ by up to
  ``ratio^2`` sit side by side in every block of consecutive rows.

Every random stream comes from ``numpy.random.SeedSequence(base).spawn``; the
noise is drawn in fixed row chunks, each from its own spawned stream, so the
result does not depend on how many threads generate it.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os
from typing import Optional

import numpy as np
import torch

__all__ = ["WORKLOADS", "Workload", "make_workload", "make_multiscale", "raw_bits", "DTYPES"]

DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}

# The five workloads: shapes, dtypes and mixtures of the benchmark configurations.
WORKLOADS = {
    1: dict(name="blobs_n65536_d64_k256_f32", B=1, N=65_536, D=64, K=256, dtype="f32",
            iters=5, kind="blobs", n_blobs=256, box=1.0, sigma=0.1, weights="equal",
            init="first", seed=0x2608_0001),
    2: dict(name="blobs_n1048576_d128_k1024_bf16", B=1, N=1_048_576, D=128, K=1024,
            dtype="bf16", iters=10, kind="blobs", n_blobs=1024, box=1.0, sigma=0.2,
            weights="equal", init="sample", seed=0x2608_0002),
    3: dict(name="zipf_blobs_n8388608_d128_k4096_bf16", B=1, N=8_388_608, D=128, K=4096,
            dtype="bf16", iters=10, kind="blobs", n_blobs=4096, box=1.0, sigma=0.15,
            weights="zipf1.1", init="sample", seed=0x2608_0003),
    4: dict(name="batched_b64_n16384_d64_k64_f16", B=64, N=16_384, D=64, K=64, dtype="f16",
            iters=20, kind="blobs", n_blobs=64, box=2.0, sigma=0.3, weights="equal",
            init="sample", seed=0x2608_0004),
    5: dict(name="subspace_n2097152_d1024_k16384_bf16", B=1, N=2_097_152, D=1024, K=16_384,
            dtype="bf16", iters=5, kind="subspace", rank=32, noise=0.05, init="sample",
            seed=0x2608_0005),
    # the shape the paper times its assignment kernels on (Section 5: B = 32,
    # N = 65,536, K = 1,024, D = 128, bf16), as 32 independent instances
    6: dict(name="paper_b32_n65536_d128_k1024_bf16", B=32, N=65_536, D=128, K=1024,
            dtype="bf16", iters=10, kind="blobs", n_blobs=1024, box=1.0, sigma=0.2,
            weights="equal", init="sample", seed=0x2608_0006),
}

_CHUNK_ROWS = 1 << 16


@dataclasses.dataclass
class Workload:
    name: str
    B: int
    N: int
    D: int
    K: int
    dtype: str            # "f32" | "bf16" | "f16"
    iters: int
    X: torch.Tensor       # [B, N, D] CPU tensor in the storage dtype
    C0: torch.Tensor      # [B, K, D] CPU float32 (exact widening of K rows of X)
    labels: Optional[np.ndarray]   # [B, N] generating blob of each point (blobs only)
    centres: Optional[np.ndarray]  # [B, n_blobs, D] float32 (blobs only)
    spec: dict


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _blob_weights(kind: str, n: int) -> np.ndarray:
    if kind == "equal":
        return np.full(n, 1.0 / n)
    if kind.startswith("zipf"):
        s = float(kind[4:])
        w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
        return w / w.sum()
    raise ValueError(f"unknown weights {kind!r}")


def _fill_rows(out: torch.Tensor, n_rows: int, seeds, make_chunk) -> None:
    """Fill out[0:n_rows] chunk by chunk; chunk c uses its own spawned seed."""
    n_chunks = (n_rows + _CHUNK_ROWS - 1) // _CHUNK_ROWS

    def job(c):
        r0 = c * _CHUNK_ROWS
        r1 = min(n_rows, r0 + _CHUNK_ROWS)
        rng = np.random.default_rng(seeds[c])
        chunk = make_chunk(rng, r0, r1)                     # fp32 numpy [r1-r0, D]
        out[r0:r1].copy_(torch.from_numpy(chunk))           # one RNE cast to out.dtype

    if n_chunks == 1:
        job(0)
        return
    with _cf.ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(job, range(n_chunks)))


def _make_instance(spec: dict, N: int, D: int, K: int, seed_seq: np.random.SeedSequence,
                   out: torch.Tensor):
    s_centre, s_label, s_noise, s_init = seed_seq.spawn(4)
    n_chunks = (N + _CHUNK_ROWS - 1) // _CHUNK_ROWS
    noise_seeds = s_noise.spawn(n_chunks)
    labels = centres = None
    if spec["kind"] == "blobs":
        n_blobs = spec.get("n_blobs_override") or spec["n_blobs"]
        box, sigma = spec["box"], spec["sigma"]
        centres = np.random.default_rng(s_centre).uniform(-box, box, size=(n_blobs, D)).astype(np.float32)
        p = _blob_weights(spec["weights"], n_blobs)
        labels = np.random.default_rng(s_label).choice(n_blobs, size=N, p=p).astype(np.int32)
        sig = np.float32(sigma)

        def make_chunk(rng, r0, r1):
            x = rng.standard_normal((r1 - r0, D), dtype=np.float32)
            x *= sig
            x += centres[labels[r0:r1]]
            return x
    elif spec["kind"] == "subspace":
        rank, nz = spec["rank"], np.float32(spec["noise"])
        g = np.random.default_rng(s_centre).standard_normal((D, rank))
        basis = np.linalg.qr(g)[0].astype(np.float32)       # D x rank, orthonormal columns

        def make_chunk(rng, r0, r1):
            z = rng.standard_normal((r1 - r0, rank), dtype=np.float32)
            x = z @ basis.T
            x += nz * rng.standard_normal((r1 - r0, D), dtype=np.float32)
            x /= np.linalg.norm(x, axis=1, keepdims=True)
            return x
    else:
        raise ValueError(spec["kind"])

    _fill_rows(out, N, noise_seeds, make_chunk)
    if spec["init"] == "first":
        rows = np.arange(K)
    else:
        rows = np.random.default_rng(s_init).choice(N, size=K, replace=False)
    return labels, centres, rows


def make_workload(index: int, *, N: Optional[int] = None, K: Optional[int] = None,
                  B: Optional[int] = None, D: Optional[int] = None,
                  n_blobs: Optional[int] = None, seed: Optional[int] = None) -> Workload:
    """Build workload ``index`` of WORKLOADS (1..6), optionally with smaller sizes.

    Overrides keep the recipe and change only the sizes; ``K`` also sets the
    number of blobs unless ``n_blobs`` is given.  The returned tensors live on
    the CPU.
    """
    spec = dict(WORKLOADS[index])
    B = B or spec["B"]
    N = N or spec["N"]
    D = D or spec["D"]
    if K is not None:
        spec["n_blobs_override"] = n_blobs or K
    elif n_blobs is not None:
        spec["n_blobs_override"] = n_blobs
    K = K or spec["K"]
    if K > N:
        raise ValueError("K must not exceed N")
    base = spec["seed"] if seed is None else seed
    dt = DTYPES[spec["dtype"]]
    X = torch.empty((B, N, D), dtype=dt)
    C0 = torch.empty((B, K, D), dtype=torch.float32)
    per_inst = np.random.SeedSequence([base, N, D, K]).spawn(B)
    labels = np.empty((B, N), np.int32) if spec["kind"] == "blobs" else None
    centres = []
    for b in range(B):
        lab, cen, rows = _make_instance(spec, N, D, K, per_inst[b], X[b])
        C0[b] = X[b][torch.from_numpy(np.asarray(rows, dtype=np.int64))].float()
        if labels is not None:
            labels[b] = lab
            centres.append(cen)
    name = spec["name"] if (N, K, B, D) == (WORKLOADS[index]["N"], WORKLOADS[index]["K"],
                                            WORKLOADS[index]["B"], WORKLOADS[index]["D"]) \
        else f"{spec['name']}@B{B}N{N}D{D}K{K}"
    return Workload(name=name, B=B, N=N, D=D, K=K, dtype=spec["dtype"], iters=spec["iters"],
                    X=X, C0=C0, labels=labels,
                    centres=np.stack(centres) if centres else None, spec=spec)


def make_multiscale(B: int, N: int, D: int, K: int, dtype: str, *, ratio: float = 100.0,
                    n_blobs: int = 64, sigma: float = 0.15, seed: int = 0x2608_00F0) -> Workload:
    """Blob points with per-point scales spread over ``[1, ratio]`` (log-uniform).

    x = s * (centre[label] + sigma * N(0, I)) in fp32, s = ratio ** u with
    u ~ U[0, 1), then one RNE cast; centroids are a seeded sample of K points.
    Consecutive rows mix all scales, so any block of a few hundred points holds
    squared norms over about ``ratio^2``.
    """
    if K > N:
        raise ValueError("K must not exceed N")
    dt = DTYPES[dtype]
    X = torch.empty((B, N, D), dtype=dt)
    C0 = torch.empty((B, K, D), dtype=torch.float32)
    labels = np.empty((B, N), np.int32)
    for b, ss in enumerate(np.random.SeedSequence([seed, B, N, D, K]).spawn(B)):
        s_centre, s_label, s_scale, s_noise, s_init = ss.spawn(5)
        centres = np.random.default_rng(s_centre).uniform(-1, 1, size=(n_blobs, D)).astype(np.float32)
        lab = np.random.default_rng(s_label).integers(0, n_blobs, size=N).astype(np.int32)
        scale = (ratio ** np.random.default_rng(s_scale).random(N)).astype(np.float32)
        x = np.random.default_rng(s_noise).standard_normal((N, D), dtype=np.float32)
        x *= np.float32(sigma)
        x += centres[lab]
        x *= scale[:, None]
        X[b].copy_(torch.from_numpy(x))
        rows = np.random.default_rng(s_init).choice(N, size=K, replace=False)
        C0[b] = X[b][torch.from_numpy(rows.astype(np.int64))].float()
        labels[b] = lab
    return Workload(name=f"multiscale_r{ratio:g}_b{B}_n{N}_d{D}_k{K}_{dtype}", B=B, N=N, D=D, K=K,
                    dtype=dtype, iters=2, X=X, C0=C0, labels=labels, centres=None,
                    spec=dict(kind="multiscale", ratio=ratio, n_blobs=n_blobs, sigma=sigma,
                              seed=seed))


def raw_bits(t: torch.Tensor) -> np.ndarray:
    """The stored bits of a CPU tensor as a numpy array (uint16 for 16-bit types)."""
    t = t.contiguous()
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.numpy()
    raise TypeError(t.dtype)
