"""Exact-rational k-means for tiny inputs (pure Python, ``fractions.Fraction``).

TEST INFRASTRUCTURE ONLY.  Every quantity here is exact, so it pins the fp64
oracle without sharing its rounding: for dyadic inputs the fp64 oracle must
agree bit for bit, and for general inputs up to fp64 rounding.

Also enumerates every labelling of a tiny point set to find the global minimum
of the k-means objective, which Lloyd's local search can only approach from
above, and sorts exact distances for KNN search.
"""
from __future__ import annotations

import itertools
from fractions import Fraction
from typing import List, Sequence, Tuple

Vec = List[Fraction]


def to_frac(rows) -> List[Vec]:
    """Exact rational copy of a 2-D array of floats (floats are dyadic rationals)."""
    return [[Fraction(float(v)) for v in row] for row in rows]


def sqdist(x: Sequence[Fraction], c: Sequence[Fraction]) -> Fraction:
    return sum(((a - b) ** 2 for a, b in zip(x, c)), Fraction(0))


def assign(X: List[Vec], C: List[Vec]) -> Tuple[List[int], List[Fraction], List[Fraction]]:
    """Nearest centroid of each point; ties to the lowest index; gap to the runner-up."""
    idx, md, gap = [], [], []
    for x in X:
        d = [sqdist(x, c) for c in C]
        best = min(d)
        k = d.index(best)                      # first (lowest) index attaining the minimum
        rest = d[:k] + d[k + 1:]
        idx.append(k)
        md.append(best)
        gap.append(min(rest) - best if rest else None)
    return idx, md, gap


def update(X: List[Vec], idx: List[int], C_prev: List[Vec]) -> Tuple[List[Vec], List[int]]:
    """Mean of each cluster's points; an empty cluster keeps its previous centroid."""
    K, D = len(C_prev), len(C_prev[0])
    S = [[Fraction(0)] * D for _ in range(K)]
    n = [0] * K
    for x, k in zip(X, idx):
        n[k] += 1
        S[k] = [s + v for s, v in zip(S[k], x)]
    return [[s / n[k] for s in S[k]] if n[k] else list(C_prev[k]) for k in range(K)], n


def lloyd(X: List[Vec], C0: List[Vec], iters: int):
    C = [list(c) for c in C0]
    objective = []
    idx = md = n = None
    for _ in range(iters):
        idx, md, _ = assign(X, C)
        objective.append(sum(md, Fraction(0)))
        C, n = update(X, idx, C)
    return C, idx, md, n, objective


def partition_cost(X: List[Vec], labels: Sequence[int], K: int) -> Fraction:
    """k-means objective of a labelling with each centroid at its cluster's mean."""
    D = len(X[0])
    total = Fraction(0)
    for k in range(K):
        members = [x for x, l in zip(X, labels) if l == k]
        if not members:
            continue
        mean = [sum((m[j] for m in members), Fraction(0)) / len(members) for j in range(D)]
        total += sum((sqdist(m, mean) for m in members), Fraction(0))
    return total


def global_minimum(X: List[Vec], K: int) -> Fraction:
    """Minimum objective over all K^N labellings (tiny N only)."""
    return min(partition_cost(X, lab, K) for lab in itertools.product(range(K), repeat=len(X)))


def knn(Q: List[Vec], R: List[Vec], k: int):
    """k nearest rows of R for each query: (indices, distances, next distance),
    ordered by (distance, index); the next distance is None when k == len(R)."""
    out_i, out_d, out_n = [], [], []
    for q in Q:
        d = [sqdist(q, r) for r in R]
        order = sorted(range(len(R)), key=lambda j: (d[j], j))
        out_i.append(order[:k])
        out_d.append([d[j] for j in order[:k]])
        out_n.append(d[order[k]] if k < len(R) else None)
    return out_i, out_d, out_n
