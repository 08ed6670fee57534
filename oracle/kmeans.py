"""Prefill key clustering in fp64 (test infrastructure only).

Sec. 4.2: per (layer, KV head), K-means on the key vectors, started from
SeqLen / (average cluster size) randomly sampled tokens, alternating an
assignment to the nearest centroid and an update of each centroid to the mean
of its members, until convergence or at most 10 iterations.

Readings: the distance is the squared Euclidean one; the sampled starting
tokens are passed in (init_idx); convergence means that an assignment step
changed no assignment; an empty cluster keeps its previous centroid; ties in
distance go to the smaller cluster id.  Centroids are stored in bf16 like the
key cache, so with round_storage=True each update rounds the mean to bf16 and
the next assignment measures distances to the stored values.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List

import numpy as np

from .numerics import round_bf16


def sq_distances(K: np.ndarray, C: np.ndarray) -> np.ndarray:
    """||k_i - c_j||^2 for all pairs (n, C), expanded as
    ||k_i||^2 - 2 k_i . c_j + ||c_j||^2 with a matrix product for the middle
    term."""
    kk = np.einsum("ij,ij->i", K, K)
    cc = np.einsum("ij,ij->i", C, C)
    return kk[:, None] - 2.0 * (K @ C.T) + cc[None, :]


def assign_step(K: np.ndarray, C: np.ndarray) -> np.ndarray:
    """Nearest centroid of every key; np.argmin returns the first (smallest
    id) of equal minima."""
    return np.argmin(sq_distances(K, C), axis=1).astype(np.int64)


def update_step(K: np.ndarray, assign: np.ndarray, C_prev: np.ndarray,
                round_storage: bool = True) -> np.ndarray:
    """Each centroid becomes the mean of the keys assigned to it; a cluster
    with no member keeps its previous centroid."""
    nc, d = C_prev.shape
    sums = np.zeros((nc, d))
    np.add.at(sums, assign, K)
    cnt = np.bincount(assign, minlength=nc)
    C = C_prev.copy()
    nz = cnt > 0
    C[nz] = sums[nz] / cnt[nz][:, None]
    if round_storage:
        C[nz] = round_bf16(C[nz])
    return C


@dataclass
class KMeansResult:
    assign: np.ndarray          # (n,) cluster id per token
    centroids: np.ndarray       # (C, d)
    iters: int                  # assignment steps taken
    inertia: List[float] = field(default_factory=list)  # sum of squared distances after each assignment


def kmeans(K: np.ndarray, init_idx, max_iters: int = 10, round_storage: bool = True,
           prev_centroids=None) -> KMeansResult:
    """Lloyd iterations from the keys of the sampled tokens (Sec. 4.2).

    prev_centroids (re-clustering, Sec. 1): the stored centroids of a previous
    clustering; centroid j starts from prev_centroids[j] for j below both
    counts and from the key of token init_idx[j] otherwise."""
    init_idx = np.asarray(init_idx, dtype=np.int64)
    m = 0 if prev_centroids is None else min(len(init_idx), len(prev_centroids))
    C = np.empty((len(init_idx), K.shape[1]))
    if m:
        C[:m] = np.asarray(prev_centroids, dtype=np.float64)[:m]
    C[m:] = K[init_idx[m:]]
    prev = None
    inertia = []
    it = 0
    for it in range(1, max_iters + 1):
        D = sq_distances(K, C)
        a = np.argmin(D, axis=1).astype(np.int64)
        inertia.append(float(D[np.arange(len(a)), a].sum()))
        if prev is not None and np.array_equal(a, prev):
            return KMeansResult(assign=a, centroids=C, iters=it, inertia=inertia)
        C = update_step(K, a, C, round_storage)
        prev = a
    return KMeansResult(assign=prev, centroids=C, iters=it, inertia=inertia)


def cluster_layout(assign: np.ndarray, n_clusters: int):
    """Cluster-contiguous order of the tokens: cluster j owns rows
    offsets[j]..offsets[j+1]-1 and perm[row] is the token stored there, in
    ascending token order within a cluster (a stable counting sort)."""
    assign = np.asarray(assign, dtype=np.int64)
    cnt = np.bincount(assign, minlength=n_clusters)
    offsets = np.zeros(n_clusters + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(cnt)
    fill = offsets[:-1].copy()
    perm = np.empty(len(assign), dtype=np.int64)
    for t, c in enumerate(assign):
        perm[fill[c]] = t
        fill[c] += 1
    return offsets, perm


def inertia(K: np.ndarray, assign: np.ndarray, C: np.ndarray) -> float:
    """Sum over tokens of the squared distance to the assigned centroid."""
    diff = K - C[np.asarray(assign, dtype=np.int64)]
    return float(np.einsum("ij,ij->", diff, diff))
