"""Decode-loop KV cache with recent tokens and periodic re-clustering.

Tactic clusters the keys once (K-means at prefill), then attends in full to
the tokens generated since and re-clusters every fixed number of decoding
steps (Sec. 1 gives 2048).  This module keeps one layer's cache in the layout
the library reads: sequence b owns a span of `capacities[b]` rows of the
per-KV-head K and V arrays, holds its first seq_len[b] rows, the first c_b of
them cluster-sorted (the clusters' offsets end at c_b) and the rest the
recent tokens in arrival order.  Every computation runs in libtactic.so;
this class only moves tokens into their rows and keeps the bookkeeping.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np
import torch

from .tactic import (ClusterBuilder, ClusterSet, DenseDecoder, RaggedBatch, SparseDecoder, decode_params,
                     sparse_decode_workspace_bytes)


class RecentTailCache:
    """One layer's cluster-sorted KV cache for a batch decoded in lockstep.

    prefill() stores each sequence's prompt and clusters it; append() adds one
    token per sequence and re-clusters the whole batch once a sequence has
    `recluster_every` recent tokens; decode() runs Tactic's sparse decode with
    every recent token attended (max_tail = recluster_every)."""

    def __init__(self, n_q_heads: int, n_kv_heads: int, capacities: Sequence[int], recluster_every: int = 2048,
                 cluster_div: int = 16, kmeans_iters: int = 10, target_frac: float = 0.9, seed: int = 0,
                 warm_start: bool = True, device="cuda"):
        self.capacities = [int(c) for c in capacities]
        self.Hq, self.Hkv = int(n_q_heads), int(n_kv_heads)
        self.recluster_every = int(recluster_every)
        self.cluster_div = int(cluster_div)
        self.kmeans_iters = int(kmeans_iters)
        self.target_frac = float(target_frac)
        self.warm_start = bool(warm_start)
        self.device = device
        self.rng = np.random.default_rng(seed)
        B = len(self.capacities)
        self.lens = [0] * B
        self.clustered = [0] * B
        self.batch = RaggedBatch(self.lens, self.Hq, self.Hkv, device=device, capacities=self.capacities)
        self.starts = torch.as_tensor(self.batch.kv_indptr_host[:-1], device=device)
        self.K = torch.zeros(self.Hkv, self.batch.total, 128, dtype=torch.bfloat16, device=device)
        self.V = torch.zeros_like(self.K)
        self.K_alt = torch.empty_like(self.K)  # the next clustering writes here, then the two swap
        self.V_alt = torch.empty_like(self.V)
        self.clusters: Optional[ClusterSet] = None
        self.decoder: Optional[SparseDecoder] = None
        self.builder: Optional[ClusterBuilder] = None
        self.dense = DenseDecoder(self.batch, device=device)
        self.reclusterings = 0

    # ------------------------------------------------------------------ tokens
    def _set_lens(self, lens: List[int]) -> None:
        if any(n > c for n, c in zip(lens, self.capacities)):
            raise ValueError("a sequence outgrew its capacity")
        self.lens = list(lens)
        self.batch.seq_lens = list(lens)
        self.batch.seq_len.copy_(torch.as_tensor(np.asarray(lens, dtype=np.int64)))

    def prefill(self, K: Sequence[torch.Tensor], V: Sequence[torch.Tensor]) -> None:
        """K[b], V[b]: bf16 [Hkv][n_b][128], the prompt of sequence b in token order."""
        lens = []
        for b, (k, v) in enumerate(zip(K, V)):
            n = int(k.shape[1])
            s = int(self.batch.kv_indptr_host[b])
            if n > self.capacities[b]:
                raise ValueError(f"prompt of sequence {b} exceeds its capacity")
            self.K[:, s:s + n] = k
            self.V[:, s:s + n] = v
            lens.append(n)
        self._set_lens(lens)
        self.recluster()

    def append(self, k: torch.Tensor, v: torch.Tensor) -> bool:
        """k, v: bf16 [B][Hkv][128], the new token of every sequence.  Returns
        True when the call re-clustered the batch.  Only device work is
        enqueued (no host-device copy): the rows come from the device lengths,
        which are then advanced in place."""
        lens = [n + 1 for n in self.lens]
        if any(n > c for n, c in zip(lens, self.capacities)):
            raise ValueError("a sequence outgrew its capacity")
        rows = self.starts + self.batch.seq_len  # the next free row of every sequence
        self.K[:, rows] = k.transpose(0, 1).to(self.K.dtype)
        self.V[:, rows] = v.transpose(0, 1).to(self.V.dtype)
        self.batch.seq_len += 1
        self.lens = lens
        self.batch.seq_lens = list(lens)
        if max(n - c for n, c in zip(self.lens, self.clustered)) >= self.recluster_every:
            self.recluster()
            return True
        return False

    # ------------------------------------------------------------------ clustering
    def n_clusters(self, n: int) -> int:
        return max(1, n // self.cluster_div)

    def recluster(self) -> None:
        """K-means over every held token of every sequence (prompt and recent),
        then the cache is the cluster-sorted copy and no token is recent.

        With warm_start and a previous clustering, centroid j of every
        (sequence, KV head) starts from the previous centroid j (j below both
        cluster counts) and the added clusters from distinct recent tokens, so
        the iterations only have to absorb the recent tokens; otherwise every
        centroid starts from a distinct sampled token."""
        ncl = [self.n_clusters(n) for n in self.lens]
        prev = self.clusters if (self.warm_start and self.clusters is not None) else None
        init = np.zeros((self.Hkv, int(sum(ncl))), dtype=np.int32)
        c0 = 0
        for b, (n, C) in enumerate(zip(self.lens, ncl)):
            m = min(C, prev.n_clusters[b]) if prev is not None else 0
            lo = self.clustered[b] if C - m <= n - self.clustered[b] else 0  # seed from the recent tokens
            for g in range(self.Hkv):
                if n and C > m:
                    init[g, c0 + m:c0 + C] = lo + self.rng.choice(n - lo, size=C - m, replace=n - lo < C - m)
            c0 += C
        if self.builder is None:  # one workspace, sized for the counts of full sequences
            self.builder = ClusterBuilder(self.batch, ncl, max_iters=self.kmeans_iters, device=self.device,
                                          workspace_clusters=[self.n_clusters(c) for c in self.capacities])
        res = self.builder(self.K, self.V, torch.as_tensor(init, device=self.device), prev=prev, n_clusters=ncl,
                           K_out=self.K_alt, V_out=self.V_alt)
        self.K, self.K_alt = self.K_alt, self.K
        self.V, self.V_alt = self.V_alt, self.V
        self.clusters = res.clusters
        self.clustered = list(self.lens)
        params = decode_params(self.target_frac, max_tail=self.recluster_every)
        if self.decoder is None:  # one workspace, sized for the counts of full sequences
            cap = [self.n_clusters(c) for c in self.capacities]
            ws = torch.empty(sparse_decode_workspace_bytes(self.batch, cap, params), dtype=torch.uint8,
                             device=self.device)
        else:
            ws = self.decoder.workspace
        self.decoder = SparseDecoder(self.batch, ncl, params, device=self.device, workspace=ws)
        self.reclusterings += 1

    # ------------------------------------------------------------------ attention
    def decode(self, q: torch.Tensor, target_frac: Optional[float] = None):
        """Sparse decode of q (bf16 [B][Hq][128]) over the cache: (out fp32
        [B][Hq][128], tokens attended per query head, K/V rows per KV head)."""
        return self.decoder(q, self.K, self.V, self.clusters, target_frac=target_frac)

    def decode_dense(self, q: torch.Tensor) -> torch.Tensor:
        return self.dense(q, self.K, self.V)

    @property
    def recent(self) -> List[int]:
        return [n - c for n, c in zip(self.lens, self.clustered)]
