"""Seeded synthetic inputs for the Tactic decode path.

This module builds inputs only: Gaussian-mixture keys, random values and
queries, the K-means initial token indices, and a cluster-contiguous layout
derived from the mixture labels that the generator itself drew.  It holds
none of the method's arithmetic (no scoring, sorting by score, fitting,
cutoff, union, attention or K-means step), so both the CPU oracle and the
HIP path may consume what it produces.

Recipe (per sequence b, layer l, KV head g; n tokens, d = 128):

* M mixture centres c_j ~ N(0, I_d).  Token i draws a label z_i uniformly from
  the M centres, and its key is c_{z_i} + sigma * eps_i with sigma = 0.3.
* A fraction rho of tokens are outliers: the key is multiplied by lambda,
  which keeps its direction and scales its norm (lambda = 3, or a
  heavy-tailed lambda = min(16, 3 U^(-1/2)) for the 1M-token workload).
* Values are N(0, 1).
* Query head h of group g picks k_h distinct centres S_h of group g and is
  q_h = beta_h * (sum_{j in S_h} c_j + sigma * eps).  k_h is fixed (3) for the
  smallest workload and uniform in {1..8} otherwise; beta_h = 2, or
  2 * LogNormal(0, 1) per (layer, head) for the 32-layer workload.  The
  "mean of centres" reading (q_mean) divides the centre sum by k_h.
* The concentration sweep (sweep_workloads): one 131072-token sequence, 32 /
  8 heads, fixed beta in {0.25, 0.5, 1, 2} under both readings, all points on
  the same keys, values and centres (one workload id), so only the query's
  concentration changes from point to point.
* Everything is cast to bf16 (round to nearest even) before use.

Sub-seeds are derived from (workload id, b, layer, head, tag) with NumPy's
SeedSequence, so every piece can be regenerated independently.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np
import torch

_BASE_SEED = 2502_12216


def sub_seed(*keys: int) -> int:
    """A 63-bit seed derived from integer keys (stable across runs)."""
    ss = np.random.SeedSequence([_BASE_SEED, *[int(k) for k in keys]])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & np.uint64(0x7FFF_FFFF_FFFF_FFFF))


@dataclass(frozen=True)
class Workload:
    """Shape and generation parameters of one synthetic workload."""

    name: str
    wid: int                          # workload id, part of every sub-seed
    seq_lens: tuple                   # tokens per sequence
    n_q_heads: int
    n_kv_heads: int
    head_dim: int = 128
    layers: int = 1
    cluster_div: int = 16             # clusters per sequence = n // cluster_div ...
    fixed_clusters: Optional[int] = None  # ... unless fixed
    noise: float = 0.3
    outlier_frac: float = 0.01
    heavy_tail: bool = False          # lambda = min(16, 3 U^-1/2) instead of 3
    q_k_range: tuple = (1, 8)         # centres mixed into one query head
    beta: float = 2.0
    beta_lognormal: bool = False      # beta = 2 * LogNormal(0, 1) per (layer, head)
    q_mean: bool = False              # query = beta * (mean of its centres + noise) instead of the sum
    target_fracs: tuple = (0.9,)
    kmeans_iters: int = 10

    @property
    def batch(self) -> int:
        return len(self.seq_lens)

    def n_clusters(self, n: int) -> int:
        if self.fixed_clusters is not None:
            return min(self.fixed_clusters, n)
        return max(1, n // self.cluster_div)

    @property
    def cluster_counts(self) -> tuple:
        return tuple(self.n_clusters(n) for n in self.seq_lens)

    def with_seq_lens(self, seq_lens: Sequence[int], name: Optional[str] = None) -> "Workload":
        d = dict(self.__dict__)
        d["seq_lens"] = tuple(int(x) for x in seq_lens)
        if name:
            d["name"] = name
        return Workload(**d)


def _ragged_lens(wid: int, count: int, lo: int, hi: int) -> tuple:
    rng = np.random.default_rng(sub_seed(wid, 99))
    return tuple(int(x) for x in rng.integers(lo, hi + 1, size=count))


# The five workloads: the smallest one (4K) is the oracle-sized case; the
# 32-layer batch-4 128K decode step is the timed one.
WORKLOADS = {
    "ctx4k_gqa4": Workload(
        name="ctx4k_gqa4", wid=1, seq_lens=(4096,), n_q_heads=8, n_kv_heads=2,
        fixed_clusters=256, q_k_range=(3, 3)),
    "ctx32k_llama8b": Workload(
        name="ctx32k_llama8b", wid=2, seq_lens=(32768,), n_q_heads=32, n_kv_heads=8,
        target_fracs=(0.8, 0.9, 0.95)),
    "ragged16_16k_128k": Workload(
        name="ragged16_16k_128k", wid=3, seq_lens=_ragged_lens(3, 16, 16384, 131072),
        n_q_heads=32, n_kv_heads=8),
    "ctx1m": Workload(
        name="ctx1m", wid=4, seq_lens=(1048576,), n_q_heads=32, n_kv_heads=8,
        cluster_div=32, outlier_frac=0.005, heavy_tail=True),
    "ctx128k_b4_32layer": Workload(
        name="ctx128k_b4_32layer", wid=5, seq_lens=(131072,) * 4, n_q_heads=32,
        n_kv_heads=8, layers=32, beta_lognormal=True),
}


SWEEP_BETAS = (0.25, 0.5, 1.0, 2.0)


def sweep_workloads(batch: int = 1, betas=SWEEP_BETAS, readings=(False, True)) -> list:
    """The concentration sweep: selected fraction, and so the speedup, as a
    function of how concentrated the queries are (not one of the workloads
    above: every point shares workload id 6, so sequence b has the same keys
    at every point and batch size)."""
    out = []
    for mean in readings:
        for beta in betas:
            name = f"sweep_b{beta:g}_{'mean' if mean else 'sum'}" + (f"_x{batch}" if batch > 1 else "")
            out.append(Workload(name=name, wid=6, seq_lens=(131072,) * batch, n_q_heads=32, n_kv_heads=8,
                                beta=beta, q_mean=mean))
    return out


def indptr(lengths: Sequence[int]) -> np.ndarray:
    out = np.zeros(len(lengths) + 1, dtype=np.int64)
    out[1:] = np.cumsum(np.asarray(lengths, dtype=np.int64))
    return out


@dataclass
class LayerInputs:
    """One layer's synthetic inputs (tensors live on `device`)."""

    wl: Workload
    layer: int
    q: torch.Tensor            # bf16 [B][Hq][d]
    K: torch.Tensor            # bf16 [Hkv][total][d], original token order
    V: torch.Tensor            # bf16 [Hkv][total][d]
    labels: torch.Tensor       # int64 [Hkv][total], mixture component of each token
    centers: torch.Tensor      # fp32 [Hkv][total_components][d]
    kv_indptr: np.ndarray      # int64 [B+1]
    comp_indptr: np.ndarray    # int64 [B+1] (components per sequence = clusters)
    q_centres: list = field(default_factory=list)  # per (b, h): centre ids mixed in
    betas: list = field(default_factory=list)      # per (b, h)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def make_layer(wl: Workload, layer: int = 0, device="cpu", seq_subset=None) -> LayerInputs:
    """Generate one layer of `wl` on `device` (seeded, deterministic per device).

    `seq_subset` (list of sequence indices) generates only those sequences,
    each with the seeds it has in the full batch.
    """
    d = wl.head_dim
    G = wl.n_q_heads // wl.n_kv_heads
    seqs = list(range(wl.batch)) if seq_subset is None else list(seq_subset)
    lens = [wl.seq_lens[b] for b in seqs]
    comps = [wl.n_clusters(n) for n in lens]
    kv_ip = indptr(lens)
    cp_ip = indptr(comps)
    total, total_c = int(kv_ip[-1]), int(cp_ip[-1])
    K = torch.empty(wl.n_kv_heads, total, d, dtype=torch.bfloat16, device=device)
    V = torch.empty_like(K)
    labels = torch.empty(wl.n_kv_heads, total, dtype=torch.int64, device=device)
    centers = torch.empty(wl.n_kv_heads, total_c, d, dtype=torch.float32, device=device)
    q = torch.empty(len(seqs), wl.n_q_heads, d, dtype=torch.bfloat16, device=device)
    q_centres, betas = [], []
    for bi, b in enumerate(seqs):
        n, M = lens[bi], comps[bi]
        s0, s1 = int(kv_ip[bi]), int(kv_ip[bi + 1])
        c0, c1 = int(cp_ip[bi]), int(cp_ip[bi + 1])
        for g in range(wl.n_kv_heads):
            gen = _gen(sub_seed(wl.wid, b, layer, g), device)
            cen = torch.randn(M, d, generator=gen, device=device)
            lab = torch.randint(0, max(M, 1), (n,), generator=gen, device=device)  # M = 0 only when n = 0
            k = cen[lab]
            k += wl.noise * torch.randn(n, d, generator=gen, device=device)
            u = torch.rand(n, generator=gen, device=device)
            mask = u < wl.outlier_frac
            if wl.heavy_tail:
                lam = torch.clamp(3.0 * torch.rand(n, generator=gen, device=device).clamp_min(1e-12) ** -0.5,
                                  max=16.0)
            else:
                lam = torch.full((n,), 3.0, device=device)
            scale = torch.where(mask, lam, torch.ones_like(lam))
            k *= scale[:, None]
            K[g, s0:s1] = k.to(torch.bfloat16)
            V[g, s0:s1] = torch.randn(n, d, generator=gen, device=device).to(torch.bfloat16)
            labels[g, s0:s1] = lab
            centers[g, c0:c1] = cen
            for j in range(G):
                h = g * G + j
                rng = np.random.default_rng(sub_seed(wl.wid, b, layer, 1000 + h))
                lo, hi = wl.q_k_range
                kh = int(rng.integers(lo, hi + 1))
                S = rng.choice(M, size=min(kh, M), replace=False)
                beta = wl.beta
                if wl.beta_lognormal:
                    brng = np.random.default_rng(sub_seed(wl.wid, layer, 2000 + h))
                    beta = wl.beta * float(brng.lognormal(0.0, 1.0))
                qg = _gen(sub_seed(wl.wid, b, layer, 1000 + h), device)
                qv = cen[torch.as_tensor(S, device=device)].sum(0)
                if wl.q_mean:
                    qv = qv / float(len(S))
                qv = qv + wl.noise * torch.randn(d, generator=qg, device=device)
                q[bi, h] = (beta * qv).to(torch.bfloat16)
                q_centres.append([int(x) for x in S])
                betas.append(beta)
    return LayerInputs(wl=wl, layer=layer, q=q, K=K, V=V, labels=labels, centers=centers,
                       kv_indptr=kv_ip, comp_indptr=cp_ip, q_centres=q_centres, betas=betas)


@dataclass
class LabelLayout:
    """A cluster-contiguous layout whose clusters are the generator's own
    mixture components and whose centroids are the generator's centres
    (rounded to bf16).  It is a valid cluster description for the decode
    path that does not depend on any K-means implementation."""

    K_sorted: torch.Tensor     # bf16 [Hkv][total][d]
    V_sorted: torch.Tensor     # bf16 [Hkv][total][d]
    centroids: torch.Tensor    # bf16 [Hkv][total_clusters][d]
    offsets: torch.Tensor      # int32 [Hkv][total_clusters + B] per-(b,g) CSR offsets, sequence-relative
    perm: torch.Tensor         # int32 [Hkv][total]: original (sequence-relative) token id of each sorted row
    kv_indptr: np.ndarray
    cl_indptr: np.ndarray


def label_layout(inp: LayerInputs, tail: Optional[Sequence[int]] = None) -> LabelLayout:
    """Cluster-sorted layout by the generator's own mixture labels.

    `tail[b]` (default 0) leaves the last tail[b] tokens of sequence b
    unclustered: they follow the clustered rows in their original order
    (recent tokens since the clustering) and the offsets end before them."""
    Hkv = inp.K.shape[0]
    B = len(inp.kv_indptr) - 1
    dev = inp.K.device
    total_c = int(inp.comp_indptr[-1])
    Ks = torch.empty_like(inp.K)
    Vs = torch.empty_like(inp.V)
    perm = torch.empty(Hkv, inp.K.shape[1], dtype=torch.int32, device=dev)
    offsets = torch.empty(Hkv, total_c + B, dtype=torch.int32, device=dev)
    for b in range(B):
        s0, s1 = int(inp.kv_indptr[b]), int(inp.kv_indptr[b + 1])
        c0, c1 = int(inp.comp_indptr[b]), int(inp.comp_indptr[b + 1])
        M = c1 - c0
        t = int(tail[b]) if tail is not None else 0
        t = min(max(t, 0), s1 - s0)
        for g in range(Hkv):
            lab = inp.labels[g, s0:s1 - t]
            p = torch.cat([torch.argsort(lab, stable=True),
                           torch.arange(s1 - s0 - t, s1 - s0, device=dev, dtype=torch.int64)])
            cnt = torch.bincount(lab, minlength=M)
            off = torch.zeros(M + 1, dtype=torch.int64, device=dev)
            off[1:] = torch.cumsum(cnt, 0)
            Ks[g, s0:s1] = inp.K[g, s0:s1][p]
            Vs[g, s0:s1] = inp.V[g, s0:s1][p]
            perm[g, s0:s1] = p.to(torch.int32)
            offsets[g, c0 + b:c1 + b + 1] = off.to(torch.int32)
    cent = inp.centers.to(torch.bfloat16)
    return LabelLayout(K_sorted=Ks, V_sorted=Vs, centroids=cent, offsets=offsets, perm=perm,
                       kv_indptr=inp.kv_indptr.copy(), cl_indptr=inp.comp_indptr.copy())


def kmeans_init_idx(wl: Workload, b: int, layer: int, g: int, n: int, C: int) -> np.ndarray:
    """C distinct token ids (sequence-relative) sampled uniformly without
    replacement: the K-means starting centroids are these tokens' keys."""
    rng = np.random.default_rng(sub_seed(wl.wid, b, layer, g, 7))
    return rng.choice(n, size=C, replace=False).astype(np.int32)


def kmeans_init_all(wl: Workload, layer: int, seq_subset=None) -> np.ndarray:
    """Initial indices for every (b, g) of one layer, laid out
    [Hkv][total_clusters] to match the centroid array."""
    seqs = list(range(wl.batch)) if seq_subset is None else list(seq_subset)
    lens = [wl.seq_lens[b] for b in seqs]
    comps = [wl.n_clusters(n) for n in lens]
    out = np.empty((wl.n_kv_heads, int(sum(comps))), dtype=np.int32)
    c = 0
    for bi, b in enumerate(seqs):
        for g in range(wl.n_kv_heads):
            out[g, c:c + comps[bi]] = kmeans_init_idx(wl, b, layer, g, lens[bi], comps[bi])
        c += comps[bi]
    return out


def small_workload(base: Workload, seq_lens: Sequence[int], name: Optional[str] = None) -> Workload:
    """A copy of `base` with other sequence lengths (for oracle-sized tests)."""
    return base.with_seq_lens(seq_lens, name or f"{base.name}_n{'-'.join(map(str, seq_lens))}")
