"""Thin torch-facing wrappers over the C ABI (include/tactic.h).

Torch supplies device memory and the current stream; every step of the
decode and of the clustering runs in libtactic.so.  There is no fallback: a
missing library or a failing call raises.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np
import torch

from . import _capi as C


def _stream(stream=None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _check_tensor(t: torch.Tensor, name: str, dtype, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must live on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _indptr(lengths: Sequence[int]) -> np.ndarray:
    ip = np.zeros(len(lengths) + 1, dtype=np.int64)
    ip[1:] = np.cumsum(np.asarray(lengths, dtype=np.int64))
    return ip


class RaggedBatch:
    """A ragged decode batch: sequence lengths, head counts, device indptr.

    With `capacities`, sequence b owns a span of capacities[b] rows of the
    per-KV-head arrays and holds its first seq_lens[b] of them (room for new
    tokens); the lengths live in a device array the caller may update in
    place (`seq_len`)."""

    def __init__(self, seq_lens: Sequence[int], n_q_heads: int, n_kv_heads: int, head_dim: int = 128,
                 device="cuda", capacities: Optional[Sequence[int]] = None):
        self.seq_lens = [int(x) for x in seq_lens]
        self.n_q_heads, self.n_kv_heads, self.head_dim = int(n_q_heads), int(n_kv_heads), int(head_dim)
        spans = self.seq_lens if capacities is None else [int(x) for x in capacities]
        if capacities is not None and any(n > c for n, c in zip(self.seq_lens, spans)):
            raise ValueError("a sequence is longer than its capacity")
        self.kv_indptr_host = _indptr(spans)
        self.kv_indptr = torch.as_tensor(self.kv_indptr_host, device=device)
        self.seq_len = (None if capacities is None
                        else torch.as_tensor(np.asarray(self.seq_lens, dtype=np.int64), device=device))
        self.total = int(self.kv_indptr_host[-1])
        self.max_len = max(spans) if spans else 0

    @property
    def batch(self) -> int:
        return len(self.seq_lens)

    def struct(self) -> C.KVShape:
        return C.KVShape(self.batch, self.n_q_heads, self.n_kv_heads, self.head_dim, self.total, self.max_len,
                         self.kv_indptr.data_ptr(), None if self.seq_len is None else self.seq_len.data_ptr())


class ClusterSet:
    """Cluster description of a cluster-sorted cache (see tactic_cluster_meta)."""

    def __init__(self, centroids: torch.Tensor, offsets: torch.Tensor, n_clusters: Sequence[int]):
        self.n_clusters = [int(x) for x in n_clusters]
        self.cl_indptr_host = _indptr(self.n_clusters)
        self.cl_indptr = torch.as_tensor(self.cl_indptr_host, device=centroids.device)
        self.total = int(self.cl_indptr_host[-1])
        self.max = max(self.n_clusters) if self.n_clusters else 0
        _check_tensor(centroids, "centroids", torch.bfloat16)
        _check_tensor(offsets, "offsets", torch.int32)
        if centroids.shape[1:] != (self.total, 128):
            raise ValueError(f"centroids must be [Hkv][{self.total}][128], got {tuple(centroids.shape)}")
        if offsets.shape[1:] != (self.total + len(self.n_clusters),):
            raise ValueError("offsets must be [Hkv][total_clusters + B]")
        self.centroids, self.offsets = centroids, offsets

    def struct(self) -> C.ClusterMeta:
        return C.ClusterMeta(self.total, self.max, self.cl_indptr.data_ptr(), self.centroids.data_ptr(),
                             self.offsets.data_ptr())


def decode_params(target_frac: float = 0.9, **kw) -> C.DecodeParams:
    p = C.DecodeParams()
    C.lib().tactic_decode_params_default(ctypes.byref(p))
    p.target_frac = float(target_frac)
    for k, v in kw.items():
        setattr(p, k, int(v))
    return p


class PagedCache:
    """A paged K/V cache (see tactic_paged_kv): K_pages, V_pages bf16
    [num_pages][Hkv][page_size][128], page_table int32 [B][max_pages], and
    optionally perm int32 [Hkv][total] mapping cluster-sorted rows to tokens."""

    def __init__(self, K_pages: torch.Tensor, V_pages: torch.Tensor, page_table: torch.Tensor,
                 perm: Optional[torch.Tensor] = None):
        _check_tensor(K_pages, "K_pages", torch.bfloat16)
        _check_tensor(V_pages, "V_pages", torch.bfloat16, tuple(K_pages.shape))
        _check_tensor(page_table, "page_table", torch.int32)
        if perm is not None:
            _check_tensor(perm, "perm", torch.int32)
        self.K_pages, self.V_pages, self.page_table, self.perm = K_pages, V_pages, page_table, perm
        self.num_pages, _, self.page_size, _ = K_pages.shape
        self.max_pages = page_table.shape[1]

    @staticmethod
    def from_token_order(K: torch.Tensor, V: torch.Tensor, batch: RaggedBatch, page_size: int,
                         page_order: Optional[torch.Tensor] = None, perm: Optional[torch.Tensor] = None
                         ) -> "PagedCache":
        """Pages holding K, V [Hkv][total][128] (token order per sequence), placed
        at the page ids `page_order` gives (default: in order)."""
        B, Hkv = batch.batch, batch.n_kv_heads
        lens = ([int(batch.kv_indptr_host[b + 1] - batch.kv_indptr_host[b]) for b in range(B)]
                if batch.seq_len is None else list(batch.seq_lens))
        npg = [(n + page_size - 1) // page_size for n in lens]
        max_pages = max(1, max(npg) if npg else 1)
        total_pages = max(1, sum(npg))
        ids = (torch.arange(total_pages, dtype=torch.int64) if page_order is None
               else page_order.cpu().long()).to(K.device)
        table = torch.zeros(B, max_pages, dtype=torch.int32, device=K.device)
        Kp = torch.zeros(total_pages, Hkv, page_size, 128, dtype=torch.bfloat16, device=K.device)
        Vp = torch.zeros_like(Kp)
        nxt = 0
        for b in range(B):
            if npg[b] == 0:
                continue
            s0, n = int(batch.kv_indptr_host[b]), lens[b]
            pid = ids[nxt:nxt + npg[b]]
            nxt += npg[b]
            table[b, :npg[b]] = pid.to(torch.int32)
            for X, Xp in ((K, Kp), (V, Vp)):
                seq = torch.zeros(Hkv, npg[b] * page_size, 128, dtype=X.dtype, device=X.device)
                seq[:, :n] = X[:, s0:s0 + n]
                Xp[pid] = seq.view(Hkv, npg[b], page_size, 128).transpose(0, 1)
        return PagedCache(Kp, Vp, table.to(K.device), perm)

    def struct(self) -> C.PagedKV:
        return C.PagedKV(self.K_pages.data_ptr(), self.V_pages.data_ptr(), self.page_table.data_ptr(),
                         None if self.perm is None else self.perm.data_ptr(), int(self.page_size),
                         int(self.max_pages), int(self.num_pages))


def sparse_decode_workspace_bytes(batch: RaggedBatch, n_clusters: Sequence[int],
                                  params: Optional[C.DecodeParams] = None) -> int:
    """Workspace bytes tactic_sparse_decode needs for this shape (its plan call)."""
    params = params if params is not None else decode_params()
    ncl = [int(x) for x in n_clusters]
    meta = C.ClusterMeta(int(sum(ncl)), max(ncl), None, None, None)
    plan, nbytes = C.DecodePlan(), ctypes.c_size_t()
    shape = batch.struct()
    C.check(C.lib().tactic_sparse_decode_plan(ctypes.byref(shape), ctypes.byref(meta), ctypes.byref(params),
                                              ctypes.byref(plan), ctypes.byref(nbytes)), "tactic_sparse_decode_plan")
    return int(nbytes.value)


def stream_read_gbps(buf: torch.Tensor, reps: int = 10, workgroups=(0, 2048, 4096, 8192, 16384),
                     stream=None) -> dict:
    """Streaming-read rate (GB/s) of the device over `buf` (tactic_probe_stream_read):
    the median of `reps` timed reads for each launch shape, and the best of them.
    A measurement helper, not part of the method."""
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous device tensor")
    nbytes = buf.numel() * buf.element_size() // 16 * 16
    sink = torch.zeros(1, dtype=torch.int32, device=buf.device)
    s = stream if stream is not None else torch.cuda.current_stream()
    rates = {}
    for wg in workgroups:
        times = []
        for _ in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            C.check(C.lib().tactic_probe_stream_read(buf.data_ptr(), nbytes, int(wg), sink.data_ptr(),
                                                     int(s.cuda_stream)), "tactic_probe_stream_read")
            e1.record(s)
            e1.synchronize()
            times.append(e0.elapsed_time(e1))
        rates[int(wg)] = nbytes / (float(np.median(times[1:])) * 1e6)
    return {"best_gbps": max(rates.values()), "gbps_by_workgroups": rates, "bytes": nbytes}


class SparseDecoder:
    """Tactic's decode for one batch shape: holds the launch plan and the
    workspace, so repeated calls (layers, decode steps) allocate nothing."""

    def __init__(self, batch: RaggedBatch, n_clusters: Sequence[int], params: Optional[C.DecodeParams] = None,
                 device="cuda", workspace: Optional[torch.Tensor] = None):
        """workspace: a uint8 device tensor to use if it is large enough (for
        instance a previous decoder's), else a new one is allocated."""
        self.batch = batch
        self.params = params if params is not None else decode_params()
        self.n_clusters = [int(x) for x in n_clusters]
        meta = C.ClusterMeta(int(sum(self.n_clusters)), max(self.n_clusters), None, None, None)
        self.plan = C.DecodePlan()
        nbytes = ctypes.c_size_t()
        self._shape = batch.struct()
        C.check(C.lib().tactic_sparse_decode_plan(ctypes.byref(self._shape), ctypes.byref(meta),
                                                  ctypes.byref(self.params), ctypes.byref(self.plan),
                                                  ctypes.byref(nbytes)), "tactic_sparse_decode_plan")
        need = max(1, nbytes.value)
        if workspace is not None and workspace.dtype == torch.uint8 and workspace.is_cuda and workspace.numel() >= need:
            self.workspace = workspace
        else:
            self.workspace = torch.empty(need, dtype=torch.uint8, device=device)
        B, Hq, Hkv = batch.batch, batch.n_q_heads, batch.n_kv_heads
        self.out = torch.empty(B, Hq, 128, dtype=torch.float32, device=device)
        self.sel_q = torch.empty(B, Hq, dtype=torch.int32, device=device)
        self.sel_kv = torch.empty(B, Hkv, dtype=torch.int32, device=device)

    def __call__(self, q: torch.Tensor, K_sorted: torch.Tensor, V_sorted: torch.Tensor, clusters: ClusterSet,
                 target_frac: Optional[float] = None, stream=None, out=None, sel_q=None, sel_kv=None):
        b = self.batch
        _check_tensor(q, "q", torch.bfloat16, (b.batch, b.n_q_heads, 128))
        _check_tensor(K_sorted, "K_sorted", torch.bfloat16, (b.n_kv_heads, b.total, 128))
        _check_tensor(V_sorted, "V_sorted", torch.bfloat16, (b.n_kv_heads, b.total, 128))
        if clusters.n_clusters != self.n_clusters:
            raise ValueError("cluster counts differ from the ones the decoder was planned for")
        out = self.out if out is None else out
        sel_q = self.sel_q if sel_q is None else sel_q
        sel_kv = self.sel_kv if sel_kv is None else sel_kv
        if target_frac is not None:
            self.params.target_frac = float(target_frac)
        meta = clusters.struct()
        C.check(C.lib().tactic_sparse_decode(
            q.data_ptr(), K_sorted.data_ptr(), V_sorted.data_ptr(), ctypes.byref(self._shape),
            ctypes.byref(meta), ctypes.byref(self.params), ctypes.byref(self.plan), out.data_ptr(),
            sel_q.data_ptr(), sel_kv.data_ptr(), self.workspace.data_ptr(), self.workspace.numel(),
            _stream(stream)), "tactic_sparse_decode")
        return out, sel_q, sel_kv

    def noalloc(self, q: torch.Tensor, K_sorted: torch.Tensor, V_sorted: torch.Tensor, clusters: ClusterSet,
                target_frac: Optional[float] = None, stream=None, out=None, sel_q=None, sel_kv=None):
        """The same decode through tactic_sparse_decode_noalloc: the library's
        static scratch instead of this decoder's workspace (calls on one GPU
        must not overlap)."""
        b = self.batch
        _check_tensor(q, "q", torch.bfloat16, (b.batch, b.n_q_heads, 128))
        _check_tensor(K_sorted, "K_sorted", torch.bfloat16, (b.n_kv_heads, b.total, 128))
        _check_tensor(V_sorted, "V_sorted", torch.bfloat16, (b.n_kv_heads, b.total, 128))
        if clusters.n_clusters != self.n_clusters:
            raise ValueError("cluster counts differ from the ones the decoder was planned for")
        out = self.out if out is None else out
        sel_q = self.sel_q if sel_q is None else sel_q
        sel_kv = self.sel_kv if sel_kv is None else sel_kv
        if target_frac is not None:
            self.params.target_frac = float(target_frac)
        meta = clusters.struct()
        C.check(C.lib().tactic_sparse_decode_noalloc(
            q.data_ptr(), K_sorted.data_ptr(), V_sorted.data_ptr(), ctypes.byref(self._shape),
            ctypes.byref(meta), ctypes.byref(self.params), ctypes.byref(self.plan), out.data_ptr(),
            sel_q.data_ptr(), sel_kv.data_ptr(), _stream(stream)), "tactic_sparse_decode_noalloc")
        return out, sel_q, sel_kv

    def paged(self, q: torch.Tensor, cache: PagedCache, clusters: ClusterSet, target_frac: Optional[float] = None,
              stream=None, out=None, sel_q=None, sel_kv=None):
        """The same decode over a paged cache (tactic_sparse_decode_paged)."""
        b = self.batch
        _check_tensor(q, "q", torch.bfloat16, (b.batch, b.n_q_heads, 128))
        if clusters.n_clusters != self.n_clusters:
            raise ValueError("cluster counts differ from the ones the decoder was planned for")
        if cache.perm is not None:
            _check_tensor(cache.perm, "perm", torch.int32, (b.n_kv_heads, b.total))
        out = self.out if out is None else out
        sel_q = self.sel_q if sel_q is None else sel_q
        sel_kv = self.sel_kv if sel_kv is None else sel_kv
        if target_frac is not None:
            self.params.target_frac = float(target_frac)
        meta = clusters.struct()
        kv = cache.struct()
        C.check(C.lib().tactic_sparse_decode_paged(
            q.data_ptr(), ctypes.byref(kv), ctypes.byref(self._shape), ctypes.byref(meta),
            ctypes.byref(self.params), ctypes.byref(self.plan), out.data_ptr(), sel_q.data_ptr(),
            sel_kv.data_ptr(), self.workspace.data_ptr(), self.workspace.numel(), _stream(stream)),
            "tactic_sparse_decode_paged")
        return out, sel_q, sel_kv

    def view(self) -> dict:
        """Intermediate stages of the last call, as tensors over the workspace."""
        v = C.DecodeView()
        C.check(C.lib().tactic_sparse_decode_view(ctypes.byref(self.plan), self.workspace.data_ptr(),
                                                  ctypes.byref(v)), "tactic_sparse_decode_view")
        base = self.workspace.data_ptr()
        b = self.batch
        BH = b.batch * b.n_q_heads
        Cm = max(self.n_clusters)
        Ct = int(sum(self.n_clusters))
        nv = b.n_kv_heads if self.params.use_union else b.n_q_heads  # selection groups per sequence

        def sl(ptr, count, dtype, shape):
            off = ptr - base
            nbytes = count * torch.empty(0, dtype=dtype).element_size()
            return self.workspace[off:off + nbytes].view(dtype).view(*shape)

        return {
            "scores": sl(v.scores, BH * Cm, torch.float32, (b.batch, b.n_q_heads, Cm)),
            "order": sl(v.order, BH * Cm, torch.int32, (b.batch, b.n_q_heads, Cm)),
            "rank_prefix": sl(v.rank_prefix, BH * (Cm + 1), torch.int32, (b.batch, b.n_q_heads, Cm + 1)),
            "fit": sl(v.fit, BH * C.FIT_FIELDS, torch.float64, (b.batch, b.n_q_heads, C.FIT_FIELDS)),
            "union_len": sl(v.union_len, nv * Ct, torch.int32, (nv, Ct)),
            "sample_rows": sl(v.sample_rows, BH * v.sample_cap, torch.int32, (b.batch, b.n_q_heads, v.sample_cap)),
        }


class DenseDecoder:
    """Dense decode attention (the baseline) over every cached token."""

    def __init__(self, batch: RaggedBatch, device="cuda"):
        self.batch = batch
        self._shape = batch.struct()
        n = C.lib().tactic_dense_decode_workspace_size(ctypes.byref(self._shape))
        if n == 0:
            C.check(1, "tactic_dense_decode_workspace_size")
        self.workspace = torch.empty(n, dtype=torch.uint8, device=device)
        self.out = torch.empty(batch.batch, batch.n_q_heads, 128, dtype=torch.float32, device=device)

    def __call__(self, q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, stream=None, out=None):
        b = self.batch
        _check_tensor(q, "q", torch.bfloat16, (b.batch, b.n_q_heads, 128))
        _check_tensor(K, "K", torch.bfloat16, (b.n_kv_heads, b.total, 128))
        _check_tensor(V, "V", torch.bfloat16, (b.n_kv_heads, b.total, 128))
        out = self.out if out is None else out
        C.check(C.lib().tactic_dense_decode(q.data_ptr(), K.data_ptr(), V.data_ptr(), ctypes.byref(self._shape),
                                            out.data_ptr(), self.workspace.data_ptr(), self.workspace.numel(),
                                            _stream(stream)), "tactic_dense_decode")
        return out

    def paged(self, q: torch.Tensor, cache: PagedCache, stream=None, out=None):
        """Dense decode over a paged cache (tactic_dense_decode_paged)."""
        b = self.batch
        _check_tensor(q, "q", torch.bfloat16, (b.batch, b.n_q_heads, 128))
        out = self.out if out is None else out
        kv = cache.struct()
        C.check(C.lib().tactic_dense_decode_paged(q.data_ptr(), ctypes.byref(kv), ctypes.byref(self._shape),
                                                  out.data_ptr(), self.workspace.data_ptr(),
                                                  self.workspace.numel(), _stream(stream)),
                "tactic_dense_decode_paged")
        return out


@dataclass
class ClusterBuild:
    clusters: ClusterSet
    assign: torch.Tensor       # int32 [Hkv][total]
    perm: torch.Tensor         # int32 [Hkv][total]
    K_sorted: Optional[torch.Tensor]
    V_sorted: Optional[torch.Tensor]


class ClusterBuilder:
    """Prefill K-means (tactic_build_clusters) for one batch shape."""

    def __init__(self, batch: RaggedBatch, n_clusters: Sequence[int], max_iters: int = 10, device="cuda",
                 workspace_clusters: Optional[Sequence[int]] = None):
        """workspace_clusters: the largest cluster counts later calls will use
        (default n_clusters); the workspace is sized for them once."""
        self.batch = batch
        self.device = device
        self.params = C.KMeansParams(int(max_iters))
        self._shape = batch.struct()
        ws = [int(x) for x in (workspace_clusters if workspace_clusters is not None else n_clusters)]
        n = C.lib().tactic_build_clusters_workspace_size(ctypes.byref(self._shape), int(sum(ws)), max(ws))
        if n == 0:
            raise C.TacticError("tactic_build_clusters_workspace_size rejected the shape")
        self.workspace = torch.empty(n, dtype=torch.uint8, device=device)
        self._set_clusters(n_clusters)

    def _set_clusters(self, n_clusters: Sequence[int]) -> None:
        self.n_clusters = [int(x) for x in n_clusters]
        self.total_c = int(sum(self.n_clusters))
        self.max_c = max(self.n_clusters)
        self.cl_indptr_host = _indptr(self.n_clusters)
        self.cl_indptr = torch.as_tensor(self.cl_indptr_host, device=self.device)

    def __call__(self, K: torch.Tensor, V: Optional[torch.Tensor], init_idx: torch.Tensor, sort_kv: bool = True,
                 stream=None, prev: Optional[ClusterSet] = None, n_clusters: Optional[Sequence[int]] = None,
                 K_out: Optional[torch.Tensor] = None, V_out: Optional[torch.Tensor] = None) -> ClusterBuild:
        """prev: a previous clustering of the same sequences to start from (its
        centroid j of every (sequence, KV head) for j below both cluster counts;
        see tactic_kmeans_params).  n_clusters: this call's cluster counts (the
        workspace must have room for them).  K_out, V_out: where the
        cluster-sorted rows go (default: new tensors; never K or V)."""
        if n_clusters is not None and [int(x) for x in n_clusters] != self.n_clusters:
            self._set_clusters(n_clusters)
        b = self.batch
        Hkv = b.n_kv_heads
        _check_tensor(K, "K", torch.bfloat16, (Hkv, b.total, 128))
        if V is not None:
            _check_tensor(V, "V", torch.bfloat16, (Hkv, b.total, 128))
        _check_tensor(init_idx, "init_idx", torch.int32, (Hkv, self.total_c))
        if prev is not None:
            if len(prev.n_clusters) != b.batch:
                raise ValueError("prev clustering has another batch size")
            _check_tensor(prev.centroids, "prev.centroids", torch.bfloat16, (Hkv, prev.total, 128))
            self.params.prev_centroids = prev.centroids.data_ptr()
            self.params.prev_cl_indptr = prev.cl_indptr.data_ptr()
        else:
            self.params.prev_centroids = None
            self.params.prev_cl_indptr = None
        dev = K.device
        cent = torch.empty(Hkv, self.total_c, 128, dtype=torch.bfloat16, device=dev)
        assign = torch.empty(Hkv, b.total, dtype=torch.int32, device=dev)
        offsets = torch.empty(Hkv, self.total_c + b.batch, dtype=torch.int32, device=dev)
        perm = torch.empty(Hkv, b.total, dtype=torch.int32, device=dev)
        Ks = Vs = None
        if sort_kv:
            Ks = torch.empty_like(K) if K_out is None else K_out
            if V is not None:
                Vs = torch.empty_like(V) if V_out is None else V_out
            for name, out in (("K_out", Ks), ("V_out", Vs)):
                if out is not None:
                    _check_tensor(out, name, torch.bfloat16, (Hkv, b.total, 128))
                    if out.data_ptr() in (K.data_ptr(), V.data_ptr() if V is not None else 0):
                        raise ValueError(f"{name} must not be the input it is sorted from")
        C.check(C.lib().tactic_build_clusters(
            K.data_ptr(), V.data_ptr() if V is not None else None, ctypes.byref(self._shape),
            self.cl_indptr.data_ptr(), self.total_c, self.max_c, init_idx.data_ptr(), ctypes.byref(self.params),
            cent.data_ptr(), assign.data_ptr(), offsets.data_ptr(), perm.data_ptr(),
            Ks.data_ptr() if Ks is not None else None, Vs.data_ptr() if Vs is not None else None,
            self.workspace.data_ptr(), self.workspace.numel(), _stream(stream)), "tactic_build_clusters")
        return ClusterBuild(ClusterSet(cent, offsets, self.n_clusters), assign, perm, Ks, Vs)
