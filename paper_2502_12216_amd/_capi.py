"""ctypes declarations of include/tactic.h and the library loader.

Argument marshalling only: every computation happens in libtactic.so.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int, c_int32, c_int64, c_size_t, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtactic.so")

TACTIC_OK = 0
NOALLOC_SCRATCH_BYTES = 64 << 20  # TACTIC_NOALLOC_SCRATCH_BYTES
FIT_FIELDS = 16
FIT_NAMES = ("m", "mu1", "mu2", "a", "b", "S_n", "T", "k", "N", "n", "exact", "samples", "E_N",
             "cut_rank", "cut_len", "unused")

# every symbol include/tactic.h declares
EXPORTS = (
    "tactic_decode_params_default", "tactic_sparse_decode_plan", "tactic_sparse_decode",
    "tactic_sparse_decode_plan_set_events",
    "tactic_sparse_decode_view", "tactic_dense_decode_workspace_size", "tactic_dense_decode",
    "tactic_sparse_decode_paged", "tactic_dense_decode_paged", "tactic_sparse_decode_noalloc",
    "tactic_probe_stream_read",
    "tactic_build_clusters_workspace_size", "tactic_build_clusters", "tactic_status_string",
    "tactic_last_error",
)


class KVShape(ctypes.Structure):
    _fields_ = [("batch", c_int32), ("n_q_heads", c_int32), ("n_kv_heads", c_int32),
                ("head_dim", c_int32), ("total_tokens", c_int64), ("max_seq_len", c_int64),
                ("kv_indptr", c_void_p), ("seq_len", c_void_p)]


class ClusterMeta(ctypes.Structure):
    _fields_ = [("total_clusters", c_int64), ("max_clusters", c_int32), ("cl_indptr", c_void_p),
                ("centroids", c_void_p), ("offsets", c_void_p)]


class DecodeParams(ctypes.Structure):
    _fields_ = [("target_frac", c_float), ("exact_bp", c_int32), ("win_bp", c_int32),
                ("win_min", c_int32), ("p1_bp", c_int32), ("p2_bp", c_int32), ("use_union", c_int32),
                ("max_tail", c_int32)]


class DecodePlan(ctypes.Structure):
    _fields_ = [("v", c_int64 * 64)]


class DecodeView(ctypes.Structure):
    _fields_ = [("scores", c_void_p), ("order", c_void_p), ("rank_prefix", c_void_p),
                ("fit", c_void_p), ("union_len", c_void_p), ("sample_rows", c_void_p), ("sample_cap", c_int64)]


class PagedKV(ctypes.Structure):
    _fields_ = [("K_pages", c_void_p), ("V_pages", c_void_p), ("page_table", c_void_p), ("perm", c_void_p),
                ("page_size", c_int32), ("max_pages", c_int32), ("num_pages", c_int64)]


class KMeansParams(ctypes.Structure):
    _fields_ = [("max_iters", c_int32), ("reserved", c_int32), ("prev_centroids", c_void_p),
                ("prev_cl_indptr", c_void_p)]


class TacticError(RuntimeError):
    pass


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built (no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (load torch's HIP runtime first so both share one)
    if not os.path.exists(LIB_PATH):
        raise TacticError(f"{LIB_PATH} is missing: build it with `python -m paper_2502_12216_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    L.tactic_decode_params_default.argtypes = [POINTER(DecodeParams)]
    L.tactic_decode_params_default.restype = None
    L.tactic_sparse_decode_plan.argtypes = [POINTER(KVShape), POINTER(ClusterMeta), POINTER(DecodeParams),
                                            POINTER(DecodePlan), POINTER(c_size_t)]
    L.tactic_sparse_decode_plan.restype = c_int
    L.tactic_sparse_decode.argtypes = [c_void_p, c_void_p, c_void_p, POINTER(KVShape), POINTER(ClusterMeta),
                                       POINTER(DecodeParams), POINTER(DecodePlan), c_void_p, c_void_p,
                                       c_void_p, c_void_p, c_size_t, c_void_p]
    L.tactic_sparse_decode.restype = c_int
    L.tactic_sparse_decode_paged.argtypes = [c_void_p, POINTER(PagedKV), POINTER(KVShape), POINTER(ClusterMeta),
                                             POINTER(DecodeParams), POINTER(DecodePlan), c_void_p, c_void_p,
                                             c_void_p, c_void_p, c_size_t, c_void_p]
    L.tactic_sparse_decode_paged.restype = c_int
    L.tactic_sparse_decode_noalloc.argtypes = [c_void_p, c_void_p, c_void_p, POINTER(KVShape), POINTER(ClusterMeta),
                                               POINTER(DecodeParams), POINTER(DecodePlan), c_void_p, c_void_p,
                                               c_void_p, c_void_p]
    L.tactic_sparse_decode_noalloc.restype = c_int
    L.tactic_sparse_decode_plan_set_events.argtypes = [POINTER(DecodePlan), c_void_p]
    L.tactic_sparse_decode_plan_set_events.restype = c_int
    L.tactic_sparse_decode_view.argtypes = [POINTER(DecodePlan), c_void_p, POINTER(DecodeView)]
    L.tactic_sparse_decode_view.restype = c_int
    L.tactic_dense_decode_workspace_size.argtypes = [POINTER(KVShape)]
    L.tactic_dense_decode_workspace_size.restype = c_size_t
    L.tactic_dense_decode.argtypes = [c_void_p, c_void_p, c_void_p, POINTER(KVShape), c_void_p, c_void_p,
                                      c_size_t, c_void_p]
    L.tactic_dense_decode.restype = c_int
    L.tactic_dense_decode_paged.argtypes = [c_void_p, POINTER(PagedKV), POINTER(KVShape), c_void_p, c_void_p,
                                            c_size_t, c_void_p]
    L.tactic_dense_decode_paged.restype = c_int
    L.tactic_build_clusters_workspace_size.argtypes = [POINTER(KVShape), c_int64, c_int32]
    L.tactic_build_clusters_workspace_size.restype = c_size_t
    L.tactic_build_clusters.argtypes = [c_void_p, c_void_p, POINTER(KVShape), c_void_p, c_int64, c_int32,
                                        c_void_p, POINTER(KMeansParams), c_void_p, c_void_p, c_void_p,
                                        c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
    L.tactic_build_clusters.restype = c_int
    L.tactic_probe_stream_read.argtypes = [c_void_p, c_size_t, c_int32, c_void_p, c_void_p]
    L.tactic_probe_stream_read.restype = c_int
    L.tactic_status_string.argtypes = [c_int]
    L.tactic_status_string.restype = c_char_p
    L.tactic_last_error.argtypes = []
    L.tactic_last_error.restype = c_char_p
    _lib = L
    return L


def check(status: int, what: str) -> None:
    if status != TACTIC_OK:
        L = lib()
        raise TacticError(f"{what}: {L.tactic_status_string(status).decode()}: "
                          f"{L.tactic_last_error().decode()} (status {status})")


__all__ = ["KVShape", "ClusterMeta", "DecodeParams", "DecodePlan", "DecodeView", "KMeansParams", "PagedKV",
           "TacticError", "lib", "check", "EXPORTS", "LIB_PATH", "FIT_FIELDS", "FIT_NAMES", "NOALLOC_SCRATCH_BYTES",
           "c_double"]
