"""MI355X (gfx950) implementation of Tactic's decode-time sparse attention.

The computation lives in libtactic.so (HIP kernels behind the C ABI of
include/tactic.h); this package only marshals torch tensors into those calls.
"""
from ._capi import TacticError, lib, LIB_PATH, EXPORTS  # noqa: F401
from .tactic import (ClusterBuild, ClusterBuilder, ClusterSet, DenseDecoder, PagedCache, RaggedBatch,  # noqa: F401
                     SparseDecoder, decode_params, sparse_decode_workspace_bytes, stream_read_gbps)
from .cache import RecentTailCache  # noqa: F401
