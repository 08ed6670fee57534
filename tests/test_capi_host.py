"""Host-only checks of the C ABI: the library loads, exports every function
include/tactic.h declares, and rejects bad arguments before any device work
(no GPU is needed: every call here fails validation, which runs first)."""
import ctypes
import os
import re

import pytest

from paper_2502_12216_amd import _capi as C

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x1000  # never dereferenced: validation fails before any launch


def header_functions():
    src = open(os.path.join(ROOT, "include", "tactic.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tactic_[a-z_]+)\s*\(", src)))


def test_exports_match_header():
    L = C.lib()
    names = header_functions()
    assert sorted(C.EXPORTS) == names
    for n in names:
        assert hasattr(L, n), n


def _shape(B=1, Hq=8, Hkv=2, d=128, total=4096, nmax=4096, indptr=FAKE):
    return C.KVShape(B, Hq, Hkv, d, total, nmax, indptr)


def _params(P=0.9):
    p = C.DecodeParams()
    C.lib().tactic_decode_params_default(ctypes.byref(p))
    p.target_frac = P
    return p


def _plan(shape, meta, params):
    plan = C.DecodePlan()
    n = ctypes.c_size_t()
    st = C.lib().tactic_sparse_decode_plan(ctypes.byref(shape), ctypes.byref(meta), ctypes.byref(params),
                                           ctypes.byref(plan), ctypes.byref(n))
    return st, plan, n.value


def test_defaults():
    p = _params()
    assert abs(p.target_frac - 0.9) < 1e-7
    assert (p.exact_bp, p.win_bp, p.win_min, p.p1_bp, p.p2_bp, p.use_union) == (100, 50, 8, 1000, 6000, 1)


@pytest.mark.parametrize("kw,code", [
    (dict(d=64), 2), (dict(Hq=6, Hkv=4), 1), (dict(Hq=24, Hkv=2), 2), (dict(B=0), 1),
    (dict(indptr=None), 1), (dict(total=10, nmax=20), 1),
])
def test_plan_rejects_bad_shapes(kw, code):
    meta = C.ClusterMeta(256, 256, FAKE, FAKE, FAKE)
    st, _, _ = _plan(_shape(**kw), meta, _params())
    assert st == code, C.lib().tactic_last_error()


@pytest.mark.parametrize("P", [0.0, -0.1, 1.5, float("nan")])
def test_plan_rejects_bad_target(P):
    meta = C.ClusterMeta(256, 256, FAKE, FAKE, FAKE)
    st, _, _ = _plan(_shape(), meta, _params(P))
    assert st == 1


def test_plan_rejects_inconsistent_clusters_and_bad_union_flag():
    st, _, _ = _plan(_shape(), C.ClusterMeta(100, 256, FAKE, FAKE, FAKE), _params())
    assert st == 1
    p = _params()
    p.use_union = 2
    st, _, _ = _plan(_shape(), C.ClusterMeta(256, 256, FAKE, FAKE, FAKE), p)
    assert st == 1


def test_per_head_plan_sizes_selection_groups_per_query_head():
    """use_union = 0 plans one selection group per query head (range tables
    per query head, partials of one head per slot), so the layout differs."""
    meta = C.ClusterMeta(256, 256, FAKE, FAKE, FAKE)
    pu = _params()
    ph = _params()
    ph.use_union = 0
    st1, plan_u, n_u = _plan(_shape(), meta, pu)
    st2, plan_h, n_h = _plan(_shape(), meta, ph)
    assert st1 == 0 and st2 == 0
    assert n_h != n_u


def test_plan_workspace_grows_with_shape():
    meta = C.ClusterMeta(256, 256, FAKE, FAKE, FAKE)
    st, plan, n1 = _plan(_shape(), meta, _params())
    assert st == 0 and n1 > 0
    st, _, n2 = _plan(_shape(B=2, total=8192), C.ClusterMeta(512, 256, FAKE, FAKE, FAKE), _params())
    assert st == 0 and n2 > n1


def test_decode_rejects_small_workspace_and_mismatched_plan():
    L = C.lib()
    shape = _shape()
    meta = C.ClusterMeta(256, 256, FAKE, FAKE, FAKE)
    params = _params()
    st, plan, nbytes = _plan(shape, meta, params)
    assert st == 0
    st = L.tactic_sparse_decode(FAKE, FAKE, FAKE, ctypes.byref(shape), ctypes.byref(meta), ctypes.byref(params),
                                ctypes.byref(plan), FAKE, FAKE, FAKE, FAKE, nbytes - 1, None)
    assert st == 3
    other = _shape(B=2, total=8192)
    st = L.tactic_sparse_decode(FAKE, FAKE, FAKE, ctypes.byref(other), ctypes.byref(meta), ctypes.byref(params),
                                ctypes.byref(plan), FAKE, FAKE, FAKE, FAKE, nbytes, None)
    assert st == 1
    st = L.tactic_sparse_decode(None, FAKE, FAKE, ctypes.byref(shape), ctypes.byref(meta), ctypes.byref(params),
                                ctypes.byref(plan), FAKE, FAKE, FAKE, FAKE, nbytes, None)
    assert st == 1
    assert "null" in L.tactic_last_error().decode()


def test_plan_rejects_more_selection_groups_than_the_attention_holds():
    """The attention keeps one prefix entry per selection group in LDS (at most
    4096 groups): per-head mode has B * Hq groups and is rejected at plan time,
    before any kernel runs, where the union's B * Hkv groups still fit."""
    B, Hq, Hkv = 200, 32, 8
    shape = _shape(B=B, Hq=Hq, Hkv=Hkv, total=B * 64, nmax=64)
    meta = C.ClusterMeta(B * 4, 4, FAKE, FAKE, FAKE)
    st, _, _ = _plan(shape, meta, _params())
    assert st == 0, C.lib().tactic_last_error()
    ph = _params()
    ph.use_union = 0
    st, _, _ = _plan(shape, meta, ph)
    assert st == 2 and b"selection groups" in C.lib().tactic_last_error()


def test_noalloc_decode_rejects_a_plan_beyond_its_scratch():
    """tactic_sparse_decode_noalloc checks the plan's workspace against its
    static scratch before any device work: 16 x 131072 tokens need ~100 MiB."""
    L = C.lib()
    B, n = 16, 131072
    shape = _shape(B=B, Hq=32, Hkv=8, total=B * n, nmax=n)
    meta = C.ClusterMeta(B * 8192, 8192, FAKE, FAKE, FAKE)
    params = _params()
    st, plan, nbytes = _plan(shape, meta, params)
    assert st == 0 and nbytes > C.NOALLOC_SCRATCH_BYTES
    st = L.tactic_sparse_decode_noalloc(FAKE, FAKE, FAKE, ctypes.byref(shape), ctypes.byref(meta),
                                        ctypes.byref(params), ctypes.byref(plan), FAKE, FAKE, FAKE, None)
    assert st == 3 and b"static scratch" in L.tactic_last_error()
    st = L.tactic_sparse_decode_noalloc(FAKE, FAKE, FAKE, ctypes.byref(shape), ctypes.byref(meta),
                                        ctypes.byref(params), None, FAKE, FAKE, FAKE, None)
    assert st == 1
    # the timed shape (4 x 131072 tokens, 8192 clusters) fits
    shape = _shape(B=4, Hq=32, Hkv=8, total=4 * n, nmax=n)
    st, _, nbytes = _plan(shape, C.ClusterMeta(4 * 8192, 8192, FAKE, FAKE, FAKE), params)
    assert st == 0 and nbytes <= C.NOALLOC_SCRATCH_BYTES


def test_dense_and_kmeans_validation():
    L = C.lib()
    shape = _shape()
    n = L.tactic_dense_decode_workspace_size(ctypes.byref(shape))
    assert n > 0
    assert L.tactic_dense_decode(FAKE, FAKE, FAKE, ctypes.byref(shape), FAKE, FAKE, n - 1, None) == 3
    bad = _shape(d=96)
    assert L.tactic_dense_decode_workspace_size(ctypes.byref(bad)) == 0
    kp = C.KMeansParams(0)
    m = L.tactic_build_clusters_workspace_size(ctypes.byref(shape), 256, 256)
    assert m > 0
    st = L.tactic_build_clusters(FAKE, FAKE, ctypes.byref(shape), FAKE, 256, 256, FAKE, ctypes.byref(kp),
                                 FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, m, None)
    assert st == 1
    kp.max_iters = 10
    st = L.tactic_build_clusters(FAKE, FAKE, ctypes.byref(shape), FAKE, 100, 256, FAKE, ctypes.byref(kp),
                                 FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, m, None)
    assert st == 1
    # a warm start needs both the previous centroids and their cluster offsets
    for pc, pi in ((FAKE, None), (None, FAKE)):
        kp2 = C.KMeansParams(10, 0, pc, pi)
        st = L.tactic_build_clusters(FAKE, FAKE, ctypes.byref(shape), FAKE, 256, 256, FAKE, ctypes.byref(kp2),
                                     FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, m, None)
        assert st == 1
        assert b"together" in L.tactic_last_error()


def test_status_strings():
    L = C.lib()
    for s in range(5):
        assert len(L.tactic_status_string(s)) > 0


@pytest.mark.parametrize("field,value", [("exact_bp", -1), ("exact_bp", 10001), ("win_bp", 10001), ("win_min", 0),
                                         ("p1_bp", -5), ("p2_bp", 20000), ("max_tail", -1)])
def test_plan_rejects_fit_parameters_out_of_range(field, value):
    """Basis-point fractions outside [0, 10000], a window below one token and a
    negative recent-token capacity are rejected at plan time."""
    p = _params()
    setattr(p, field, value)
    st, _, _ = _plan(_shape(), C.ClusterMeta(256, 256, FAKE, FAKE, FAKE), p)
    assert st == 1, (field, value)


def test_plan_shape_and_cluster_limits():
    """A sequence of 2^31 tokens, more (sequence, KV head) groups than the
    attention's work list holds (4096), and more than 2^24 clusters per
    sequence are unsupported (status 2), before any device work."""
    L = C.lib()
    meta = C.ClusterMeta(256, 256, FAKE, FAKE, FAKE)
    st, _, _ = _plan(_shape(total=1 << 31, nmax=1 << 31), meta, _params())
    assert st == 2 and b"2^31" in L.tactic_last_error()
    B = 1000
    st, _, _ = _plan(_shape(B=B, Hq=64, Hkv=8, total=B * 64, nmax=64), C.ClusterMeta(B * 4, 4, FAKE, FAKE, FAKE),
                     _params())
    assert st == 2 and b"n_kv_heads" in L.tactic_last_error()
    big = (1 << 24) + 1
    st, _, _ = _plan(_shape(total=1 << 25, nmax=1 << 25), C.ClusterMeta(big, big, FAKE, FAKE, FAKE), _params())
    assert st == 2 and b"2^24" in L.tactic_last_error()


@pytest.mark.parametrize("case,code", [("null_table", 1), ("page_size", 1), ("few_pages", 1), ("huge_pages", 2),
                                       ("too_many_rows", 2)])
def test_paged_decode_validates_its_page_table(case, code):
    """The paged calls check the page table before any device work: null
    pointers, a zero page size, fewer pages per sequence than its longest
    sequence needs, and page counts whose rows overflow 32-bit indices."""
    L = C.lib()
    shape = _shape()  # longest sequence 4096 tokens, 2 KV heads
    kv = C.PagedKV(FAKE, FAKE, FAKE, None, 16, 256, 512)  # 16 x 256 = 4096 tokens per sequence
    if case == "null_table":
        kv.page_table = None
    elif case == "page_size":
        kv.page_size = 0
    elif case == "few_pages":
        kv.max_pages = 100
    elif case == "huge_pages":
        kv.max_pages = 1 << 27  # 2^27 pages x 16 tokens = 2^31 positions
    else:
        kv.num_pages = 1 << 26  # 2^26 pages x 2 heads x 16 rows = 2^31 rows
    n = L.tactic_dense_decode_workspace_size(ctypes.byref(shape))
    st = L.tactic_dense_decode_paged(FAKE, ctypes.byref(kv), ctypes.byref(shape), FAKE, FAKE, n, None)
    assert st == code, (case, L.tactic_last_error())


def test_build_clusters_rejects_bad_requests():
    """K-means build: V_sorted without V, max_iters outside [1, 1000], 2^21 or
    more clusters per sequence (status 2) and a workspace one byte short
    (status 3) are rejected before any device work."""
    L = C.lib()
    shape = _shape()
    m = L.tactic_build_clusters_workspace_size(ctypes.byref(shape), 256, 256)
    kp = C.KMeansParams(10)

    def build(V=FAKE, total=256, cmax=256, params=kp, V_sorted=FAKE, nbytes=m):
        return L.tactic_build_clusters(FAKE, V, ctypes.byref(shape), FAKE, total, cmax, FAKE, ctypes.byref(params),
                                       FAKE, FAKE, FAKE, FAKE, FAKE, V_sorted, FAKE, nbytes, None)

    assert build(V=None) == 1 and b"without V" in L.tactic_last_error()
    assert build(params=C.KMeansParams(1001)) == 1
    big = 1 << 21
    assert build(total=big, cmax=big) == 2 and b"2^21" in L.tactic_last_error()
    assert build(nbytes=m - 1) == 3


def test_stream_read_probe_validation():
    """The read-ceiling probe rejects a null buffer, a size that is not a
    multiple of 16 bytes and a negative workgroup count."""
    L = C.lib()
    assert L.tactic_probe_stream_read(None, 1 << 20, 0, FAKE, None) == 1
    assert L.tactic_probe_stream_read(FAKE, (1 << 20) + 8, 0, FAKE, None) == 1
    assert L.tactic_probe_stream_read(FAKE, 1 << 20, -1, FAKE, None) == 1
