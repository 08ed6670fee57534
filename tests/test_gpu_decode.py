"""GPU parity of the sparse and dense decode against the fp64 oracle.

Inputs are the seeded synthetic workloads (synth), laid out by the
generator's own mixture labels, so no input of the oracle comes from the HIP
path.  Every call goes through the C ABI of libtactic.so.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from oracle import tactic as OT
from tests.parity import check_group, fit_params, group_inputs, np64

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _tactic():
    import paper_2502_12216_amd as P
    return P


def _p32(P: float) -> float:
    """The library takes P as fp32; the oracle gets the same value."""
    return float(np.float32(P))


def run_sparse(inp, lay, P, params=None):
    T = _tactic()
    wl = inp.wl
    lens = [int(inp.kv_indptr[i + 1] - inp.kv_indptr[i]) for i in range(len(inp.kv_indptr) - 1)]
    ncl = [int(lay.cl_indptr[i + 1] - lay.cl_indptr[i]) for i in range(len(lay.cl_indptr) - 1)]
    batch = T.RaggedBatch(lens, wl.n_q_heads, wl.n_kv_heads)
    params = params or T.decode_params(P)
    dec = T.SparseDecoder(batch, ncl, params)
    cl = T.ClusterSet(lay.centroids.to(DEV).contiguous(), lay.offsets.to(DEV).contiguous(), ncl)
    out, sq, skv = dec(inp.q.to(DEV).contiguous(), lay.K_sorted.to(DEV).contiguous(),
                       lay.V_sorted.to(DEV).contiguous(), cl, target_frac=P)
    torch.cuda.synchronize()
    view = {k: v.clone().cpu() for k, v in dec.view().items()}
    return dict(out=out.clone().cpu(), sel_q=sq.clone().cpu(), sel_kv=skv.clone().cpu(), view=view,
                params=params, decoder=dec)


def check_layer(inp, lay, P, res, groups=None, label=""):
    wl = inp.wl
    G = wl.n_q_heads // wl.n_kv_heads
    union = bool(res["params"].use_union)
    B = len(inp.kv_indptr) - 1
    prm = fit_params(res["params"])
    todo = groups if groups is not None else [(b, g) for b in range(B) for g in range(wl.n_kv_heads)]
    allstats = []
    for b, g in todo:
        gi = group_inputs(inp.q, lay.K_sorted, lay.V_sorted, lay.centroids, lay.offsets, lay.kv_indptr,
                          lay.cl_indptr, b, g, G)
        c0, c1 = int(lay.cl_indptr[b]), int(lay.cl_indptr[b + 1])
        v = res["view"]
        gpu = dict(scores=np64(v["scores"][b, g * G:(g + 1) * G]),
                   order=v["order"][b, g * G:(g + 1) * G].numpy(),
                   k=res["sel_q"][b, g * G:(g + 1) * G].numpy(),
                   union_len=(v["union_len"][g, c0:c1].numpy() if union
                              else v["union_len"][g * G:(g + 1) * G, c0:c1].numpy()),
                   out=np64(res["out"][b, g * G:(g + 1) * G]),
                   sel_kv=int(res["sel_kv"][b, g]))
        allstats.append(check_group(gi, _p32(P), prm, gpu, label=f"{label} b={b} g={g}", use_union=union))
    return allstats


def _small(base, lens, name=None):
    return synth.small_workload(synth.WORKLOADS[base], lens, name)


@pytest.mark.parametrize("P", [0.5, 0.8, 0.9, 0.95, 1.0])
def test_sparse_ctx4k_full_parity(P):
    inp = synth.make_layer(synth.WORKLOADS["ctx4k_gqa4"], 0)
    lay = synth.label_layout(inp)
    res = run_sparse(inp, lay, P)
    st = check_layer(inp, lay, P, res, label=f"ctx4k P={P}")
    print(f"ctx4k P={P}: k={[s['k'] for s in st]} union={[s['union'] for s in st]} "
          f"err={max(s['out_err'] for s in st):.2e}")
    if P == 1.0:
        assert all(s["union"] == s["n"] for s in st)


@pytest.mark.parametrize("P", [0.5, 0.9])
def test_sparse_per_head_parity_and_union_saving(P):
    """use_union = 0: every head attends over its own selection (the ablation
    partner of the GQA union).  Same budgets as the union path; the union
    never loads more rows than the per-head sum."""
    T = _tactic()
    wl = _small("ctx32k_llama8b", [4096, 2500, 0, 3])
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp)
    ph = run_sparse(inp, lay, P, T.decode_params(P, use_union=0))
    check_layer(inp, lay, P, ph, label=f"per-head P={P}")
    un = run_sparse(inp, lay, P)
    assert torch.equal(ph["sel_q"], un["sel_q"])
    assert torch.all(un["sel_kv"] <= ph["sel_kv"])
    G = wl.n_q_heads // wl.n_kv_heads
    assert torch.equal(ph["sel_kv"], ph["sel_q"].view(len(wl.seq_lens), wl.n_kv_heads, G).sum(-1))


@pytest.mark.parametrize("P", [0.3, 0.9, 1.0])
def test_sparse_recent_tail_parity(P):
    """Recent unclustered tokens at the end of each sequence (Sec. 1): always
    selected, exact mass counted toward the target.  Tails of 0, 1, a few
    hundred, one longer than its clustered part, and a whole sequence."""
    T = _tactic()
    wl = _small("ctx32k_llama8b", [3000, 700, 1500, 257, 900])
    inp = synth.make_layer(wl, 0)
    tail = [0, 1, 300, 200, 900]
    lay = synth.label_layout(inp, tail=tail)
    for union in (1, 0):
        res = run_sparse(inp, lay, P, T.decode_params(P, max_tail=1024, use_union=union))
        st = check_layer(inp, lay, P, res, label=f"tail P={P} union={union}")
        G = wl.n_q_heads // wl.n_kv_heads
        for b, t in enumerate(tail):
            assert torch.all(res["sel_q"][b] >= t)
        if P == 1.0:
            assert all(s["union"] >= s["n"] for s in st)


def test_sparse_ragged_small_with_empty_and_tiny_sequences():
    # lengths straddle tiles, a 1-token and a 5-token sequence (exact mode) and an empty one
    wl = _small("ctx32k_llama8b", [700, 0, 1, 5, 1300, 64, 3000])
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp)
    for P in (0.3, 0.9):
        res = run_sparse(inp, lay, P)
        check_layer(inp, lay, P, res, label=f"ragged P={P}")
        B = len(inp.kv_indptr) - 1
        G = wl.n_q_heads // wl.n_kv_heads
        assert torch.all(res["out"][1] == 0) and torch.all(res["sel_q"][1] == 0)
        assert torch.all(res["sel_kv"][1] == 0)


def test_sparse_one_cluster_per_token_is_top_p():
    """Every token its own cluster (centroid = key) and every score exact:
    the selection of each head must be the exact top-P prefix (Sec. 3.4)."""
    T = _tactic()
    torch.manual_seed(0)
    n, Hq, Hkv = 2000, 4, 1
    K = (torch.randn(Hkv, n, 128) * 0.6).to(torch.bfloat16)
    V = torch.randn(Hkv, n, 128).to(torch.bfloat16)
    q = (torch.randn(1, Hq, 128) * 1.5).to(torch.bfloat16)
    offsets = torch.arange(n + 1, dtype=torch.int32)[None].contiguous()
    batch = T.RaggedBatch([n], Hq, Hkv)
    for P in (0.5, 0.9, 0.99):
        params = T.decode_params(P, exact_bp=10000)
        dec = T.SparseDecoder(batch, [n], params)
        cl = T.ClusterSet(K.to(DEV).contiguous(), offsets.to(DEV), [n])
        out, sq, skv = dec(q.to(DEV), K.to(DEV), V.to(DEV), cl)
        torch.cuda.synchronize()
        Kd, Vd, qd = np64(K[0]), np64(V[0]), np64(q[0])
        U = set()
        for h in range(Hq):
            ref = OA.optimal_selection(qd[h], Kd, _p32(P))
            kg = int(sq[0, h])
            if kg != len(ref):  # accept only a cutoff tie
                s = OA.softmax_weights(OA.logits(qd[h], Kd))
                cs = np.add.accumulate(np.sort(s)[::-1])
                assert abs(cs[kg - 1] - _p32(P)) <= 1e-5 or abs(cs[len(ref) - 1] - _p32(P)) <= 1e-5
            U |= set(OA.optimal_selection(qd[h], Kd, _p32(P))[:kg].tolist())
        assert int(skv[0, 0]) == len(U)
        for h in range(Hq):
            ref = OA.sparse_attention(qd[h], Kd, Vd, np.array(sorted(U)))
            assert float(np.max(np.abs(np64(out[0, h]) - ref))) <= 2e-3


def test_sparse_single_cluster_and_target_one_is_dense():
    T = _tactic()
    wl = _small("ctx4k_gqa4", [1500, 333])
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp)
    res = run_sparse(inp, lay, 1.0)
    G = wl.n_q_heads // wl.n_kv_heads
    for b, n in enumerate([1500, 333]):
        for h in range(wl.n_q_heads):
            g = h // G
            s0 = int(inp.kv_indptr[b])
            ref = OA.dense_attention(np64(inp.q[b, h]), np64(inp.K[g, s0:s0 + n]), np64(inp.V[g, s0:s0 + n]))
            assert float(np.max(np.abs(np64(res["out"][b, h]) - ref))) <= 2e-3
            assert int(res["sel_q"][b, h]) == n
    # one cluster holding every token
    K1 = lay.K_sorted.clone()
    n = 1500
    cent = inp.K[:, :1].clone().contiguous()
    off = torch.tensor([[0, n]] * wl.n_kv_heads, dtype=torch.int32)
    lay1 = synth.LabelLayout(K_sorted=K1[:, :n].contiguous(), V_sorted=lay.V_sorted[:, :n].contiguous(),
                             centroids=cent, offsets=off, perm=lay.perm[:, :n].contiguous(),
                             kv_indptr=np.array([0, n]), cl_indptr=np.array([0, 1]))
    inp1 = synth.make_layer(_small("ctx4k_gqa4", [n]), 0)
    inp1.q = inp.q[:1].clone()
    res1 = run_sparse(inp1, lay1, 0.9)
    check_layer(inp1, lay1, 0.9, res1, label="one cluster")


@pytest.mark.parametrize("case", ["lds", "shared"])
def test_sparse_is_deterministic(case):
    """Two calls give bit-identical outputs and counts: the in-LDS sort, and
    12000 clusters per sequence, where workgroups share each head's sort (a
    cluster's place inside its bucket follows the order of atomic arrivals,
    which may differ between calls) and each group's union runs in slices."""
    import dataclasses
    if case == "lds":
        wl = _small("ctx32k_llama8b", [5000, 2500])
    else:
        base = _small("ctx32k_llama8b", [30000, 12000])
        wl = dataclasses.replace(base, fixed_clusters=12000, name=f"{base.name}_c12000_det")
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp)
    a = run_sparse(inp, lay, 0.9)
    b = run_sparse(inp, lay, 0.9)
    assert torch.equal(a["out"], b["out"]) and torch.equal(a["sel_q"], b["sel_q"])
    assert torch.equal(a["sel_kv"], b["sel_kv"])


@pytest.mark.parametrize("P", [0.8, 0.9, 0.95])
def test_sparse_ctx32k_full_parity(P):
    inp = synth.make_layer(synth.WORKLOADS["ctx32k_llama8b"], 0, device=DEV)
    lay = synth.label_layout(inp)
    res = run_sparse(inp, lay, P)
    st = check_layer(inp, lay, P, res, label=f"ctx32k P={P}")
    ks = np.array([s["k"] for s in st]).ravel()
    us = np.array([s["union"] for s in st])
    print(f"ctx32k P={P}: k median {np.median(ks):.0f} max {ks.max()} union median {np.median(us):.0f}"
          f" max {us.max()} ties(order)={sum(s['order_ties'] for s in st)} ties(cut)={sum(s['cut_ties'] for s in st)}")


def test_sparse_ctx128k_b4_layer_sampled_parity():
    """The timed workload's shape (batch 4 x 128K, 32q/8kv, 8192 clusters per
    head), one layer, parity on a seeded sample of (b, g) groups."""
    wl = synth.WORKLOADS["ctx128k_b4_32layer"]
    inp = synth.make_layer(wl, 3, device=DEV)
    lay = synth.label_layout(inp)
    res = run_sparse(inp, lay, 0.9)
    rng = np.random.default_rng(5)
    groups = [(int(b), int(g)) for b, g in zip(rng.integers(0, 4, 4), rng.integers(0, 8, 4))]
    st = check_layer(inp, lay, 0.9, res, groups=groups, label="ctx128k")
    print("ctx128k sampled:", [(s["k"], s["union"]) for s in st])


@pytest.mark.slow
def test_sparse_ctx1m_global_sort_sampled_parity():
    """1M tokens with 32768 clusters per head: the cluster sort runs out of
    the workspace instead of LDS."""
    wl = synth.WORKLOADS["ctx1m"]
    inp = synth.make_layer(wl, 0, device=DEV)
    lay = synth.label_layout(inp)
    res = run_sparse(inp, lay, 0.9)
    st = check_layer(inp, lay, 0.9, res, groups=[(0, 2), (0, 5)], label="ctx1m")
    print("ctx1m sampled:", [(s["k"], s["union"]) for s in st])


def test_sparse_ragged16_sampled_parity():
    wl = synth.WORKLOADS["ragged16_16k_128k"]
    inp = synth.make_layer(wl, 0, device=DEV, seq_subset=[0, 3, 7, 11])
    lay = synth.label_layout(inp)
    res = run_sparse(inp, lay, 0.9)
    st = check_layer(inp, lay, 0.9, res, groups=[(0, 1), (1, 6), (2, 0), (3, 7)], label="ragged16")
    print("ragged16 sampled:", [(s["n"], s["k"], s["union"]) for s in st])


# ------------------------------------------------------------------ dense

@pytest.mark.parametrize("lens", [[4096], [700, 0, 1, 5, 1300], [33000, 1000]])
def test_dense_decode_matches_oracle(lens):
    T = _tactic()
    wl = _small("ctx32k_llama8b", lens)
    inp = synth.make_layer(wl, 0, device=DEV)
    batch = T.RaggedBatch(lens, wl.n_q_heads, wl.n_kv_heads)
    dec = T.DenseDecoder(batch)
    out = dec(inp.q, inp.K, inp.V)
    out2 = dec(inp.q, inp.K, inp.V).clone()  # counters reset after a call
    torch.cuda.synchronize()
    G = wl.n_q_heads // wl.n_kv_heads
    err = 0.0
    for b, n in enumerate(lens):
        s0 = int(batch.kv_indptr_host[b])
        for h in range(wl.n_q_heads):
            if n == 0:
                assert torch.all(out2[b, h] == 0)
                continue
            g = h // G
            ref = OA.dense_attention(np64(inp.q[b, h]), np64(inp.K[g, s0:s0 + n]), np64(inp.V[g, s0:s0 + n]))
            err = max(err, float(np.max(np.abs(np64(out2[b, h]) - ref))))
    assert err <= 2e-3, err


def test_spare_room_layout_matches_packed_layout():
    """Sequences with spare rows after their tokens (seq_len < span): every
    kernel reads only the first seq_len rows, so results equal the packed
    layout's bit for bit even when the spare rows hold huge values."""
    T = _tactic()
    wl = _small("ctx32k_llama8b", [1800, 0, 700, 2500])
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp, tail=[100, 0, 0, 40])
    lens = list(wl.seq_lens)
    caps = [n + extra for n, extra in zip(lens, [300, 5, 0, 77])]
    ncl = [int(lay.cl_indptr[i + 1] - lay.cl_indptr[i]) for i in range(len(lens))]
    Hkv = wl.n_kv_heads
    packed = T.RaggedBatch(lens, wl.n_q_heads, Hkv)
    spaced = T.RaggedBatch(lens, wl.n_q_heads, Hkv, capacities=caps)

    def spread(X):
        Y = torch.full((Hkv, spaced.total, 128), 3e4, dtype=torch.bfloat16)
        for b, n in enumerate(lens):
            s0, d0 = packed.kv_indptr_host[b], spaced.kv_indptr_host[b]
            Y[:, d0:d0 + n] = X[:, s0:s0 + n]
        return Y.to(DEV)

    q = inp.q.to(DEV)
    cl = T.ClusterSet(lay.centroids.to(DEV), lay.offsets.to(DEV), ncl)
    for P in (0.6, 1.0):
        params = T.decode_params(P, max_tail=256)
        o1, q1, k1 = T.SparseDecoder(packed, ncl, params)(q, lay.K_sorted.to(DEV), lay.V_sorted.to(DEV), cl)
        o2, q2, k2 = T.SparseDecoder(spaced, ncl, params)(q, spread(lay.K_sorted), spread(lay.V_sorted), cl)
        torch.cuda.synchronize()
        assert torch.equal(q1, q2) and torch.equal(k1, k2)
        assert torch.equal(o1, o2)
    d1 = T.DenseDecoder(packed)(q, inp.K.to(DEV), inp.V.to(DEV))
    d2 = T.DenseDecoder(spaced)(q, spread(inp.K), spread(inp.V))
    torch.cuda.synchronize()
    assert torch.allclose(d1, d2, atol=1e-5, rtol=0)


@pytest.mark.parametrize("page_size", [16, 1, 64])
def test_paged_cache_matches_cluster_sorted_copy(page_size):
    """Decode from a paged cache in token order (cluster order reached through
    perm, pages scattered at random) and from pages already in cluster order:
    the same rows in the same order as the cluster-sorted copy, so the same
    bits.  Includes recent tokens past the clusters and an empty sequence."""
    T = _tactic()
    wl = _small("ctx32k_llama8b", [2100, 0, 900, 1337])
    inp = synth.make_layer(wl, 0)
    tail = [50, 0, 0, 137]
    lay = synth.label_layout(inp, tail=tail)
    lens = list(wl.seq_lens)
    ncl = [int(lay.cl_indptr[i + 1] - lay.cl_indptr[i]) for i in range(len(lens))]
    batch = T.RaggedBatch(lens, wl.n_q_heads, wl.n_kv_heads)
    g = torch.Generator().manual_seed(page_size)
    npg = sum((n + page_size - 1) // page_size for n in lens)
    scattered = torch.randperm(npg, generator=g)
    q = inp.q.to(DEV)
    K, V, Ks, Vs = (x.to(DEV) for x in (inp.K, inp.V, lay.K_sorted, lay.V_sorted))
    perm = lay.perm.to(DEV).contiguous()
    token_pages = T.PagedCache.from_token_order(K, V, batch, page_size, page_order=scattered, perm=perm)
    sorted_pages = T.PagedCache.from_token_order(Ks, Vs, batch, page_size)
    cl = T.ClusterSet(lay.centroids.to(DEV), lay.offsets.to(DEV), ncl)
    for P in (0.5, 0.95):
        params = T.decode_params(P, max_tail=256)
        dec = T.SparseDecoder(batch, ncl, params)
        ref = [x.clone() for x in dec(q, Ks, Vs, cl)]
        for name, pages in (("token order + perm", token_pages), ("cluster order", sorted_pages)):
            got = dec.paged(q, pages, cl)
            torch.cuda.synchronize()
            for a, b in zip(ref, got):
                assert torch.equal(a, b)
            # and the paged call's own selection and output against the oracle
            res = dict(out=got[0].clone().cpu(), sel_q=got[1].clone().cpu(), sel_kv=got[2].clone().cpu(),
                       view={k: v.clone().cpu() for k, v in dec.view().items()}, params=params)
            check_layer(inp, lay, P, res, label=f"paged ps={page_size} {name} P={P}")
    den = T.DenseDecoder(batch)
    d_ref = den(q, K, V).clone()
    d_pg = den.paged(q, token_pages)
    torch.cuda.synchronize()
    assert torch.equal(d_ref, d_pg)


@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (8, 4), (16, 2)])
def test_sparse_other_group_sizes(Hq, Hkv):
    """Group sizes G = 1 (multi-head), 2 and 8: the kernels' per-group code
    (head-splitting reduction, per-head broadcasts, union over G heads) for
    every G they support, in union and per-head modes, with a recent tail."""
    import dataclasses
    T = _tactic()
    base = _small("ctx32k_llama8b", [1500, 640])
    wl = dataclasses.replace(base, n_q_heads=Hq, n_kv_heads=Hkv, name=f"{base.name}_h{Hq}x{Hkv}")
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp, tail=[40, 0])
    for union in (1, 0):
        for P in (0.6, 0.95):
            res = run_sparse(inp, lay, P, T.decode_params(P, use_union=union, max_tail=64))
            check_layer(inp, lay, P, res, label=f"G={Hq // Hkv} union={union} P={P}")
    den = T.DenseDecoder(T.RaggedBatch(list(wl.seq_lens), Hq, Hkv))
    out = den(inp.q.to(DEV), lay.K_sorted.to(DEV), lay.V_sorted.to(DEV)).cpu()
    for b in range(len(wl.seq_lens)):
        s0, s1 = int(inp.kv_indptr[b]), int(inp.kv_indptr[b + 1])
        for h in range(Hq):
            g = h // (Hq // Hkv)
            ref = OA.dense_attention(np64(inp.q[b, h]), np64(lay.K_sorted[g, s0:s1]), np64(lay.V_sorted[g, s0:s1]))
            assert float(np.max(np.abs(np64(out[b, h]) - ref))) <= 2e-3


@pytest.mark.parametrize("P", [0.5, 0.9])
def test_sparse_degenerate_scores(P):
    """Score ties end to end: a zero query (every cluster score 0: the sort's
    equal-scores shortcut, uniform logits, a flat fit with a = 0) and
    centroids repeated every 8 clusters (each score shared by an eighth of
    the clusters: crowded sort buckets, order by cluster id within a tie)."""
    wl = _small("ctx32k_llama8b", [3000, 1500])
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp)
    G = wl.n_q_heads // wl.n_kv_heads
    q = inp.q.clone()
    q[0, ::G] = 0  # the first query head of every group of sequence 0
    inp.q = q
    cent = lay.centroids.clone()
    c0, c1 = int(lay.cl_indptr[1]), int(lay.cl_indptr[2])
    idx = c0 + (torch.arange(c1 - c0) % 8)
    cent[:, c0:c1] = cent[:, idx]
    lay.centroids = cent
    res = run_sparse(inp, lay, P)
    st = check_layer(inp, lay, P, res, label=f"degenerate P={P}")
    order = res["view"]["order"]
    for g in range(wl.n_kv_heads):  # equal scores: the order is the cluster id
        C0 = int(lay.cl_indptr[1] - lay.cl_indptr[0])
        assert torch.equal(order[0, g * G, :C0], torch.arange(C0, dtype=order.dtype))
    print(f"degenerate P={P}: ties(order)={sum(s['order_ties'] for s in st)} k={[s['k'] for s in st][:2]}")


def test_sparse_empty_clusters_parity():
    """Empty clusters (Sec. 4.2 keeps a centroid that lost its members): the
    tokens of every odd mixture component are filed under the even one below
    it, so half the clusters hold no token but keep their centroid and are
    ranked like the others (the query's own centres among them)."""
    wl = _small("ctx32k_llama8b", [3000, 1700, 260])
    inp = synth.make_layer(wl, 0)
    inp.labels = (inp.labels // 2) * 2
    lay = synth.label_layout(inp, tail=[0, 45, 0])
    off = lay.offsets.long()
    empty = int(((off[:, 1:] - off[:, :-1]) == 0).sum())
    assert empty >= lay.centroids.shape[1] // 2 - 1
    T = _tactic()
    for P in (0.5, 0.9, 1.0):
        res = run_sparse(inp, lay, P, T.decode_params(P, max_tail=64))
        check_layer(inp, lay, P, res, label=f"empty clusters P={P}")


def test_sparse_target_one_at_128k_matches_dense_and_paged():
    """P = 1 selects every token (Eq. 2 from Eq. 3): at the timed shape
    (4 x 131072 tokens, one layer) the sparse decode must agree with the
    dense decode and with the fp64 oracle on sampled heads.  Every
    attention workgroup then streams ~5.5K tokens of one group, several
    2048-row sub-ranges starting inside a 256-position chunk, so the
    sub-range walk and the paged row lookups past position 256 are
    exercised; paged and contiguous caches give the same bits."""
    T = _tactic()
    wl = synth.WORKLOADS["ctx128k_b4_32layer"]
    inp = synth.make_layer(wl, 0, device=DEV)
    lay = synth.label_layout(inp)
    ncl = list(wl.cluster_counts)
    batch = T.RaggedBatch(wl.seq_lens, wl.n_q_heads, wl.n_kv_heads)
    cl = T.ClusterSet(lay.centroids.contiguous(), lay.offsets.contiguous(), ncl)
    dec = T.SparseDecoder(batch, ncl, T.decode_params(1.0))
    out, sq, skv = (x.clone() for x in dec(inp.q, lay.K_sorted, lay.V_sorted, cl))
    den = T.DenseDecoder(batch)
    d_sorted = den(inp.q, lay.K_sorted, lay.V_sorted).clone()
    d_tok = den(inp.q, inp.K, inp.V).clone()
    torch.cuda.synchronize()
    n = wl.seq_lens[0]
    assert torch.all(sq == n) and torch.all(skv == n)
    assert float((out - d_sorted).abs().max()) <= 1e-4
    assert float((out - d_tok).abs().max()) <= 1e-4
    # paged: 16-token pages at random page ids, cluster order through perm
    npg = sum((x + 15) // 16 for x in wl.seq_lens)
    pages = T.PagedCache.from_token_order(inp.K, inp.V, batch, 16,
                                          page_order=torch.randperm(npg, generator=torch.Generator().manual_seed(3)),
                                          perm=lay.perm.contiguous())
    got = [x.clone() for x in dec.paged(inp.q, pages, cl)]
    d_pg = den.paged(inp.q, pages).clone()
    torch.cuda.synchronize()
    assert torch.equal(got[0], out) and torch.equal(got[1], sq) and torch.equal(got[2], skv)
    assert torch.equal(d_pg, d_tok)
    # the fp64 oracle on a seeded sample of heads
    G = wl.n_q_heads // wl.n_kv_heads
    rng = np.random.default_rng(17)
    err = 0.0
    for b, h in zip(rng.integers(0, 4, 6), rng.integers(0, wl.n_q_heads, 6)):
        g = int(h) // G
        s0 = int(batch.kv_indptr_host[b])
        ref = OA.dense_attention(np64(inp.q[b, h]), np64(inp.K[g, s0:s0 + n]), np64(inp.V[g, s0:s0 + n]))
        err = max(err, float(np.max(np.abs(np64(out[b, h]) - ref))))
    assert err <= 2e-3, err
    print(f"128k P=1: sparse-dense {float((out - d_tok).abs().max()):.2e}, oracle max-abs {err:.2e}")


@pytest.mark.parametrize("case", ["c34000", "big_bucket", "big_cluster", "empty_seq"])
def test_sparse_sort_general_workspace_path(case):
    """Heads that the LDS-piece sort of 8192 < C <= 32768 clusters hands to
    the general workspace path: more than 32768 clusters (34000 clusters of
    about two tokens), a bucket larger than a piece (7000 of 9000 clusters of
    sequence 0 share one centroid, so 7000 equal scores), and a cluster of
    more than 65535 tokens (cluster 0 of every KV head holds 70000 of 90000
    tokens); and an empty sequence with no clusters between two of 9000
    clusters (its heads take no piece and must return zeros).  Staged parity
    on every group at P = 0.9."""
    import dataclasses
    P = 0.9
    lens, C = {"c34000": ([70000], 34000), "big_bucket": ([20000, 12000], 9000),
               "big_cluster": ([90000], 9000), "empty_seq": ([20000, 0, 12000], 9000)}[case]
    base = _small("ctx32k_llama8b", lens)
    wl = dataclasses.replace(base, fixed_clusters=C, name=f"{base.name}_{case}")
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp)
    if case == "big_bucket":
        cent = lay.centroids.clone()
        c0 = int(lay.cl_indptr[0])
        cent[:, c0:c0 + 7000] = cent[:, c0:c0 + 1]
        lay.centroids = cent
    if case == "big_cluster":
        # a valid layout with other cluster boundaries: cluster 0 takes the
        # first 70000 sorted rows, the other 8999 share the rest evenly
        n = lens[0]
        rest = np.round(np.linspace(70000, n, C)).astype(np.int32)
        off = np.concatenate([[0], rest]).astype(np.int32)
        assert off[1] == 70000 and off[-1] == n and np.all(np.diff(off) >= 0)
        lay.offsets = torch.as_tensor(np.tile(off, (wl.n_kv_heads, 1)))
    res = run_sparse(inp, lay, P)
    st = check_layer(inp, lay, P, res, label=f"sort general path {case}")
    print(f"sort general path {case}: k={[s['k'] for s in st][:2]} union={[s['union'] for s in st][:4]}")


@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (16, 2)])
def test_sparse_union_range_writers(Hq, Hkv):
    """Unions of more than 8192 clusters. With 8 heads per group (16 / 2) the
    group's one workgroup writes the ranges one of two ways: from each
    thread's 32-cluster segment when at most an eighth of the clusters are
    non-empty, else in a coalesced pass over the clusters; with 4 heads (32 /
    8) and in per-head mode the union runs in slices with a second kernel for
    the ranges. 9000 clusters of about two tokens at a low and a high target
    give both densities (asserted from the union lengths), in union and
    per-head modes and with 300 recent tokens after the clusters of sequence
    0 (their range follows the clusters' ranges), with staged parity on
    every group."""
    import dataclasses
    T = _tactic()
    base = _small("ctx32k_llama8b", [20000, 12000])
    wl = dataclasses.replace(base, n_q_heads=Hq, n_kv_heads=Hkv, fixed_clusters=9000,
                             name=f"{base.name}_c9000_h{Hq}x{Hkv}")
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp, tail=[300, 0])
    for union in (1, 0):
        seen = set()
        for P in (0.3, 0.99):
            res = run_sparse(inp, lay, P, T.decode_params(P, use_union=union, max_tail=512))
            check_layer(inp, lay, P, res, label=f"range writers G={Hq // Hkv} union={union} P={P}")
            ulen = res["view"]["union_len"]
            for b in range(len(wl.seq_lens)):
                c0, c1 = int(lay.cl_indptr[b]), int(lay.cl_indptr[b + 1])
                for row in range(Hkv if union else Hq):  # one row per selection group
                    nz = int((ulen[row, c0:c1] > 0).sum())
                    seen.add("segment" if nz * 8 <= c1 - c0 else "coalesced")
        assert seen == {"segment", "coalesced"}, (union, seen)


@pytest.mark.parametrize("case", ["pieces", "workspace", "mixed", "odd_split"])
def test_sparse_large_sort_paths_with_recent_tail(case):
    """Recent tokens after the clusters on the sorts of more than 8192
    clusters: 12000 clusters (LDS pieces) and 34000 clusters (workspace
    path), with a tail of 200 and 150 tokens on the first sequence (its
    sampled rows follow the windows', its range follows the union's), and a
    batch that mixes 12000 clusters with 3000 (the smaller sequence's heads
    then take the pieces, shared by the same number of workgroups, with a
    tail of 100), and three sequences of 16 / 4 heads at 9000 clusters (48
    heads: five workgroups share each head's sort, five slices of 1800
    clusters each per-head union), in union and per-head modes, staged parity
    on every group at P = 0.9."""
    import dataclasses
    T = _tactic()
    P = 0.9
    lens, C, tail = {"pieces": ([30000, 12000], 12000, [200, 0]), "workspace": ([70000], 34000, [150]),
                     "mixed": ([30000, 3000], 12000, [0, 100]),
                     "odd_split": ([20000, 15000, 12000], 9000, [0, 50, 0])}[case]
    base = _small("ctx32k_llama8b", lens)
    heads = {"n_q_heads": 16, "n_kv_heads": 4} if case == "odd_split" else {}
    wl = dataclasses.replace(base, fixed_clusters=C, name=f"{base.name}_{case}_tail", **heads)
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp, tail=tail)
    for union in (1, 0):
        res = run_sparse(inp, lay, P, T.decode_params(P, use_union=union, max_tail=256))
        st = check_layer(inp, lay, P, res, label=f"{case} tail union={union}")
        print(f"{case} tail union={union}: k={[s['k'] for s in st][:2]}")


@pytest.mark.parametrize("P", [0.5, 0.9])
def test_sparse_degenerate_scores_out_of_lds_sort(P):
    """The sort of more than 8192 clusters per head runs out of the
    workspace: a zero query (all scores equal: identity order), centroids
    repeated every 8 clusters (eight scores shared by an eighth of the
    clusters each: crowded buckets, ties by cluster id) and ordinary heads,
    with 9000 clusters of about two tokens each (many empty)."""
    import dataclasses
    base = _small("ctx32k_llama8b", [20000, 12000])
    wl = dataclasses.replace(base, fixed_clusters=9000, name=base.name + "_c9000")
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp)
    G = wl.n_q_heads // wl.n_kv_heads
    q = inp.q.clone()
    q[0, ::G] = 0
    inp.q = q
    cent = lay.centroids.clone()
    c0, c1 = int(lay.cl_indptr[1]), int(lay.cl_indptr[2])
    cent[:, c0:c1] = cent[:, c0 + (torch.arange(c1 - c0) % 8)]
    lay.centroids = cent
    res = run_sparse(inp, lay, P)
    st = check_layer(inp, lay, P, res, label=f"degenerate C=9000 P={P}")
    order = res["view"]["order"]
    for g in range(wl.n_kv_heads):
        assert torch.equal(order[0, g * G, :9000], torch.arange(9000, dtype=order.dtype))
    print(f"degenerate C=9000 P={P}: k={[s['k'] for s in st][:2]}")
