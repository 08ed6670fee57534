"""Staged GPU-vs-oracle comparison for one (sequence, KV head) group.

Stages (each later stage is evaluated on the GPU's own result of the earlier
ones, so a tie resolved differently upstream cannot fail a later stage):
  1. cluster scores q . c within fp32 accumulation error;
  2. cluster order: exactly the order of the GPU's own fp32 scores (score
     descending, ties by ascending cluster id); against the oracle's fp64
     scores it may differ only inside blocks of near-tied scores (within the
     score tolerance 1e-5 * |q| * max |c|);
  3. budget k of every head, with the oracle run on the GPU's order: equal,
     or the oracle's cumulative sum at the GPU's k is within 1e-5 (relative)
     of the target on both sides of the cutoff;
  4. union: per-cluster selected prefix lengths identical to the oracle's
     union of the GPU's per-head selections (per-head mode: each head's own
     selection, and the loaded count is the sum of the k_h);
  5. output: max |out_gpu - o~(U_gpu)| <= 2e-3 with o~ the oracle's fp64
     attention over the GPU's union (Eq. 3), or over each head's own
     selection in per-head mode.
Rows of the cache past the last cluster are recent tokens: every head's
selection holds all of them and the GPU's per-head count includes them.
"""
from __future__ import annotations

import numpy as np

from oracle import attention as OA
from oracle import tactic as OT

ORDER_TIE_REL = 1e-5
CUT_TIE_REL = 1e-5
OUT_ATOL = 2e-3


def np64(t) -> np.ndarray:
    return t.detach().to("cpu").double().numpy()


def fit_params(params) -> OT.FitParams:
    return OT.FitParams(exact_bp=params.exact_bp, win_bp=params.win_bp, win_min=params.win_min,
                        p1_bp=params.p1_bp, p2_bp=params.p2_bp)


def group_inputs(q, Ks, Vs, cent, offsets, kv_indptr, cl_indptr, b, g, G):
    """fp64 host copies of one group's inputs (bf16 upcast exactly)."""
    s0, s1 = int(kv_indptr[b]), int(kv_indptr[b + 1])
    c0, c1 = int(cl_indptr[b]), int(cl_indptr[b + 1])
    return dict(
        Q=np64(q[b, g * G:(g + 1) * G]),
        Ks=np64(Ks[g, s0:s1]),
        Vs=np64(Vs[g, s0:s1]),
        cent=np64(cent[g, c0:c1]),
        off=offsets[g, c0 + b:c1 + b + 1].to("cpu").numpy().astype(np.int64),
    )


def _cluster_lengths(rows: np.ndarray, off: np.ndarray, C: int) -> np.ndarray:
    """Selected rows per cluster of a set of rows of the cluster-sorted cache."""
    if len(rows) == 0:
        return np.zeros(C, np.int64)
    clus = np.searchsorted(off, rows, side="right") - 1
    return np.bincount(clus, minlength=C)[:C]


def check_group(inp: dict, P: float, prm: OT.FitParams, gpu: dict, label: str = "",
                use_union: bool = True) -> dict:
    """gpu: scores (G, C), order (G, C), k (G,), union_len (C,) or per head (G, C)
    when not use_union, out (G, d), sel_kv (int)."""
    Q, Ks, Vs, cent, off = inp["Q"], inp["Ks"], inp["Vs"], inp["cent"], inp["off"]
    G = Q.shape[0]
    C = cent.shape[0]
    n = int(off[-1])
    tail_rows = np.arange(n, len(Ks), dtype=np.int64)
    stats = dict(order_ties=0, cut_ties=0, order_equal=0)
    cmax = float(np.max(np.linalg.norm(cent, axis=1))) if C else 0.0
    orders = []
    for h in range(G):
        s_or = cent @ Q[h]
        tol = ORDER_TIE_REL * float(np.linalg.norm(Q[h])) * cmax + 1e-30
        sg = gpu["scores"][h][:C]
        err = float(np.max(np.abs(sg - s_or))) if C else 0.0
        assert err <= tol, f"{label} head {h}: score error {err} > {tol}"
        og = np.asarray(gpu["order"][h][:C], dtype=np.int64)
        # the GPU sorts its own fp32 scores: that order is unique (ties by id)
        own = np.lexsort((np.arange(C), -np.asarray(sg, dtype=np.float64)))
        assert np.array_equal(og, own), \
            f"{label} head {h}: order differs from the sort of the GPU's scores at {int(np.argmax(og != own))}"
        _, oo = OT.rank_clusters(Q[h], cent)
        if np.array_equal(oo, og):
            stats["order_equal"] += 1
        else:
            # every disagreement must sit inside a block of near-tied scores
            d = np.nonzero(oo != og)[0]
            assert np.all(np.abs(s_or[oo[d]] - s_or[og[d]]) <= 2 * tol), f"{label} head {h}: order differs"
            stats["order_ties"] += 1
        orders.append(og)
    r = OT.decode_group(Q, Ks, Vs, cent, off, P, prm, orders=orders)
    k_gpu = np.asarray(gpu["k"], dtype=np.int64) - len(tail_rows)  # the GPU counts the recent tokens
    for h in range(G):
        kg, ko = int(k_gpu[h]), int(r.k[h])
        if kg == ko:
            continue
        info = r.infos[h]
        S, T = info["S"], info.get("T", None)
        assert T is not None and 0 <= kg <= n, f"{label} head {h}: k gpu {kg} oracle {ko}"
        E_t = info.get("E_t", 0.0)

        def reach(k):  # mass of the recent tokens and the first k listed ones
            return S[k - 1] if k >= 1 else E_t
        ok = reach(kg) >= T * (1 - CUT_TIE_REL) and (kg == 0 or reach(kg - 1) < T * (1 + CUT_TIE_REL))
        assert ok, f"{label} head {h}: k gpu {kg} oracle {ko} (S_kg={S[kg-1]}, T={T})"
        stats["cut_ties"] += 1
    # union of the GPU's per-head selections, as per-cluster prefix lengths
    sel_rows = [np.concatenate([r.rows[h][:int(k_gpu[h])], tail_rows]) for h in range(G)]
    if not use_union:
        loaded = 0
        err = 0.0
        for h in range(G):
            I = np.sort(sel_rows[h])
            ug = np.asarray(gpu["union_len"][h][:C], dtype=np.int64)
            assert np.array_equal(_cluster_lengths(I, off, C), ug), f"{label} head {h}: selection differs"
            loaded += len(I)
            ref = OA.sparse_attention(Q[h], Ks, Vs, I) if len(I) else np.zeros(Q.shape[1])
            err = max(err, float(np.max(np.abs(gpu["out"][h] - ref))))
        assert int(gpu["sel_kv"]) == loaded, f"{label}: loaded gpu {int(gpu['sel_kv'])} oracle {loaded}"
        assert err <= OUT_ATOL, f"{label}: output max-abs error {err} > {OUT_ATOL}"
        stats.update(out_err=err, k=k_gpu.tolist(), union=loaded, n=n, result=r)
        return stats
    U = np.unique(np.concatenate(sel_rows)) if G else np.zeros(0, np.int64)
    clus = np.searchsorted(off, U, side="right") - 1 if len(U) else np.zeros(0, np.int64)
    ulen = np.bincount(clus, minlength=C)[:C] if len(U) else np.zeros(C, np.int64)
    ug = np.asarray(gpu["union_len"][:C], dtype=np.int64)
    assert np.array_equal(ulen, ug), f"{label}: union differs in {int(np.sum(ulen != ug))} clusters"
    assert int(gpu["sel_kv"]) == len(U), f"{label}: |U| gpu {int(gpu['sel_kv'])} oracle {len(U)}"
    # output over the GPU's union
    err = 0.0
    for h in range(G):
        ref = OA.sparse_attention(Q[h], Ks, Vs, U) if len(U) else np.zeros(Q.shape[1])
        err = max(err, float(np.max(np.abs(gpu["out"][h] - ref))))
    assert err <= OUT_ATOL, f"{label}: output max-abs error {err} > {OUT_ATOL}"
    stats["out_err"] = err
    stats["k"] = k_gpu.tolist()
    stats["union"] = len(U)
    stats["n"] = n
    stats["result"] = r  # the oracle's decode on the GPU's order (GroupResult)
    return stats
