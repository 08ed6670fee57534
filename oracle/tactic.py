"""Tactic decode path in plain fp64 (test infrastructure only).

Follows the method section (Sec. 4.3 querying, Sec. 4.4 distribution fitting
with Algorithm 1, Sec. 4.5 GQA union, Sec. 4.6 attention on the selected
tokens).  Readings of points the paper leaves open are stated where they are
used; each is a parameter or a rule, never a tuning.

Layout of one (sequence, KV head): the cache rows are stored cluster by
cluster (cluster j owns rows offsets[j] .. offsets[j+1]-1, its tokens in
ascending original token order), so a token is named by its row in that
cluster-sorted cache.  Rows past the last cluster (offsets[-1] .. n-1) are
the recent tokens generated since the clustering: they are not clustered and
every head attends to all of them (Sec. 1: full attention on newly generated
tokens until the next re-clustering).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from .attention import logits as _logits, sparse_attention, softmax_weights


@dataclass(frozen=True)
class FitParams:
    """Integer parameters of the distribution fit, in basis points (1e-4).

    exact_bp  exact head N = ceil(n * exact_bp / 1e4), at least 1 (Sec. 4.4:
              the first 1-2% of tokens are outliers and get exact scores).
    win_bp,   window width W = max(win_min, ceil(n * win_bp / 1e4)); the paper
    win_min   does not size its windows, this reading makes the centroids plus
              the sampled keys about 2.5% of the KV bytes (Sec. 1).
    p1_bp,    window centres at 10% and 60% of the token list (Sec. 4.4):
    p2_bp     c = floor((n * p_bp + 5000) / 1e4), 1-based.
    """

    exact_bp: int = 100
    win_bp: int = 50
    win_min: int = 8
    p1_bp: int = 1000
    p2_bp: int = 6000


def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


@dataclass(frozen=True)
class Geometry:
    n: int
    N: int
    W: int
    s1: int
    t1: int
    s2: int
    t2: int
    exact: bool


def geometry(n: int, prm: FitParams = FitParams()) -> Geometry:
    """Exact head and the two sampling windows for a list of n tokens.

    Window j spans 1-based positions s_j..t_j with s_j = max(c_j - floor(W/2),
    N + 1) and t_j = min(s_j + W - 1, n).  When a window is empty, the two
    overlap, or the exact head covers every token, the fit is skipped and all
    n scores are computed exactly ("exact mode")."""
    N = min(n, max(1, _ceil_div(n * prm.exact_bp, 10000)))
    W = max(prm.win_min, _ceil_div(n * prm.win_bp, 10000))
    c1 = (n * prm.p1_bp + 5000) // 10000
    c2 = (n * prm.p2_bp + 5000) // 10000
    s1 = max(c1 - W // 2, N + 1)
    t1 = min(s1 + W - 1, n)
    s2 = max(c2 - W // 2, N + 1)
    t2 = min(s2 + W - 1, n)
    exact = (N == n) or (s1 > t1) or (s2 > t2) or (t1 >= s2)
    return Geometry(n, N, W, s1, t1, s2, t2, exact)


def rank_clusters(q: np.ndarray, centroids: np.ndarray):
    """Cluster criticality is the dot product of the query with the centroid
    (Sec. 4.3 and its footnote).  Returns (scores, order) with order sorted by
    descending score, ties broken by ascending cluster id.  Empty clusters
    are ranked like any other (they contribute no tokens)."""
    s = centroids @ q
    order = np.lexsort((np.arange(len(s)), -s))
    return s, order


def unpack(order: np.ndarray, offsets: np.ndarray) -> np.ndarray:
    """The partially sorted token list x_1..x_n (Sec. 4.3; Algorithm 1's
    input): the tokens of the ranked clusters in rank order, each cluster's
    tokens in stored order.  Returns cache rows, position i-1 -> row."""
    parts = [np.arange(offsets[c], offsets[c + 1], dtype=np.int64) for c in order]
    if not parts:
        return np.zeros(0, dtype=np.int64)
    return np.concatenate(parts)


def estimate_budget(l_pos: np.ndarray, P: float, prm: FitParams = FitParams(),
                    l_tail: Optional[np.ndarray] = None):
    """Algorithm 1: the token budget k for one query head.

    l_pos are the logits x_i . Q / sqrt(d) of the unpacked list, in position
    order.  Scores are handled relative to m = max of the exact head (and of
    the recent tokens, when there are any); every quantity below scales by
    exp(-m), which leaves k unchanged.

    l_tail, if given, are the logits of the recent unclustered tokens.  They
    are always selected, so their exact mass E_t counts toward the target:
    the total is E_t + S_n and k is the minimal k >= 0 with
    E_t + S_k >= P * (E_t + S_n) (reading: the paper attends to these tokens
    in full but does not say how they enter the budget).

    1. Means mu_1, mu_2 of exp(l - m) over the two windows, at x-coordinates
       x_j = (s_j + t_j) / 2; solve y = a/x + b through (x_1, mu_1), (x_2, mu_2).
    2. w_i = exp(l_i - m) for i <= N, else max(0, a/i + b) (a negative fitted
       score is read as zero).
    3. k = minimal k with sum_{i<=k} w_i >= P * sum_{i<=n} w_i, sums taken
       sequentially.  P >= 1 selects all n tokens.
    """
    n = len(l_pos)
    geo = geometry(n, prm)
    info = dict(n=n, N=geo.N, W=geo.W, s1=geo.s1, t1=geo.t1, s2=geo.s2, t2=geo.t2,
                exact=geo.exact)
    has_tail = l_tail is not None and len(l_tail) > 0
    if n == 0:
        info["k"] = 0
        info["E_t"] = 0.0
        return 0, info
    m = float(np.max(l_pos[:geo.N]))
    if has_tail:
        m = max(m, float(np.max(l_tail)))
    E_t = float(np.sum(np.exp(l_tail - m))) if has_tail else 0.0
    info["m"] = m
    info["E_t"] = E_t
    if geo.exact:
        w = np.exp(l_pos - m)
    else:
        e = np.exp(l_pos[:geo.N] - m)
        mu1 = float(np.mean(np.exp(l_pos[geo.s1 - 1:geo.t1] - m)))
        mu2 = float(np.mean(np.exp(l_pos[geo.s2 - 1:geo.t2] - m)))
        x1 = (geo.s1 + geo.t1) / 2.0
        x2 = (geo.s2 + geo.t2) / 2.0
        a = (mu1 - mu2) / (1.0 / x1 - 1.0 / x2)
        b = mu1 - a / x1
        i = np.arange(geo.N + 1, n + 1, dtype=np.float64)
        w = np.concatenate([e, np.maximum(0.0, a / i + b)])
        info.update(mu1=mu1, mu2=mu2, x1=x1, x2=x2, a=a, b=b)
    S = np.add.accumulate(w)
    if has_tail:
        S = E_t + S  # cumulative mass of the recent tokens plus the first k listed ones
    info["S_n"] = float(S[-1])
    if P >= 1.0:
        k = n
    else:
        T = P * S[-1]
        info["T"] = float(T)
        k = 0 if (has_tail and E_t >= T) else int(np.argmax(S >= T)) + 1
    info["k"] = k
    info["w"] = w
    info["S"] = S
    return k, info


@dataclass
class GroupResult:
    out: np.ndarray                  # (G, d) attention output per query head
    k: np.ndarray                    # (G,) token budget per query head
    sel: List[np.ndarray]            # per head: selected rows, in position order
    union: np.ndarray                # sorted rows of the union
    orders: List[np.ndarray]         # per head: cluster order
    rows: List[np.ndarray]           # per head: unpacked list (position -> row)
    infos: List[dict] = field(default_factory=list)

    @property
    def union_count(self) -> int:
        return int(len(self.union))


def decode_group(Q: np.ndarray, Ks: np.ndarray, Vs: np.ndarray, centroids: np.ndarray,
                 offsets: np.ndarray, P: float, prm: FitParams = FitParams(),
                 use_union: bool = True, orders: Optional[List[np.ndarray]] = None) -> GroupResult:
    """Tactic's decode for the G query heads sharing one KV head (Sec. 4.3-4.6).

    Q (G, d) queries; Ks, Vs (n, d) the cluster-sorted cache of this sequence
    and KV head; centroids (C, d); offsets (C+1,).  `orders`, if given,
    replaces the computed cluster order of each head (used to evaluate the
    rest of the path on an order produced elsewhere).

    Each head ranks the clusters, unpacks them, estimates its budget k_h and
    selects the first k_h tokens I_h.  With the union (Sec. 4.5) every head of
    the group attends over U = union of the I_h, loaded once; without it each
    head attends over its own I_h.  Rows of Ks past offsets[-1] are the recent
    tokens: every I_h contains them and they enter the budget with their exact
    mass (estimate_budget).  An empty sequence yields zeros."""
    G, d = Q.shape
    n = int(offsets[-1])
    n_all = int(Ks.shape[0])
    tail = np.arange(n, n_all, dtype=np.int64)
    if n_all == 0:
        z = np.zeros(0, dtype=np.int64)
        return GroupResult(out=np.zeros((G, d)), k=np.zeros(G, dtype=np.int64), sel=[z] * G,
                           union=z, orders=[np.zeros(0, dtype=np.int64)] * G, rows=[z] * G)
    ks, sels, ords, rowss, infos = [], [], [], [], []
    for h in range(G):
        q = Q[h]
        if orders is None:
            _, order = rank_clusters(q, centroids)
        else:
            order = np.asarray(orders[h], dtype=np.int64)
        rows = unpack(order, offsets)
        l_pos = _logits(q, Ks[rows])
        k, info = estimate_budget(l_pos, P, prm, _logits(q, Ks[tail]) if len(tail) else None)
        if n == 0:  # nothing is clustered: the recent tokens are the whole selection
            k = 0
        ks.append(k)
        sels.append(np.concatenate([rows[:k], tail]))
        ords.append(order)
        rowss.append(rows)
        infos.append(info)
    union = np.unique(np.concatenate(sels))
    out = np.zeros((G, d))
    for h in range(G):
        idx = union if use_union else np.sort(sels[h])
        out[h] = sparse_attention(Q[h], Ks, Vs, idx)
    return GroupResult(out=out, k=np.asarray(ks, dtype=np.int64), sel=sels, union=union,
                       orders=ords, rows=rowss, infos=infos)


def decode(q: np.ndarray, K_sorted: np.ndarray, V_sorted: np.ndarray, centroids: np.ndarray,
           offsets: np.ndarray, kv_indptr, cl_indptr, P: float, prm: FitParams = FitParams(),
           use_union: bool = True, groups=None):
    """Batched decode over a ragged batch.

    q (B, Hq, d); K_sorted, V_sorted (Hkv, total, d); centroids
    (Hkv, total_clusters, d); offsets (Hkv, total_clusters + B): sequence b's
    C_b + 1 offsets start at cl_indptr[b] + b.  Query head h uses KV head
    h // (Hq / Hkv).  `groups` restricts the work to a list of (b, g).

    Returns (out (B, Hq, d), k (B, Hq), union_count (B, Hkv), results dict
    keyed by (b, g))."""
    B, Hq, d = q.shape
    Hkv = K_sorted.shape[0]
    G = Hq // Hkv
    out = np.zeros((B, Hq, d))
    kq = np.zeros((B, Hq), dtype=np.int64)
    ukv = np.zeros((B, Hkv), dtype=np.int64)
    res = {}
    todo = groups if groups is not None else [(b, g) for b in range(B) for g in range(Hkv)]
    for b, g in todo:
        s0, s1 = int(kv_indptr[b]), int(kv_indptr[b + 1])
        c0, c1 = int(cl_indptr[b]), int(cl_indptr[b + 1])
        off = np.asarray(offsets[g, c0 + b:c1 + b + 1], dtype=np.int64)
        r = decode_group(q[b, g * G:(g + 1) * G], K_sorted[g, s0:s1], V_sorted[g, s0:s1],
                         centroids[g, c0:c1], off, P, prm, use_union)
        out[b, g * G:(g + 1) * G] = r.out
        kq[b, g * G:(g + 1) * G] = r.k
        ukv[b, g] = r.union_count
        res[(b, g)] = r
    return out, kq, ukv, res


def selection_report(q: np.ndarray, Ks: np.ndarray, Vs: np.ndarray, r: GroupResult, P: float,
                     h: int) -> dict:
    """Diagnostics for one head (not compared with the GPU): the true
    cumulative score of I_h and of the union (Eq. 5), the optimal budget
    (exact top-P, Sec. 3.4), the "cluster optimal" budget (true scores taken
    in cluster order), the attention distance (Eq. 4) and its bound (Eq. 6)."""
    s = softmax_weights(_logits(q, Ks))
    p_sel = float(s[r.sel[h]].sum())
    p_union = float(s[r.union].sum())

    def first_reaching(cum: np.ndarray, target: float) -> int:
        # fewest leading tokens whose mass reaches the target; all of them
        # when rounding leaves the full sum a hair below it (P = 1)
        hit = np.nonzero(cum >= target)[0]
        return int(hit[0]) + 1 if len(hit) else len(cum)

    k_opt = first_reaching(np.add.accumulate(np.sort(s)[::-1]), P)
    # Cluster-Optimal: the true scores of the clustered tokens taken in the
    # head's cluster order, against P of their total
    cs = np.add.accumulate(s[r.rows[h]])
    k_cluster = first_reaching(cs, P * cs[-1]) if len(cs) else 0
    o = s @ Vs
    eps = float(np.linalg.norm(o - r.out[h]))
    bound = 2.0 * (1.0 - p_union) * float(np.max(np.linalg.norm(Vs, axis=1)))
    return dict(k=int(r.k[h]), union=r.union_count, p_sel=p_sel, p_union=p_union,
                k_optimal=k_opt, k_cluster_optimal=k_cluster, eps=eps, bound=bound)
