"""Pins of the fp64 oracle against what the paper and the mathematics fix.

CPU only.  Each test names the passage it pins.  None of them re-types the
oracle's own formula: they use hand-derived values (tests/golden), exact
rational arithmetic, brute force on tiny inputs, an independent library
(torch SDPA, scipy K-means, torch's bf16 cast, NumPy's stable sort) or an
invariant that must hold for any input.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import kmeans as KM
from oracle import numerics as NUM
from oracle import tactic as T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _frac(s):
    return float(Fraction(s))


# ---------------------------------------------------------------- numerics

def test_round_bf16_matches_torch_cast():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000),
                        [0.0, 1.0, -1.0, 1.00390625, 1.001953125, 1.005859375]])
    x32 = x.astype(np.float32).astype(np.float64)
    ref = torch.tensor(x32, dtype=torch.float32).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(NUM.round_bf16(x32), ref)


# ---------------------------------------------------------------- attention (Eq. 2-6)

def test_dense_attention_matches_torch_sdpa():
    rng = np.random.default_rng(1)
    for n in (1, 7, 300):
        q = rng.standard_normal(128) * 2
        K = rng.standard_normal((n, 128))
        V = rng.standard_normal((n, 128))
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.tensor(q)[None, None, None], torch.tensor(K)[None, None],
            torch.tensor(V)[None, None])[0, 0, 0].numpy()
        np.testing.assert_allclose(A.dense_attention(q, K, V), ref, rtol=0, atol=1e-12)


def test_error_bound_eq6_holds_for_any_subset():
    """Appendix A: eps(I) <= 2 (1 - p(I)) max ||v|| for every I."""
    rng = np.random.default_rng(2)
    for trial in range(200):
        n = int(rng.integers(1, 40))
        q = rng.standard_normal(128) * rng.uniform(0.1, 3)
        K = rng.standard_normal((n, 128))
        V = rng.standard_normal((n, 128)) * rng.uniform(0.1, 5)
        idx = rng.choice(n, size=int(rng.integers(1, n + 1)), replace=False)
        assert A.attention_distance(q, K, V, idx) <= A.error_bound(q, K, V, idx) + 1e-12


def test_optimal_selection_is_minimum_cardinality_bruteforce():
    """Sec. 1 / 3.4: the descending-score prefix is a smallest set reaching P."""
    rng = np.random.default_rng(3)
    for trial in range(60):
        n = int(rng.integers(1, 11))
        q = rng.standard_normal(128) * rng.uniform(0.2, 3)
        K = rng.standard_normal((n, 128))
        P = float(rng.uniform(0.05, 0.99))
        s = A.softmax_weights(A.logits(q, K))
        best = None
        for size in range(1, n + 1):
            if any(s[list(c)].sum() >= P for c in itertools.combinations(range(n), size)):
                best = size
                break
        sel = A.optimal_selection(q, K, P)
        assert len(sel) == best
        assert s[sel].sum() >= P


# ---------------------------------------------------------------- geometry (Sec. 4.4 reading)

@pytest.mark.parametrize("n,expect", [
    (4096, (41, 21, 400, 420, 2448, 2468, False)),
    (131072, (1311, 656, 12779, 13434, 78315, 78970, False)),
    (10, (1, 8, 2, 9, 2, 9, True)),
    (1, (1, 8, 2, 1, 2, 1, True)),
])
def test_geometry_hand_values(n, expect):
    g = T.geometry(n)
    assert (g.N, g.W, g.s1, g.t1, g.s2, g.t2, g.exact) == expect


# ---------------------------------------------------------------- Algorithm 1

def _harmonic_sum(a: Fraction, b: Fraction, lo: int, hi: int) -> Fraction:
    return sum((max(Fraction(0), a / i + b) for i in range(lo, hi + 1)), Fraction(0))


def test_fit_recovers_exact_curve_and_cutoff_matches_rational_arithmetic():
    """Algorithm 1 on a list whose tail follows y = a/x + b exactly.

    With one-token windows the two sampled means lie on the curve, so the fit
    must recover (a, b) and the budget must equal the one obtained with exact
    rational arithmetic on the closed-form scores."""
    prm = T.FitParams(exact_bp=100, win_bp=0, win_min=1)
    a, b = Fraction(1, 2), Fraction(1, 100)
    for n in (200, 1000, 5000):
        g = T.geometry(n, prm)
        assert not g.exact and g.s1 == g.t1 and g.s2 == g.t2
        m = 5.0
        head = [m] + [m - 1.0 - 0.01 * i for i in range(1, g.N)]
        tail = [m + math.log(float(a) / i + float(b)) for i in range(g.N + 1, n + 1)]
        l_pos = np.array(head + tail)
        for P in (0.3, 0.5, 0.8, 0.9, 0.97):
            k, info = T.estimate_budget(l_pos, P, prm)
            assert abs(info["a"] - float(a)) < 1e-9 and abs(info["b"] - float(b)) < 1e-9
            E = [Fraction(math.exp(x - m)) for x in head]
            S_n = sum(E, Fraction(0)) + _harmonic_sum(a, b, g.N + 1, n)
            target = Fraction(P) * S_n
            acc, k_exact = Fraction(0), None
            for i in range(1, n + 1):
                acc += E[i - 1] if i <= g.N else a / i + b
                if acc >= target:
                    k_exact = i
                    break
            # no rational S_k lies within 1e-9 of the target for these inputs
            assert k == k_exact, (n, P, k, k_exact)


def _window_mean_exact(a: Fraction, b: Fraction, s: int, t: int) -> Fraction:
    """Mean of a/i + b over the integers s..t: (a (H_t - H_{s-1}) + b W) / W."""
    W = t - s + 1
    return (a * sum((Fraction(1, i) for i in range(s, t + 1)), Fraction(0)) + b * W) / W


WINDOWED_CASES = [
    (600, dict()),                                     # W = 8 (the minimum)
    (1700, dict()),                                    # W = 9
    (2000, dict(win_bp=400)),                          # W = 80
    (1200, dict(exact_bp=200, win_bp=300, p1_bp=1500, p2_bp=5000)),
]


def pin_windowed_fit_exact(T):
    """Algorithm 1 with real windows (W >= 8) on a list whose tail follows
    y = a/x + b exactly.  Each window's point is the mean of the scores over
    its positions placed at the window's middle position (Sec. 4.4: means
    within windows around p1 and p2).  Since 1/x is convex that mean is not
    a/x_mid + b, so the fit gives other coefficients (a', b'); they, the two
    means and the budget must equal the values exact rational arithmetic
    gives from those definitions."""
    checked = 0
    for n, kw in WINDOWED_CASES:
        prm = T.FitParams(**kw)
        g = T.geometry(n, prm)
        assert not g.exact and g.t1 - g.s1 + 1 >= 8 and g.t2 - g.s2 + 1 >= 8
        a, b = Fraction(g.N, 2), Fraction(1, 64)
        m = 3.0
        head = [m] + [m - 0.05 - 0.6 * i / g.N for i in range(1, g.N)]
        tail = [m + math.log(float(a) / i + float(b)) for i in range(g.N + 1, n + 1)]
        l_pos = np.array(head + tail)
        mu1 = _window_mean_exact(a, b, g.s1, g.t1)
        mu2 = _window_mean_exact(a, b, g.s2, g.t2)
        x1, x2 = Fraction(g.s1 + g.t1, 2), Fraction(g.s2 + g.t2, 2)
        a2 = (mu1 - mu2) / (1 / x1 - 1 / x2)
        b2 = mu1 - a2 / x1
        E = [Fraction(math.exp(x - m)) for x in head]
        w = E + [max(Fraction(0), a2 / i + b2) for i in range(g.N + 1, n + 1)]
        S, acc = [], Fraction(0)
        for x in w:
            acc += x
            S.append(acc)
        for P in (0.3, 0.5, 0.7, 0.8, 0.9, 0.97):
            k, info = T.estimate_budget(l_pos, P, prm)
            assert abs(info["mu1"] - float(mu1)) <= 1e-12 * float(mu1), (n, kw, info["mu1"], float(mu1))
            assert abs(info["mu2"] - float(mu2)) <= 1e-12 * float(mu2), (n, kw, info["mu2"], float(mu2))
            assert abs(info["a"] - float(a2)) <= 1e-9 * abs(float(a2)), (n, kw, info["a"], float(a2))
            assert abs(info["b"] - float(b2)) <= 1e-9 * abs(float(a2)) / n, (n, kw, info["b"], float(b2))
            target = Fraction(P) * S[-1]
            k_exact = next(i for i, x in enumerate(S, start=1) if x >= target)
            # compare only where no cumulative sum lies within 1e-9 of the target
            margin = min(abs(S[k_exact - 1] - target), abs(target - S[k_exact - 2]) if k_exact > 1 else 1)
            if margin > Fraction(1, 10 ** 9) * S[-1]:
                assert k == k_exact, (n, kw, P, k, k_exact)
                checked += 1
    assert checked >= 20


def test_windowed_fit_matches_exact_arithmetic():
    pin_windowed_fit_exact(T)


def test_constant_tail_budget_closed_form():
    """a = 0: w is constant b beyond the head, so the budget is
    N + ceil((P S_n - E_N) / b) when the target lies beyond the head."""
    n = 3000
    g = T.geometry(n)
    m = 2.0
    head = np.array([m] + [m - 0.5] * (g.N - 1))
    lb = m + math.log(0.25)
    l_pos = np.concatenate([head, np.full(n - g.N, lb)])
    for P in (0.2, 0.6, 0.95):
        k, info = T.estimate_budget(l_pos, P, T.FitParams())
        assert abs(info["a"]) < 1e-12
        E_N = 1.0 + (g.N - 1) * math.exp(-0.5)
        S_n = E_N + 0.25 * (n - g.N)
        assert k == g.N + math.ceil((P * S_n - E_N) / 0.25)


def test_budget_invariants_random():
    """Algorithm 1: S_k >= P S_n and S_{k-1} < P S_n (minimality); P = 1 takes all."""
    rng = np.random.default_rng(4)
    for trial in range(300):
        n = int(rng.integers(1, 3000))
        l_pos = np.sort(rng.standard_normal(n) * rng.uniform(0.1, 6))[::-1] + rng.standard_normal(n) * 0.3
        P = float(rng.uniform(0.01, 0.999))
        k, info = T.estimate_budget(l_pos, P)
        S = info["S"]
        assert 1 <= k <= n
        assert S[k - 1] >= P * S[-1]
        if k > 1:
            assert S[k - 2] < P * S[-1]
        assert np.all(info["w"] >= 0)
        k1, _ = T.estimate_budget(l_pos, 1.0)
        assert k1 == n


def test_one_cluster_per_token_exact_mode_is_top_p():
    """One cluster per token (centroid = key) ranks tokens exactly; with every
    score exact the selection must be the textbook top-P prefix."""
    rng = np.random.default_rng(5)
    prm = T.FitParams(exact_bp=10000)
    for trial in range(40):
        n = int(rng.integers(1, 200))
        q = rng.standard_normal(128) * rng.uniform(0.3, 3)
        K = rng.standard_normal((n, 128))
        V = rng.standard_normal((n, 128))
        P = float(rng.uniform(0.05, 0.99))
        offsets = np.arange(n + 1)
        r = T.decode_group(q[None], K, V, K, offsets, P, prm)
        ref = A.optimal_selection(q, K, P)
        assert r.k[0] == len(ref)
        assert set(r.sel[0].tolist()) == set(ref.tolist())
        np.testing.assert_allclose(r.out[0], A.sparse_attention(q, K, V, np.sort(ref)), atol=1e-12)


# ---------------------------------------------------------------- whole group (Sec. 4.3-4.6)

def _golden_inputs(fx):
    d = fx["d"]
    key0 = [{"ln4": math.log(4), "ln2": math.log(2), "0": 0.0}[s] for s in fx["key0"]]
    n = len(key0)
    K = np.zeros((n, d))
    K[:, 0] = key0
    V = np.zeros((n, d))
    V[np.arange(n), np.arange(n)] = 1.0
    Q = np.zeros((len(fx["q_signs"]), d))
    Q[:, 0] = np.array(fx["q_signs"]) * math.sqrt(d)
    cent = np.zeros((2, d))
    cent[0, 0] = 1.0
    return Q, K, V, cent, np.array(fx["offsets"])


def pin_golden_pipeline(T):
    with open(os.path.join(GOLDEN, "tiny_exact.json")) as f:
        fx = json.load(f)
    Q, K, V, cent, off = _golden_inputs(fx)
    for case in fx["cases"]:
        for use_union, key in ((True, "out_union"), (False, "out_per_head")):
            r = T.decode_group(Q, K, V, cent, off, case["P"], use_union=use_union)
            assert r.k.tolist() == case["k"]
            assert r.union.tolist() == case["union"]
            exp = np.array([[_frac(x) for x in row] for row in case[key]])
            np.testing.assert_allclose(r.out[:, :4], exp, rtol=0, atol=1e-12)
            assert np.all(r.out[:, 4:] == 0)


def pin_golden_report(T):
    """Sec. 5.2's diagnostics on the worked example: p(I_h) and p(U) (Eq. 5),
    the Optimal and Cluster-Optimal budgets, the attention distance (Eq. 4)
    and its bound (Eq. 6), each derived by hand in tests/golden."""
    with open(os.path.join(GOLDEN, "tiny_exact.json")) as f:
        fx = json.load(f)
    Q, K, V, cent, off = _golden_inputs(fx)
    for case in fx["cases"]:
        r = T.decode_group(Q, K, V, cent, off, case["P"])
        for h, want in enumerate(case["report"]):
            got = T.selection_report(Q[h], K, V, r, case["P"], h)
            assert got["k_optimal"] == want["k_optimal"], (case["P"], h, got)
            assert got["k_cluster_optimal"] == want["k_cluster_optimal"], (case["P"], h, got)
            assert abs(got["p_sel"] - _frac(want["p_sel"])) <= 1e-12, (case["P"], h, got)
            assert abs(got["p_union"] - _frac(want["p_union"])) <= 1e-12, (case["P"], h, got)
            assert abs(got["eps"] ** 2 - _frac(want["eps_sq"])) <= 1e-12, (case["P"], h, got)
            assert abs(got["bound"] - _frac(want["bound"])) <= 1e-12, (case["P"], h, got)


def test_golden_tiny_exact_pipeline():
    pin_golden_pipeline(T)


def test_golden_tiny_exact_report():
    pin_golden_report(T)


def _random_clustered_group(rng, n, C, G=4, d=128):
    cen = rng.standard_normal((C, d))
    lab = rng.integers(0, C, n)
    K = cen[lab] + 0.3 * rng.standard_normal((n, d))
    perm = np.argsort(lab, kind="stable")
    Ks = K[perm]
    Vs = rng.standard_normal((n, d))
    offsets = np.zeros(C + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(np.bincount(lab, minlength=C))
    Q = np.stack([2.0 * (cen[rng.choice(C, min(3, C), replace=False)].sum(0) + 0.3 * rng.standard_normal(d))
                  for _ in range(G)])
    return Q, Ks, Vs, cen, offsets


def test_union_invariants():
    """Sec. 4.5: U contains every I_h, |U| <= sum k_h, and U meets every
    cluster in a prefix of its stored rows; each I_h is a prefix of the
    head's unpacked list."""
    rng = np.random.default_rng(6)
    for trial in range(20):
        n = int(rng.integers(50, 3000))
        C = max(1, n // 16)
        Q, Ks, Vs, cen, off = _random_clustered_group(rng, n, C)
        r = T.decode_group(Q, Ks, Vs, cen, off, float(rng.uniform(0.5, 0.99)))
        U = set(r.union.tolist())
        for h in range(len(Q)):
            assert set(r.sel[h].tolist()) <= U
            np.testing.assert_array_equal(r.sel[h], r.rows[h][:r.k[h]])
        assert len(U) <= int(r.k.sum())
        for j in range(C):
            inside = [row for row in range(off[j], off[j + 1]) if row in U]
            assert inside == list(range(off[j], off[j] + len(inside)))


def test_target_one_equals_dense_attention():
    """P = 1 selects all tokens; the output is dense attention (Eq. 2), here
    checked against torch's SDPA."""
    rng = np.random.default_rng(7)
    n, C = 700, 40
    Q, Ks, Vs, cen, off = _random_clustered_group(rng, n, C)
    r = T.decode_group(Q, Ks, Vs, cen, off, 1.0)
    assert r.k.tolist() == [n] * len(Q)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(Q)[None, :, None], torch.tensor(Ks)[None, None].expand(1, len(Q), n, 128),
        torch.tensor(Vs)[None, None].expand(1, len(Q), n, 128))[0, :, 0].numpy()
    np.testing.assert_allclose(r.out, ref, atol=1e-12)


def test_decode_matches_loop_reimplementation_tiny():
    """A loop-only re-implementation (pairwise ranking, explicit position
    walk, explicit window sums) for n <= 64 agrees with the vectorised
    oracle on k and on the union."""
    rng = np.random.default_rng(8)
    for trial in range(30):
        n = int(rng.integers(1, 65))
        C = int(rng.integers(1, min(n, 9) + 1))
        Q, Ks, Vs, cen, off = _random_clustered_group(rng, n, C, G=2)
        P = float(rng.uniform(0.2, 0.98))
        r = T.decode_group(Q, Ks, Vs, cen, off, P)
        d = Ks.shape[1]
        union = set()
        for h in range(2):
            q = Q[h]
            sc = [float(np.dot(q, cen[j])) for j in range(C)]
            rank = sorted(range(C), key=lambda j: (-sc[j], j))
            pos_rows = []
            for j in rank:
                for row in range(off[j], off[j + 1]):
                    pos_rows.append(row)
            lg = [float(np.dot(q, Ks[row])) / math.sqrt(d) for row in pos_rows]
            N = min(n, max(1, -(-n * 100 // 10000)))
            W = max(8, -(-n * 50 // 10000))
            c1, c2 = (n * 1000 + 5000) // 10000, (n * 6000 + 5000) // 10000
            s1 = max(c1 - W // 2, N + 1); t1 = min(s1 + W - 1, n)
            s2 = max(c2 - W // 2, N + 1); t2 = min(s2 + W - 1, n)
            m = max(lg[:N])
            if N == n or s1 > t1 or s2 > t2 or t1 >= s2:
                w = [math.exp(x - m) for x in lg]
            else:
                mu1 = sum(math.exp(lg[i - 1] - m) for i in range(s1, t1 + 1)) / (t1 - s1 + 1)
                mu2 = sum(math.exp(lg[i - 1] - m) for i in range(s2, t2 + 1)) / (t2 - s2 + 1)
                x1, x2 = (s1 + t1) / 2, (s2 + t2) / 2
                a = (mu1 - mu2) / (1 / x1 - 1 / x2)
                b = mu1 - a / x1
                w = [math.exp(lg[i - 1] - m) if i <= N else max(0.0, a / i + b) for i in range(1, n + 1)]
            tot = 0.0
            for x in w:
                tot += x
            acc, k = 0.0, n
            for i, x in enumerate(w, start=1):
                acc += x
                if acc >= P * tot:
                    k = i
                    break
            assert r.k[h] == k
            union |= set(pos_rows[:k])
        assert set(r.union.tolist()) == union


def test_empty_sequence_yields_zeros():
    Q = np.ones((4, 128))
    r = T.decode_group(Q, np.zeros((0, 128)), np.zeros((0, 128)), np.ones((1, 128)),
                       np.array([0, 0]), 0.9)
    assert r.k.tolist() == [0, 0, 0, 0] and r.union_count == 0 and np.all(r.out == 0)


# ---------------------------------------------------------------- K-means (Sec. 4.2)

def test_kmeans_single_cluster_is_mean():
    rng = np.random.default_rng(9)
    K = rng.standard_normal((500, 128))
    r = KM.kmeans(K, [17], round_storage=False)
    assert np.all(r.assign == 0)
    np.testing.assert_allclose(r.centroids[0], K.mean(0), atol=1e-14)
    r2 = KM.kmeans(K, [17], round_storage=True)
    np.testing.assert_array_equal(r2.centroids[0], NUM.round_bf16(K.mean(0)))


def test_kmeans_one_cluster_per_token_is_identity():
    rng = np.random.default_rng(10)
    K = rng.standard_normal((64, 128))
    r = KM.kmeans(K, np.arange(64))
    np.testing.assert_array_equal(r.assign, np.arange(64))
    assert r.iters == 2


def test_kmeans_matches_scipy_lloyd():
    """Without bf16 storage the iteration is Lloyd's algorithm, which
    scipy.cluster.vq.kmeans2(minit='matrix') also runs.  Its default for a
    cluster that loses all members (missing='warn': warn, keep the previous
    centroid) is the empty-cluster reading of Sec. 4.2 taken here, so trials
    with and without an emptied cluster must both give identical results;
    the seeds below produce both kinds."""
    import warnings
    from scipy.cluster.vq import kmeans2
    rng = np.random.default_rng(11)
    kinds = set()
    for trial in range(5):
        C, per = 12, 30
        cen = rng.standard_normal((C, 16)) * 4
        K = np.concatenate([cen[j] + rng.standard_normal((per, 16)) for j in range(C)])
        K = K[rng.permutation(len(K))]
        init = rng.choice(len(K), C, replace=False)
        r = KM.kmeans(K, init, max_iters=10, round_storage=False)
        with warnings.catch_warnings(record=True) as caught:
            warnings.simplefilter("always")
            cb, lab = kmeans2(K, K[init].copy(), iter=10, minit="matrix")
        emptied = any("empty" in str(w.message) for w in caught)
        kinds.add(emptied)
        if not emptied:
            assert np.bincount(r.assign, minlength=C).min() > 0
        np.testing.assert_array_equal(r.assign, lab)
        np.testing.assert_allclose(r.centroids, cb, atol=1e-12)
    assert kinds == {True, False}


def test_kmeans_warm_start_from_converged_clustering_is_a_fixed_point():
    """Re-clustering (Sec. 1) from a clustering that has converged (its last
    assignment step changed nothing) must stop at the second assignment of
    the new run with the same assignment and the same stored centroids."""
    rng = np.random.default_rng(21)
    C, per = 16, 40
    cen = rng.standard_normal((C, 16)) * 3
    K = NUM.round_bf16(np.concatenate([cen[j] + rng.standard_normal((per, 16)) for j in range(C)]))
    r0 = KM.kmeans(K, rng.choice(len(K), C, replace=False), max_iters=200)
    assert r0.iters < 200, "the cold run must converge for this pin"
    garbage = np.full(C, len(K) - 1)  # ignored: every centroid is warm-started
    r1 = KM.kmeans(K, garbage, max_iters=10, prev_centroids=r0.centroids)
    assert r1.iters == 2
    np.testing.assert_array_equal(r1.assign, r0.assign)
    np.testing.assert_array_equal(r1.centroids, r0.centroids)


def test_kmeans_warm_start_takes_the_prefix_from_the_previous_centroids():
    """Centroid j starts from the previous clustering's centroid j below both
    counts and from init_idx above: previous centroids equal to the keys of
    the first init tokens reproduce the cold run whatever init_idx holds
    there, with previous clusterings shorter and longer than the new one."""
    rng = np.random.default_rng(22)
    K = NUM.round_bf16(rng.standard_normal((600, 32)))
    C = 24
    init = rng.choice(len(K), C, replace=False)
    cold = KM.kmeans(K, init, max_iters=6)
    for m in (1, 10, C):
        init2 = init.copy()
        init2[:m] = rng.integers(0, len(K), m)  # ignored entries
        prev = np.concatenate([K[init[:m]], rng.standard_normal((3, 32))]) if m == C else K[init[:m]]
        warm = KM.kmeans(K, init2, max_iters=6, prev_centroids=prev)
        np.testing.assert_array_equal(warm.assign, cold.assign)
        np.testing.assert_array_equal(warm.centroids, cold.centroids)
    # and a previous centroid that differs from the key changes the run
    prev = K[init[:1]] + 5.0
    assert not np.array_equal(KM.kmeans(K, init, max_iters=1, prev_centroids=prev).assign,
                              KM.kmeans(K, init, max_iters=1).assign)


def test_kmeans_inertia_non_increasing():
    rng = np.random.default_rng(12)
    K = rng.standard_normal((2000, 128))
    r = KM.kmeans(K, rng.choice(2000, 64, replace=False), max_iters=10, round_storage=False)
    assert all(b <= a + 1e-9 for a, b in zip(r.inertia, r.inertia[1:]))


def test_kmeans_stored_centroids_are_rounded_means():
    rng = np.random.default_rng(13)
    K = NUM.round_bf16(rng.standard_normal((3000, 128)))
    r = KM.kmeans(K, rng.choice(3000, 100, replace=False), max_iters=10)
    np.testing.assert_array_equal(NUM.round_bf16(r.centroids), r.centroids)
    for j in range(100):
        mem = r.assign == j
        if mem.any():
            np.testing.assert_array_equal(r.centroids[j], NUM.round_bf16(K[mem].mean(0)))


def test_sq_distances_matches_direct_form():
    rng = np.random.default_rng(14)
    K = rng.standard_normal((50, 128))
    C = rng.standard_normal((7, 128))
    direct = ((K[:, None, :] - C[None, :, :]) ** 2).sum(-1)
    np.testing.assert_allclose(KM.sq_distances(K, C), direct, rtol=1e-12, atol=1e-10)


def test_cluster_layout_is_stable_sort():
    rng = np.random.default_rng(15)
    a = rng.integers(0, 37, 5000)
    off, perm = KM.cluster_layout(a, 40)
    np.testing.assert_array_equal(perm, np.argsort(a, kind="stable"))
    np.testing.assert_array_equal(np.diff(off), np.bincount(a, minlength=40))


def test_budget_reaching_target_exactly_counts():
    """Algorithm 1 asks for the cumulative sum to reach P times the total
    (>=).  Equal logits give w = 1 exactly, so S_k = k and P S_n = P n: the
    budget is exactly ceil(P n), including when P n is an integer."""
    for n in (10, 16, 40, 64):
        l_pos = np.full(n, 0.75)
        for P in (0.25, 0.5, 0.75, 0.3):
            k, _ = T.estimate_budget(l_pos, P, T.FitParams(exact_bp=10000))
            assert k == math.ceil(P * n - 1e-12) if (P * n) != int(P * n) else k == int(P * n)


# ---------------------------------------------------------------- recent-token tail (Sec. 1)

def test_tail_only_is_dense_attention():
    """Nothing clustered yet: the recent tokens are the whole selection."""
    rng = np.random.default_rng(31)
    n, G = 50, 4
    Q = rng.standard_normal((G, 128))
    K = rng.standard_normal((n, 128))
    V = rng.standard_normal((n, 128))
    r = T.decode_group(Q, K, V, np.zeros((1, 128)), np.array([0, 0]), 0.5)
    assert list(r.k) == [0] * G and r.union_count == n
    for h in range(G):
        np.testing.assert_allclose(r.out[h], A.dense_attention(Q[h], K, V), atol=1e-12)


def test_tail_with_target_one_is_dense_attention():
    rng = np.random.default_rng(32)
    Q, K, V, cent, off = _random_clustered_group(rng, 400, 24)
    tail = rng.standard_normal((37, 128))
    K2, V2 = np.vstack([K, tail]), np.vstack([V, rng.standard_normal((37, 128))])
    r = T.decode_group(Q, K2, V2, cent, off, 1.0)
    assert r.union_count == len(K2)
    for h in range(len(Q)):
        np.testing.assert_allclose(r.out[h], A.dense_attention(Q[h], K2, V2), atol=1e-12)


def test_tail_budget_is_top_p_given_the_recent_mass():
    """One cluster per token and every score exact: head h selects every recent
    token plus the fewest clustered tokens, taken by descending score (ties by
    id), whose mass with the recent tokens' reaches P of the total (brute force)."""
    rng = np.random.default_rng(33)
    prm = T.FitParams(exact_bp=10000)
    for trial in range(30):
        n, t = int(rng.integers(1, 120)), int(rng.integers(1, 40))
        q = rng.standard_normal(128) * rng.uniform(0.3, 3)
        K = rng.standard_normal((n + t, 128))
        V = rng.standard_normal((n + t, 128))
        P = float(rng.uniform(0.05, 0.99))
        off = np.arange(n + 1)
        r = T.decode_group(q[None], K, V, K[:n], off, P, prm)
        w = A.softmax_weights(A.logits(q, K))
        order = np.lexsort((np.arange(n), -A.logits(q, K[:n])))
        mass, k = float(w[n:].sum()), 0
        while mass < P * (1 - 1e-12) and k < n:
            mass += w[order[k]]
            k += 1
        assert r.k[0] == k, (trial, r.k[0], k)
        assert set(r.sel[0].tolist()) == set(order[:k].tolist()) | set(range(n, n + t))


def test_tail_holding_the_mass_selects_no_cluster():
    """A recent token that carries more than P of the mass leaves k = 0."""
    rng = np.random.default_rng(34)
    Q, K, V, cent, off = _random_clustered_group(rng, 300, 20, G=1)
    hot = Q[0] / np.linalg.norm(Q[0]) * 40.0  # logit ~ 40 * |q| / sqrt(d)
    K2 = np.vstack([K, hot[None]])
    V2 = np.vstack([V, rng.standard_normal((1, 128))])
    r = T.decode_group(Q, K2, V2, cent, off, 0.9)
    assert r.k[0] == 0 and list(r.sel[0]) == [len(K)]


def test_tail_of_length_zero_changes_nothing():
    rng = np.random.default_rng(35)
    Q, K, V, cent, off = _random_clustered_group(rng, 500, 30)
    _, info_a = T.estimate_budget(A.logits(Q[0], K[T.unpack(T.rank_clusters(Q[0], cent)[1], off)]), 0.8)
    _, info_b = T.estimate_budget(A.logits(Q[0], K[T.unpack(T.rank_clusters(Q[0], cent)[1], off)]), 0.8,
                                  l_tail=np.zeros(0))
    assert info_a["k"] == info_b["k"] and info_a["S_n"] == info_b["S_n"]
