"""GPU parity of the prefill K-means (tactic_build_clusters) with the fp64 oracle.

Procedure (the two trajectories may drift apart after a near-tie, so they are
compared step by step from shared states, then on the final objective):
  * one assignment from the shared starting centroids: identical except near
    ties (|d1 - d2| <= 1e-4 (|k|^2 + |c|^2));
  * the update from the GPU's own assignment: centroids within 1 bf16 ulp of
    the oracle's rounded means; the layout (offsets, perm) is exactly the
    stable counting sort of the GPU's assignment, and K_sorted = K[perm];
  * after 10 iterations the inertia is within 0.1% of the oracle's.
Starting tokens come from the seeded generator, never from the GPU.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import kmeans as OK
from oracle import numerics as ON
from tests.parity import np64

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _tactic():
    import paper_2502_12216_amd as P
    return P


def _build(inp, wl, iters):
    T = _tactic()
    lens = [int(inp.kv_indptr[i + 1] - inp.kv_indptr[i]) for i in range(len(inp.kv_indptr) - 1)]
    ncl = [wl.n_clusters(n) for n in lens]
    batch = T.RaggedBatch(lens, wl.n_q_heads, wl.n_kv_heads)
    builder = T.ClusterBuilder(batch, ncl, max_iters=iters)
    init = torch.as_tensor(synth.kmeans_init_all(wl, inp.layer), device=DEV)
    res = builder(inp.K.to(DEV).contiguous(), inp.V.to(DEV).contiguous(), init)
    torch.cuda.synchronize()
    return res, lens, ncl, init.cpu().numpy()


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    return torch.tensor(x, dtype=torch.float64).to(torch.bfloat16).view(torch.int16).numpy().astype(np.int64)


def _groups(lens, Hkv):
    return [(b, g) for b in range(len(lens)) for g in range(Hkv) if lens[b] > 0]


def _slices(inp, res, lens, ncl, b, g):
    kv = np.concatenate([[0], np.cumsum(lens)])
    cl = np.concatenate([[0], np.cumsum(ncl)])
    s0, s1, c0, c1 = int(kv[b]), int(kv[b + 1]), int(cl[b]), int(cl[b + 1])
    K = np64(inp.K[g, s0:s1])
    return dict(K=K, s0=s0, s1=s1, c0=c0, c1=c1,
                assign=res.assign[g, s0:s1].cpu().numpy().astype(np.int64),
                cent=np64(res.clusters.centroids[g, c0:c1]),
                off=res.clusters.offsets[g, c0 + b:c1 + b + 1].cpu().numpy().astype(np.int64),
                perm=res.perm[g, s0:s1].cpu().numpy().astype(np.int64))


@pytest.mark.parametrize("lens", [[4096], [3000, 1500, 700], [1, 3, 97, 5000]])
def test_kmeans_one_step_parity(lens):
    wl = synth.small_workload(synth.WORKLOADS["ctx4k_gqa4"], lens)
    inp = synth.make_layer(wl, 0)
    res, lens, ncl, init = _build(inp, wl, 1)
    cl = np.concatenate([[0], np.cumsum(ncl)])
    ties = 0
    for b, g in _groups(lens, wl.n_kv_heads):
        sl = _slices(inp, res, lens, ncl, b, g)
        K = sl["K"]
        c0 = K[init[g, int(cl[b]):int(cl[b + 1])]]
        D = OK.sq_distances(K, c0)
        a_or = np.argmin(D, axis=1)
        a_gpu = sl["assign"]
        diff = np.nonzero(a_or != a_gpu)[0]
        if len(diff):
            kk = np.einsum("ij,ij->i", K[diff], K[diff])
            cc = np.einsum("ij,ij->i", c0[a_or[diff]], c0[a_or[diff]])
            gap = np.abs(D[diff, a_gpu[diff]] - D[diff, a_or[diff]])
            assert np.all(gap <= 1e-4 * (kk + cc)), f"b={b} g={g}: {len(diff)} assignments differ beyond ties"
            ties += len(diff)
        # update from the GPU's own assignment
        c_or = OK.update_step(K, a_gpu, c0, round_storage=True)
        bits_o, bits_g = _bf16_bits(c_or), _bf16_bits(sl["cent"])
        assert np.max(np.abs(bits_o - bits_g)) <= 1, f"b={b} g={g}: centroid differs by more than 1 bf16 ulp"
        # layout = stable counting sort of the GPU's assignment
        off_or, perm_or = OK.cluster_layout(a_gpu, len(c0))
        np.testing.assert_array_equal(sl["off"], off_or)
        np.testing.assert_array_equal(sl["perm"], perm_or)
        Ks = np64(res.K_sorted[g, sl["s0"]:sl["s1"]])
        np.testing.assert_array_equal(Ks, K[perm_or])
        Vs = np64(res.V_sorted[g, sl["s0"]:sl["s1"]])
        np.testing.assert_array_equal(Vs, np64(inp.V[g, sl["s0"]:sl["s1"]])[perm_or])
    print(f"kmeans one step {lens}: near-tie assignment differences {ties}")


@pytest.mark.parametrize("base,lens", [("ctx4k_gqa4", [4096]), ("ctx32k_llama8b", [32768])])
def test_kmeans_ten_iterations_inertia(base, lens):
    wl = synth.small_workload(synth.WORKLOADS[base], lens)
    inp = synth.make_layer(wl, 0, device=DEV)
    res, lens, ncl, init = _build(inp, wl, 10)
    cl = np.concatenate([[0], np.cumsum(ncl)])
    groups = _groups(lens, wl.n_kv_heads)[:2]
    for b, g in groups:
        sl = _slices(inp, res, lens, ncl, b, g)
        K = sl["K"]
        r = OK.kmeans(K, init[g, int(cl[b]):int(cl[b + 1])], max_iters=10)
        in_or = OK.inertia(K, r.assign, r.centroids)
        in_gpu = OK.inertia(K, sl["assign"], sl["cent"])
        assert abs(in_gpu - in_or) <= 1e-3 * in_or, f"b={b} g={g}: inertia gpu {in_gpu} oracle {in_or}"
        # the returned layout always matches the returned assignment
        off_or, perm_or = OK.cluster_layout(sl["assign"], len(sl["cent"]))
        np.testing.assert_array_equal(sl["off"], off_or)
        np.testing.assert_array_equal(sl["perm"], perm_or)
        # every non-empty centroid is the (bf16) mean of its members
        for j in range(0, len(sl["cent"]), max(1, len(sl["cent"]) // 64)):
            mem = sl["assign"] == j
            if mem.any():
                d = np.abs(_bf16_bits(ON.round_bf16(K[mem].mean(0))) - _bf16_bits(sl["cent"][j]))
                assert d.max() <= 1
        print(f"kmeans 10 it {base} b={b} g={g}: inertia gpu {in_gpu:.6e} oracle {in_or:.6e} "
              f"(oracle iters {r.iters})")


def test_kmeans_is_deterministic():
    wl = synth.small_workload(synth.WORKLOADS["ctx32k_llama8b"], [6000, 2500])
    inp = synth.make_layer(wl, 0, device=DEV)
    r1, *_ = _build(inp, wl, 10)
    r2, *_ = _build(inp, wl, 10)
    assert torch.equal(r1.assign, r2.assign) and torch.equal(r1.perm, r2.perm)
    assert torch.equal(r1.clusters.centroids, r2.clusters.centroids)
    assert torch.equal(r1.K_sorted, r2.K_sorted)


def test_decode_on_kmeans_clusters_invariants():
    """Decode over the library's own clusters (no oracle input comes from the
    GPU here): properties that hold for any valid cluster layout."""
    T = _tactic()
    wl = synth.small_workload(synth.WORKLOADS["ctx32k_llama8b"], [9000, 4000])
    inp = synth.make_layer(wl, 0, device=DEV)
    res, lens, ncl, _ = _build(inp, wl, 10)
    batch = T.RaggedBatch(lens, wl.n_q_heads, wl.n_kv_heads)
    for P in (0.5, 0.9, 1.0):
        dec = T.SparseDecoder(batch, ncl, T.decode_params(P))
        out, sq, skv = dec(inp.q, res.K_sorted, res.V_sorted, res.clusters)
        torch.cuda.synchronize()
        G = wl.n_q_heads // wl.n_kv_heads
        sq, skv = sq.cpu().numpy(), skv.cpu().numpy()
        for b, n in enumerate(lens):
            for g in range(wl.n_kv_heads):
                k = sq[b, g * G:(g + 1) * G]
                assert np.all(k >= 1) and np.all(k <= n)
                assert k.max() <= skv[b, g] <= min(n, k.sum())
                if P == 1.0:
                    assert skv[b, g] == n
        assert torch.isfinite(out).all()


def test_decode_on_kmeans_clusters_128k_sampled_parity():
    """The timed shape as the benchmark runs it: one 4 x 131072-token layer
    clustered by tactic_build_clusters (10 iterations, 8192 clusters per
    sequence and KV head, some of them emptied by the iterations), then the
    sparse decode at P = 0.9, staged parity on sampled groups (those with the
    most empty clusters first).  The oracle reads the library's cluster
    layout as its input, as a decode loop would hand it over."""
    from tests.test_gpu_decode import check_layer
    T = _tactic()
    wl = synth.WORKLOADS["ctx128k_b4_32layer"]
    inp = synth.make_layer(wl, 3, device=DEV)
    res, lens, ncl, _ = _build(inp, wl, wl.kmeans_iters)
    batch = T.RaggedBatch(lens, wl.n_q_heads, wl.n_kv_heads)
    P = 0.9
    params = T.decode_params(P)
    dec = T.SparseDecoder(batch, ncl, params)
    out, sq, skv = dec(inp.q, res.K_sorted, res.V_sorted, res.clusters)
    torch.cuda.synchronize()
    run = dict(out=out.clone().cpu(), sel_q=sq.clone().cpu(), sel_kv=skv.clone().cpu(),
               view={k: v.clone().cpu() for k, v in dec.view().items()}, params=params)
    kv_ip = np.concatenate([[0], np.cumsum(lens)])
    cl_ip = np.concatenate([[0], np.cumsum(ncl)])
    lay = synth.LabelLayout(K_sorted=res.K_sorted, V_sorted=res.V_sorted, centroids=res.clusters.centroids,
                            offsets=res.clusters.offsets, perm=res.perm, kv_indptr=kv_ip, cl_indptr=cl_ip)
    off = res.clusters.offsets.long().cpu()
    empties = {}
    for b in range(len(lens)):
        o = off[:, cl_ip[b] + b:cl_ip[b + 1] + b + 1]
        for g in range(wl.n_kv_heads):
            empties[(b, g)] = int(((o[g, 1:] - o[g, :-1]) == 0).sum())
    ranked = sorted(empties, key=lambda bg: -empties[bg])
    rng = np.random.default_rng(23)
    rest = [ranked[i] for i in rng.choice(np.arange(2, len(ranked)), 3, replace=False)]
    groups = ranked[:2] + rest
    st = check_layer(inp, lay, P, run, groups=groups, label="kmeans 128k")
    print("kmeans 128k sampled:", [(bg, empties[bg], s["k"], s["union"]) for bg, s in zip(groups, st)],
          "empty clusters in the layer:", sum(empties.values()))


def test_kmeans_spare_room_layout_matches_packed():
    """K-means over sequences with spare rows (seq_len < span) touches only
    the sequences' tokens: same clusters and cluster-sorted rows as packed."""
    T = _tactic()
    wl = synth.small_workload(synth.WORKLOADS["ctx32k_llama8b"], [3000, 1200])
    inp = synth.make_layer(wl, 0)
    lens = list(wl.seq_lens)
    caps = [lens[0] + 333, lens[1] + 64]
    ncl = [wl.n_clusters(n) for n in lens]
    Hkv = wl.n_kv_heads
    packed = T.RaggedBatch(lens, wl.n_q_heads, Hkv)
    spaced = T.RaggedBatch(lens, wl.n_q_heads, Hkv, capacities=caps)

    def spread(X):
        Y = torch.full((Hkv, spaced.total, 128), -7.0, dtype=torch.bfloat16)
        for b, n in enumerate(lens):
            s0, d0 = packed.kv_indptr_host[b], spaced.kv_indptr_host[b]
            Y[:, d0:d0 + n] = X[:, s0:s0 + n]
        return Y.to(DEV)

    init = torch.as_tensor(synth.kmeans_init_all(wl, 0), device=DEV)
    r1 = T.ClusterBuilder(packed, ncl, max_iters=5)(inp.K.to(DEV), inp.V.to(DEV), init)
    r2 = T.ClusterBuilder(spaced, ncl, max_iters=5)(spread(inp.K), spread(inp.V), init)
    torch.cuda.synchronize()
    assert torch.equal(r1.clusters.centroids, r2.clusters.centroids)
    assert torch.equal(r1.clusters.offsets, r2.clusters.offsets)
    for b, n in enumerate(lens):
        s0, d0 = packed.kv_indptr_host[b], spaced.kv_indptr_host[b]
        assert torch.equal(r1.assign[:, s0:s0 + n], r2.assign[:, d0:d0 + n])
        assert torch.equal(r1.K_sorted[:, s0:s0 + n], r2.K_sorted[:, d0:d0 + n])


@pytest.mark.parametrize("iters", [1, 10])
def test_kmeans_warm_start_parity(iters):
    """Re-clustering from a previous clustering (tactic_kmeans_params
    prev_centroids / prev_cl_indptr): centroid j of (b, g) starts from the
    previous centroid j below both cluster counts, from the init_idx key
    otherwise.  The previous centroids are the oracle's own CPU clustering
    (3 iterations, bf16 storage) with fewer, more and as many clusters as the
    new one, so no oracle input comes from the GPU.  One step: assignment
    from the warm start identical except near ties, update within 1 bf16 ulp;
    ten steps: inertia within 0.1% of the oracle's warm run."""
    T = _tactic()
    wl = synth.small_workload(synth.WORKLOADS["ctx4k_gqa4"], [3000, 1500, 700])
    inp = synth.make_layer(wl, 0)
    lens = [int(inp.kv_indptr[i + 1] - inp.kv_indptr[i]) for i in range(len(inp.kv_indptr) - 1)]
    ncl = [wl.n_clusters(n) for n in lens]
    prev_ncl = [ncl[0] - 7, ncl[1] + 5, ncl[2]]
    Hkv = wl.n_kv_heads
    kv = np.concatenate([[0], np.cumsum(lens)])
    pcl = np.concatenate([[0], np.cumsum(prev_ncl)])
    cl = np.concatenate([[0], np.cumsum(ncl)])
    rng = np.random.default_rng(31)
    prev_cent = np.zeros((Hkv, int(pcl[-1]), 128))
    for b in range(len(lens)):
        for g in range(Hkv):
            K = np64(inp.K[g, int(kv[b]):int(kv[b + 1])])
            r = OK.kmeans(K, rng.choice(lens[b], prev_ncl[b], replace=False), max_iters=3)
            prev_cent[g, int(pcl[b]):int(pcl[b + 1])] = r.centroids
    prev = T.ClusterSet(torch.tensor(prev_cent, dtype=torch.bfloat16, device=DEV),
                        torch.zeros(Hkv, int(pcl[-1]) + len(lens), dtype=torch.int32, device=DEV), prev_ncl)
    batch = T.RaggedBatch(lens, wl.n_q_heads, Hkv)
    builder = T.ClusterBuilder(batch, ncl, max_iters=iters)
    init_np = synth.kmeans_init_all(wl, inp.layer)
    res = builder(inp.K.to(DEV).contiguous(), inp.V.to(DEV).contiguous(), torch.as_tensor(init_np, device=DEV),
                  prev=prev)
    torch.cuda.synchronize()
    ties = 0
    for b, g in _groups(lens, Hkv):
        sl = _slices(inp, res, lens, ncl, b, g)
        K = sl["K"]
        ini = init_np[g, int(cl[b]):int(cl[b + 1])].astype(np.int64)
        pc = prev_cent[g, int(pcl[b]):int(pcl[b + 1])]
        m = min(ncl[b], prev_ncl[b])
        c_start = np.concatenate([pc[:m], K[ini[m:]]])
        if iters == 1:
            D = OK.sq_distances(K, c_start)
            a_or = np.argmin(D, axis=1)
            a_gpu = sl["assign"]
            diff = np.nonzero(a_or != a_gpu)[0]
            if len(diff):
                kk = np.einsum("ij,ij->i", K[diff], K[diff])
                cc = np.einsum("ij,ij->i", c_start[a_or[diff]], c_start[a_or[diff]])
                gap = np.abs(D[diff, a_gpu[diff]] - D[diff, a_or[diff]])
                assert np.all(gap <= 1e-4 * (kk + cc)), f"b={b} g={g}: {len(diff)} assignments differ beyond ties"
                ties += len(diff)
            c_or = OK.update_step(K, a_gpu, c_start, round_storage=True)
            assert np.max(np.abs(_bf16_bits(c_or) - _bf16_bits(sl["cent"]))) <= 1, f"b={b} g={g}"
        else:
            r = OK.kmeans(K, ini, max_iters=10, prev_centroids=pc)
            in_or = OK.inertia(K, r.assign, r.centroids)
            in_gpu = OK.inertia(K, sl["assign"], sl["cent"])
            assert abs(in_gpu - in_or) <= 1e-3 * in_or, f"b={b} g={g}: inertia gpu {in_gpu} oracle {in_or}"
    print(f"kmeans warm start, {iters} iteration(s): near-tie assignment differences {ties}")

