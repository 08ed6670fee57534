"""Synthetic analog of the paper's token-budget table (Sec. 5.2.1, Tab. token_budget),
with the Tactic column taken from the library.

Workload: the timed 4 x 131072-token decode (32 query / 8 KV heads, per-head
sharpness from the workload's log-normal distribution), clustered by the
library's K-means (8192 clusters, 10 iterations), 3 layers x 4 sequences x 2
KV groups per (layer, sequence) = 96 query heads per target fraction.  For
every head and P in {0.5, ..., 0.9}:
  Tactic           sel_count_q of tactic_sparse_decode (Algorithm 1's budget k),
                   which must equal the fp64 oracle's k on the GPU's cluster
                   order except at a cutoff tie (staged parity of tests/parity.py);
  Optimal          fewest tokens in descending order of the true attention
                   scores whose mass reaches P (Sec. 3.4);
  Cluster Optimal  fewest tokens along the cluster order, true scores known;
  Achieved         true cumulative score p(I_h) of the library's selection (Eq. 5);
  Success          share of heads whose selection reaches P.
The table is printed (run with -s).  Checks: parity of every k, Optimal <=
Cluster Optimal for every head, budgets that grow with P, and the fit
reaching the target on average and for most heads.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import attention as OA
from oracle import tactic as OT
from tests.parity import check_group, fit_params, group_inputs, np64

pytestmark = pytest.mark.gpu

DEV = "cuda"
PS = (0.5, 0.6, 0.7, 0.8, 0.9)
LAYERS = (0, 9, 21)
GROUPS_PER_SEQ = 2


def test_token_budget_table_from_the_library():
    import paper_2502_12216_amd as T
    wl = synth.WORKLOADS["ctx128k_b4_32layer"]
    lens = list(wl.seq_lens)
    ncl = list(wl.cluster_counts)
    G = wl.n_q_heads // wl.n_kv_heads
    batch = T.RaggedBatch(lens, wl.n_q_heads, wl.n_kv_heads)
    builder = T.ClusterBuilder(batch, ncl, max_iters=wl.kmeans_iters)
    params = T.decode_params(0.9)
    dec = T.SparseDecoder(batch, ncl, params)
    prm = fit_params(params)
    kv_ip = np.concatenate([[0], np.cumsum(lens)])
    cl_ip = np.concatenate([[0], np.cumsum(ncl)])
    cols = {P: {"opt": [], "cl": [], "tac": [], "p": []} for P in PS}
    ties = 0
    for layer in LAYERS:
        inp = synth.make_layer(wl, layer, device=DEV)
        cb = builder(inp.K, inp.V, torch.as_tensor(synth.kmeans_init_all(wl, layer), device=DEV))
        lay = synth.LabelLayout(K_sorted=cb.K_sorted, V_sorted=cb.V_sorted, centroids=cb.clusters.centroids,
                                offsets=cb.clusters.offsets, perm=cb.perm, kv_indptr=kv_ip, cl_indptr=cl_ip)
        rng = np.random.default_rng([layer, 31])
        groups = [(b, int(g)) for b in range(len(lens))
                  for g in rng.choice(wl.n_kv_heads, GROUPS_PER_SEQ, replace=False)]
        gin = {bg: group_inputs(inp.q, lay.K_sorted, lay.V_sorted, lay.centroids, lay.offsets, kv_ip, cl_ip,
                                bg[0], bg[1], G) for bg in groups}
        for P in PS:
            P32 = float(np.float32(P))
            out, sq, skv = dec(inp.q, cb.K_sorted, cb.V_sorted, cb.clusters, target_frac=P)
            torch.cuda.synchronize()
            view = {k: v.cpu() for k, v in dec.view().items()}
            out, sq, skv = out.cpu(), sq.cpu(), skv.cpu()
            for b, g in groups:
                c0, c1 = int(cl_ip[b]), int(cl_ip[b + 1])
                gpu = dict(scores=np64(view["scores"][b, g * G:(g + 1) * G]),
                           order=view["order"][b, g * G:(g + 1) * G].numpy(),
                           k=sq[b, g * G:(g + 1) * G].numpy(), union_len=view["union_len"][g, c0:c1].numpy(),
                           out=np64(out[b, g * G:(g + 1) * G]), sel_kv=int(skv[b, g]))
                gi = gin[(b, g)]
                st = check_group(gi, P32, prm, gpu, label=f"budget layer={layer} b={b} g={g} P={P}")
                ties += st["cut_ties"]
                r = st["result"]
                for h in range(G):
                    rep = OT.selection_report(gi["Q"][h], gi["Ks"], gi["Vs"], r, P32, h)
                    k_lib = int(gpu["k"][h])
                    s = OA.softmax_weights(OA.logits(gi["Q"][h], gi["Ks"]))
                    cols[P]["opt"].append(rep["k_optimal"])
                    cols[P]["cl"].append(rep["k_cluster_optimal"])
                    cols[P]["tac"].append(k_lib)
                    cols[P]["p"].append(float(s[r.rows[h][:k_lib]].sum()))
        print(f"token budget: layer {layer} done", flush=True)
    n = lens[0]
    heads = len(cols[PS[0]]["tac"])
    print(f"\n| P | Optimal | Cluster Optimal | Tactic (library) | Achieved | Success |  "
          f"(means over {heads} heads, n = {n}; cutoff ties {ties})")
    print("|---|---|---|---|---|---|")
    summary = []
    for P in PS:
        c = {k: np.asarray(v, dtype=np.float64) for k, v in cols[P].items()}
        row = dict(P=P, opt=c["opt"].mean(), cl=c["cl"].mean(), tac=c["tac"].mean(), ach=c["p"].mean(),
                   succ=float(np.mean(c["p"] >= P - 1e-12)),
                   med=(np.median(c["opt"]), np.median(c["cl"]), np.median(c["tac"])))
        summary.append(row)
        print(f"| {P:.0%} | {row['opt']:.0f} | {row['cl']:.0f} | {row['tac']:.0f} | {row['ach']:.1%} | "
              f"{row['succ']:.0%} |  medians {row['med'][0]:.0f} / {row['med'][1]:.0f} / {row['med'][2]:.0f}")
        assert np.all(c["opt"] <= c["cl"])
        assert row["ach"] >= P - 0.02, row
        assert row["succ"] >= 0.75, row
    for a, b in zip(summary, summary[1:]):
        assert a["opt"] <= b["opt"] and a["cl"] <= b["cl"] and a["tac"] <= b["tac"]
