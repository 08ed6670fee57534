"""Synthetic analog of the paper's token-budget table (Sec. 5.2, Tab. token_budget).

For every query head of one 128K-token sequence of the 4 x 128K workload (layer 0,
clusters = the generator's mixture labels, per-head sharpness drawn from the
workload's log-normal distribution) and P in {0.5, ..., 0.9}, the oracle gives:
  Optimal          tokens needed in descending order of the true attention
                   scores (Sec. 3.4);
  Cluster Optimal  tokens needed along the cluster order when the true scores
                   are known (Eq. 5 summed in cluster order);
  Tactic           the budget k of Algorithm 1 (exact head + fitted tail);
  Achieved         the true cumulative score of Tactic's selection;
  Success          the share of heads whose selection reaches P.
The test checks what holds by construction (Optimal <= Cluster Optimal for
every head, budgets grow with P) and that the fit reaches the target on
average and for most heads; run with -s to print the table.
"""
import numpy as np
import pytest

import synth
from oracle import tactic as OT

PS = (0.5, 0.6, 0.7, 0.8, 0.9)


def token_budget_rows(wl_name="ctx128k_b4_32layer", layer=0, Ps=PS):
    wl = synth.WORKLOADS[wl_name]
    inp = synth.make_layer(wl, layer, seq_subset=[0])
    lay = synth.label_layout(inp)
    G = wl.n_q_heads // wl.n_kv_heads
    b = 0
    s0, s1 = int(lay.kv_indptr[0]), int(lay.kv_indptr[1])
    c0, c1 = int(lay.cl_indptr[0]), int(lay.cl_indptr[1])
    rows = []
    for P in Ps:
        rep = []
        for g in range(wl.n_kv_heads):
            Q = inp.q[b, g * G:(g + 1) * G].double().numpy()
            Ks = lay.K_sorted[g, s0:s1].double().numpy()
            Vs = lay.V_sorted[g, s0:s1].double().numpy()
            cent = lay.centroids[g, c0:c1].double().numpy()
            off = lay.offsets[g, c0 + b:c1 + b + 1].numpy().astype(np.int64)
            r = OT.decode_group(Q, Ks, Vs, cent, off, P)
            for h in range(G):
                rep.append(OT.selection_report(Q[h], Ks, Vs, r, P, h))
        k_opt = np.array([x["k_optimal"] for x in rep])
        k_cl = np.array([x["k_cluster_optimal"] for x in rep])
        k_t = np.array([x["k"] for x in rep])
        p_sel = np.array([x["p_sel"] for x in rep])
        rows.append(dict(P=P, optimal=float(k_opt.mean()), cluster_optimal=float(k_cl.mean()),
                         tactic=float(k_t.mean()), achieved=float(p_sel.mean()),
                         success=float(np.mean(p_sel >= P - 1e-12)), n=s1 - s0, heads=len(rep),
                         k_opt=k_opt, k_cl=k_cl, k_t=k_t, p_sel=p_sel))
    return rows


@pytest.mark.slow
def test_token_budget_table():
    rows = token_budget_rows()
    print(f"\n| P | Optimal | Cluster Optimal | Tactic | Achieved | Success |  (n = {rows[0]['n']}, "
          f"{rows[0]['heads']} heads)")
    print("|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {r['P']:.0%} | {r['optimal']:.0f} | {r['cluster_optimal']:.0f} | {r['tactic']:.0f} | "
              f"{r['achieved']:.1%} | {r['success']:.0%} |")
    for r in rows:
        # optimal is the minimum over all orders; cluster optimal follows one order
        assert np.all(r["k_opt"] <= r["k_cl"])
        # the fit reaches the target on average and for most heads (the paper
        # reports 84-92% success); whole clusters make it overshoot, not
        # undershoot
        assert r["achieved"] >= r["P"] - 0.02, r
        assert r["success"] >= 0.75, r
        # and it estimates the cluster-order budget within a factor of two
        assert 0.5 <= r["tactic"] / r["cluster_optimal"] <= 2.0, r
    # more mass needs more tokens, in every column
    for a, b in zip(rows, rows[1:]):
        assert a["optimal"] <= b["optimal"] and a["cluster_optimal"] <= b["cluster_optimal"]
        assert a["tactic"] <= b["tactic"]
