"""Host-side checks of the seeded input generator (CPU only)."""
import numpy as np
import torch

import synth


def test_small_workload_is_deterministic_and_layout_valid():
    wl = synth.small_workload(synth.WORKLOADS["ctx32k_llama8b"], [700, 0, 1300])
    a = synth.make_layer(wl, 0)
    b = synth.make_layer(wl, 0)
    assert torch.equal(a.K, b.K) and torch.equal(a.q, b.q) and torch.equal(a.V, b.V)
    lay = synth.label_layout(a)
    Hkv = a.K.shape[0]
    B = len(a.kv_indptr) - 1
    for bb in range(B):
        s0, s1 = int(a.kv_indptr[bb]), int(a.kv_indptr[bb + 1])
        c0, c1 = int(lay.cl_indptr[bb]), int(lay.cl_indptr[bb + 1])
        for g in range(Hkv):
            off = lay.offsets[g, c0 + bb:c1 + bb + 1].long()
            assert int(off[0]) == 0 and int(off[-1]) == s1 - s0
            perm = lay.perm[g, s0:s1].long()
            assert sorted(perm.tolist()) == list(range(s1 - s0))
            assert torch.equal(lay.K_sorted[g, s0:s1], a.K[g, s0:s1][perm])
            lab = a.labels[g, s0:s1][perm]
            for j in range(c1 - c0):
                seg = lab[off[j]:off[j + 1]]
                assert torch.all(seg == j)
                p = perm[off[j]:off[j + 1]]
                assert torch.all(p[1:] > p[:-1])


def test_kmeans_init_is_distinct():
    wl = synth.WORKLOADS["ctx4k_gqa4"]
    idx = synth.kmeans_init_idx(wl, 0, 0, 1, 4096, 256)
    assert len(set(idx.tolist())) == 256 and idx.min() >= 0 and idx.max() < 4096


def test_concentration_sweep_readings():
    """The sweep's points share keys, values and centres; the mean reading
    divides the query's centre sum by k_h (same noise draw), so
    q_sum - q_mean = beta (1 - 1/k_h) sum_j c_j up to bf16 rounding."""
    ws = synth.sweep_workloads()
    assert len(ws) == 8 and len({w.wid for w in ws}) == 1
    by = {w.name: w.with_seq_lens([1024]) for w in ws}
    a = synth.make_layer(by["sweep_b2_sum"], 0)
    m = synth.make_layer(by["sweep_b2_mean"], 0)
    assert torch.equal(a.K, m.K) and torch.equal(a.V, m.V) and torch.equal(a.centers, m.centers)
    G = a.q.shape[1] // a.K.shape[0]
    for h in range(a.q.shape[1]):
        S = a.q_centres[h]
        assert S == m.q_centres[h]
        csum = a.centers[h // G][torch.as_tensor(S)].double().sum(0)
        diff = a.q[0, h].double() - m.q[0, h].double()
        expect = 2.0 * (1.0 - 1.0 / len(S)) * csum
        scale = a.q[0, h].double().abs() + m.q[0, h].double().abs()
        assert torch.all((diff - expect).abs() <= 2 ** -8 * scale + 1e-6), h
    # beta scales the whole query
    q1 = synth.make_layer(by["sweep_b1_sum"], 0).q.double()
    assert torch.allclose(a.q.double(), 2.0 * q1, rtol=2 ** -7, atol=1e-6)
