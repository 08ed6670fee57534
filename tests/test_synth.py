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
