"""Decode loop with recent tokens and periodic re-clustering (Sec. 1), on the
GPU through the C ABI, checked against the fp64 oracle at every kind of step:
right after prefill, with a growing recent tail, and right after a
re-clustering.  The tokens are the seeded generator's; the cache layout the
oracle reads is the GPU's own cluster-sorted rows, and every check is of the
selection and attention over that layout (stages as in tests/parity.py)."""
import numpy as np
import pytest
import torch

import synth
from tests.parity import check_group, fit_params, np64

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _row_multiset(X: torch.Tensor):
    return sorted(map(bytes, X.contiguous().view(torch.int16).cpu().numpy()))


def test_recent_tail_cache_decode_loop_matches_oracle():
    import paper_2502_12216_amd as T
    wl = synth.small_workload(synth.WORKLOADS["ctx4k_gqa4"], [900, 610])
    inp = synth.make_layer(wl, 0)
    lens = list(wl.seq_lens)
    new = 100
    G = wl.n_q_heads // wl.n_kv_heads
    cache = T.RecentTailCache(wl.n_q_heads, wl.n_kv_heads, [n + 8 for n in lens], recluster_every=48,
                              kmeans_iters=5, seed=3)
    kvp = [int(x) for x in inp.kv_indptr]
    cache.prefill([inp.K[:, kvp[b]:kvp[b] + lens[b] - new].to(DEV) for b in range(len(lens))],
                  [inp.V[:, kvp[b]:kvp[b] + lens[b] - new].to(DEV) for b in range(len(lens))])
    q = inp.q.to(DEV)
    P = 0.8
    prm = fit_params(T.decode_params(P))
    checked = 0
    # buffers the re-clusterings reuse: two K/V buffers in turn, one builder and one decoder workspace
    kv_bufs = {cache.K.data_ptr(), cache.K_alt.data_ptr()}
    ws_ptrs = (cache.builder.workspace.data_ptr(), cache.decoder.workspace.data_ptr())
    for step in range(new + 1):
        if step in (0, 1, 30, 47, 48, 49, 96, new):
            out, sq, skv = cache.decode(q, target_frac=P)
            torch.cuda.synchronize()
            v = {k: t.clone().cpu() for k, t in cache.decoder.view().items()}
            out, sq, skv = out.clone().cpu(), sq.clone().cpu(), skv.clone().cpu()
            cl = cache.clusters
            for b in range(len(lens)):
                s0 = int(cache.batch.kv_indptr_host[b])
                n = cache.lens[b]
                c0, c1 = int(cl.cl_indptr_host[b]), int(cl.cl_indptr_host[b + 1])
                for g in range(wl.n_kv_heads):
                    gi = dict(Q=np64(inp.q[b, g * G:(g + 1) * G]), Ks=np64(cache.K[g, s0:s0 + n]),
                              Vs=np64(cache.V[g, s0:s0 + n]), cent=np64(cl.centroids[g, c0:c1]),
                              off=cl.offsets[g, c0 + b:c1 + b + 1].cpu().numpy().astype(np.int64))
                    assert int(gi["off"][-1]) == cache.clustered[b]
                    gpu = dict(scores=np64(v["scores"][b, g * G:(g + 1) * G]),
                               order=v["order"][b, g * G:(g + 1) * G].numpy(),
                               k=sq[b, g * G:(g + 1) * G].numpy(), union_len=v["union_len"][g, c0:c1].numpy(),
                               out=np64(out[b, g * G:(g + 1) * G]), sel_kv=int(skv[b, g]))
                    check_group(gi, float(np.float32(P)), prm, gpu, label=f"step {step} b={b} g={g}")
                    checked += 1
        if step == new:
            break
        kt = torch.stack([inp.K[:, kvp[b] + lens[b] - new + step] for b in range(len(lens))]).to(DEV)
        vt = torch.stack([inp.V[:, kvp[b] + lens[b] - new + step] for b in range(len(lens))]).to(DEV)
        reclustered = cache.append(kt, vt)
        assert reclustered == ((step + 1) % 48 == 0)
        if reclustered:
            assert cache.recent == [0, 0]
            assert {cache.K.data_ptr(), cache.K_alt.data_ptr()} == kv_bufs
            assert (cache.builder.workspace.data_ptr(), cache.decoder.workspace.data_ptr()) == ws_ptrs
    assert cache.reclusterings == 1 + new // 48
    # every token is still held once, in the cluster-sorted rows or the recent tail
    for b in range(len(lens)):
        s0 = int(cache.batch.kv_indptr_host[b])
        for g in range(wl.n_kv_heads):
            assert _row_multiset(cache.K[g, s0:s0 + lens[b]]) == _row_multiset(inp.K[g, kvp[b]:kvp[b] + lens[b]])
    assert checked == 8 * len(lens) * wl.n_kv_heads
