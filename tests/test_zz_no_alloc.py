"""tactic_sparse_decode_noalloc (the library's static scratch instead of a
caller workspace) against tactic_sparse_decode (a workspace from torch).

Both run the same kernels on the same inputs, so the outputs must be
identical bit for bit.  Two calls in a row on different shapes, the second
smaller, check that nothing the first left in the scratch leaks into the
second; a third call repeats the first.
"""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _case(lens, tail, P, union):
    import paper_2502_12216_amd as T
    wl = synth.small_workload(synth.WORKLOADS["ctx32k_llama8b"], lens)
    inp = synth.make_layer(wl, 0)
    lay = synth.label_layout(inp, tail=tail)
    ncl = [int(lay.cl_indptr[i + 1] - lay.cl_indptr[i]) for i in range(len(lens))]
    batch = T.RaggedBatch(lens, wl.n_q_heads, wl.n_kv_heads)
    dec = T.SparseDecoder(batch, ncl, T.decode_params(P, max_tail=256, use_union=union))
    cl = T.ClusterSet(lay.centroids.to(DEV).contiguous(), lay.offsets.to(DEV).contiguous(), ncl)
    args = (inp.q.to(DEV).contiguous(), lay.K_sorted.to(DEV).contiguous(), lay.V_sorted.to(DEV).contiguous(), cl)
    return dec, args


def _run(dec, args, noalloc):
    B, Hq, Hkv = dec.batch.batch, dec.batch.n_q_heads, dec.batch.n_kv_heads
    out = torch.full((B, Hq, 128), float("nan"), device=DEV)
    sq = torch.full((B, Hq), -7, dtype=torch.int32, device=DEV)
    skv = torch.full((B, Hkv), -7, dtype=torch.int32, device=DEV)
    call = dec.noalloc if noalloc else dec.__call__
    call(*args, out=out, sel_q=sq, sel_kv=skv)
    torch.cuda.synchronize()
    return out.cpu(), sq.cpu(), skv.cpu()


def test_noalloc_matches_workspace_decode_on_two_calls_in_a_row():
    big = _case([5000, 2600, 0, 3100], [120, 0, 0, 7], 0.9, 1)
    small = _case([900, 1], [30, 0], 0.6, 0)
    ref_big = _run(*big, noalloc=False)
    ref_small = _run(*small, noalloc=False)
    got_big = _run(*big, noalloc=True)
    got_small = _run(*small, noalloc=True)  # smaller shape right after the larger one
    again = _run(*big, noalloc=True)
    for ref, got in ((ref_big, got_big), (ref_small, got_small), (ref_big, again)):
        for a, b in zip(ref, got):
            assert torch.equal(a, b)
    assert torch.isfinite(got_big[0]).all() and int(got_big[1].min()) >= 0
    print("noalloc: identical to the workspace decode on", [tuple(x.shape) for x in got_big + got_small])
