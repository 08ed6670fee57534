"""Benchmark of Tactic's sparse decode attention on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one full decode step of the workload: every layer runs the whole
hot path (centroid scoring, cluster sort, sampled logits + fit + cutoff +
union, gather split-K attention) on its own cluster-sorted cache.  The
default workload is 32 layers of a batch of 4 sequences of 131072 tokens
(32 query / 8 KV heads, head_dim 128, bf16, 8192 clusters per sequence and
KV head, target fraction 0.9) on seeded synthetic Gaussian-mixture keys.
Its clusters come from the library's own K-means (10 iterations, timed
separately), or from the generator's mixture labels with --clusters labels.

Prints one JSON line: sparse microseconds per layer (lower is better), the
same-GPU dense decode time and speedup, the HBM rate on the bytes the
kernels must read, a roofline record of the dominant kernel and the CPU
oracle's time on a bounded sample.  The same line carries one record per
other workload (4K, 32K at three target fractions, the ragged batch of 16,
1M tokens) and for one layer of the timed shape at five target fractions:
single-layer timings with the caches flushed before every rep, and the
device's measured streaming-read ceiling.

Bytes "touched" per layer: every centroid row and cluster offset, every K and
V row of each group's union, and the distinct sampled key rows of a group
that lie outside its union (the ones inside are read again by the attention).
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

HBM_PEAK_GBPS = 8000.0
METRIC = "sparse decode-attn µs/layer + HBM GB/s at 128K ctx; speedup vs dense"


def log(msg: str) -> None:
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def profiled_traffic(stage: str):
    """HBM bytes per launch of a decode kernel from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary (scaled by the reference copy), or None
    when no summary matches the kernel source as it is now."""
    import glob
    import hashlib
    import re
    src = {n: hashlib.sha256(open(os.path.join(ROOT, "paper_2502_12216_amd", "csrc", n), "rb").read()).hexdigest()[:16]
           for n in ("decode_attn.hip", "decode_select.hip")}
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
        if not m:
            continue
        summ = json.loads(m.group(1))
        shas = summ.get("_source_sha256", {})
        if any(shas.get(n) != h for n, h in src.items()):
            continue
        for k, v in summ.items():
            if k.startswith(stage) and "[dense]" not in k:
                return v.get("traffic_bytes")
    return None


class TimingEvents:
    """HIP events for timing only, created with hipEventDisableSystemFence:
    recording one does not write back and invalidate the caches (which would
    also slow the kernel after it), and they are read after a full device
    synchronisation.  `array` is what tactic_sparse_decode_plan_set_events
    takes."""

    FLAGS = 0x20000000  # hipEventDisableSystemFence

    def __init__(self, n: int):
        import ctypes
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.events = []
        for _ in range(n):
            ev = ctypes.c_void_p()
            if self.hip.hipEventCreateWithFlags(ctypes.byref(ev), ctypes.c_uint(self.FLAGS)) != 0:
                raise RuntimeError("hipEventCreateWithFlags failed")
            self.events.append(ev)
        self.array = (ctypes.c_void_p * n)(*[e.value for e in self.events])

    def elapsed(self, i: int, j: int) -> float:
        """Milliseconds from event i to event j (both recorded and complete)."""
        import ctypes
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), self.events[i], self.events[j]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value


class Flusher:
    """Evicts L2 and the 256 MB Infinity Cache between timed reps by writing a
    1 GiB buffer (untimed: it runs between the events of two reps)."""

    def __init__(self, dev, nbytes: int = 1 << 30):
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        self.v = 0

    def __call__(self):
        self.v ^= 1
        self.buf.fill_(self.v)


def timed_reps(fn, reps: int, flush=None) -> list:
    """Milliseconds of each of `reps` calls of fn, from events around the call
    alone on the current stream; `flush`, if given, runs before every rep."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    torch.cuda.synchronize()
    for e0, e1 in evs:
        if flush is not None:
            flush()
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    return [e0.elapsed_time(e1) for e0, e1 in evs]


def samples_outside_union(view: dict, clusters, G: int) -> int:
    """Distinct sampled key rows of every (sequence, KV head) group that lie
    outside the group's union: the sampled rows the attention does not read
    again.  Rows past a sequence's clusters (recent tokens) are always in it."""
    rows = view["sample_rows"].cpu().numpy()
    cnt = view["fit"][..., 11].cpu().numpy().astype(np.int64)
    ulen = view["union_len"].cpu().numpy()
    off = clusters.offsets.cpu().numpy()
    clp = clusters.cl_indptr_host
    B, Hq = cnt.shape
    total = 0
    for b in range(B):
        c0, c1 = int(clp[b]), int(clp[b + 1])
        for g in range(Hq // G):
            o = off[g, c0 + b:c1 + b + 1].astype(np.int64)
            r = np.unique(np.concatenate([rows[b, g * G + j, :cnt[b, g * G + j]] for j in range(G)]))
            r = r[r < o[-1]]
            c = np.searchsorted(o, r, side="right") - 1
            total += int(np.count_nonzero((r - o[c]) >= ulen[g, c0 + c]))
    return total


def touched_bytes(view: dict, clusters, sel_kv: torch.Tensor, G: int) -> dict:
    """Bytes one sparse decode call must move: centroids and offsets, the
    union's K and V rows, and the sampled key rows outside the union."""
    Hkv, Ct = clusters.centroids.shape[0], clusters.total
    B = len(clusters.n_clusters)
    cent = Hkv * Ct * 256 + Hkv * (Ct + B) * 4
    samples = samples_outside_union(view, clusters, G) * 256
    union = float(sel_kv.sum()) * 512
    return {"centroids": float(cent), "samples_outside_union": float(samples), "union_kv": union,
            "total": float(cent + samples + union)}


def dense_sdpa(q, K, V, wl, reps: int, own_out=None) -> dict:
    """torch's scaled_dot_product_attention (GQA) as a second dense decode on
    one layer's bf16 inputs, restricted to the fused flash / memory-efficient
    backends; the result says why when neither takes the shape."""
    if len(set(wl.seq_lens)) != 1:
        return {"us_per_layer": None, "error": "ragged batch: SDPA needs equal lengths"}
    try:
        from torch.nn.attention import SDPBackend, sdpa_kernel
        B, Hq, d = q.shape
        Hkv, n = K.shape[0], wl.seq_lens[0]
        qS = q.view(B, Hq, 1, d)
        KS = K.view(Hkv, B, n, d).transpose(0, 1).contiguous()
        VS = V.view(Hkv, B, n, d).transpose(0, 1).contiguous()
        backends = [SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]

        def call():
            with sdpa_kernel(backends):
                return torch.nn.functional.scaled_dot_product_attention(qS, KS, VS, enable_gqa=True)

        o = call().view(B, Hq, d).float()
        diff = float((o - own_out).abs().max()) if own_out is not None else None
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            call()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1000 / reps
        del KS, VS
        return {"us_per_layer": round(us, 2), "backends": "flash, efficient", "reps": reps,
                "max_abs_diff_vs_own_dense": diff}
    except Exception as e:  # no fused backend for this shape in the installed torch
        return {"us_per_layer": None, "error": f"{type(e).__name__}: {str(e)[:160]}"}


# the decode's kernels in launch order (one library event after each)
STAGE_NAMES = ["score_clusters", "sort_clusters", "sample_logits", "fit_union", "attn_splitk", "combine"]
STAGE_KERNEL = {n: n for n in STAGE_NAMES}
SEL, ATT, COMB = STAGE_NAMES.index("sample_logits"), STAGE_NAMES.index("attn_splitk"), STAGE_NAMES.index("combine")


def config_record(T, wl, Ps, dev, flush, reps: int, stage_ev, ceiling, host_groups=None, union_ab=None):
    """One layer of workload `wl` on the library's K-means clusters: sparse and
    dense decode times (medians of `reps` calls, caches flushed before each),
    per-kernel times (library events, flushed), touched bytes and rates,
    selected fractions.  host_groups: (sequence, KV head) groups whose fp64
    inputs are returned for the CPU oracle legs.  union_ab: a target fraction
    (one of Ps) at which every query head also attends over its own selection
    (the GQA-union ablation, Sec. 4.5)."""
    import ctypes
    from paper_2502_12216_amd import _capi as C
    B, Hq, Hkv = wl.batch, wl.n_q_heads, wl.n_kv_heads
    G = Hq // Hkv
    ncl = list(wl.cluster_counts)
    lens = np.asarray(wl.seq_lens, dtype=np.float64)
    batch = T.RaggedBatch(wl.seq_lens, Hq, Hkv)
    inp = synth.make_layer(wl, 0, device=dev)
    init = torch.as_tensor(synth.kmeans_init_all(wl, 0), device=dev)
    bld = T.ClusterBuilder(batch, ncl, max_iters=wl.kmeans_iters)
    built = []
    km_ms = timed_reps(lambda: built.append(bld(inp.K, inp.V, init)), 1)[0]
    cb = built[0]
    q, Ks, Vs, cl = inp.q, cb.K_sorted, cb.V_sorted, cb.clusters
    host = None
    if host_groups:
        kvp, clp = batch.kv_indptr_host, cl.cl_indptr_host
        host = {"G": G, "groups": []}
        for b, g in host_groups:
            s0, s1, c0, c1 = int(kvp[b]), int(kvp[b + 1]), int(clp[b]), int(clp[b + 1])
            host["groups"].append(dict(
                Q=q[b, g * G:(g + 1) * G].double().cpu().numpy(), Ks=Ks[g, s0:s1].double().cpu().numpy(),
                Vs=Vs[g, s0:s1].double().cpu().numpy(), cent=cl.centroids[g, c0:c1].double().cpu().numpy(),
                off=cl.offsets[g, c0 + b:c1 + b + 1].cpu().numpy().astype(np.int64),
                K=inp.K[g, s0:s1].double().cpu().numpy(), init=init[g, c0:c1].cpu().numpy().astype(np.int64)))
        host["groups_per_layer"] = B * Hkv
    del inp, built
    den = T.DenseDecoder(batch)
    for _ in range(3):
        den(q, Ks, Vs)
    us_dense = float(np.median(timed_reps(lambda: den(q, Ks, Vs), reps, flush))) * 1000
    dense_bytes = float(lens.sum()) * Hkv * 512
    def timed_and_staged(dec):
        """Flushed median time of one call (us) and per-kernel event times (us)."""
        for _ in range(3):
            dec(q, Ks, Vs, cl)
        us = float(np.median(timed_reps(lambda: dec(q, Ks, Vs, cl), reps, flush))) * 1000
        C.check(C.lib().tactic_sparse_decode_plan_set_events(ctypes.byref(dec.plan), stage_ev.array), "set_events")
        acc = np.zeros(len(STAGE_NAMES))
        n_ev = 5
        for _ in range(n_ev):
            flush()
            dec(q, Ks, Vs, cl)
            torch.cuda.synchronize()
            acc += [stage_ev.elapsed(i, i + 1) for i in range(len(STAGE_NAMES))]
        C.check(C.lib().tactic_sparse_decode_plan_set_events(ctypes.byref(dec.plan), None), "set_events")
        return us, acc / n_ev * 1000

    points = []
    ab_union = None
    for P in Ps:
        dec = T.SparseDecoder(batch, ncl, T.decode_params(P))
        us, stage_us = timed_and_staged(dec)
        _, sq, skv = dec(q, Ks, Vs, cl)
        torch.cuda.synchronize()
        tb = touched_bytes(dec.view(), cl, skv, G)
        kq = sq.cpu().numpy() / lens[:, None]
        ku = skv.cpu().numpy() / lens[:, None]
        gbps = tb["total"] / (us * 1e3)
        rec = {"target_frac": P, "sparse_us": round(us, 2), "dense_us": round(us_dense, 2),
               "speedup_vs_dense": round(us_dense / us, 3),
               "touched_mb": round(tb["total"] / 1e6, 3),
               "touched_parts_mb": {k: round(v / 1e6, 3) for k, v in tb.items() if k != "total"},
               "hbm_gbps": round(gbps, 1), "hbm_frac_peak": round(gbps / HBM_PEAK_GBPS, 4),
               "hbm_frac_read_ceiling": round(gbps / ceiling, 4) if ceiling else None,
               "byte_bound_speedup": round(dense_bytes / tb["total"], 3),
               "stages_us": {n: round(float(t), 2) for n, t in zip(STAGE_NAMES, stage_us)},
               "attn_gbps": round(tb["union_kv"] / (float(stage_us[ATT]) * 1e3), 1),
               "selected_frac": {"head_mean": round(float(kq.mean()), 5),
                                 "head_median": round(float(np.median(kq)), 5),
                                 "head_max": round(float(kq.max()), 5), "union_mean": round(float(ku.mean()), 5),
                                 "union_max": round(float(ku.max()), 5)}}
        if B == 1 and Hq <= 32 and lens[0] >= 1 << 20:
            rec["k_per_query_head"] = [int(x) for x in sq.cpu().numpy()[0]]
            rec["union_per_kv_head"] = [int(x) for x in skv.cpu().numpy()[0]]
        points.append(rec)
        if union_ab is not None and P == union_ab:
            ab_union = (us, float(stage_us[ATT] + stage_us[COMB]), int(skv.sum()))
        del dec
    ablation = None
    if ab_union is not None:
        dph = T.SparseDecoder(batch, ncl, T.decode_params(union_ab, use_union=0))
        us_ph, st_ph = timed_and_staged(dph)
        _, _, skv_ph = dph(q, Ks, Vs, cl)
        att_ph = float(st_ph[ATT] + st_ph[COMB])
        ablation = {"target_frac": union_ab, "per_head_us": round(us_ph, 2), "union_us": round(ab_union[0], 2),
                    "per_head_attn_us": round(att_ph, 2), "union_attn_us": round(ab_union[1], 2),
                    "attn_speedup_from_union": round(att_ph / ab_union[1], 3),
                    "kv_rows_per_head_over_union": round(int(skv_ph.sum()) / max(1, ab_union[2]), 3)}
        del dph
    sort_path = "LDS" if max(ncl) <= 8192 else ("LDS pieces" if max(ncl) <= 32768 else "workspace")
    out = {"batch": B, "seq_lens": (list(map(int, wl.seq_lens)) if B > 1 else int(wl.seq_lens[0])),
           "n_q_heads": Hq, "n_kv_heads": Hkv, "clusters_per_seq": (list(map(int, ncl)) if B > 1 else int(ncl[0])),
           "cluster_sort": sort_path, "kmeans_ms": round(km_ms, 2), "dense_us": round(us_dense, 2),
           "dense_gbps": round(dense_bytes / (us_dense * 1e3), 1), "points": points}
    if ablation is not None:
        out["union_ablation"] = ablation
    del den, q, Ks, Vs, cl, cb
    torch.cuda.empty_cache()
    return out, host


def oracle_config_timings(hosts: dict, P: float) -> dict:
    """The fp64 oracle's decode (per group, scaled to one layer) on the host
    cores, with all BLAS threads and with one, and its K-means (10
    iterations) on one group, for the small workloads."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import kmeans as OK
    from oracle import tactic as OT
    all_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    res = {}
    for name, host in hosts.items():
        r = {"groups_timed": len(host["groups"]), "groups_per_layer": host["groups_per_layer"]}
        for label, th in (("all_threads", all_threads), ("one_thread", 1)):
            with threadpool_limits(limits=th):
                t = 0.0
                for gi in host["groups"]:
                    t0 = time.perf_counter()
                    OT.decode_group(gi["Q"], gi["Ks"], gi["Vs"], gi["cent"], gi["off"], P)
                    t += time.perf_counter() - t0
            r[f"decode_us_per_layer_{label}"] = round(t / len(host["groups"]) * host["groups_per_layer"] * 1e6, 1)
        gi = host["groups"][0]
        with threadpool_limits(limits=all_threads):
            t0 = time.perf_counter()
            km = OK.kmeans(gi["K"], gi["init"], max_iters=10)
            t = time.perf_counter() - t0
        r["kmeans_s_per_group_all_threads"] = round(t, 3)
        r["kmeans_iters"] = int(km.iters)
        r["threads"] = {"all": int(all_threads), "one": 1}
        res[name] = r
    return res


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="ctx128k_b4_32layer", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--layers", type=int, default=0, help="override the layer count (0: the workload's)")
    ap.add_argument("--target-frac", type=float, default=0.9)
    ap.add_argument("--clusters", choices=["kmeans", "labels"], default="kmeans")
    ap.add_argument("--cpu-groups", type=int, default=96,
                    help="(sequence, KV head) groups the CPU oracle times, all groups of layer 0, then layer 1, ...")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-ablation", action="store_true", help="skip the per-head (no-union) comparison")
    ap.add_argument("--no-paged", action="store_true", help="skip the paged-cache comparison")
    ap.add_argument("--no-recent", action="store_true", help="skip the recent-token / re-clustering run")
    ap.add_argument("--no-sweep", action="store_true", help="skip the query-concentration sweep")
    ap.add_argument("--calibrate", action="store_true",
                    help="also run a plain 1 GiB device copy (reference dispatch for HBM counters)")
    ap.add_argument("--no-configs", action="store_true", help="skip the records of the other workloads")
    ap.add_argument("--config-reps", type=int, default=20, help="timed calls per point of those records")
    ap.add_argument("--no-ceiling", action="store_true", help="skip the streaming-read ceiling measurement")
    return ap.parse_args()


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library runs on a single MI355X and has no multi-GPU path "
              "(the decode shards by (sequence, KV head) with no exchange, so each GPU would run its share "
              "of the KV heads at the same shape).",
              file=sys.stderr)
        sys.exit(2)
    import paper_2502_12216_amd as T

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = "cuda"
    wl = synth.WORKLOADS[args.workload]
    layers = args.layers or wl.layers
    B, Hq, Hkv = wl.batch, wl.n_q_heads, wl.n_kv_heads
    G = Hq // Hkv
    ncl = list(wl.cluster_counts)
    batch = T.RaggedBatch(wl.seq_lens, Hq, Hkv)
    P = float(np.float32(args.target_frac))

    # ---------------------------------------------------------------- inputs + clustering
    qs, Ks, Vs, cls = [], [], [], []
    keep = 0 if args.no_paged else min(layers, 4)  # layers whose token-order K/V the paged run needs
    K_tok, V_tok, perms = [], [], []
    kmeans_ms = 0.0
    builder = T.ClusterBuilder(batch, ncl, max_iters=wl.kmeans_iters) if args.clusters == "kmeans" else None
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_gen = time.time()
    for l in range(layers):
        inp = synth.make_layer(wl, l, device=dev)
        if builder is not None:
            init = torch.as_tensor(synth.kmeans_init_all(wl, l), device=dev)
            ev0.record()
            cb = builder(inp.K, inp.V, init)
            ev1.record()
            torch.cuda.synchronize()
            kmeans_ms += ev0.elapsed_time(ev1)
            qs.append(inp.q)
            Ks.append(cb.K_sorted)
            Vs.append(cb.V_sorted)
            cls.append(cb.clusters)
            if l < keep:
                K_tok.append(inp.K)
                V_tok.append(inp.V)
                perms.append(cb.perm)
            del cb
        else:
            lay = synth.label_layout(inp)
            qs.append(inp.q)
            Ks.append(lay.K_sorted)
            Vs.append(lay.V_sorted)
            cls.append(T.ClusterSet(lay.centroids, lay.offsets, ncl))
            if l < keep:
                K_tok.append(inp.K)
                V_tok.append(inp.V)
                perms.append(lay.perm)
            del lay
        del inp
        if l % 4 == 3 or l == layers - 1:
            log(f"layer {l + 1}/{layers} ready ({time.time() - t_gen:.1f}s, k-means {kmeans_ms / 1000:.2f}s)")
    torch.cuda.synchronize()

    if args.calibrate:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("calibration copy of 1 GiB done")

    params = T.decode_params(P)
    dec = T.SparseDecoder(batch, ncl, params)
    dense = T.DenseDecoder(batch)
    flush = Flusher(dev)

    def sparse_step():
        for l in range(layers):
            dec(qs[l], Ks[l], Vs[l], cls[l])

    def dense_step():
        for l in range(layers):
            dense(qs[l], Ks[l], Vs[l])

    def timed(step, n, per_step=None):
        """Mean milliseconds per step over n steps; per_step, if given, receives
        every step's own time (events between the steps, same stream)."""
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
        torch.cuda.synchronize()
        ev0.record()
        evs[0].record()
        for i in range(n):
            step()
            evs[i + 1].record()
        ev1.record()
        torch.cuda.synchronize()
        if per_step is not None:
            per_step.extend(evs[i].elapsed_time(evs[i + 1]) for i in range(n))
        return ev0.elapsed_time(ev1) / n

    for _ in range(args.warmup):
        sparse_step()
        dense_step()
    step_ms = []
    ms_sparse = timed(sparse_step, args.steps, step_ms)
    log(f"sparse step {ms_sparse:.3f} ms")
    ms_dense = timed(dense_step, args.steps)
    log(f"dense step {ms_dense:.3f} ms")
    sdpa = dense_sdpa(qs[0], Ks[0], Vs[0], wl, max(3, args.steps), dense(qs[0], Ks[0], Vs[0]).clone())
    log(f"torch SDPA dense layer: {sdpa}")

    # ---------------------------------------------------------------- per-stage timing (HIP events)
    NS = len(STAGE_NAMES)
    import ctypes
    from paper_2502_12216_amd import _capi as C
    stage_ev = TimingEvents(NS + 1)
    arr = stage_ev.array

    def stage_times(decoder, call=None, n_layers=None, per_layer=None):
        """Mean per-kernel milliseconds over args.steps passes of every layer, from
        events the library records between its launches on the decode stream;
        per_layer, if given, receives each call's first-to-last event time."""
        call = call or (lambda l: decoder(qs[l], Ks[l], Vs[l], cls[l]))
        C.check(C.lib().tactic_sparse_decode_plan_set_events(ctypes.byref(decoder.plan), arr), "set_events")
        acc = np.zeros(NS)
        nrep = 0
        for _ in range(args.steps):
            for l in range(n_layers or layers):
                call(l)
                torch.cuda.synchronize()
                for i in range(NS):
                    acc[i] += stage_ev.elapsed(i, i + 1)
                if per_layer is not None:
                    per_layer.append(stage_ev.elapsed(0, NS))
                nrep += 1
        C.check(C.lib().tactic_sparse_decode_plan_set_events(ctypes.byref(decoder.plan), None), "set_events")
        return acc / nrep

    layer_ms = []
    stage_ms = stage_times(dec, per_layer=layer_ms)
    stage_names = STAGE_NAMES

    # ---------------------------------------------------------------- GQA-union ablation (Sec. 4.5)
    ablation = None
    if not args.no_ablation:
        dec_ph = T.SparseDecoder(batch, ncl, T.decode_params(P, use_union=0))

        def per_head_step():
            for l in range(layers):
                dec_ph(qs[l], Ks[l], Vs[l], cls[l])

        per_head_step()
        ms_ph = timed(per_head_step, args.steps)
        st_ph = stage_times(dec_ph)
        rows_ph = rows_un = 0
        for l in range(layers):
            _, _, skv_ph = dec_ph(qs[l], Ks[l], Vs[l], cls[l])
            _, _, skv_un = dec(qs[l], Ks[l], Vs[l], cls[l])
            rows_ph += int(skv_ph.sum())
            rows_un += int(skv_un.sum())
        ablation = {"per_head_us_per_layer": round(ms_ph * 1000 / layers, 2),
                    "per_head_attn_us": round(float(st_ph[ATT] + st_ph[COMB]) * 1000, 2),
                    "union_attn_us": round(float(stage_ms[ATT] + stage_ms[COMB]) * 1000, 2),
                    "attn_speedup_from_union": round(float((st_ph[ATT] + st_ph[COMB]) /
                                                           (stage_ms[ATT] + stage_ms[COMB])), 3),
                    "kv_rows_per_head_over_union": round(rows_ph / max(1, rows_un), 3)}
        del dec_ph
        log(f"per-head step {ms_ph:.3f} ms")

    # ---------------------------------------------------------------- paged cache (Sec. 4.6)
    paged = None
    if keep:
        PS = 16
        g_pages = torch.Generator().manual_seed(11)
        pcs = []
        for l in range(keep):
            npg = sum((n + PS - 1) // PS for n in wl.seq_lens)
            pcs.append(T.PagedCache.from_token_order(K_tok[l], V_tok[l], batch, PS,
                                                     page_order=torch.randperm(npg, generator=g_pages),
                                                     perm=perms[l].contiguous()))
        del K_tok, V_tok

        def contiguous_part():
            for l in range(keep):
                dec(qs[l], Ks[l], Vs[l], cls[l])

        def paged_part():
            for l in range(keep):
                dec.paged(qs[l], pcs[l], cls[l])

        paged_part()
        ms_c = timed(contiguous_part, args.steps)
        ms_p = timed(paged_part, args.steps)
        st_c = stage_times(dec, n_layers=keep)
        st_p = stage_times(dec, call=lambda l: dec.paged(qs[l], pcs[l], cls[l]), n_layers=keep)
        ub = []
        for l in range(keep):
            _, _, skv = dec(qs[l], Ks[l], Vs[l], cls[l])
            ub.append(float(skv.sum()) * 512)
        ub = float(np.mean(ub))
        paged = {"page_size": PS, "layers": keep, "placement": "pages in token order at random page ids, "
                 "cluster order through perm",
                 "sparse_us_per_layer": round(ms_p * 1000 / keep, 2),
                 "sparse_us_per_layer_cluster_sorted": round(ms_c * 1000 / keep, 2),
                 "attn_us": round(float(st_p[ATT]) * 1000, 2),
                 "attn_us_cluster_sorted": round(float(st_c[ATT]) * 1000, 2),
                 "sample_us": round(float(st_p[SEL]) * 1000, 2),
                 "sample_us_cluster_sorted": round(float(st_c[SEL]) * 1000, 2),
                 "attn_gbps": round(ub / (float(st_p[ATT]) * 1e6), 1),
                 "attn_gbps_cluster_sorted": round(ub / (float(st_c[ATT]) * 1e6), 1)}
        del pcs
        log(f"paged step ({keep} layers) {ms_p:.3f} ms vs {ms_c:.3f} ms cluster-sorted")

    # ---------------------------------------------------------------- recent tokens + re-clustering (Sec. 1)
    recent = None
    if not args.no_recent and len(set(wl.seq_lens)) == 1:
        T_rec = 2048
        n = int(wl.seq_lens[0])
        kvp = batch.kv_indptr_host
        inp0 = synth.make_layer(wl, 0, device=dev)  # layer 0 in token order
        cache = T.RecentTailCache(Hq, Hkv, list(wl.seq_lens), recluster_every=T_rec, cluster_div=n // ncl[0],
                                  kmeans_iters=wl.kmeans_iters, target_frac=P, seed=5, device=dev)
        cut = n - T_rec

        def timed_once(fn):
            torch.cuda.synchronize()
            ev0.record()
            fn()
            ev1.record()
            torch.cuda.synchronize()
            return ev0.elapsed_time(ev1)

        ms_prefill = timed_once(lambda: cache.prefill([inp0.K[:, kvp[b]:kvp[b] + cut] for b in range(B)],
                                                      [inp0.V[:, kvp[b]:kvp[b] + cut] for b in range(B)]))
        for i in range(T_rec - 1):
            rows = [int(kvp[b]) + cut + i for b in range(B)]
            cache.append(inp0.K[:, rows].transpose(0, 1), inp0.V[:, rows].transpose(0, 1))
        q0 = qs[0]

        def decode_us():
            for _ in range(20):  # warm-up (the appends before leave the GPU lightly loaded)
                cache.decode(q0)
            return float(np.median(timed_reps(lambda: cache.decode(q0), 30, flush))) * 1000

        us_tail = decode_us()
        tail_now = cache.recent[0]
        rows = [int(kvp[b]) + n - 1 for b in range(B)]
        ms_warm = timed_once(lambda: cache.append(inp0.K[:, rows].transpose(0, 1), inp0.V[:, rows].transpose(0, 1)))
        assert cache.recent[0] == 0, "the last append re-clusters"
        us_fresh = decode_us()
        cache.warm_start = False
        ms_cold = timed_once(cache.recluster)
        us_cold_fresh = decode_us()
        recent = {"layer": 0, "tail_tokens": tail_now, "recluster_every": T_rec,
                  "sparse_us_with_tail": round(us_tail, 2), "sparse_us_after_recluster": round(us_fresh, 2),
                  "sparse_us_after_cold_recluster": round(us_cold_fresh, 2),
                  "prefill_cluster_ms": round(ms_prefill, 2),
                  "recluster_warm_ms": round(ms_warm, 2), "recluster_cold_ms": round(ms_cold, 2),
                  "amortized_us_per_step_warm": round(ms_warm * 1000 / T_rec, 2),
                  "amortized_us_per_step_cold": round(ms_cold * 1000 / T_rec, 2),
                  "note": "one layer of the workload; prefill of n - 2048 tokens, 2047 appended, the 2048th "
                          "append re-clusters from the previous centroids (warm), then a cold re-clustering of "
                          "the same cache for comparison; the warm time includes the append; decode times are "
                          "medians of 30 calls, caches flushed before each"}
        del cache, inp0
        log(f"recent tail: decode {us_tail:.1f} us with {tail_now} recent tokens, re-clustering warm {ms_warm:.1f} ms "
            f"cold {ms_cold:.1f} ms")

    # ---------------------------------------------------------------- query-concentration sweep
    sweep = None
    if not args.no_sweep:
        points = []
        # one sequence at every point, then the two concentrated points at the timed batch of 4
        for wl_s in synth.sweep_workloads() + synth.sweep_workloads(4, betas=(1.0, 2.0), readings=(False,)):
            inp_s = synth.make_layer(wl_s, 0, device=dev)
            ncl_s = list(wl_s.cluster_counts)
            n_s = int(wl_s.seq_lens[0])
            B_s = len(wl_s.seq_lens)
            batch_s = T.RaggedBatch(wl_s.seq_lens, wl_s.n_q_heads, wl_s.n_kv_heads)
            bld = T.ClusterBuilder(batch_s, ncl_s, max_iters=wl_s.kmeans_iters)
            cb_s = bld(inp_s.K, inp_s.V, torch.as_tensor(synth.kmeans_init_all(wl_s, 0), device=dev))
            dec_s = T.SparseDecoder(batch_s, ncl_s, T.decode_params(P))
            den_s = T.DenseDecoder(batch_s)
            args_s = (inp_s.q, cb_s.K_sorted, cb_s.V_sorted)
            for _ in range(5):
                dec_s(*args_s, cb_s.clusters)
                den_s(*args_s)
            us_s = float(np.median(timed_reps(lambda: dec_s(*args_s, cb_s.clusters), 30, flush))) * 1000
            us_d = float(np.median(timed_reps(lambda: den_s(*args_s), 30, flush))) * 1000
            _, sq_s, skv_s = dec_s(*args_s, cb_s.clusters)
            b_sparse = touched_bytes(dec_s.view(), cb_s.clusters, skv_s, wl_s.n_q_heads // wl_s.n_kv_heads)["total"]
            b_dense = float(n_s) * B_s * wl_s.n_kv_heads * 512
            points.append({"batch": B_s, "beta": wl_s.beta, "reading": "mean" if wl_s.q_mean else "sum",
                           "head_frac_mean": round(float(sq_s.double().mean()) / n_s, 5),
                           "union_frac_mean": round(float(skv_s.double().mean()) / n_s, 5),
                           "sparse_us": round(us_s, 2), "dense_us": round(us_d, 2),
                           "speedup": round(us_d / us_s, 3), "byte_bound_speedup": round(b_dense / b_sparse, 3)})
            del inp_s, cb_s, dec_s, den_s, bld, args_s
        sweep = {"workload": "batch x 131072 tokens (batch 1 at every point, 4 at two), 32 query / 8 KV heads, "
                             "8192 K-means clusters per sequence (10 iterations), P = 0.9; query = beta (sum or "
                             "mean of k_h in 1..8 centres + noise)",
                 "timing": "median of 30 calls of one layer, L2 and Infinity Cache flushed before each",
                 "points": points}
        log("concentration sweep: " + ", ".join(f"B={p['batch']} b={p['beta']:g}/{p['reading']} U={p['union_frac_mean']:.3f} "
                                                f"x{p['speedup']:.2f}" for p in points))

    # ---------------------------------------------------------------- selection statistics, bytes
    sel_q, sel_kv, tb = [], [], []
    for l in range(layers):
        _, sq, skv = dec(qs[l], Ks[l], Vs[l], cls[l])
        torch.cuda.synchronize()
        sel_q.append(sq.cpu().numpy().copy())
        sel_kv.append(skv.cpu().numpy().copy())
        v = dec.view()
        tb.append(touched_bytes(v, cls[l], skv, G))
        tb[-1]["sampled_all"] = float(v["fit"][..., 11].sum()) * 256  # what the sampling kernel reads
    sel_q, sel_kv = np.array(sel_q), np.array(sel_kv)
    lens = np.array(wl.seq_lens, dtype=np.float64)
    bytes_centroids = tb[0]["centroids"]
    bytes_samples = np.array([t["samples_outside_union"] for t in tb])   # per layer
    bytes_union = np.array([t["union_kv"] for t in tb])                  # per layer
    bytes_layer = bytes_centroids + bytes_samples + bytes_union
    dense_bytes_layer = float(lens.sum()) * Hkv * 512
    us_sparse = ms_sparse * 1000 / layers
    us_dense = ms_dense * 1000 / layers
    us_dense_best = min(us_dense, sdpa["us_per_layer"]) if sdpa.get("us_per_layer") else us_dense
    gbps = float(bytes_layer.mean()) / (us_sparse * 1e3)
    stage_us = stage_ms * 1000
    # each kernel's own algorithmic bytes: the sampler reads every sampled row
    stage_bytes = [0.0] * len(STAGE_NAMES)
    stage_bytes[0] = bytes_centroids
    stage_bytes[SEL] = float(np.mean([t["sampled_all"] for t in tb]))
    stage_bytes[ATT] = float(bytes_union.mean())
    dom = int(np.argmax(stage_us))
    dom_bytes = stage_bytes[dom]
    roof = {
        "kernel": stage_names[dom],
        "bound": "hbm",
        "achieved": round(dom_bytes / (stage_us[dom] * 1e3), 1),
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(dom_bytes / (stage_us[dom] * 1e3) / HBM_PEAK_GBPS, 4),
        "traffic": None,
    }
    if stage_bytes[dom] == 0.0:
        roof["bound"] = "alu"
    roof["traffic"] = profiled_traffic(STAGE_KERNEL[stage_names[dom]])
    kq = sel_q.astype(np.float64) / lens[None, :, None]
    ku = sel_kv.astype(np.float64) / lens[None, :, None]

    # ---------------------------------------------------------------- streaming-read ceiling
    ceiling = None
    if not args.no_ceiling:
        buf = torch.zeros(4 << 30, dtype=torch.uint8, device=dev)
        probe = T.stream_read_gbps(buf, reps=10)
        ceiling = probe["best_gbps"]
        del buf
        log(f"streaming-read ceiling {ceiling:.0f} GB/s (by workgroups: "
            f"{ {k: round(v) for k, v in probe['gbps_by_workgroups'].items()} })")

    # ---------------------------------------------------------------- the other workloads (and the timed shape over P), one layer each
    configs, hosts = None, {}
    if not args.no_configs:
        configs = {}
        for name, Ps, hg, ab in (("ctx4k_gqa4", (0.9,), [(0, 0), (0, 1)], None),
                                 ("ctx32k_llama8b", (0.8, 0.9, 0.95), [(0, 0), (0, 5)], 0.9),
                                 ("ragged16_16k_128k", (0.9,), None, None),
                                 ("ctx1m", (0.9,), None, None),
                                 # the timed shape, one layer, over the target fraction
                                 ("ctx128k_b4_32layer", (0.5, 0.8, 0.9, 0.95, 0.99), None, None)):
            rec, host = config_record(T, synth.WORKLOADS[name], Ps, dev, flush, args.config_reps, stage_ev, ceiling,
                                      host_groups=None if args.no_cpu else hg, union_ab=ab)
            configs[name] = rec
            if host is not None:
                hosts[name] = host
            log(f"{name}: " + ", ".join(f"P={p['target_frac']} {p['sparse_us']:.1f} us vs dense {p['dense_us']:.1f} us "
                                        f"(x{p['speedup_vs_dense']:.2f}, union {p['selected_frac']['union_mean']:.3f})"
                                        for p in rec["points"]))

    # ---------------------------------------------------------------- CPU oracle on a bounded sample
    cpu = None
    if not args.no_cpu:
        from oracle import tactic as OT
        n_groups = max(1, min(args.cpu_groups, layers * B * Hkv))
        kvp = batch.kv_indptr_host
        t_or = 0.0
        for idx in range(n_groups):
            l, r = divmod(idx, B * Hkv)
            b, g = divmod(r, Hkv)
            cl_l = cls[l]
            clp = cl_l.cl_indptr_host
            s0, s1 = int(kvp[b]), int(kvp[b + 1])
            c0, c1 = int(clp[b]), int(clp[b + 1])
            Qg = qs[l][b, g * G:(g + 1) * G].double().cpu().numpy()
            Kg = Ks[l][g, s0:s1].double().cpu().numpy()
            Vg = Vs[l][g, s0:s1].double().cpu().numpy()
            cent = cl_l.centroids[g, c0:c1].double().cpu().numpy()
            off = cl_l.offsets[g, c0 + b:c1 + b + 1].cpu().numpy().astype(np.int64)
            t0 = time.perf_counter()
            OT.decode_group(Qg, Kg, Vg, cent, off, P)
            t_or += time.perf_counter() - t0
            del Qg, Kg, Vg, cent, off
        per_group = t_or / n_groups
        try:
            from threadpoolctl import threadpool_info
            blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        except Exception:
            blas_threads = 1
        cpu = {"value": round(per_group * B * Hkv * 1e6, 1), "unit": "us/layer", "cores": int(blas_threads),
               "kind": "oracle",
               "sample": f"{n_groups} (sequence, KV head) groups (every group of layer 0, then layer 1, ...; "
                         f"{B * Hkv} per layer), fp64 NumPy oracle decode_group each, {t_or:.1f} s in total, "
                         f"mean per group x {B * Hkv} groups = one layer; "
                         f"host {platform.processor() or platform.machine()}, "
                         f"{len(os.sched_getaffinity(0))} cores visible"}
        log(f"cpu oracle {per_group:.2f} s per group")
        if hosts:
            cpu["configs"] = oracle_config_timings(hosts, P)
            log(f"cpu oracle on the small workloads: {cpu['configs']}")

    res = {
        "metric": METRIC,
        "value": round(us_sparse, 2),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_sparse, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "seq_len": int(wl.seq_lens[0]), "layers": layers,
                   "n_q_heads": Hq, "n_kv_heads": Hkv, "head_dim": 128, "clusters_per_seq": int(ncl[0]),
                   "target_frac": args.target_frac, "clustering": args.clusters},
        "us_per_layer_dist": {
            "steps_p10": round(float(np.percentile(step_ms, 10)) * 1000 / layers, 2),
            "steps_median": round(float(np.median(step_ms)) * 1000 / layers, 2),
            "steps_p90": round(float(np.percentile(step_ms, 90)) * 1000 / layers, 2),
            "layer_calls_p10": round(float(np.percentile(layer_ms, 10)) * 1000, 2),
            "layer_calls_median": round(float(np.median(layer_ms)) * 1000, 2),
            "layer_calls_p90": round(float(np.percentile(layer_ms, 90)) * 1000, 2),
            "note": "steps: each timed step / layers; layer_calls: one layer's six launches between "
                    "library events, synchronised per call (layers differ in their selected fraction)"},
        "dense_us_per_layer": round(us_dense, 2),
        "dense_sdpa": sdpa,
        "speedup_vs_dense": round(us_dense_best / us_sparse, 3),
        "speedup_vs_own_dense": round(us_dense / us_sparse, 3),
        "hbm_gbps": round(gbps, 1),
        "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
        "dense_hbm_gbps": round(dense_bytes_layer / (us_dense * 1e3), 1),
        "bytes_per_layer": {"centroids": bytes_centroids, "samples_outside_union": float(bytes_samples.mean()),
                            "union_kv": float(bytes_union.mean()), "dense_kv": dense_bytes_layer,
                            "note": "touched bytes: centroids + offsets, distinct sampled key rows of a group "
                                    "outside its union, and the union's K and V rows; mean over layers"},
        "stages_us_per_layer": {n: round(float(t), 2) for n, t in zip(stage_names, stage_us)},
        "stage_timing": "HIP events recorded by the library between its launches on the decode stream, "
                        "created with hipEventDisableSystemFence (no cache flush at each event)",
        "selected_frac": {"head_mean": round(float(kq.mean()), 5), "head_median": round(float(np.median(kq)), 5),
                          "head_max": round(float(kq.max()), 5), "union_mean": round(float(ku.mean()), 5),
                          "union_max": round(float(ku.max()), 5)},
        "roofline": roof,
        "hbm_read_ceiling_gbps": round(ceiling, 1) if ceiling else None,
        "hbm_read_ceiling_note": ("best median of 10 reads of a 4 GiB buffer by tactic_probe_stream_read over "
                                  "launch shapes " + str({k: round(v, 1) for k, v in probe["gbps_by_workgroups"].items()})
                                  if ceiling else None),
        "attn_frac_of_read_ceiling": (round(stage_bytes[ATT] / (stage_us[ATT] * 1e3) / ceiling, 4) if ceiling else None),
        "cpu_baseline": cpu,
        "configs": configs,
        "union_ablation": ablation,
        "paged_kv": paged,
        "recent_tail": recent,
        "concentration_sweep": sweep,
    }
    if args.clusters == "kmeans":
        res["kmeans"] = {"seconds_all_layers": round(kmeans_ms / 1000, 3), "layers": layers,
                         "iters": wl.kmeans_iters}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
