#!/usr/bin/env python3
"""Benchmark of the vector-index output head on one MI355X.

Workload: the Qwen3-0.6B-shaped head (|V| = 151936, d = 1024, bf16 rows,
fp32 accumulation), M = 32, ef_construction = 200, k = 50, 1024 seeded
synthetic queries, each served at batch size 1.

A step is one pass of the head over the 1024 queries, one call per query on
one stream: HNSW search (greedy upper layers + layer-0 beam, ef = 128) and
scatter of the 50 retrieved logits into a -inf-filled 151936-wide row.  The
exact dense head (GEMV + fused top-k, then the same scatter) runs as the
baseline leg in the same run, with the same protocol.  `value` is the HNSW
head's queries per second; the dense leg, the ef sweep, recall@50 (against
the exact dense head) and the per-kernel roofline figures are reported next
to it.  The CPU baseline is the plain-C oracle's HNSW search on the same
graph (one thread, a bounded sample of the same queries).

The batch-graph leg builds a single-layer graph over W_out on the GPU
(vie_index_build_gpu: exact 128 nearest rows by inner product, the
neighbour-selection heuristic, reverse edges) and searches it at B = 1 with
the same protocol, next to the HNSW graph built on the host CPUs.

The recall-target leg finds, for each traversal (sequential beam, 8
expansions per step, 8 per step on int8 rows with the exact re-rank; on the
HNSW graph and on the batch graph), the smallest beam width in 128 .. 4096
whose recall@k reaches 0.95 on the first 128 queries, and its per-call time
next to the dense head's.

The other workloads (--workload tiny | llama3.2-1b | gemma3-270m |
llama3.2-3b) run the same protocol at their own shapes, ef and k; the Gemma
shape adds a k sweep (20, 50, 100) and the Llama-3.2-3B shape a sweep of
queries per call (1, 4, 16, 64: HNSW with one workgroup per query against
the dense head, which switches to the matrix cores from 3 queries on).

    python bench.py [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

METRIC = "us/query and queries/s of top-k output head at B=1 (HNSW vs dense), %HBM peak"
HBM_PEAK_GBS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
KERNEL_SRC = os.path.join(ROOT, "paper_2608_27460_amd", "csrc", "kernels.hip")


def measured_traffic(workload):
    """HBM bytes per launch from the committed counter summary of this workload
    (FETCH_SIZE + WRITE_SIZE, each scaled by the same counter's reading of a
    plain device copy of known size).  None when no summary exists or when the
    kernel source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "hbm_traffic_%s.txt" % workload)
    if not os.path.exists(path):
        return {}
    sha = hashlib.sha1(open(KERNEL_SRC, "rb").read()).hexdigest()
    out, src = {}, None
    for line in open(path):
        f = line.split()
        if len(f) == 2 and f[0] == "source_sha1":
            src = f[1]
        elif len(f) == 3 and f[0] == "traffic_bytes":
            out[f[1]] = float(f[2])
    return out if src == sha else {}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="qwen3-0.6b")
    ap.add_argument("--ef", type=int, default=0, help="beam width (default: the workload's middle ef)")
    ap.add_argument("--k", type=int, default=0, help="results per query (default: the workload's middle k)")
    ap.add_argument("--queries", type=int, default=0, help="queries per step (default: the workload's)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the oracle CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cache", default=os.environ.get("VIE_CACHE", "/tmp/vie_cache"))
    ap.add_argument("--sweep-ef", type=lambda x: [int(v) for v in x.split(",") if v], default=[512, 1024, 2048, 4096],
                    help="extra beam widths of the ef sweep (comma separated)")
    ap.add_argument("--sweep-queries", type=int, default=128, help="queries per extra sweep point")
    ap.add_argument("--int8-widths", type=lambda x: [int(v) for v in x.split(",") if v], default=[1, 4, 8],
                    help="expansion widths of the int8-row sweep (comma separated; empty: skip)")
    ap.add_argument("--forced", type=int, default=64,
                    help="forced-inclusion tokens of the forced leg (ids 0..n-1 stand in for special tokens)")
    ap.add_argument("--widths", type=lambda x: [int(v) for v in x.split(",") if v], default=[2, 4, 8],
                    help="expansion widths of the vie_query_ex sweep (comma separated)")
    ap.add_argument("--batch-graph-k", type=int, default=128,
                    help="candidates per node of the GPU-built batch graph leg (0: skip the leg)")
    ap.add_argument("--batch-graph-ef", type=lambda x: [int(v) for v in x.split(",") if v], default=[512, 1024],
                    help="extra beam widths searched on the batch graph (first --sweep-queries queries)")
    ap.add_argument("--target-recall", type=float, default=0.95,
                    help="recall@k that the beam-width search of each traversal aims for (0 skips it)")
    ap.add_argument("--target-ef", type=lambda x: [int(v) for v in x.split(",") if v],
                    default=[128, 256, 512, 1024, 2048, 4096], help="beam widths tried, in order, for the target")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="finish with a device copy of this many MiB (a known-size reference for HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the head is a single-GPU path (sharding it over several "
              "GPUs is designed but not built), so --gpus %d is not supported." % args.gpus, file=sys.stderr)
        return 2

    import torch

    from paper_2608_27460_amd import synth
    from paper_2608_27460_amd import vie

    if not torch.cuda.is_available():
        print("bench.py needs an MI355X", file=sys.stderr)
        return 2
    wl = synth.WORKLOADS[args.workload]
    Q = args.queries or wl.Q
    k = args.k or wl.k[len(wl.k) // 2]
    ef = args.ef or wl.ef[len(wl.ef) // 2]
    s = wl.elem_bytes
    dev = torch.device("cuda:0")

    t0 = time.time()
    W = wl.make_w()
    H, _ = wl.make_queries(W, Q=Q)
    log("[bench] inputs %s: %.1fs" % (wl.name, time.time() - t0))

    os.makedirs(args.cache, exist_ok=True)
    gpath = os.path.join(args.cache, "%s-M%d-efC%d-seed%d.vie" % (wl.name, wl.M, wl.efC, wl.seed_levels))
    t0 = time.time()
    ix = None
    cpu_build_s = None
    if os.path.exists(gpath):
        try:
            ix = vie.Index.load(gpath, W)
            log("[bench] graph loaded from %s" % gpath)
        except vie.VieError as e:
            log("[bench] cached graph rejected (%s); rebuilding" % e)
    if ix is None:
        nt = min(16, os.cpu_count() or 1)
        ix = vie.Index.build(W, wl.dtype, wl.M, wl.efC, seed=wl.seed_levels, n_threads=nt)
        ix.save(gpath)
        cpu_build_s = time.time() - t0
        log("[bench] graph built with %d threads in %.1fs" % (nt, cpu_build_s))
    info = ix.info()

    Wd = vie.host_to_torch(W, wl.dtype).to(dev)
    Hd = vie.host_to_torch(H, wl.dtype).to(dev)
    ix.to_device(Wd)
    head = vie.DenseHead(Wd, max_batch=1, max_k=k)
    ids = torch.empty((Q, k), dtype=torch.int32, device=dev)
    lg = torch.empty((Q, k), dtype=torch.float32, device=dev)
    st = torch.empty((Q, 2), dtype=torch.int32, device=dev)
    dids = torch.empty((Q, k), dtype=torch.int32, device=dev)
    dlg = torch.empty((Q, k), dtype=torch.float32, device=dev)
    row = torch.empty((1, wl.V), dtype=torch.float32, device=dev)  # the step's full-vocab logits
    hv = [Hd[q:q + 1] for q in range(Q)]
    iv, lv, sv = [ids[q:q + 1] for q in range(Q)], [lg[q:q + 1] for q in range(Q)], [st[q:q + 1] for q in range(Q)]
    div, dlv = [dids[q:q + 1] for q in range(Q)], [dlg[q:q + 1] for q in range(Q)]
    stream = torch.cuda.current_stream(dev)

    def hnsw_step(ef_=ef):
        for q in range(Q):
            ix.query_into(hv[q], k, ef_, iv[q], lv[q], sv[q])
            vie.scatter_into(iv[q], lv[q], wl.V, row)

    def dense_step():
        for q in range(Q):
            vie.dense_topk_into(Wd, hv[q], k, div[q], dlv[q], head.workspace)
            vie.scatter_into(div[q], dlv[q], wl.V, row)

    def timed(step, K, W_):
        # K steps between two events on the launch stream (nothing else recorded inside)
        for _ in range(W_):
            step()
        torch.cuda.synchronize()
        outer = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        t = time.perf_counter()
        outer[0].record(stream)
        for i in range(K):
            step()
        outer[1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t
        return outer[0].elapsed_time(outer[1]), wall

    def per_call_us(fn, n_calls):
        # mean event-timed duration of n_calls back-to-back calls (after one warm-up call)
        fn(0)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for c in range(n_calls):
            fn(c)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / n_calls

    # ---- HNSW head (the method) ----------------------------------------
    log("[bench] HNSW head: %d steps x %d queries, ef=%d" % (args.steps, Q, ef))
    h_ms, h_wall = timed(hnsw_step, args.steps, args.warmup)
    stats = st.cpu().numpy().astype(np.int64)
    hnsw_ids = ids.cpu().numpy()
    # ---- dense head (the baseline) -------------------------------------
    log("[bench] dense head: %d steps x %d queries" % (args.steps, Q))
    d_ms, d_wall = timed(dense_step, args.steps, args.warmup)
    exact_ids = dids.cpu().numpy()
    # ---- per-launch kernel time: Q back-to-back calls between two events ----
    # (the roofline figures; the kernels alone, no scatter and no events in between)
    h_us = per_call_us(lambda c: ix.query_into(hv[c], k, ef, iv[c], lv[c], sv[c]), Q)
    d_us = per_call_us(lambda c: vie.dense_topk_into(Wd, hv[c], k, div[c], dlv[c], head.workspace), Q)

    def recall(a, b, kk=None):
        kk = kk or a.shape[1]
        return float(np.mean([len(set(x[:kk].tolist()) & set(y[:kk].tolist())) / kk for x, y in zip(a, b)]))

    def reach(index, width, int8, nq):
        # the smallest beam of --target-ef whose recall@k on the first nq
        # queries reaches --target-recall; per-call kernel time as per_call_us
        ri = torch.empty((nq, k), dtype=torch.int32, device=dev)
        rl = torch.empty((nq, k), dtype=torch.float32, device=dev)
        tried = {}
        for e in sorted(v for v in args.target_ef if v >= k):
            us = per_call_us(lambda c: index.query_into(hv[c], k, e, ri[c:c + 1], rl[c:c + 1], None, width, int8), nq)
            r = recall(ri.cpu().numpy(), exact_ids[:nq])
            tried[str(e)] = [round(us, 2), round(r, 4)]
            if r >= args.target_recall:
                return {"ef": e, "us_per_query": round(us, 2), "recall_at_k": round(r, 4), "tried": tried}
        return {"ef": None, "us_per_query": None, "recall_at_k": None, "tried": tried}

    target = {}
    tq = min(Q, args.sweep_queries)

    # ---- ef sweep (same protocol; one warm-up and one timed pass each) ----
    # Beams wider than the workload's own ef values run on the first
    # --sweep-queries queries only.
    sweep = {}
    for e in sorted(set(wl.ef) | {ef} | set(args.sweep_ef)):
        nq = Q if e <= max(max(wl.ef), ef) else min(Q, args.sweep_queries)

        def step_e(e=e, nq=nq):
            for q in range(nq):
                ix.query_into(hv[q], k, e, iv[q], lv[q], sv[q])
                vie.scatter_into(iv[q], lv[q], wl.V, row)

        ms_e, _ = timed(step_e, 1, 1)
        sweep[str(e)] = {"us_per_query": round(ms_e * 1e3 / nq, 2), "queries": nq,
                         "recall_at_k": round(recall(ids.cpu().numpy()[:nq], exact_ids[:nq]), 4),
                         "recall_at_2": round(recall(ids.cpu().numpy()[:nq], exact_ids[:nq], 2), 4),
                         "mean_n_dist": float(st.cpu().numpy()[:nq, 0].mean())}
    # ---- all queries in one launch (one workgroup each) -------------------
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ix.query_into(Hd, k, ef, ids, lg, st)
    a.record(stream)
    ix.query_into(Hd, k, ef, ids, lg, st)
    b.record(stream)
    torch.cuda.synchronize()
    batched_s = a.elapsed_time(b) * 1e-3
    batched_qps = Q / batched_s
    bst = st.cpu().numpy().astype(np.float64)
    batched_bytes = float((bst[:, 0] * wl.d * s + bst[:, 1] * wl.M0 * 4 + wl.d * s + k * 8).sum())
    batched_gbs = batched_bytes / batched_s / 1e9

    # ---- expansion-width sweep (vie_query_ex; B = 1, first 256 queries) ---
    w_sweep = {}
    for wd in args.widths:
        nq = min(Q, 256)
        wi = torch.empty((nq, k), dtype=torch.int32, device=dev)
        wlg = torch.empty((nq, k), dtype=torch.float32, device=dev)
        ws = torch.empty((nq, 2), dtype=torch.int32, device=dev)
        w_us = per_call_us(lambda c: ix.query_into(hv[c], k, ef, wi[c:c + 1], wlg[c:c + 1], ws[c:c + 1], wd), nq)
        wst = ws.cpu().numpy().astype(np.int64)
        w_sweep[str(wd)] = {"us_per_query": round(w_us, 2), "queries": nq,
                            "recall_at_k": round(recall(wi.cpu().numpy(), exact_ids[:nq]), 4),
                            "recall_at_2": round(recall(wi.cpu().numpy(), exact_ids[:nq], 2), 4),
                            "mean_n_dist": float(wst[:, 0].mean()), "mean_n_expand": float(wst[:, 1].mean())}

    if args.target_recall > 0:
        log("[bench] beam widths reaching recall@k %.2f" % args.target_recall)
        target["hnsw"] = reach(ix, 1, False, tq)
        target["hnsw_width_8"] = reach(ix, 8, False, tq)

    # ---- int8 rows for layer 0, exact re-rank (B = 1, first 256 queries) ----
    q_sweep = {}
    if args.int8_widths and wl.d % 16 == 0:
        qrows, qscale = vie.quantize_rows(Wd, wl.dtype)
        ix.attach_int8(qrows, qscale)
        for wd in args.int8_widths:
            nq = min(Q, 256)
            wi = torch.empty((nq, k), dtype=torch.int32, device=dev)
            wlg = torch.empty((nq, k), dtype=torch.float32, device=dev)
            ws = torch.empty((nq, 2), dtype=torch.int32, device=dev)
            w_us = per_call_us(lambda c: ix.query_into(hv[c], k, ef, wi[c:c + 1], wlg[c:c + 1], ws[c:c + 1], wd,
                                                       True), nq)
            wst = ws.cpu().numpy().astype(np.int64)
            q_sweep[str(wd)] = {"us_per_query": round(w_us, 2), "queries": nq,
                                "recall_at_k": round(recall(wi.cpu().numpy(), exact_ids[:nq]), 4),
                                "recall_at_2": round(recall(wi.cpu().numpy(), exact_ids[:nq], 2), 4),
                                "mean_n_dist": float(wst[:, 0].mean()), "mean_n_expand": float(wst[:, 1].mean()),
                                "row_bytes_per_query": float(wst[:, 0].mean() * wl.d)}
        wb = max(args.int8_widths)
        torch.cuda.synchronize()
        ix.query_into(Hd, k, ef, ids, lg, st, wb, True)
        a.record(stream)
        ix.query_into(Hd, k, ef, ids, lg, st, wb, True)
        b.record(stream)
        torch.cuda.synchronize()
        q_sweep["batched_width_%d" % wb] = {"queries_per_s": round(Q / (a.elapsed_time(b) * 1e-3), 1),
                                             "recall_at_k": round(recall(ids.cpu().numpy(), exact_ids), 4)}
        if args.target_recall > 0:
            target["hnsw_int8_width_8"] = reach(ix, 8, True, tq)
        ix.attach_int8(None, None)
        if not args.batch_graph_k:
            del qrows, qscale

    # ---- batch graph built on the GPU (vie_index_build_gpu), searched at B = 1 ----
    batch = None
    if args.batch_graph_k:
        Kb = min(args.batch_graph_k, wl.V - 1)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        bix = vie.Index.build_gpu(Wd, Kb, wl.M0)  # first call: includes the GEMM library's set-up
        first_s = time.perf_counter() - t0
        del bix
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        bix = vie.Index.build_gpu(Wd, Kb, wl.M0)
        build_s = time.perf_counter() - t0
        bsweep = {}
        for e in sorted(set(wl.ef) | {ef} | set(args.batch_graph_ef)):
            nq = Q if e <= max(max(wl.ef), ef) else min(Q, args.sweep_queries)
            bi = torch.empty((nq, k), dtype=torch.int32, device=dev)
            bl = torch.empty((nq, k), dtype=torch.float32, device=dev)
            bs = torch.empty((nq, 2), dtype=torch.int32, device=dev)
            b_us = per_call_us(lambda c: bix.query_into(hv[c], k, e, bi[c:c + 1], bl[c:c + 1], bs[c:c + 1]), nq)
            bst = bs.cpu().numpy().astype(np.int64)
            bsweep[str(e)] = {"us_per_query": round(b_us, 2), "queries": nq,
                              "recall_at_k": round(recall(bi.cpu().numpy(), exact_ids[:nq]), 4),
                              "recall_at_2": round(recall(bi.cpu().numpy(), exact_ids[:nq], 2), 4),
                              "mean_n_dist": float(bst[:, 0].mean()), "mean_n_expand": float(bst[:, 1].mean())}
        bix.query_into(Hd, k, ef, ids, lg, st)
        torch.cuda.synchronize()
        a.record(stream)
        bix.query_into(Hd, k, ef, ids, lg, st)
        b.record(stream)
        torch.cuda.synchronize()
        if args.target_recall > 0:
            target["batch_graph"] = reach(bix, 1, False, tq)
            target["batch_graph_width_8"] = reach(bix, 8, False, tq)
            if args.int8_widths and wl.d % 16 == 0:
                bix.attach_int8(qrows, qscale)
                target["batch_graph_int8_width_8"] = reach(bix, 8, True, tq)
                bix.attach_int8(None, None)
        batch = {"K": Kb, "M0": wl.M0, "build_s": round(build_s, 4), "first_build_s": round(first_s, 4),
                 "cpu_hnsw_build_s": None if cpu_build_s is None else round(cpu_build_s, 2),
                 "entry": bix.info()["entry"], "ef_sweep": bsweep,
                 "batched_queries_per_s": round(Q / (a.elapsed_time(b) * 1e-3), 1),
                 "batched_recall_at_k": round(recall(ids.cpu().numpy(), exact_ids), 4)}
        del bix

    # ---- forced-inclusion tokens (stand-in: the first 64 ids; B = 1) -------
    forced = None
    if args.forced:
        nq = min(Q, 256)
        fids = torch.arange(args.forced, dtype=torch.int32, device=dev)
        fi = torch.empty((nq, k + args.forced), dtype=torch.int32, device=dev)
        fl = torch.empty((nq, k + args.forced), dtype=torch.float32, device=dev)
        f_us = per_call_us(lambda c: ix.query_forced_into(hv[c], k, ef, fids, fi[c:c + 1], fl[c:c + 1]), nq)
        p_us = per_call_us(lambda c: ix.query_into(hv[c], k, ef, iv[c], lv[c]), nq)
        forced = {"n": args.forced, "ids": "0..%d" % (args.forced - 1), "queries": nq,
                  "us_per_query": round(f_us, 2), "search_only_us_per_query": round(p_us, 2)}

    # ---- k sweep (workloads quoted at several k; B = 1, first 256 queries) --
    k_sweep = {}
    if len(wl.k) > 1:
        nq = min(Q, 256)
        for kk in wl.k:
            ik = torch.empty((nq, kk), dtype=torch.int32, device=dev)
            lk = torch.empty((nq, kk), dtype=torch.float32, device=dev)
            dk = torch.empty((nq, kk), dtype=torch.int32, device=dev)
            dlk = torch.empty((nq, kk), dtype=torch.float32, device=dev)
            hk = vie.DenseHead(Wd, max_batch=1, max_k=kk)
            h_us_k = per_call_us(lambda c: ix.query_into(hv[c], kk, ef, ik[c:c + 1], lk[c:c + 1]), nq)
            d_us_k = per_call_us(lambda c: vie.dense_topk_into(Wd, hv[c], kk, dk[c:c + 1], dlk[c:c + 1],
                                                               hk.workspace), nq)
            k_sweep[str(kk)] = {"hnsw_us_per_query": round(h_us_k, 2), "dense_us_per_query": round(d_us_k, 2),
                                "recall_at_k": round(recall(ik.cpu().numpy(), dk.cpu().numpy()), 4),
                                "queries": nq}
            del hk

    # ---- batch sweep (queries per call; HNSW: one workgroup per query) ----
    b_sweep = {}
    if len(wl.B) > 1:
        bdense = vie.DenseHead(Wd, max_batch=max(wl.B), max_k=k)
        for Bc in wl.B:
            ncall = Q // Bc
            bi = torch.empty((ncall * Bc, k), dtype=torch.int32, device=dev)
            bl = torch.empty((ncall * Bc, k), dtype=torch.float32, device=dev)
            di = torch.empty((ncall * Bc, k), dtype=torch.int32, device=dev)
            dl = torch.empty((ncall * Bc, k), dtype=torch.float32, device=dev)
            hs = [Hd[c * Bc:(c + 1) * Bc] for c in range(ncall)]
            h_call = per_call_us(lambda c: ix.query_into(hs[c], k, ef, bi[c * Bc:(c + 1) * Bc],
                                                         bl[c * Bc:(c + 1) * Bc]), ncall)
            d_call = per_call_us(lambda c: vie.dense_topk_into(Wd, hs[c], k, di[c * Bc:(c + 1) * Bc],
                                                               dl[c * Bc:(c + 1) * Bc], bdense.workspace), ncall)
            b_sweep[str(Bc)] = {"hnsw_us_per_call": round(h_call, 2), "dense_us_per_call": round(d_call, 2),
                                "hnsw_queries_per_s": round(Bc * 1e6 / h_call, 1),
                                "dense_queries_per_s": round(Bc * 1e6 / d_call, 1),
                                "dense_hbm_frac": round(wl.V * wl.d * s / (d_call * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                                "recall_at_k": round(recall(bi.cpu().numpy(), di.cpu().numpy()), 4),
                                "calls": ncall}
        del bdense

    # ---- roofline figures ----------------------------------------------------
    n_dist, n_exp = stats[:, 0].astype(np.float64), stats[:, 1].astype(np.float64)
    hnsw_bytes = n_dist * wl.d * s + n_exp * wl.M0 * 4 + wl.d * s + k * 8  # per launch (one query)
    hnsw_gbs = float(hnsw_bytes.mean()) / (h_us * 1e-6) / 1e9
    dense_bytes = wl.V * wl.d * s + wl.d * s + k * 8
    dense_gbs = dense_bytes / (d_us * 1e-6) / 1e9

    traffic = measured_traffic(args.workload)
    h_qps = Q * args.steps / (h_ms * 1e-3)
    d_qps = Q * args.steps / (d_ms * 1e-3)

    # ---- CPU baseline: the oracle on the host cores ----------------------
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import oracle as O
        g, _ = O.load_graph(gpath)
        O.check_graph(g)
        done, t = 0, time.perf_counter()
        while time.perf_counter() - t < args.cpu_seconds and done < Q:
            O.hnsw_search(W, wl.dtype, g, H[done:done + 8], k, ef, validate=False)
            done += min(8, Q - done)
        cpu_s = time.perf_counter() - t
        t = time.perf_counter()
        O.topk(W, wl.dtype, H[:1], k)
        bf_s = time.perf_counter() - t
        cpu = {"value": round(done / cpu_s, 2), "unit": "queries/s", "cores": 1, "kind": "oracle",
               "sample": "HNSW search (ef=%d, k=%d) of the first %d of the %d queries on the same graph, one "
                         "thread; exact brute-force top-k of 1 query: %.2f s" % (ef, k, done, Q, bf_s),
               "brute_force_queries_per_s": round(1.0 / bf_s, 3)}

    out = {
        "metric": METRIC,
        "value": round(h_qps, 1),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(h_ms / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == synth.BF16 else "f32",
        "data": "synthetic, seeded: rows N(0, I/d) x LogNormal(0, 0.25) norms, h = sum of 3 rows + N(0, 0.1/d)",
        "config": {"workload": wl.name, "V": wl.V, "d": wl.d, "B": 1, "k": k, "ef": ef, "M": wl.M, "M0": wl.M0,
                   "ef_construction": wl.efC, "queries_per_step": Q, "accumulate": "fp32",
                   "graph": {"maxlevel": info["maxlevel"], "entry": info["entry"]}},
        "hnsw": {"us_per_query": round(h_ms * 1e3 / (Q * args.steps), 2), "queries_per_s": round(h_qps, 1),
                 "kernel_us": round(h_us, 2), "recall_at_k": round(recall(hnsw_ids, exact_ids), 4),
                 "recall_at_2": round(recall(hnsw_ids, exact_ids, 2), 4),
                 "mean_n_dist": float(n_dist.mean()), "mean_n_expand": float(n_exp.mean()),
                 "row_bytes_per_query": float((n_dist * wl.d * s).mean()),
                 "batched_queries_per_s": round(batched_qps, 1), "wall_s": round(h_wall, 3), "ef_sweep": sweep,
                 "width_sweep": w_sweep or None, "k_sweep": k_sweep or None, "batch_sweep": b_sweep or None,
                 "int8_sweep": q_sweep or None, "forced": forced, "batch_graph": batch,
                 "recall_target": ({"recall_at_k": args.target_recall, "queries": tq,
                                    "dense_us_per_query": round(d_us, 2), **target} if target else None)},
        "dense": {"us_per_query": round(d_ms * 1e3 / (Q * args.steps), 2), "queries_per_s": round(d_qps, 1),
                  "kernel_us": round(d_us, 2), "wall_s": round(d_wall, 3)},
        "roofline": {"kernel": "hnsw_kernel", "bound": "hbm", "achieved": round(hnsw_gbs, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(hnsw_gbs / HBM_PEAK_GBS, 5),
                     "traffic": traffic.get("hnsw_kernel")},
        "roofline_batched": {"kernel": "hnsw_kernel, all %d queries in one launch" % Q, "bound": "hbm",
                             "achieved": round(batched_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": round(batched_gbs / HBM_PEAK_GBS, 4), "traffic": None},
        "roofline_dense": {"kernel": "dense_stream_kernel+dense_merge_kernel", "bound": "hbm", "achieved": round(dense_gbs, 1),
                           "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(dense_gbs / HBM_PEAK_GBS, 4),
                           "traffic": traffic.get("dense_head")},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
    return 0


if __name__ == "__main__":
    sys.exit(main())
