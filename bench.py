#!/usr/bin/env python3
"""Benchmark of the vector-index output head on one MI355X.

Workload (default): the Llama-3.2-3B-shaped head, |V| = 128256 rows of
d = 3072 bf16 values (fp32 accumulation), k = 50, 1024 seeded synthetic
queries served one per call (B = 1), HNSW graph with M = 32 (M0 = 64),
ef_construction = 200, built by the library on the host CPUs.

The beam width is the one the method needs: for each traversal (the
sequential search; 8, 32 or 64 expansions per step; 8, 16, 32 or 64 per step
on int8 rows with the exact re-rank; 128 per step in teams only) the smallest ef of 128, 256, ..., 4096 whose recall@50 reaches
0.95 on the first 128 queries (recall against the exact dense head, itself
parity-tested against the oracle).  The team traversals (128 workgroups
sharing each query's row scoring) walk exactly the path of their
one-workgroup twin and take its ef.  The fastest of them at its ef is the
headline traversal.

A step is 128 queries, each a call of the head at B = 1 on one stream: the
search and the scatter of its 50 logits into a -inf-filled 128256-wide row;
successive steps take successive blocks of the 1024 queries.  `value` is the
headline traversal's queries per second over the timed steps.  Beside it, in
the same run and with the same protocol: the sequential traversal at its own
ef, the exact dense head (GEMV + fused top-k + scatter; calls alternate
between two copies of W_out so that no call finds the matrix in the 256 MB
Infinity Cache), per-call percentiles (p10/p50/p90), an fp32-row leg of the
same shape (the paper's precision), queries per call B = 1/4/16/64, the
batch graph built on the GPU, forced-inclusion tokens, the per-launch kernel
times and algorithmic bytes behind the roofline figures, and the oracle on
the host cores: its queries/s, and its ids, counts and expansion order
compared with the GPU's for every query it ran.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--quick]

Other workloads: --workload tiny | qwen3-0.6b | llama3.2-1b | gemma3-270m.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import json
import os
import platform
import sys
import time

import numpy as np

METRIC = "us/query and queries/s of top-k output head at B=1 (HNSW vs dense), %HBM peak"
HBM_PEAK_GBS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
KERNEL_SRC = os.path.join(ROOT, "paper_2608_27460_amd", "csrc", "kernels.hip")
NODE_MASK = (1 << 26) - 1

TEAM = 128  # workgroups per query of the team traversals
TRAVERSALS = {  # name -> (expansions per layer-0 step, int8 rows for layer 0, workgroups per query)
    "sequential": (1, False, 1),
    "width8": (8, False, 1),
    "width32": (32, False, 1),
    "width64": (64, False, 1),
    "int8_width8": (8, True, 1),
    "int8_width16": (16, True, 1),
    "int8_width32": (32, True, 1),
    "int8_width64": (64, True, 1),
    "width64_team%d" % TEAM: (64, False, TEAM),
    "width128_team%d" % TEAM: (128, False, TEAM),
    "int8_width32_team%d" % TEAM: (32, True, TEAM),
    "int8_width64_team%d" % TEAM: (64, True, TEAM),
    "int8_width128_team%d" % TEAM: (128, True, TEAM),
}


def solo_of(trav):
    """The one-workgroup traversal a team traversal reproduces exactly (None
    when there is none: 128 per step needs a team's smaller LDS)."""
    width, int8, _ = TRAVERSALS[trav]
    return next((t for t, v in TRAVERSALS.items() if v == (width, int8, 1)), None)


def kernel_of(trav):
    width, int8, team = TRAVERSALS[trav]
    if width == 1 and not int8 and team == 1:
        return "hnsw_kernel"
    return "hnsw_multi_kernel (%s rows, %d per step%s%s)" % (
        "int8" if int8 else "stored", width, ", exact re-rank" if int8 else "",
        ", %d workgroups per query" % team if team > 1 else "")


def measured_traffic(workload):
    """HBM bytes per launch from the committed counter summary of this workload
    (FETCH_SIZE + WRITE_SIZE, each scaled by the same counter's reading of a
    plain device copy of known size).  Empty when no summary exists or when
    the kernel source has changed since the counters were taken."""
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


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def pct(a):
    a = np.asarray(a, np.float64)
    return {"p10": round(float(np.percentile(a, 10)), 2), "p50": round(float(np.percentile(a, 50)), 2),
            "p90": round(float(np.percentile(a, 90)), 2), "mean": round(float(a.mean()), 2)}


def layer_counts(trace, graph, M):
    """(upper-layer expansions, layer-0 expansions, distance evaluations above
    layer 0) of one query, replayed from its expansion record on the graph:
    on each upper layer the search visits its entry point and every
    neighbour of the nodes it expands; the first entry point is scored once."""
    t = trace[trace >= 0]
    node, lay = t & NODE_MASK, t >> 27
    up_exp = int((lay >= 1).sum())
    n_up = 1
    for L in sorted(set(lay[lay >= 1].tolist()), reverse=True):
        nodes = node[lay == L]
        vis = {int(nodes[0])}
        for u in nodes:
            lst = graph["upper"][graph["upper_off"][u] + L - 1]
            vis.update(int(x) for x in lst if x >= 0)
        n_up += len(vis) - 1
    return up_exp, int((lay == 0).sum()), n_up


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="llama3.2-3b")
    ap.add_argument("--k", type=int, default=0, help="results per query (default: the workload's middle k)")
    ap.add_argument("--step-queries", type=int, default=128, help="queries per timed step")
    ap.add_argument("--target-recall", type=float, default=0.95)
    ap.add_argument("--calib-queries", type=int, default=128, help="queries that choose each traversal's ef")
    ap.add_argument("--ef-ladder", type=lambda x: [int(v) for v in x.split(",") if v],
                    default=[128, 256, 512, 1024, 2048, 4096])
    ap.add_argument("--traversal", default="", help="force the headline traversal (default: the fastest)")
    ap.add_argument("--ef", type=int, default=0, help="force the headline beam width (skips the calibration)")
    ap.add_argument("--quick", action="store_true",
                    help="headline and dense legs only (no fp32, batch, graph, forced or CPU legs): for profilers")
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="wall-clock budget of the oracle leg")
    ap.add_argument("--cpu-threads", type=int, default=0, help="oracle threads (default: min(16, nproc))")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-fp32", action="store_true")
    ap.add_argument("--forced", type=int, default=64,
                    help="forced-inclusion tokens of the forced leg (ids 0..n-1 stand in for special tokens)")
    ap.add_argument("--share-groups", type=lambda x: [int(v) for v in x.split(",") if v], default=[2, 4],
                    help="row-sharing group sizes of the one-launch leg (empty: skip the leg)")
    ap.add_argument("--batch-graph-k", type=int, default=128,
                    help="candidates per node of the GPU-built batch graph leg (0: skip the leg)")
    ap.add_argument("--cache", default=os.environ.get("VIE_CACHE", "/tmp/vie_cache"))
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
    Q = wl.Q
    k = args.k or wl.k[len(wl.k) // 2]
    s = wl.elem_bytes
    SQ = min(args.step_queries, Q)
    nthreads = min(16, os.cpu_count() or 1)
    dev = torch.device("cuda:0")

    t0 = time.time()
    W = wl.make_w()
    H, _ = wl.make_queries(W)
    log("[bench] inputs %s: %.1fs" % (wl.name, time.time() - t0))

    def graph_for(Wh, dtype, tag):
        os.makedirs(args.cache, exist_ok=True)
        path = os.path.join(args.cache, "%s-%s-M%d-efC%d-seed%d.vie" % (wl.name, tag, wl.M, wl.efC, wl.seed_levels))
        t = time.time()
        if os.path.exists(path):
            try:
                ix_ = vie.Index.load(path, Wh)
                log("[bench] graph loaded from %s" % path)
                return ix_, None
            except vie.VieError as e:
                log("[bench] cached graph rejected (%s); rebuilding" % e)
        ix_ = vie.Index.build(Wh, dtype, wl.M, wl.efC, seed=wl.seed_levels, n_threads=nthreads)
        ix_.save(path)
        log("[bench] %s graph built with %d threads in %.1fs" % (tag, nthreads, time.time() - t))
        return ix_, time.time() - t

    ix, cpu_build_s = graph_for(W, wl.dtype, synth.DTYPE_NAMES[wl.dtype])
    info = ix.info()
    graph = ix.export()

    Wd = vie.host_to_torch(W, wl.dtype).to(dev)
    Hd = vie.host_to_torch(H, wl.dtype).to(dev)
    ix.to_device(Wd)
    stream = torch.cuda.current_stream(dev)
    row = torch.empty((1, wl.V), dtype=torch.float32, device=dev)  # a call's full-vocabulary logits
    hv = [Hd[q:q + 1] for q in range(Q)]
    qrows = qscale = None
    if wl.d % 16 == 0:
        qrows, qscale = vie.quantize_rows(Wd, wl.dtype)
        ix.attach_int8(qrows, qscale)
    travs = [t for t in TRAVERSALS if not TRAVERSALS[t][1] or qrows is not None]

    def out_bufs(n, kk=k):
        return (torch.empty((n, kk), dtype=torch.int32, device=dev), torch.empty((n, kk), dtype=torch.float32,
                                                                                device=dev),
                torch.empty((n, 2), dtype=torch.int32, device=dev))

    def events(n):
        return [torch.cuda.Event(enable_timing=True) for _ in range(n)]

    def back_to_back(fn, n):
        """Mean event-timed duration (us) of n back-to-back calls after one warm-up call."""
        fn(0)
        torch.cuda.synchronize()
        e0, e1 = events(2)
        e0.record(stream)
        for c in range(n):
            fn(c)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / n

    def per_call(fn, n):
        """Event-timed duration (us) of each of n calls (an event between calls)."""
        fn(0)
        torch.cuda.synchronize()
        ev = events(n + 1)
        ev[0].record(stream)
        for c in range(n):
            fn(c)
            ev[c + 1].record(stream)
        torch.cuda.synchronize()
        return [ev[c].elapsed_time(ev[c + 1]) * 1e3 for c in range(n)]

    def timed_steps(step, K, Wu):
        """K steps between two events on the launch stream (nothing recorded inside)."""
        for i in range(Wu):
            step(i)
        torch.cuda.synchronize()
        e0, e1 = events(2)
        t = time.perf_counter()
        e0.record(stream)
        for i in range(K):
            step(Wu + i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1), time.perf_counter() - t

    def recall(a, b, kk=None):
        kk = kk or a.shape[1]
        return float(np.mean([len(set(x[:kk].tolist()) & set(y[:kk].tolist())) / kk for x, y in zip(a, b)]))

    # ---- exact top-k of every query (the dense head; parity-tested) --------
    dense = vie.DenseHead(Wd, max_batch=64, max_k=max(k, max(wl.k)))
    ex_ids = torch.empty((Q, k), dtype=torch.int32, device=dev)
    ex_lg = torch.empty((Q, k), dtype=torch.float32, device=dev)
    for q0 in range(0, Q, 64):
        vie.dense_topk_into(Wd, Hd[q0:q0 + 64], k, ex_ids[q0:q0 + 64], ex_lg[q0:q0 + 64], dense.workspace)
    exact_ids = ex_ids.cpu().numpy()

    def search_into(index, trav, ef, q, ids_, lg_, st_=None, trace=None):
        width, int8, team = TRAVERSALS[trav]
        index.query_into(hv[q], k, ef, ids_, lg_, st_, width, int8, trace, team)

    # ---- each traversal's beam width for the recall target ----------------
    nc = min(Q, args.calib_queries)
    ci, cl, cs = out_bufs(nc)
    calib = {}
    chosen = {}
    for trav in travs:
        if args.ef:
            chosen[trav] = args.ef
            continue
        tried = {}
        if TRAVERSALS[trav][2] > 1 and solo_of(trav):  # the results of its one-workgroup twin: time it at that ef
            ef = chosen.get(solo_of(trav))
            if ef:
                us = back_to_back(lambda c: search_into(ix, trav, ef, c, ci[c:c + 1], cl[c:c + 1]), nc)
                r = recall(ci.cpu().numpy(), exact_ids[:nc])
                tried[str(ef)] = {"us_per_query": round(us, 2), "recall_at_k": round(r, 4)}
                chosen[trav] = ef
            calib[trav] = {"ef": ef, "tried": tried, "same_results_as": solo_of(trav)}
            log("[bench] %s: ef %s (as %s)" % (trav, ef, solo_of(trav)))
            continue
        for ef in args.ef_ladder:
            if ef < k:
                continue
            us = back_to_back(lambda c: search_into(ix, trav, ef, c, ci[c:c + 1], cl[c:c + 1]), nc)
            r = recall(ci.cpu().numpy(), exact_ids[:nc])
            tried[str(ef)] = {"us_per_query": round(us, 2), "recall_at_k": round(r, 4)}
            if r >= args.target_recall:
                chosen[trav] = ef
                break
        calib[trav] = {"ef": chosen.get(trav), "tried": tried}
        log("[bench] %s: ef %s reaches recall@%d %.2f" % (trav, chosen.get(trav), k, args.target_recall))
    reachable = [t for t in travs if chosen.get(t)]
    if not reachable:
        log("[bench] no traversal reaches the recall target; the headline falls back to the widest beam")
        chosen = {t: max(args.ef_ladder) for t in travs}
        reachable = travs
    if args.traversal:
        head_trav = args.traversal
    elif args.ef:
        head_trav = "int8_width128_team%d" % TEAM if qrows is not None else "width128_team%d" % TEAM
    else:
        head_trav = min(reachable, key=lambda t: calib[t]["tried"][str(chosen[t])]["us_per_query"])
    ef = chosen[head_trav]

    # ---- headline: K steps of SQ queries at B = 1 --------------------------
    hi, hl, hs = out_bufs(Q)
    iv = [hi[q:q + 1] for q in range(Q)]
    lv = [hl[q:q + 1] for q in range(Q)]
    sv = [hs[q:q + 1] for q in range(Q)]

    def head_step(i, trav=head_trav, ef_=None):
        ef_ = ef_ or chosen[trav]
        q0 = (i * SQ) % Q
        for q in range(q0, min(Q, q0 + SQ)):
            search_into(ix, trav, ef_, q, iv[q], lv[q], sv[q])
            vie.scatter_into(iv[q], lv[q], wl.V, row)

    log("[bench] headline %s at ef=%d: %d steps x %d queries" % (head_trav, ef, args.steps, SQ))
    h_ms, h_wall = timed_steps(head_step, args.steps, args.warmup)
    # every query once (untimed) for recall, counts and expansion records
    cap = max(ef, k) + 1024
    trace = torch.full((Q, cap), -1, dtype=torch.int32, device=dev)
    width, int8, team = TRAVERSALS[head_trav]
    tb = max(1, 256 // team)  # queries per launch: every team member resident at once
    for q0 in range(0, Q, tb):
        ix.query_into(Hd[q0:q0 + tb], k, ef, hi[q0:q0 + tb], hl[q0:q0 + tb], hs[q0:q0 + tb], width, int8,
                      trace[q0:q0 + tb], team)
    head_ids, head_lg = hi.cpu().numpy(), hl.cpu().numpy()
    head_st = hs.cpu().numpy().astype(np.int64)
    head_tr = trace.cpu().numpy()
    head_calls = per_call(lambda c: (search_into(ix, head_trav, ef, c, iv[c], lv[c]),
                                     vie.scatter_into(iv[c], lv[c], wl.V, row)), min(Q, 256))
    head_kernel_us = back_to_back(lambda c: search_into(ix, head_trav, ef, c, iv[c], lv[c]), SQ)

    # ---- the sequential traversal at its own ef (the paper's search) -------
    seq = None
    if head_trav != "sequential" and not args.quick and chosen.get("sequential"):
        ef_s = chosen["sequential"]
        nseq = min(Q, 64)
        calls = per_call(lambda c: (search_into(ix, "sequential", ef_s, c, iv[c], lv[c], sv[c]),
                                    vie.scatter_into(iv[c], lv[c], wl.V, row)), nseq)
        seq = {"ef": ef_s, "queries": nseq, "us_per_query": pct(calls),
               "recall_at_k": round(recall(hi.cpu().numpy()[:nseq], exact_ids[:nseq]), 4),
               "kernel": kernel_of("sequential")}

    # ---- dense head: calls alternate between two copies of W_out -----------
    Wd2 = Wd.clone()
    Ws = [Wd, Wd2]
    di, dl, _ = out_bufs(Q)
    div_, dlv_ = [di[q:q + 1] for q in range(Q)], [dl[q:q + 1] for q in range(Q)]
    dhead = vie.DenseHead(Wd, max_batch=1, max_k=k)

    def dense_call(q, scatter=True):
        vie.dense_topk_into(Ws[q & 1], hv[q], k, div_[q], dlv_[q], dhead.workspace)
        if scatter:
            vie.scatter_into(div_[q], dlv_[q], wl.V, row)

    def dense_step(i):
        q0 = (i * SQ) % Q
        for q in range(q0, min(Q, q0 + SQ)):
            dense_call(q)

    log("[bench] dense head: %d steps x %d queries" % (args.steps, SQ))
    d_ms, d_wall = timed_steps(dense_step, args.steps, args.warmup)
    dense_calls = per_call(lambda c: dense_call(c), min(Q, 256))
    d_kernel_us = back_to_back(lambda c: dense_call(c, scatter=False), SQ)
    # both copies give the same top k, bit for bit (the same kernels on equal bytes), and it is the exact top k
    # of the 64-query passes up to the order of near ties (the passes sum in another order)
    di2, dl2, _ = out_bufs(SQ)
    for q in range(SQ):
        vie.dense_topk_into(Ws[(q + 1) & 1], hv[q], k, di2[q:q + 1], dl2[q:q + 1], dhead.workspace)
    assert np.array_equal(di.cpu().numpy()[:SQ], di2.cpu().numpy()) and \
        np.array_equal(dl.cpu().numpy()[:SQ].view(np.uint32), dl2.cpu().numpy().view(np.uint32))
    assert recall(di.cpu().numpy()[:SQ], exact_ids[:SQ]) >= 0.99
    del Wd2, Ws, di2, dl2

    # ---- roofline figures --------------------------------------------------
    M, M0 = info["M"], info["M0"]
    nd, ne = head_st[:, 0].astype(np.float64), head_st[:, 1].astype(np.float64)
    lc = np.array([layer_counts(head_tr[q], graph, M) for q in range(Q)], np.float64)
    up_exp, l0_exp, nd_up = lc[:, 0], lc[:, 1], lc[:, 2]
    assert np.array_equal(up_exp + l0_exp, ne), "expansion records disagree with the counters"
    lists = up_exp * M * 4 + l0_exp * M0 * 4
    width, int8, team = TRAVERSALS[head_trav]
    if int8:
        nd_l0 = nd - nd_up
        head_bytes = nd_up * wl.d * s + nd_l0 * (wl.d + 4) + np.minimum(max(ef, k), nd_l0) * wl.d * s + lists
    else:
        head_bytes = nd * wl.d * s + lists
    head_bytes = head_bytes + wl.d * s + k * 8
    head_gbs = float(head_bytes[:SQ].mean()) / (head_kernel_us * 1e-6) / 1e9
    dense_bytes = wl.V * wl.d * s + wl.d * s + k * 8
    dense_gbs = dense_bytes / (d_kernel_us * 1e-6) / 1e9
    traffic = measured_traffic(args.workload)
    h_qps = SQ * args.steps / (h_ms * 1e-3)
    d_qps = SQ * args.steps / (d_ms * 1e-3)

    legs = {}
    if not args.quick:
        # ---- fp32 rows of the same shape (the paper's precision) ----------
        if not args.no_fp32 and wl.dtype == synth.BF16:
            W32 = synth.make_w(wl.V, wl.d, synth.F32, wl.seed_w, wl.hub_frac, seed_hub=wl.seed_hub)
            H32, _ = synth.make_queries(W32, synth.F32, Q, wl.seed_q)
            ix32, b32 = graph_for(W32, synth.F32, "f32")
            W32d = vie.host_to_torch(W32, synth.F32).to(dev)
            H32d = vie.host_to_torch(H32, synth.F32).to(dev)
            ix32.to_device(W32d)
            n32 = min(Q, 64)
            e_i, e_l, _ = out_bufs(n32)
            h32 = vie.DenseHead(W32d, max_batch=1, max_k=k)
            dcalls = per_call(lambda c: vie.dense_topk_into(W32d, H32d[c:c + 1], k, e_i[c:c + 1], e_l[c:c + 1],
                                                            h32.workspace), n32)
            ex32 = e_i.cpu().numpy()
            f_trav = head_trav
            if TRAVERSALS[f_trav][1]:
                q32, s32 = vie.quantize_rows(W32d, synth.F32)
                ix32.attach_int8(q32, s32)
            f_i, f_l, _ = out_bufs(n32)
            fw0, f8, ft = TRAVERSALS[f_trav]
            hcalls = None
            for fw in [w for w in (128, 112, 96, 80, 64) if w <= fw0]:
                # fp32 queries take twice the LDS of bf16 ones: the widest step that fits
                try:
                    hcalls = per_call(lambda c, w=fw: ix32.query_into(H32d[c:c + 1], k, ef, f_i[c:c + 1],
                                                                      f_l[c:c + 1], None, w, f8, None, ft), n32)
                    break
                except vie.VieError as e:
                    if e.status != vie.EUNSUPPORTED:
                        raise
            assert hcalls is not None, "no step width fits the fp32 search"

            legs["fp32_rows"] = {
                "W_bytes": wl.V * wl.d * 4, "queries": n32, "dense_us_per_query": pct(dcalls),
                "dense_hbm_frac": round(wl.V * wl.d * 4 / (np.median(dcalls) * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                "hnsw": {"traversal": f_trav, "expansions_per_step": fw, "ef": ef, "us_per_query": pct(hcalls),
                         "recall_at_k": round(recall(f_i.cpu().numpy(), ex32), 4)},
                "graph_build_s": None if b32 is None else round(b32, 1)}
            del ix32, W32d, H32d, h32
            torch.cuda.empty_cache()

        # ---- queries per call (HNSW: one workgroup per query) --------------
        if len(wl.B) > 1:
            bs = {}
            for Bc in wl.B:
                ncall = min(Q // Bc, 64)
                bi, bl, _ = out_bufs(ncall * Bc)
                hb = [Hd[c * Bc:(c + 1) * Bc] for c in range(ncall)]
                w8, i8, tm = TRAVERSALS[head_trav]
                tm = max(1, min(tm, 256 // Bc))  # the team shrinks as the batch grows (all resident at once)
                tm = 1 << (tm.bit_length() - 1)  # a power of two
                h_call = back_to_back(lambda c: ix.query_into(hb[c], k, ef, bi[c * Bc:(c + 1) * Bc],
                                                              bl[c * Bc:(c + 1) * Bc], None, w8, i8, None, tm),
                                      ncall)
                d_call = back_to_back(lambda c: vie.dense_topk_into(Wd, hb[c], k, bi[c * Bc:(c + 1) * Bc],
                                                                    bl[c * Bc:(c + 1) * Bc], dense.workspace), ncall)
                bs[str(Bc)] = {"team": tm, "hnsw_us_per_call": round(h_call, 2), "dense_us_per_call": round(d_call, 2),
                               "hnsw_queries_per_s": round(Bc * 1e6 / h_call, 1),
                               "dense_queries_per_s": round(Bc * 1e6 / d_call, 1),
                               "dense_hbm_frac": round(wl.V * wl.d * s / (d_call * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                               "calls": ncall}
            legs["queries_per_call"] = {"traversal": head_trav, "ef": ef, "B": bs}

        # ---- all queries in one launch --------------------------------------
        torch.cuda.synchronize()
        a, b = events(2)
        w8, i8, _ = TRAVERSALS[head_trav]  # one workgroup per query: 1024 queries fill the device
        w8 = min(w8, 64)  # (128 per step fits only a team's LDS)
        ix.query_into(Hd, k, ef, hi, hl, hs, w8, i8)
        a.record(stream)
        ix.query_into(Hd, k, ef, hi, hl, hs, w8, i8)
        b.record(stream)
        torch.cuda.synchronize()
        one_launch_s = a.elapsed_time(b) * 1e-3
        # its algorithmic bytes: the headline's, scaled by this walk's distance evaluations
        ol_bytes = float(head_bytes.sum()) * float(hs[:, 0].double().mean()) / float(nd.mean())
        legs["one_launch"] = {"queries": Q, "expansions_per_step": w8, "queries_per_s": round(Q / one_launch_s, 1),
                              "hbm_frac": round(ol_bytes / one_launch_s / 1e9 / HBM_PEAK_GBS, 4)}

        # ---- row sharing between the queries of one launch ------------------
        if args.share_groups:
            rs = {}
            w8, i8, _ = TRAVERSALS[head_trav]
            w8 = min(w8, 64)
            for Bc in [b for b in (64, 256, 1024) if b <= Q]:
                row, ref = {}, None
                for sh in [1] + args.share_groups:
                    def launch(_c, sh=sh, Bc=Bc):
                        ix.query_into(Hd[:Bc], k, ef, hi[:Bc], hl[:Bc], hs[:Bc], w8, i8, None, 1, sh)
                    try:
                        ms = back_to_back(launch, 3) / 1e3
                    except vie.VieError as e:  # a group's queries that do not fit in LDS
                        row[str(sh)] = {"error": str(e)[:120]}
                        continue
                    out = (hi[:Bc].cpu().numpy(), hl[:Bc].cpu().numpy().view(np.uint32), hs[:Bc].cpu().numpy())
                    if ref is None:
                        ref = out
                    row[str(sh)] = {"ms_per_launch": round(ms, 3), "queries_per_s": round(Bc / ms * 1e3, 1),
                                    "same_results": all(np.array_equal(a, b) for a, b in zip(out, ref))}
                rs[str(Bc)] = row
            legs["row_sharing"] = {"traversal": "%swidth%d, one workgroup per query" % ("int8_" if i8 else "", w8),
                                   "ef": ef, "share": rs}

        # ---- batch graph built on the GPU, searched at B = 1 ----------------
        if args.batch_graph_k:
            Kb = min(args.batch_graph_k, wl.V - 1)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            bix = vie.Index.build_gpu(Wd, Kb, wl.M0)
            torch.cuda.synchronize()
            first_s = time.perf_counter() - t0
            del bix
            t0 = time.perf_counter()
            bix = vie.Index.build_gpu(Wd, Kb, wl.M0)
            torch.cuda.synchronize()
            build_s = time.perf_counter() - t0
            if qrows is not None:
                bix.attach_int8(qrows, qscale)
            bi, bl, _ = out_bufs(nc)
            tried, bef = {}, None
            for e in args.ef_ladder:
                if e < k:
                    continue
                us = back_to_back(lambda c: search_into(bix, head_trav, e, c, bi[c:c + 1], bl[c:c + 1]), nc)
                r = recall(bi.cpu().numpy(), exact_ids[:nc])
                tried[str(e)] = {"us_per_query": round(us, 2), "recall_at_k": round(r, 4)}
                if r >= args.target_recall:
                    bef = e
                    break
            legs["batch_graph"] = {"K": Kb, "M0": wl.M0, "build_s": round(build_s, 4),
                                   "first_build_s": round(first_s, 4), "traversal": head_trav, "ef": bef,
                                   "tried": tried}
            del bix

        # ---- forced-inclusion tokens (stand-in: the first ids) --------------
        if args.forced:
            nf = min(Q, 128)
            fids = torch.arange(args.forced, dtype=torch.int32, device=dev)
            fi = torch.empty((nf, k + args.forced), dtype=torch.int32, device=dev)
            fl = torch.empty((nf, k + args.forced), dtype=torch.float32, device=dev)
            w8, i8, tm = TRAVERSALS[head_trav]
            f_us = back_to_back(lambda c: ix.query_forced_into(hv[c], k, ef, fids, fi[c:c + 1], fl[c:c + 1], None, w8,
                                                               i8, tm), nf)
            legs["forced"] = {"n": args.forced, "ids": "0..%d" % (args.forced - 1), "queries": nf,
                              "us_per_query": round(f_us, 2), "search_only_us_per_query": round(head_kernel_us, 2)}

    # ---- the oracle on the host cores: throughput and parity ---------------
    cpu = None
    if not args.no_cpu_baseline and not args.quick:
        cpu = oracle_leg(args, wl, W, H, ix, graph, info, head_trav, ef, k, head_ids, head_lg, head_st, head_tr,
                         cap, nthreads)

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
        "config": {"workload": wl.name, "V": wl.V, "d": wl.d, "B": 1, "k": k, "traversal": head_trav, "ef": ef,
                   "M": M, "M0": M0, "ef_construction": wl.efC, "queries": Q, "queries_per_step": SQ,
                   "recall_target": args.target_recall, "accumulate": "fp32",
                   "graph": {"maxlevel": info["maxlevel"], "entry": info["entry"],
                             "build_s_16_threads": None if cpu_build_s is None else round(cpu_build_s, 1)}},
        "hnsw": {"traversal": head_trav, "ef": ef, "kernel": kernel_of(head_trav),
                 "us_per_query": round(h_ms * 1e3 / (SQ * args.steps), 2), "queries_per_s": round(h_qps, 1),
                 "per_call_us": pct(head_calls), "kernel_us": round(head_kernel_us, 2),
                 "recall_at_k": round(recall(head_ids, exact_ids), 4),
                 "recall_at_2": round(recall(head_ids, exact_ids, 2), 4),
                 "mean_n_dist": float(nd.mean()), "mean_n_expand": float(ne.mean()),
                 "mean_upper_n_dist": float(nd_up.mean()), "bytes_per_query": float(head_bytes.mean()),
                 "wall_s": round(h_wall, 3), "sequential": seq, "ef_for_recall_target": calib},
        "dense": {"us_per_query": round(d_ms * 1e3 / (SQ * args.steps), 2), "queries_per_s": round(d_qps, 1),
                  "per_call_us": pct(dense_calls), "kernel_us": round(d_kernel_us, 2), "W_copies": 2,
                  "wall_s": round(d_wall, 3)},
        "legs": legs,
        "roofline": {"kernel": kernel_of(head_trav), "bound": "hbm", "achieved": round(head_gbs, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(head_gbs / HBM_PEAK_GBS, 5),
                     "traffic": traffic.get(head_trav)},
        "roofline_dense": {"kernel": "dense_stream_kernel+dense_merge_kernel", "bound": "hbm",
                           "achieved": round(dense_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": round(dense_gbs / HBM_PEAK_GBS, 4), "traffic": traffic.get("dense_head")},
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


def oracle_leg(args, wl, W, H, ix, graph, info, trav, ef, k, gids, glg, gst, gtr, cap, nthreads):
    """The plain-C oracle (test infrastructure) on the host cores: the same
    traversal on the same graph for as many of the same queries as fit in the
    budget, with T threads over chunks of queries (ctypes releases the GIL),
    plus a few queries on one thread; its ids, counts and expansion records
    are compared with the GPU's for every query it ran."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from oracle import oracle as O
    import parity

    g = O.Graph(wl.V, wl.d, wl.dtype, info["M"], info["M0"], wl.efC, wl.seed_levels, info["maxlevel"],
                info["entry"], graph["levels"], graph["adj0"], graph["upper_off"], graph["upper"])
    width, int8, _ = TRAVERSALS[trav]  # a team walks the one-workgroup path
    oq = osc = None
    if int8:
        oq, osc = O.quantize_rows(W, wl.dtype)

    def run(a, b):
        if int8:
            return O.hnsw_search_q(W, wl.dtype, g, oq, osc, H[a:b], k, ef, width, validate=False, trace_cap=cap)
        if width > 1:
            return O.hnsw_search_multi(W, wl.dtype, g, H[a:b], k, ef, width, validate=False, trace_cap=cap)
        r = O.hnsw_search(W, wl.dtype, g, H[a:b], k, ef, validate=False, trace_cap=cap)
        return r[0], r[1], r[2], r[4]

    T = args.cpu_threads or nthreads
    t1 = time.perf_counter()
    one = [run(q, q + 1) for q in range(2)]
    single_us = (time.perf_counter() - t1) * 1e6 / 2
    results = {}
    t = time.perf_counter()
    nxt = 2
    with cf.ThreadPoolExecutor(T) as ex:
        while time.perf_counter() - t < args.cpu_seconds and nxt < len(H):
            chunk = list(range(nxt, min(len(H), nxt + T)))
            for q, r in zip(chunk, ex.map(lambda q: run(q, q + 1), chunk)):
                results[q] = r
            nxt = chunk[-1] + 1
    wall = time.perf_counter() - t
    for q in range(2):
        results[q] = one[q]
    done = sorted(results)
    same = near = 0
    worst_gap, unexplained = 0.0, []
    ex_sc = {}
    for q in done:
        oid, olg, ost, otr = (x[0] for x in results[q])
        if np.array_equal(gst[q], ost.astype(np.int64)) and np.array_equal(gtr[q], otr):
            same += 1
            continue
        try:
            r = parity.first_divergence(W, wl.dtype, g, H[q], gtr[q], otr, max(ef, k), int8=int8)
            near += 1
            worst_gap = max(worst_gap, r[4] if r else 0.0)
        except AssertionError as e:
            unexplained.append((q, str(e)[:160]))
    ids_equal = sum(int(set(gids[q].tolist()) == set(results[q][0][0].tolist())) for q in done)
    return {"value": round((len(done) - 2) / wall, 2), "unit": "queries/s", "cores": T, "kind": "oracle",
            "sample": "%s search (ef=%d, k=%d) of %d of the %d queries on the same graph: %d on %d threads in "
                      "%.1f s, 2 on one thread" % (trav, ef, k, len(done), len(H), len(done) - 2, T, wall),
            "single_thread_us_per_query": round(single_us, 1), "cpu_model": cpu_model(),
            "nproc": os.cpu_count(),
            "parity": {"queries": len(done), "same_expansions_and_counts": same, "near_tie_divergences": near,
                       "worst_near_tie_gap": worst_gap, "unexplained": unexplained[:4],
                       "same_id_sets": ids_equal}}


if __name__ == "__main__":
    sys.exit(main())
