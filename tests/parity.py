"""Comparison rules between the HIP path and the oracle (shared by the GPU
tests and the benchmark's parity leg).

Tolerances (stated for the head in its specification):
* id sets: an id returned by only one side must score within 1e-4 relative of
  the oracle's k-th score (a near tie at the cut);
* logits: |gpu - exact| <= rel * max(|exact|, 1e-6 * max_j |exact_j|) with
  rel = 1e-5 for fp32 storage and 2e-2 for bf16; the floor (a millionth of
  the query's largest returned logit) only keeps the bound finite for logits
  at zero;
* order: logits non-increasing, ids distinct;
* HNSW traversal: the GPU walked the oracle's path when its expansion record
  (the nodes it expanded, in order) and its counts equal the oracle's; a
  query that parts from the path must do so at a near tie (first_divergence
  below), and is counted instead of compared by ids.
"""
from __future__ import annotations

import concurrent.futures as cf
import os

import numpy as np

from oracle import oracle as O

REL_LOGIT = {0: 1e-5, 1: 2e-2}
REL_CUT = 1e-4


def exact_scores(W, dtype, H, ids):
    B, k = ids.shape
    q = np.repeat(np.arange(B, dtype=np.int32), k)
    return O.pair_scores(W, dtype, H, q, ids.ravel()).reshape(B, k)


def check_logits(W, dtype, H, ids, logits, what=""):
    """Returned logits agree with the exact scores of the returned ids."""
    valid = ids >= 0
    safe = np.where(valid, ids, 0)
    ex = exact_scores(W, dtype, H, safe)
    B, k = ids.shape
    rel = REL_LOGIT[dtype]
    for q in range(B):
        v = valid[q]
        if not v.any():
            continue
        err = np.abs(logits[q, v].astype(np.float64) - ex[q, v])
        floor = 1e-6 * np.abs(ex[q, v]).max()
        allowed = rel * np.maximum(np.abs(ex[q, v]), floor)
        ratio = np.where(allowed > 0, err / np.where(allowed > 0, allowed, 1.0), np.where(err > 0, np.inf, 0.0))
        worst = int(np.argmax(ratio))
        assert err[worst] <= allowed[worst], "%s query %d: logit %.9g vs exact %.9g (allowed %.3g)" % (
            what, q, logits[q, v][worst], ex[q, v][worst], allowed[worst])
        lg = logits[q, v]
        assert np.all(np.diff(lg) <= 0), "%s query %d: logits not sorted" % (what, q)
        assert len(set(ids[q, v].tolist())) == int(v.sum()), "%s query %d: duplicate ids" % (what, q)


def check_id_sets(W, dtype, H, gpu_ids, ora_ids, ora_scores_k, queries=None, what=""):
    """gpu and oracle id sets equal except for near ties at the oracle's k-th
    score.  ora_scores_k [B]: exact score of the oracle's k-th item."""
    B = gpu_ids.shape[0]
    bad = []
    for q in (range(B) if queries is None else queries):
        g = set(gpu_ids[q][gpu_ids[q] >= 0].tolist())
        o = set(ora_ids[q][ora_ids[q] >= 0].tolist())
        diff = sorted(g ^ o)
        if not diff:
            continue
        s = O.pair_scores(W, dtype, H, np.full(len(diff), q, np.int32), np.array(diff, np.int32))
        sk = ora_scores_k[q]
        if np.any(np.abs(s - sk) > REL_CUT * abs(sk)):
            bad.append((q, diff[:6], s[:6].tolist(), sk))
    assert not bad, "%s: id sets differ beyond near ties: %s" % (what, bad[:3])


def recall(found, exact):
    return float(O.recall(found, exact).mean())


def oracle_rows(fn, H, *args, threads=None, **kw):
    """An oracle function over chunks of the queries H in parallel threads
    (the oracle holds no global state and ctypes releases the GIL).  The
    None in args marks where the chunk of H goes; every output is
    concatenated along its first axis."""
    n = len(H)
    t = threads or min(16, os.cpu_count() or 1)
    cuts = np.linspace(0, n, min(t, n) + 1).astype(int)
    parts = [(a, b) for a, b in zip(cuts[:-1], cuts[1:]) if b > a]

    def one(ab):
        a, b = ab
        return fn(*[H[a:b] if x is None else x for x in args], **kw)

    with cf.ThreadPoolExecutor(len(parts)) as ex:
        outs = list(ex.map(one, parts))
    if not isinstance(outs[0], tuple):
        return np.concatenate(outs)
    return tuple(np.concatenate([o[i] for o in outs]) for i in range(len(outs[0])))


# ------------------------------------------------ traversal divergences

NODE_MASK = (1 << 26) - 1


def _decode(trace):
    t = np.asarray(trace)
    t = t[t >= 0]
    return t & NODE_MASK, (t >> 26) & 1, t >> 27


def first_divergence(W, dtype, g, h, tg, to, ef_eff, rel=REL_CUT, int8=False):
    """Explains where a traversal left the oracle's.  tg / to: the GPU's and
    the oracle's expansion records of one query ((layer << 27) | (first of
    step << 26) | node, -1 padded); h: the query [d].

    Up to the first differing entry both walked the same nodes, so on the
    layer L of that step both hold the same visited set S (the layer's entry
    and every neighbour of a node expanded there) and the same expanded set
    E.  Each side's beam is the best ef of S in its own arithmetic (ef = 1
    above layer 0), and a step expands the best unexpanded entries of it.
    With the oracle's fp64 order, x its ef-th best score in S and y the next:
    if the GPU took a where the oracle took b, then either both lie in the
    oracle's beam and their order flipped (|s_a - s_b| small), or b left the
    GPU's beam (s_b - y small), or a entered it (x - s_a small); a side that
    stopped or ended its step earlier counts as taking nothing.  Returns
    (index, L, a, b, gap) with the smallest relative gap of those that apply
    (None if the records are equal), or raises AssertionError when none of
    them is within rel (not a near tie)."""
    ng, fg, lg_ = _decode(tg)
    no, fo, lo_ = _decode(to)
    n = min(len(ng), len(no))
    i = 0
    while i < n and ng[i] == no[i] and fg[i] == fo[i] and lg_[i] == lo_[i]:
        i += 1
    if i == len(ng) and i == len(no):
        return None
    # the step in which they part: both start one at i, or i lies inside a
    # step both began before
    g_new = i >= len(ng) or fg[i] == 1
    o_new = i >= len(no) or fo[i] == 1
    if g_new and o_new:
        s0 = i
        layers = [x[i] for x, m in ((lg_, len(ng)), (lo_, len(no))) if i < m]
        L = max(layers)
    else:
        s0 = max(j for j in range(i) if fg[j] == 1)
        L = int(lg_[s0])
    pre_nodes, pre_layers = ng[:s0], lg_[:s0]
    on_L = [int(x) for x, l in zip(pre_nodes, pre_layers) if l == L]
    assert on_L, "records part at the first expansion of layer %d (its entry point)" % L
    assert not (int8 and L == 0), "int8 layer-0 scores are computed alike on both sides"
    if L == 0:
        lists = {u: [int(x) for x in g.adj0[u] if x >= 0] for u in on_L}
    else:
        lists = {u: [int(x) for x in g.upper[g.upper_off[u] + L - 1] if x >= 0] for u in on_L}
    S = {on_L[0]}
    for u in on_L:
        S.update(lists[u])
    S = np.array(sorted(S), np.int32)
    E = set(on_L)
    sc = O.pair_scores(W, dtype, np.atleast_2d(h), np.zeros(len(S), np.int32), S)
    order = np.lexsort((S, -sc))
    S, sc = S[order], sc[order]
    ef = 1 if L >= 1 else ef_eff
    in_beam = {int(u) for u in S[:ef]}
    score = {int(u): float(v) for u, v in zip(S, sc)}
    x = float(sc[ef - 1]) if len(S) >= ef else None
    y = float(sc[ef]) if len(S) > ef else None

    def taken(nodes, flags, layers, m):
        if i >= m or layers[i] != L or (i > s0 and flags[i] == 1):
            return None  # stopped this layer, or ended this step
        return int(nodes[i])

    a, b = taken(ng, fg, lg_, len(ng)), taken(no, fo, lo_, len(no))
    assert a is None or a not in E, "GPU expanded node %d twice" % a
    gaps = []
    if a is not None and b is not None and a in in_beam and b in in_beam:
        gaps.append(abs(score[a] - score[b]) / max(abs(score[a]), abs(score[b])))
    if b is not None and b in in_beam and y is not None:
        gaps.append((score[b] - y) / max(abs(y), abs(score[b])))
    if a is not None and a not in in_beam and x is not None:
        gaps.append((x - score[a]) / max(abs(x), abs(score[a])))
    gap = min(gaps) if gaps else float("inf")
    assert gap <= rel, "expansion %d on layer %d: GPU took %s, oracle %s; the nearest tie is %.3g relative" % (
        i, L, a, b, gap)
    return i, L, a, b, gap
