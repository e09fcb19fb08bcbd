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
* HNSW traversal: equal (n_dist, n_expand) means the GPU walked the same path;
  queries whose counts differ are counted as traversal divergences (they can
  only start at a near tie of an fp32 against a float64 comparison).
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
