"""Comparison rules between the HIP path and the oracle (shared by the GPU
tests and the benchmark's parity leg).

Tolerances (stated for the head in its specification):
* id sets: an id returned by only one side must score within 1e-4 relative of
  the oracle's k-th score (a near tie at the cut);
* logits: |gpu - exact| <= rel * |exact| + d * 2^-24 * sum_j |w_j h_j| with
  rel = 1e-5 for fp32 storage and 2e-2 for bf16.  The second term is the
  worst-case rounding of any length-d fp32 sum (Higham, "Accuracy and
  Stability of Numerical Algorithms", eq. 3.5); it only matters where
  cancellation leaves |exact| far below its summands (logits near zero);
* order: logits non-increasing, ids distinct;
* HNSW traversal: equal (n_dist, n_expand) means the GPU walked the same path;
  queries whose counts differ are counted as traversal divergences (they can
  only start at a near tie of an fp32 against a float64 comparison).
"""
from __future__ import annotations

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
    q = np.repeat(np.arange(B, dtype=np.int32), k)
    mag = O.pair_abs_scores(W, dtype, H, q, safe.ravel()).reshape(B, k)
    rel = REL_LOGIT[dtype]
    d = W.shape[1]
    for q in range(B):
        v = valid[q]
        if not v.any():
            continue
        err = np.abs(logits[q, v].astype(np.float64) - ex[q, v])
        allowed = rel * np.abs(ex[q, v]) + d * 2.0 ** -24 * mag[q, v]
        worst = int(np.argmax(err / allowed))
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
