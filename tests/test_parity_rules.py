"""The comparison rules of the parity tests, checked on the CPU against cases
whose answer is known: a traversal that parts from the oracle's at a planted
near tie is explained as one, and a traversal that takes a clearly worse node
is not."""
import os
import sys

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_27460_amd import synth

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import parity  # noqa: E402


def _twins(eps):
    """1000 rows and their twins scaled by (1 + eps): every query scores a
    twin within |eps| relative of its original."""
    base = synth.make_w(1000, 16, synth.F32, 5)
    return np.concatenate([base, (base.astype(np.float64) * (1.0 + eps)).astype(np.float32)])


@pytest.mark.parametrize("width", [1, 4])
def test_planted_near_ties_are_explained(width):
    W = _twins(1e-6)
    W2 = W.copy()
    W2[1000:] = (W[:1000].astype(np.float64) * (1.0 - 1e-6)).astype(np.float32)  # every twin pair flips order
    g = O.hnsw_build(W, synth.F32, 6, 40, 3)
    H, _ = synth.make_queries(W, synth.F32, 24, 6)
    ef, k, cap = 64, 10, 1024
    if width == 1:
        ref = O.hnsw_search(W, synth.F32, g, H, k, ef, validate=False, trace_cap=cap)[4]
        alt = O.hnsw_search(W2, synth.F32, g, H, k, ef, validate=False, trace_cap=cap)[4]
    else:
        ref = O.hnsw_search_multi(W, synth.F32, g, H, k, ef, width, validate=False, trace_cap=cap)[3]
        alt = O.hnsw_search_multi(W2, synth.F32, g, H, k, ef, width, validate=False, trace_cap=cap)[3]
    parted = 0
    for q in range(len(H)):
        r = parity.first_divergence(W, synth.F32, g, H[q], alt[q], ref[q], ef)
        if r is not None:
            parted += 1
            assert r[4] <= 3e-6, r
    assert parted >= 3  # the planted ties do decide some walks


def test_a_worse_choice_is_not_a_near_tie():
    W = synth.make_w(2000, 16, synth.F32, 8)
    g = O.hnsw_build(W, synth.F32, 6, 40, 4)
    H, _ = synth.make_queries(W, synth.F32, 4, 9)
    ef, k = 32, 10
    ids, _, st, _, tr = O.hnsw_search(W, synth.F32, g, H, k, ef, validate=False, trace_cap=512)
    assert parity.first_divergence(W, synth.F32, g, H[0], tr[0], tr[0], ef) is None
    # a walk that expands, at its third layer-0 step, the worst node it has
    # seen instead of the oracle's choice
    t = tr[0][tr[0] >= 0]
    lay = t >> 27
    i = int(np.nonzero(lay == 0)[0][2])
    seen = set()
    for u in (t[:i][lay[:i] == 0] & parity.NODE_MASK):
        seen.update(int(x) for x in g.adj0[u] if x >= 0)
    seen -= set(int(x) for x in (t[:i] & parity.NODE_MASK))
    cand = np.array(sorted(seen), np.int32)
    s = O.pair_scores(W, synth.F32, H[:1], np.zeros(len(cand), np.int32), cand)
    bad = t.copy()
    bad[i] = (1 << 26) | int(cand[np.argmin(s)])
    with pytest.raises(AssertionError, match="nearest tie"):
        parity.first_divergence(W, synth.F32, g, H[0], bad, t, ef)
