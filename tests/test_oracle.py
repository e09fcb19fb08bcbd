"""Pins for the CPU oracle: each test ties it to something other than itself.

* the exact head (Section 3, z = W_out h) against an independent library
  routine (numpy float64 matmul + lexsort), closed-form special cases and a
  hand-worked fixture;
* the HNSW search (Malkov & Yashunin Alg. 2/5, the method of Sections 2-3)
  against a hand-traced fixture, against brute force where the algorithm must
  be exact (ef >= |V| on a connected layer 0; complete graphs), and against the
  "expand the best unexpanded beam entry" reformulation written independently
  here in Python;
* the HNSW build against its structural invariants and the closed-form level
  distribution P(level >= l) = M^-l;
* the invariant checker against graphs with planted violations.
"""
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_27460_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _numpy_topk(W, dtype, h, k):
    Wv = synth.stored_values_f32(W, dtype).astype(np.float64)
    hv = synth.stored_values_f32(np.atleast_2d(h), dtype).astype(np.float64)
    s = hv @ Wv.T
    ids = np.stack([np.lexsort((np.arange(W.shape[0]), -row))[:k] for row in s])
    return ids, np.take_along_axis(s, ids, 1)


# ---------------------------------------------------------------- exact head

@pytest.mark.parametrize("dtype,V,d", [(synth.F32, 1000, 32), (synth.BF16, 1531, 48), (synth.F32, 97, 5)])
def test_topk_matches_numpy(dtype, V, d):
    W = synth.make_w(V, d, dtype, 11 + V)
    H, _ = synth.make_queries(W, dtype, 6, 12 + V)
    k = min(50, V)
    ids, lg, sc = O.topk(W, dtype, H, k)
    nid, ns = _numpy_topk(W, dtype, H, k)
    np.testing.assert_array_equal(ids, nid)
    np.testing.assert_allclose(sc, ns, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(lg, sc.astype(np.float32))


def test_topk_golden_hand_example():
    W, h, k, ids, lg = [], None, None, None, None
    for line in open(os.path.join(GOLDEN, "topk_hand.txt")):
        if line.startswith("#") or not line.strip():
            continue
        tag, *vals = line.split()
        if tag == "W":
            W.append([float(v) for v in vals])
        elif tag == "h":
            h = np.array([float(v) for v in vals], np.float32)
        elif tag == "k":
            k = int(vals[0])
        elif tag == "ids":
            ids = [int(v) for v in vals]
        elif tag == "logits":
            lg = [float(v) for v in vals]
    W = np.array(W, np.float32)
    got_ids, got_lg, _ = O.topk(W, synth.F32, h, k)
    assert got_ids[0].tolist() == ids
    assert got_lg[0].tolist() == lg


def test_topk_zero_query_is_id_order():
    W = synth.make_w(300, 16, synth.BF16, 3)
    ids, lg, _ = O.topk(W, synth.BF16, np.zeros(16, np.uint16), 20)
    assert ids[0].tolist() == list(range(20))
    assert np.all(lg == 0)


def test_topk_k_equals_v_returns_everything_sorted():
    W = synth.make_w(40, 8, synth.F32, 4)
    h = synth.make_queries(W, synth.F32, 1, 5)[0]
    ids, lg, sc = O.topk(W, synth.F32, h, 40)
    assert sorted(ids[0].tolist()) == list(range(40))
    assert np.all(np.diff(sc[0]) <= 0)


def test_topk_one_hot_rows_pick_the_argmax():
    rng = np.random.default_rng(0)
    d = 24
    perm = rng.permutation(d)
    W = np.zeros((d, d), np.float32)
    W[np.arange(d), perm] = 1.0 + np.arange(d, dtype=np.float32)  # row i = (1+i) e_perm[i]
    for j in range(d):
        h = np.zeros(d, np.float32)
        h[j] = 1.0
        ids, lg, _ = O.topk(W, synth.F32, h, 1)
        i = int(np.where(perm == j)[0][0])
        assert ids[0, 0] == i and lg[0, 0] == 1.0 + i


def test_topk_rejects_bad_k():
    W = synth.make_w(10, 4, synth.F32, 1)
    with pytest.raises(ValueError):
        O.topk(W, synth.F32, W[0], 11)


def test_pair_scores_matches_numpy():
    W = synth.make_w(200, 12, synth.BF16, 9)
    H, _ = synth.make_queries(W, synth.BF16, 3, 10)
    q = np.array([0, 1, 2, 2], np.int32)
    ids = np.array([5, 199, 0, 77], np.int32)
    got = O.pair_scores(W, synth.BF16, H, q, ids)
    Wv = synth.bf16_bits_to_f32(W).astype(np.float64)
    Hv = synth.bf16_bits_to_f32(H).astype(np.float64)
    np.testing.assert_allclose(got, [Wv[i] @ Hv[j] for i, j in zip(ids, q)], rtol=1e-12)


# ------------------------------------------------------------------- scatter

def test_scatter_definition():
    ids = np.array([[3, 0, 7], [9, -1, 2]], np.int32)
    lg = np.array([[1.5, -2.0, 0.25], [4.0, 99.0, -0.5]], np.float32)
    out = O.scatter(ids, lg, 10)
    assert out.shape == (2, 10)
    assert out[0, 3] == 1.5 and out[0, 0] == -2.0 and out[0, 7] == 0.25
    assert out[1, 9] == 4.0 and out[1, 2] == -0.5
    assert np.isneginf(out).sum() == 20 - 5       # the -1 id is ignored
    assert np.all(np.isneginf(np.delete(out[0], [0, 3, 7])))


# --------------------------------------------------------------------- levels

@pytest.mark.parametrize("M", [8, 16, 32])
def test_level_distribution_closed_form(M):
    V = 400_000
    lv = O.levels(V, M, 4002).astype(np.int64)
    # P(level >= l) = M^-l because level = floor(-ln(u) / ln M), u ~ U(0, 1].
    for l in range(1, 4):
        expect = V * float(M) ** -l
        got = int((lv >= l).sum())
        if expect >= 20:
            assert abs(got - expect) < 5 * np.sqrt(expect), (l, got, expect)
    assert lv.min() == 0 and lv.max() <= 16


def test_levels_deterministic_and_seeded():
    a = O.levels(5000, 16, 1)
    assert np.array_equal(a, O.levels(5000, 16, 1))
    assert not np.array_equal(a, O.levels(5000, 16, 2))


# ---------------------------------------------------------------------- build

def _build(V=600, d=16, dtype=synth.F32, M=6, efC=40, seed=5, select="heuristic", M0=None):
    W = synth.make_w(V, d, dtype, 100 + seed)
    return W, O.hnsw_build(W, dtype, M, efC, seed, M0=M0, select=select)


@pytest.mark.parametrize("select", ["heuristic", "simple"])
@pytest.mark.parametrize("dtype,M,M0", [(synth.F32, 6, None), (synth.BF16, 4, None), (synth.F32, 5, 5)])
def test_build_invariants(select, dtype, M, M0):
    W, g = _build(dtype=dtype, M=M, M0=M0, select=select)
    assert O.check_graph(g) == ""
    assert g.M0 == (2 * M if M0 is None else M0)
    assert np.array_equal(g.levels, O.levels(g.V, M, g.seed))
    # entry: the first node to reach the top level (strictly higher levels only)
    assert g.entry == int(np.argmax(g.levels == g.levels.max()))
    deg0 = (g.adj0 >= 0).sum(1)
    assert deg0.max() <= g.M0 and deg0.min() >= 1
    if g.nb:
        assert (g.upper >= 0).sum(1).max() <= M


def test_build_is_deterministic():
    _, a = _build(seed=9)
    _, b = _build(seed=9)
    for f in ("levels", "adj0", "upper_off", "upper"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    assert (a.entry, a.maxlevel) == (b.entry, b.maxlevel)


def _build_trace_case():
    """tests/golden/build_trace.txt: rows, levels, parameters and the graph
    worked out by hand (MY18 Alg. 1 + 4 as the paper's index)."""
    lines = [l.split() for l in open(os.path.join(GOLDEN, "build_trace.txt")) if l.strip() and l[0] != "#"]
    f = {l[0]: l[1:] for l in lines}
    W = np.array([[float(x) for x in r.split(",")] for r in f["rows"]], np.float32)
    levels = np.array([int(x) for x in f["levels"]], np.uint8)
    prm = dict(x.split("=") for x in f["params"])
    lists = {}
    for layer in ("layer0", "layer1"):
        for item in f[layer]:
            node, ids = item.split(":")
            lists[(int(layer[-1]), int(node))] = [int(x) for x in ids.split(",")]
    return W, levels, int(prm["M"]), int(prm["M0"]), int(prm["efC"]), int(f["entry"][0]), \
        int(f["maxlevel"][0]), lists


def test_build_golden_hand_trace():
    """Every list (in stored order), the entry point and the top level of a
    build traced by hand: layer-0 lists overflow and are cut by the Alg. 4
    heuristic (to fewer than the cap), the whole layer-1 result of node 5 is
    its layer-0 entry set (its nearest alone would give it the list [1, 4]),
    node 1 raises the entry point and nodes 3 and 5, at the same level, do
    not move it."""
    W, levels, M, M0, efC, entry, maxlevel, lists = _build_trace_case()
    g = O.hnsw_build(W, synth.F32, M, efC, 0, M0=M0, levels=levels)
    assert O.check_graph(g) == ""
    assert (g.entry, g.maxlevel) == (entry, maxlevel)
    assert np.array_equal(g.levels, levels)
    for u in range(g.V):
        row = g.adj0[u]
        assert row[row >= 0].tolist() == lists[(0, u)], (u, row)
        if levels[u] >= 1:
            up = g.upper[g.upper_off[u]]
            assert up[up >= 0].tolist() == lists[(1, u)], (u, up)
        else:
            assert g.upper_off[u] == -1 and (1, u) not in lists
    # the heuristic is what cut the lists: the simple rule keeps the 3 nearest
    s = O.hnsw_build(W, synth.F32, M, efC, 0, M0=M0, levels=levels, select="simple")
    assert [s.adj0[u][s.adj0[u] >= 0].tolist() for u in (1, 2, 3)] == [[4, 2, 5], [4, 1, 0], [0, 6, 5]]


def test_build_levels_argument_matches_the_seeded_draw():
    W = synth.make_w(500, 12, synth.F32, 77)
    a = O.hnsw_build(W, synth.F32, 6, 30, 11)
    b = O.hnsw_build(W, synth.F32, 6, 30, 0, levels=O.levels(500, 6, 11))
    for f in ("levels", "adj0", "upper_off", "upper"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    assert (a.entry, a.maxlevel) == (b.entry, b.maxlevel)


def test_graph_size_matches_memory_formula():
    # Section 3: the index adds 8M bytes per node with 32-bit ids, i.e. 2M layer-0 ids.
    _, g = _build(M=8)
    assert g.adj0.nbytes == g.V * 8 * g.M


def _strongly_connected_l0(g):
    adj = [set(r[r >= 0].tolist()) for r in g.adj0]
    radj = [set() for _ in range(g.V)]
    for u, s in enumerate(adj):
        for v in s:
            radj[v].add(u)

    def reach(a):
        seen, st = {0}, [0]
        while st:
            u = st.pop()
            for v in a[u]:
                if v not in seen:
                    seen.add(v)
                    st.append(v)
        return len(seen)
    return reach(adj) == g.V and reach(radj) == g.V


def _reachable_l0(g, start):
    seen, st = {start}, [start]
    while st:
        u = st.pop()
        for v in g.adj0[u][g.adj0[u] >= 0].tolist():
            if v not in seen:
                seen.add(v)
                st.append(v)
    return np.array(sorted(seen))


@pytest.mark.parametrize("dtype,select", [(synth.F32, "heuristic"), (synth.BF16, "heuristic"),
                                          (synth.F32, "simple")])
def test_search_with_ef_at_least_v_is_exact_over_reachable_nodes(dtype, select):
    # With ef >= |V| nothing is ever evicted, so every node reachable at layer 0
    # from the start node is scored: the result is the brute-force top-k of
    # that set (of all of V when layer 0 is connected).
    W, g = _build(V=400, d=12, dtype=dtype, M=5, efC=30, seed=21, select=select)
    H, _ = synth.make_queries(W, dtype, 8, 22)
    ids, lg, st, l0 = O.hnsw_search(W, dtype, g, H, 10, ef=g.V)
    for q in range(H.shape[0]):
        R = _reachable_l0(g, int(l0[q]))
        eid, elg, _ = O.topk(W[R], dtype, H[q], 10)
        np.testing.assert_array_equal(ids[q], R[eid[0]])
        np.testing.assert_array_equal(lg[q], elg[0])
        assert st[q, 0] >= len(R)


@pytest.mark.parametrize("select", ["heuristic", "simple"])
def test_search_with_ef_at_least_v_is_exact_on_connected_graph(select):
    # Unit-norm rows (inner product = cosine) give a strongly connected layer 0,
    # so ef >= |V| must return the brute-force top-k of all of V.
    W = synth.make_w(400, 12, synth.F32, 121)
    W = (W / np.linalg.norm(W, axis=1, keepdims=True)).astype(np.float32)
    g = O.hnsw_build(W, synth.F32, 5, 40, 21, select=select)
    assert _strongly_connected_l0(g)
    H, _ = synth.make_queries(W, synth.F32, 8, 22)
    ids, lg, _, _ = O.hnsw_search(W, synth.F32, g, H, 10, ef=g.V)
    eid, elg, _ = O.topk(W, synth.F32, H, 10)
    np.testing.assert_array_equal(ids, eid)
    np.testing.assert_array_equal(lg, elg)


def test_complete_graph_is_exact_for_any_ef_at_least_k():
    M = 12
    W, g = _build(V=M + 1, d=8, M=M, efC=M + 1, seed=3)  # each insert sees every earlier node
    assert np.all((g.adj0 >= 0).sum(1) == g.V - 1)
    H, _ = synth.make_queries(W, synth.F32, 5, 4)
    eid, elg, _ = O.topk(W, synth.F32, H, 4)
    for ef in (1, 4, 7):
        ids, lg, _, _ = O.hnsw_search(W, synth.F32, g, H, 4, ef=ef)
        np.testing.assert_array_equal(ids, eid)


def _chain_case():
    lines = [l.split() for l in open(os.path.join(GOLDEN, "chain_search.txt")) if l.strip() and l[0] != "#"]
    vals = next(l for l in lines if l[0] == "values")[1:]
    edges = next(l for l in lines if l[0] == "edges")[1:]
    V = len(vals)
    W = np.array([[float(v)] for v in vals], np.float32)
    nbr = [[] for _ in range(V)]
    for e in edges:
        a, b = (int(x) for x in e.split("-"))
        nbr[a].append(b)
        nbr[b].append(a)
    adj0 = -np.ones((V, 2), np.int32)
    for u in range(V):
        s = sorted(nbr[u])
        adj0[u, :len(s)] = s
    g = O.Graph(V, 1, synth.F32, 1, 2, 1, 0, 0, 0, np.zeros(V, np.uint8), adj0, -np.ones(V, np.int32),
                np.zeros((0, 1), np.int32))
    cases = []
    for l in lines:
        if l[0] == "case":
            kv = dict(x.split("=") for x in l[1:])
            cases.append((int(kv["ef"]), int(kv["k"]), [int(x) for x in kv["ids"].split(",")],
                          int(kv["n_dist"]), int(kv["n_expand"]), _steps(kv["expanded"])))
    return W, g, cases


def _steps(text):
    """'0|1,2|4' -> the trace entries of layer-0 expansions 0, 1, 2, 4 with
    the first node of each step flagged (bit 26)."""
    out = []
    for step in text.split("|"):
        for j, x in enumerate(step.split(",")):
            out.append(int(x) | ((1 << 26) if j == 0 else 0))
    return out


def test_search_golden_chain_trace():
    W, g, cases = _chain_case()
    assert O.check_graph(g) == ""
    for ef, k, ids, nd, ne, order in cases:
        got, lg, st, _, tr = O.hnsw_search(W, synth.F32, g, np.ones((1, 1), np.float32), k, ef, trace_cap=16)
        assert got[0].tolist() == ids, (ef, got)
        assert st[0].tolist() == [nd, ne], (ef, st)
        assert tr[0][:ne].tolist() == order and np.all(tr[0][ne:] == -1), (ef, tr)
        # a short record keeps the first expansions
        _, _, _, _, tr2 = O.hnsw_search(W, synth.F32, g, np.ones((1, 1), np.float32), k, ef, trace_cap=2)
        assert tr2[0].tolist() == order[:2]


def _tree_case():
    lines = [l.split() for l in open(os.path.join(GOLDEN, "multi_expand_tree.txt")) if l.strip() and l[0] != "#"]
    vals = next(l for l in lines if l[0] == "values")[1:]
    edges = next(l for l in lines if l[0] == "edges")[1:]
    V = len(vals)
    W = np.array([[float(v)] for v in vals], np.float32)
    nbr = [[] for _ in range(V)]
    for e in edges:
        a, b = (int(x) for x in e.split("-"))
        nbr[a].append(b)
        nbr[b].append(a)
    adj0 = -np.ones((V, 3), np.int32)
    for u in range(V):
        s = sorted(nbr[u])
        adj0[u, :len(s)] = s
    g = O.Graph(V, 1, synth.F32, 2, 3, 1, 0, 0, 0, np.zeros(V, np.uint8), adj0, -np.ones(V, np.int32),
                np.zeros((0, 2), np.int32))
    cases = []
    for l in lines:
        if l[0] == "case":
            kv = dict(x.split("=") for x in l[1:])
            cases.append((int(kv["P"]), int(kv["ef"]), int(kv["k"]), [int(x) for x in kv["ids"].split(",")],
                          int(kv["n_dist"]), int(kv["n_expand"]), _steps(kv["expanded"])))
    return W, g, cases


def test_multi_expansion_golden_tree_trace():
    W, g, cases = _tree_case()
    assert O.check_graph(g) == ""
    for P, ef, k, ids, nd, ne, order in cases:
        got, lg, st, tr = O.hnsw_search_multi(W, synth.F32, g, np.ones((1, 1), np.float32), k, ef, P, trace_cap=16)
        assert got[0].tolist() == ids, (P, ef, got)
        assert st[0].tolist() == [nd, ne], (P, ef, st)
        assert tr[0][:ne].tolist() == order, (P, ef, tr)


@pytest.mark.parametrize("seed", [4, 5])
def test_multi_expansion_with_width_one_is_the_search(seed):
    V, d = 1500, 16
    W = synth.make_w(V, d, synth.BF16, 60 + seed)
    H, _ = synth.make_queries(W, synth.BF16, 20, 70 + seed)
    g = O.hnsw_build(W, synth.BF16, 6, 30, seed)
    a = O.hnsw_search(W, synth.BF16, g, H, 10, 40, trace_cap=512)
    b = O.hnsw_search_multi(W, synth.BF16, g, H, 10, 40, 1, trace_cap=512)
    for x, y in zip(a[:3] + a[4:], b):
        assert np.array_equal(x, y)
    # the record tags each expansion with its layer: the upper layers first,
    # then layer 0, as many as the counter says
    for q in range(len(H)):
        t = a[4][q][:a[2][q, 1]]
        assert np.all((t >> 26) & 1 == 1)  # one node per step
        lay = t >> 27
        assert np.all(np.diff(lay) <= 0) and lay[-1] == 0 and lay[0] <= g.maxlevel
        assert np.all(a[4][q][a[2][q, 1]:] == -1)


@pytest.mark.parametrize("P", [2, 3, 8])
def test_multi_expansion_with_ef_at_least_v_is_exact(P):
    W = synth.make_w(300, 8, synth.F32, 123)
    W = (W / np.linalg.norm(W, axis=1, keepdims=True)).astype(np.float32)
    g = O.hnsw_build(W, synth.F32, 5, 40, 3)
    H, _ = synth.make_queries(W, synth.F32, 12, 124)
    ids, lg, st = O.hnsw_search_multi(W, synth.F32, g, H, 10, 300, P)
    oid, olg, _ = O.topk(W, synth.F32, H, 10)
    assert np.array_equal(ids, oid)
    assert np.array_equal(lg, olg)


def test_forced_merge_golden_hand_example():
    lines = {l.split()[0]: l.split()[1:] for l in open(os.path.join(GOLDEN, "forced_hand.txt"))
             if l.strip() and l[0] != "#"}
    W = np.array([[float(x) for x in r.split(",")] for r in lines["rows"]], np.float32)
    h = np.array([[float(x) for x in lines["h"][0].split(",")]], np.float32)
    search = np.array([[int(x) for x in lines["search"][0].split(",")]], np.int32)
    forced = np.array([int(x) for x in lines["forced"][0].split(",")], np.int32)
    kv = dict(x.split("=") for x in lines["expect"])
    ids, lg = O.forced_merge(W, synth.F32, h, search, forced)
    assert ids[0].tolist() == [int(x) for x in kv["ids"].split(",")]
    assert lg[0].tolist() == [float(x) for x in kv["logits"].split(",")]


def test_forced_merge_special_cases():
    W = synth.make_w(400, 16, synth.BF16, 9)
    H, _ = synth.make_queries(W, synth.BF16, 5, 10)
    g = O.hnsw_build(W, synth.BF16, 6, 30, 2)
    ids, lg, _, _ = O.hnsw_search(W, synth.BF16, g, H, 10, 20)
    # no forced ids: the search result itself
    fi, fl = O.forced_merge(W, synth.BF16, H, ids, np.zeros(0, np.int32))
    assert np.array_equal(fi, ids) and np.array_equal(fl, lg)
    # every id forced: the exact order of the whole vocabulary, then k pads
    fi, fl = O.forced_merge(W, synth.BF16, H, ids, np.arange(400, dtype=np.int32)[::-1].copy())
    oid, olg, _ = O.topk(W, synth.BF16, H, 400)
    assert np.array_equal(fi[:, :400], oid) and np.array_equal(fl[:, :400], olg)
    assert np.all(fi[:, 400:] == -1) and np.all(np.isneginf(fl[:, 400:]))


def test_int8_quantization_closed_forms():
    rng = np.random.default_rng(3)
    ints = rng.integers(-127, 128, size=(6, 40)).astype(np.float32)
    ints[:, 0] = 127.0                       # max |x| = 127: scale exactly 1 (times the power of two below)
    W = np.concatenate([ints, ints * 0.25, np.zeros((1, 40), np.float32),
                        np.array([[127.0, 2.5, 3.5, -2.5, -3.5, 0.5] + [0.0] * 34], np.float32)])
    q, sc = O.quantize_rows(W, synth.F32)
    assert np.array_equal(sc[:6], np.ones(6, np.float32)) and np.array_equal(q[:6], ints.astype(np.int8))
    assert np.array_equal(sc[6:12], np.full(6, 0.25, np.float32)) and np.array_equal(q[6:12], ints.astype(np.int8))
    assert sc[12] == 0.0 and not q[12].any()
    assert q[13, :6].tolist() == [127, 2, 4, -2, -4, 0]    # ties round to even
    Wr = synth.make_w(300, 64, synth.BF16, 17)
    q, sc = O.quantize_rows(Wr, synth.BF16)
    x = synth.bf16_bits_to_f32(Wr).astype(np.float64)
    err = np.abs(q.astype(np.float64) * sc[:, None] - x)
    # half a step, plus the fp32 rounding of x / scale and of scale (each at most 127 * 2^-24 steps)
    assert np.all(err <= sc[:, None] * (0.5 + 2 * 127 * 2.0 ** -24))
    assert np.all(np.abs(q).max(axis=1) == 127)
    assert np.all(np.abs(q[np.arange(300), np.abs(x).argmax(axis=1)]) == 127)


def test_int8_search_with_exact_integer_data_is_the_multi_search():
    # rows and query are integers with max 127: every int8 score is exact, so
    # the traversal is the unquantized one (plus the re-scored entry point)
    rng = np.random.default_rng(11)
    V, d = 800, 12
    W = rng.integers(-20, 21, size=(V, d)).astype(np.float32)
    W[:, 0] = 127.0
    H = rng.integers(-30, 31, size=(6, d)).astype(np.float32)
    H[:, 1] = 127.0
    g = O.hnsw_build(W, synth.F32, 6, 30, 4)
    q, sc = O.quantize_rows(W, synth.F32)
    for P in (1, 3):
        a = O.hnsw_search_multi(W, synth.F32, g, H, 10, 30, P)
        b = O.hnsw_search_q(W, synth.F32, g, q, sc, H, 10, 30, P)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
        assert np.array_equal(a[2][:, 0] + 1, b[2][:, 0]) and np.array_equal(a[2][:, 1], b[2][:, 1])


@pytest.mark.parametrize("P", [1, 4])
def test_int8_search_with_ef_at_least_v_is_exact(P):
    W = synth.make_w(300, 8, synth.BF16, 125)
    Wf = synth.bf16_bits_to_f32(W)
    W = synth.f32_to_bf16_bits(Wf / np.linalg.norm(Wf, axis=1, keepdims=True))
    g = O.hnsw_build(W, synth.BF16, 5, 40, 3)
    H, _ = synth.make_queries(W, synth.BF16, 12, 126)
    q, sc = O.quantize_rows(W, synth.BF16)
    ids, lg, st = O.hnsw_search_q(W, synth.BF16, g, q, sc, H, 10, 300, P)
    oid, olg, _ = O.topk(W, synth.BF16, H, 10)
    assert np.array_equal(ids, oid) and np.array_equal(lg, olg)


def test_knn_graph_golden_star():
    lines = [l.split() for l in open(os.path.join(GOLDEN, "knn_graph_star.txt")) if l.strip() and l[0] != "#"]
    vals = next(l for l in lines if l[0] == "values")[1:]
    K = int(next(l for l in lines if l[0] == "K")[1])
    M0 = int(next(l for l in lines if l[0] == "M0")[1])
    W = np.array([[float(v)] for v in vals], np.float32)
    g = O.knn_graph(W, synth.F32, K, M0)
    assert O.check_graph(g) == ""
    for l in lines:
        if l[0] == "list":
            got = [int(x) for x in g.adj0[int(l[1])] if x >= 0]
            assert got == [int(x) for x in l[2].split(",")], (l, got)
    assert g.entry == int(next(l for l in lines if l[0] == "entry")[1])


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_knn_graph_properties(dtype):
    V, d, K, M0 = 700, 16, 24, 12
    W = synth.make_w(V, d, dtype, 31)
    g = O.knn_graph(W, dtype, K, M0)
    assert O.check_graph(g) == ""
    Wf = synth.stored_values_f32(W, dtype).astype(np.float64)
    G = Wf @ Wf.T
    np.fill_diagonal(G, -np.inf)
    nearest = np.lexsort((np.arange(V)[None, :].repeat(V, 0), -G), axis=1)[:, 0]
    # every node keeps its nearest other node (the heuristic keeps the first candidate)
    assert all(nearest[i] in g.adj0[i] for i in range(V))
    assert g.entry == int(np.argmax((Wf * Wf).sum(1)))
    # the search on this graph with ef >= |V| is exact over the nodes reachable from the entry
    H, _ = synth.make_queries(W, dtype, 8, 32)
    ids, _, _, _ = O.hnsw_search(W, dtype, g, H, 10, V)
    seen, todo = {g.entry}, [g.entry]
    while todo:
        u = todo.pop()
        for v in g.adj0[u]:
            if v >= 0 and v not in seen:
                seen.add(int(v))
                todo.append(int(v))
    reach = np.array(sorted(seen))
    sc = synth.stored_values_f32(H, dtype).astype(np.float64) @ Wf[reach].T
    for q in range(len(H)):
        order = reach[np.lexsort((reach, -sc[q]))][:10]
        assert ids[q].tolist() == order.tolist()


def test_knn_graph_forward_and_reverse_edges():
    V, d, K, M0 = 500, 8, 20, 10
    W = synth.make_w(V, d, synth.F32, 41)
    g, fwd = O.knn_graph(W, synth.F32, K, M0, with_forward=True)
    Wf = W.astype(np.float64)
    G = Wf @ Wf.T
    rev = [[] for _ in range(V)]
    for i in range(V):
        f = [int(x) for x in fwd[i] if x >= 0]
        # fwd(i) follows the heuristic over the exact K nearest: every kept e beats all kept before it,
        # every skipped candidate (before M0 kept) loses to one of them
        order = sorted((j for j in range(V) if j != i), key=lambda j: (-G[i, j], j))[:K]
        kept = []
        for e in order:
            if len(kept) == M0:
                break
            if all(G[e, i] > G[e, r] for r in kept):
                kept.append(e)
        assert f == kept, i
        assert [int(x) for x in g.adj0[i][:len(f)]] == f  # forward edges come first
        for j in f:
            rev[j].append(i)
    for j in range(V):
        lst = [int(x) for x in g.adj0[j] if x >= 0]
        f = [int(x) for x in fwd[j] if x >= 0]
        extra = sorted(set(rev[j]) - set(f), key=lambda i: (-G[j, i], i))
        assert lst == (f + extra)[:M0], j  # free slots filled by reverse edges, nearest first


def _beam_search_reformulated(W, dtype, g, h, k, ef):
    """Independent restatement: keep one beam sorted by (dist, id) with
    'expanded' flags; repeatedly expand the best unexpanded entry, scoring all
    its unseen neighbours, then keep the best ef.  Equivalent to MY18 Alg. 2."""
    Wv = synth.stored_values_f32(W, dtype).astype(np.float64)
    hv = synth.stored_values_f32(np.atleast_2d(h), dtype).astype(np.float64)[0]
    nd = ne = 0

    def dist(u):
        nonlocal nd
        nd += 1
        return -sum(float(a) * float(b) for a, b in zip(Wv[u], hv))

    def lists(u, l):
        row = g.adj0[u] if l == 0 else g.upper[g.upper_off[u] + l - 1]
        return [int(x) for x in row if x >= 0]

    def layer(ep, ef_l, l):
        nonlocal ne
        beam = [[ep[0], ep[1], False]]
        seen = {ep[1]}
        while True:
            todo = [b for b in beam if not b[2]]
            if not todo:
                return beam
            c = min(todo, key=lambda b: (b[0], b[1]))
            c[2] = True
            ne += 1
            for e in lists(c[1], l):
                if e not in seen:
                    seen.add(e)
                    beam.append([dist(e), e, False])
            beam = sorted(beam, key=lambda b: (b[0], b[1]))[:ef_l]

    ep = (dist(g.entry), g.entry)
    for l in range(g.maxlevel, 0, -1):
        b = layer(ep, 1, l)
        ep = (b[0][0], b[0][1])
    beam = layer(ep, max(ef, k), 0)[:k]
    return [b[1] for b in beam], nd, ne


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_search_equals_reformulated_beam(seed):
    W, g = _build(V=300, d=6, M=4, efC=20, seed=seed)
    H, _ = synth.make_queries(W, synth.F32, 5, 50 + seed)
    for ef in (1, 5, 17):
        ids, _, st, _ = O.hnsw_search(W, synth.F32, g, H, 5, ef)
        for q in range(H.shape[0]):
            rid, nd, ne = _beam_search_reformulated(W, synth.F32, g, H[q], 5, ef)
            assert ids[q].tolist() == rid
            assert st[q].tolist() == [nd, ne]


def test_search_output_is_sorted_unique_and_exactly_scored():
    W, g = _build(V=2000, d=24, dtype=synth.BF16, M=8, efC=60, seed=4)
    H, _ = synth.make_queries(W, synth.BF16, 10, 5)
    ids, lg, st, _ = O.hnsw_search(W, synth.BF16, g, H, 20, 32)
    for q in range(10):
        assert len(set(ids[q].tolist())) == 20
        assert np.all(np.diff(lg[q]) <= 0)
    sc = O.pair_scores(W, synth.BF16, H, np.repeat(np.arange(10), 20), ids.ravel())
    np.testing.assert_array_equal(lg.ravel(), sc.astype(np.float32))


def test_mean_recall_grows_with_ef():
    # Section 4, "Index Accuracy": recall improves monotonically with ef.
    W, g = _build(V=3000, d=32, M=6, efC=40, seed=8)
    H, _ = synth.make_queries(W, synth.F32, 60, 9)
    eid, _, _ = O.topk(W, synth.F32, H, 10)
    means = []
    for ef in (10, 20, 40, 80, 160):
        ids, _, _, _ = O.hnsw_search(W, synth.F32, g, H, 10, ef)
        means.append(O.recall(ids, eid).mean())
    assert all(b >= a for a, b in zip(means, means[1:])), means
    assert means[-1] > means[0]


# ----------------------------------------------------- invariant checker pins

def _copy(g):
    return O.Graph(**{f: (v.copy() if isinstance(v, np.ndarray) else v) for f, v in g.__dict__.items()})


def test_checker_catches_planted_violations():
    _, g = _build(V=500, M=6, seed=31)
    assert O.check_graph(g) == ""
    u = int(np.argmax((g.adj0 >= 0).sum(1) >= 2))
    bad = _copy(g); bad.adj0[u, 0] = u
    assert "self loop" in O.check_graph(bad)
    bad = _copy(g); bad.adj0[u, 1] = bad.adj0[u, 0]
    assert "duplicate" in O.check_graph(bad)
    bad = _copy(g); bad.adj0[u, 0] = g.V
    assert "out of range" in O.check_graph(bad)
    n = int((g.adj0[u] >= 0).sum())
    if n < g.M0 - 1:
        bad = _copy(g); bad.adj0[u, n + 1] = 0
        assert "padding" in O.check_graph(bad)
    bad = _copy(g); bad.entry = int(np.argmin(g.levels))
    assert "entry" in O.check_graph(bad)
    hi = int(np.argmax(g.levels))
    bad = _copy(g); bad.upper[g.upper_off[hi], 0] = int(np.argmin(g.levels))
    assert "has level" in O.check_graph(bad)


# ------------------------------------------------------------------ file form

def test_file_round_trip_and_corruption(tmp_path):
    W, g = _build(V=700, dtype=synth.BF16, seed=13)
    p = str(tmp_path / "g.vie")
    O.save_graph(g, p, W)
    g2, fp = O.load_graph(p)
    assert fp == O.fingerprint(W, synth.BF16)
    for f in ("levels", "adj0", "upper_off", "upper"):
        assert np.array_equal(getattr(g, f), getattr(g2, f))
    assert (g2.V, g2.d, g2.M, g2.M0, g2.efC, g2.seed, g2.entry, g2.maxlevel) == \
        (g.V, g.d, g.M, g.M0, g.efC, g.seed, g.entry, g.maxlevel)
    raw = bytearray(open(p, "rb").read())
    raw[200] ^= 1
    open(p, "wb").write(bytes(raw))
    with pytest.raises(ValueError, match="checksum"):
        O.load_graph(p)
    open(p, "wb").write(bytes(raw[:-20]))
    with pytest.raises(ValueError):
        O.load_graph(p)


def test_fingerprint_sees_sampled_rows():
    W = synth.make_w(3000, 8, synth.F32, 2)
    f0 = O.fingerprint(W, synth.F32)
    W2 = W.copy(); W2[0, 0] += 1
    W3 = W.copy(); W3[2999, 7] += 1
    assert O.fingerprint(W2, synth.F32) != f0 and O.fingerprint(W3, synth.F32) != f0


def test_pair_abs_scores_matches_numpy():
    W = synth.make_w(100, 9, synth.F32, 19)
    H, _ = synth.make_queries(W, synth.F32, 2, 20)
    got = O.pair_abs_scores(W, synth.F32, H, np.array([0, 1], np.int32), np.array([3, 99], np.int32))
    ref = [np.abs(W[3].astype(np.float64) * H[0]).sum(), np.abs(W[99].astype(np.float64) * H[1]).sum()]
    np.testing.assert_allclose(got, ref, rtol=1e-12)
