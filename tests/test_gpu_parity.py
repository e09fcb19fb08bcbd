"""GPU parity: every kernel, called through the C ABI, against the oracle on
the same seeded inputs (and, for HNSW, the same graph file, entry point and
ef).  Sizes span several tiles/workgroups with ragged tails; edge cases cover
k = V, B above one pass, odd row widths, zero queries and ef >= |V|."""
import os
import sys
import tempfile

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_27460_amd import synth

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import parity  # noqa: E402

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def vie():
    assert torch.cuda.is_available(), "the gpu tests need an MI355X"
    from paper_2608_27460_amd import vie as v
    return v


def dev_tensor(vie, a, dtype):
    return vie.host_to_torch(a, dtype).cuda()


def say(*a):
    print(*a, flush=True)


# ------------------------------------------------------------------ scatter

@pytest.mark.parametrize("V,B,k", [(10000, 3, 50), (4096, 1, 7), (1, 1, 1), (4097, 2, 100), (151937, 2, 50)])
def test_scatter_bitwise(vie, V, B, k):
    say("scatter", V, B, k)
    rng = np.random.default_rng(V + k)
    k = min(k, V)
    ids = np.stack([rng.choice(V, size=k, replace=False) for _ in range(B)]).astype(np.int32)
    ids[:, ::7] = -1  # padding ids are skipped
    lg = rng.standard_normal((B, k)).astype(np.float32)
    out = vie.scatter(torch.from_numpy(ids).cuda(), torch.from_numpy(lg).cuda(), V)
    torch.cuda.synchronize()
    ref = O.scatter(ids, lg, V)
    assert np.array_equal(out.cpu().numpy().view(np.uint32), ref.view(np.uint32))


# --------------------------------------------------------------- dense head

DENSE_CASES = [
    (5000, 64, synth.F32, 1, 50),
    (20011, 256, synth.BF16, 3, 100),
    (3001, 37, synth.BF16, 2, 20),     # odd bf16 row: 2-byte loads
    (2000, 5, synth.F32, 1, 16),       # 20-byte rows: 4-byte loads
    (1000, 48, synth.F32, 9, 1000),    # two passes of queries, k = V
    (777, 64, synth.BF16, 1, 777),     # k = V
    (100000, 128, synth.BF16, 2, 50),
    (262147, 96, synth.BF16, 1, 1),    # rows_per_wg > 512, k = 1
    # batched bf16 on the matrix cores
    (20011, 256, synth.BF16, 16, 50),  # one 16-query tile, ragged slab tail
    (9000, 1000, synth.BF16, 33, 64),  # three query tiles padded to four, column tail
    (9000, 1000, synth.BF16, 20, 64),  # two query tiles, stages loaded two ahead
    (5000, 1400, synth.BF16, 24, 30),  # an odd number of 128-column stages, column tail
    (2500, 40, synth.BF16, 20, 5),     # a row shorter than one 128-column step
    (3000, 64, synth.BF16, 130, 10),   # passes of 64, 64 and 2 queries
    (262147, 64, synth.BF16, 16, 20),  # several row blocks per slab
    (777, 37, synth.BF16, 17, 30),     # odd row: batched on the vector path
    (4000, 96, synth.F32, 24, 40),     # fp32 batch: vector path, passes of 8
    (1000, 64, synth.BF16, 16, 50),    # fewer slabs than k on the matrix-core path
    # one or two queries over 16-byte aligned rows: the streaming slab kernel
    (30011, 640, synth.BF16, 1, 50),   # 80 chunks: the second chunk on 16 lanes only
    (12000, 1536, synth.BF16, 1, 64),  # 3 of 4 chunks per lane
    (6007, 2048, synth.BF16, 1, 50),   # 4 of 4 chunks per lane (the Llama-3.2-1B row width)
    (9001, 3072, synth.BF16, 1, 50),   # 6 of 8 chunks per lane
    (7001, 2048, synth.BF16, 2, 50),   # two queries, 4 chunks per lane
    (5003, 3072, synth.BF16, 2, 10),   # two queries, rows too long for it: the slab kernel
    (8000, 1000, synth.F32, 1, 30),    # fp32, 250 chunks
    (3000, 3072, synth.F32, 1, 50),    # fp32 rows of 768 chunks: 12 of 12 per lane
    (2000, 2560, synth.F32, 1, 20),    # fp32, 10 of 12 chunks per lane
    (2500, 5120, synth.BF16, 1, 40),   # bf16 rows of 10 KB: 10 of 12 chunks per lane
    (1200, 6144, synth.BF16, 1, 50),   # bf16, 12 of 12 chunks per lane
    (1500, 3328, synth.F32, 1, 10),    # 13 chunks per lane: the slab kernel
    (4000, 256, synth.F32, 2, 40),     # fp32, two queries, one chunk per lane
    # fewer slabs than k over more rows than the merge holds in LDS: every
    # row is a candidate and the merge bisects the whole key space
    (5000, 64, synth.BF16, 4, 50),     # matrix cores: 40 slabs of 128 rows
    (5000, 64, synth.F32, 1, 1024),    # vector path: 1000 slabs of 5 rows
    (151936, 64, synth.BF16, 1, 1024), # vector path: 1020 slabs of 149 rows
]


@pytest.mark.parametrize("V,d,dtype,B,k", DENSE_CASES)
def test_dense_topk_matches_oracle(vie, V, d, dtype, B, k):
    say("dense", V, d, dtype, B, k)
    W = synth.make_w(V, d, dtype, 31 + V)
    H, _ = synth.make_queries(W, dtype, B, 32 + V)
    head = vie.DenseHead(dev_tensor(vie, W, dtype), max_batch=B, max_k=k)
    ids, lg = head(dev_tensor(vie, H, dtype), k)
    torch.cuda.synchronize()
    ids, lg = ids.cpu().numpy(), lg.cpu().numpy()
    oid, olg, osc = O.topk(W, dtype, H, k)
    parity.check_logits(W, dtype, H, ids, lg, "dense")
    parity.check_id_sets(W, dtype, H, ids, oid, osc[:, -1], what="dense")
    # repeated calls reuse the workspace
    for _ in range(2):
        ids2, lg2 = head(dev_tensor(vie, H, dtype), k)
        torch.cuda.synchronize()
        assert np.array_equal(ids2.cpu().numpy(), ids) and np.array_equal(lg2.cpu().numpy(), lg)


@pytest.mark.parametrize("B,k", [(1, 50), (1, 100), (16, 50), (16, 100)])
def test_dense_far_maximum_takes_the_exact_fallbacks(vie, B, k):
    # one planted row per query scores about 2^20 times the usual maximum, so
    # the merge's histogram window (eight binades below the largest slab
    # maximum) holds fewer than k slab maxima: k <= 64 takes the sorting
    # network over the maxima, larger k the radix select
    V, d = 20000, 128
    W = synth.make_w(V, d, synth.BF16, 141)
    H, _ = synth.make_queries(W, synth.BF16, B, 142)
    Wf = synth.bf16_bits_to_f32(W).copy()
    hf = synth.bf16_bits_to_f32(H)
    for b in range(B):
        Wf[7 + 100 * b] = hf[b] / (hf[b] @ hf[b]) * 2.0 ** 20
    W = synth.f32_to_bf16_bits(Wf)
    head = vie.DenseHead(dev_tensor(vie, W, synth.BF16), max_batch=B, max_k=k)
    ids, lg = head(dev_tensor(vie, H, synth.BF16), k)
    torch.cuda.synchronize()
    ids, lg = ids.cpu().numpy(), lg.cpu().numpy()
    oid, olg, osc = O.topk(W, synth.BF16, H, k)
    parity.check_logits(W, synth.BF16, H, ids, lg, "far maximum")
    parity.check_id_sets(W, synth.BF16, H, ids, oid, osc[:, -1], what="far maximum")
    assert all(ids[b, 0] == 7 + 100 * b for b in range(B))


@pytest.mark.parametrize("B", [1, 4])
def test_dense_clustered_top_keys(vie, B):
    # the best rows sit next to each other, so several slabs hold many of
    # the top k and must be read again (not just their largest key)
    V, d, k = 20000, 128, 50
    W = synth.make_w(V, d, synth.BF16, 77)
    H, _ = synth.make_queries(W, synth.BF16, B, 78)
    Wf = synth.bf16_bits_to_f32(W).copy()
    hf = synth.bf16_bits_to_f32(H)
    rng = np.random.default_rng(3)
    for b in range(B):
        rows = np.arange(1000 * b, 1000 * b + 120)
        Wf[rows] = hf[b] * (0.02 + rng.random((120, 1)))
    W = synth.f32_to_bf16_bits(Wf)
    head = vie.DenseHead(dev_tensor(vie, W, synth.BF16), max_batch=B, max_k=k)
    ids, lg = head(dev_tensor(vie, H, synth.BF16), k)
    torch.cuda.synchronize()
    ids, lg = ids.cpu().numpy(), lg.cpu().numpy()
    oid, olg, osc = O.topk(W, synth.BF16, H, k)
    parity.check_logits(W, synth.BF16, H, ids, lg, "clustered")
    parity.check_id_sets(W, synth.BF16, H, ids, oid, osc[:, -1], what="clustered")
    assert all(np.isin(ids[b], np.arange(1000 * b, 1000 * b + 120)).sum() >= 40 for b in range(B))


@pytest.mark.parametrize("B,dtype", [(1, synth.BF16), (2, synth.BF16), (1, synth.F32), (4, synth.BF16),
                                     (16, synth.BF16)])
def test_dense_slab_lists_boundary(vie, B, dtype):
    # each slab passes its four largest keys to the merge; here single slabs
    # hold exactly 3, 4 and 5 of the top k (rows 2560 apart start a slab both
    # for 20-row slabs of the vector path and 128-row slabs of the matrix
    # cores), so the merge takes a list whole, must read a slab whose fourth
    # key clears the threshold, and must find a fifth key outside the list
    V, d, k = 20000, 128, 20
    W = synth.make_w(V, d, dtype, 91)
    H, _ = synth.make_queries(W, dtype, B, 92)
    Wf = synth.stored_values_f32(W, dtype).copy()
    hf = synth.stored_values_f32(H, dtype)
    planted = np.concatenate([np.arange(0, 3), np.arange(2560, 2564), np.arange(5120, 5125)])
    Wf[planted] = hf[0] * (4.0 + 0.1 * np.arange(len(planted)))[:, None] / (hf[0] @ hf[0]) * 10.0
    W = Wf if dtype == synth.F32 else synth.f32_to_bf16_bits(Wf)
    head = vie.DenseHead(dev_tensor(vie, W, dtype), max_batch=B, max_k=k)
    ids, lg = head(dev_tensor(vie, H, dtype), k)
    torch.cuda.synchronize()
    ids, lg = ids.cpu().numpy(), lg.cpu().numpy()
    oid, olg, osc = O.topk(W, dtype, H, k)
    assert set(planted.tolist()) <= set(oid[0].tolist())
    parity.check_logits(W, dtype, H, ids, lg, "slab lists")
    parity.check_id_sets(W, dtype, H, ids, oid, osc[:, -1], what="slab lists")


@pytest.mark.parametrize("V,k", [(30000, 64), (200000, 100)])
def test_dense_zero_query_orders_by_id(vie, V, k):
    # every logit is 0, so the answer is ids 0..k-1 (ties go to the smaller
    # id); the second case has more tied keys at the threshold than the
    # merge holds in LDS, which takes its bisection path
    W = synth.make_w(V, 32, synth.BF16, 5)
    head = vie.DenseHead(dev_tensor(vie, W, synth.BF16), max_batch=1, max_k=k)
    ids, lg = head(torch.zeros((1, 32), dtype=torch.bfloat16, device="cuda"), k)
    torch.cuda.synchronize()
    assert ids.cpu().numpy()[0].tolist() == list(range(k))
    assert np.all(lg.cpu().numpy() == 0)


# --------------------------------------------------------------------- HNSW

def _load_on_gpu(vie, g, W, dtype, tmp):
    p = os.path.join(tmp, "g.vie")
    O.save_graph(g, p, W)
    ix = vie.Index.load(p, W)
    ix.to_device(dev_tensor(vie, W, dtype))
    return ix


def _compare_hnsw(vie, ix, W, dtype, g, H, k, ef, what, width=1, int8=None, team=1, share=1):
    """One launch of the search variant (width expansions per layer-0 step;
    int8 = the oracle's (rows, scales) when layer 0 walks int8 rows) against
    the oracle's search of the same variant on the same graph.  A query
    walks the oracle's path when it expands the oracle's nodes in the
    oracle's order (equal expansion records and counts); its id set must
    then equal the oracle's up to near ties at the k-th score.  A query that
    parts from the oracle's path must do so at a near tie: the first
    expansion where the records differ is traced back to the comparison that
    decided it, whose scores must lie within 1e-4 relative (an fp32 sum
    against a float64 one can order such a pair either way); it is counted,
    and its ids are not compared.  Every returned logit must agree with the
    exact score of its id.  Returns (ids, stats, parted queries)."""
    ef_eff = max(ef, k)
    cap = ef_eff + 1024
    h = dev_tensor(vie, H, dtype)
    ids, lg, st, tr = ix.query(h, k, ef, stats=True, width=width, int8=int8 is not None, trace_cap=cap, team=team,
                               share=share)
    torch.cuda.synchronize()
    ids, lg, st, tr = (ids.cpu().numpy(), lg.cpu().numpy(), st.cpu().numpy().astype(np.uint32),
                       tr.cpu().numpy())
    if int8 is not None:
        oid, olg, ost, otr = parity.oracle_rows(O.hnsw_search_q, H, W, dtype, g, int8[0], int8[1], None, k, ef,
                                                width, validate=False, trace_cap=cap)
    elif width > 1:
        oid, olg, ost, otr = parity.oracle_rows(O.hnsw_search_multi, H, W, dtype, g, None, k, ef, width,
                                                validate=False, trace_cap=cap)
    else:
        oid, olg, ost, _, otr = parity.oracle_rows(O.hnsw_search, H, W, dtype, g, None, k, ef, validate=False,
                                                   trace_cap=cap)
    assert st[:, 1].max() <= cap
    parted = []
    for q in range(len(H)):
        if st[q].tolist() == ost[q].tolist() and np.array_equal(tr[q], otr[q]):
            continue
        try:
            why = parity.first_divergence(W, dtype, g, H[q], tr[q], otr[q], ef_eff, int8=int8 is not None)
        except AssertionError as e:
            raise AssertionError("%s: query %d leaves the oracle's path, not at a near tie (counts %s vs %s): %s" %
                                 (what, q, st[q].tolist(), ost[q].tolist(), e))
        parted.append(q)
        say("  %s: query %d parts from the oracle at expansion %d (layer %d: %s vs %s), a tie within %.2g" %
            ((what, q) + tuple(why[:4]) + (why[4],)))
    parity.check_logits(W, dtype, H, ids, lg, what)
    valid = oid[:, -1] >= 0
    osk = np.where(valid, parity.exact_scores(W, dtype, H, np.where(oid >= 0, oid, 0))[:, -1], 0)
    keep = np.array([q for q in range(len(H)) if q not in parted], np.int64)
    parity.check_id_sets(W, dtype, H, ids, oid, osk, queries=keep, what=what)
    return ids, st, len(parted)


def _library_graph(ix, W, dtype, efC, seed):
    """The oracle's view (a Graph) of a graph built by the library."""
    e, info = ix.export(), ix.info()
    g = O.Graph(W.shape[0], W.shape[1], dtype, info["M"], info["M0"], efC, seed, info["maxlevel"], info["entry"],
                e["levels"], e["adj0"], e["upper_off"], e["upper"])
    assert O.check_graph(g) == ""
    return g


@pytest.mark.parametrize("V,d,dtype,M,efC", [(3000, 64, synth.F32, 8, 60), (5000, 128, synth.BF16, 12, 80),
                                             (2500, 40, synth.BF16, 6, 40)])
def test_hnsw_matches_oracle_on_oracle_graph(vie, V, d, dtype, M, efC):
    say("hnsw", V, d, dtype, M, efC)
    W = synth.make_w(V, d, dtype, 41 + V)
    H, _ = synth.make_queries(W, dtype, 48, 42 + V)
    g = O.hnsw_build(W, dtype, M, efC, 7)
    exact, _, _ = O.topk(W, dtype, H, 50)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, dtype, tmp)
        for k, ef in [(1, 1), (10, 10), (10, 50), (50, 150), (50, 20)]:
            ids, st, nd = _compare_hnsw(vie, ix, W, dtype, g, H, k, ef, "hnsw V=%d k=%d ef=%d" % (V, k, ef))
            say("  k=%d ef=%d recall@k=%.3f divergent=%d mean n_dist=%.0f" %
                (k, ef, parity.recall(ids, exact[:, :k]), nd, st[:, 0].mean()))
        # one query per launch gives the same answers as the batch
        ids_b, lg_b = ix.query(dev_tensor(vie, H, dtype), 10, 50)
        for q in range(4):
            i1, l1 = ix.query(dev_tensor(vie, H[q:q + 1], dtype), 10, 50)
            assert np.array_equal(i1.cpu().numpy()[0], ids_b.cpu().numpy()[q])


@pytest.mark.parametrize("width", [2, 3, 4, 8, 13, 32, 64, 128])
def test_hnsw_multi_expansion_matches_oracle(vie, width):
    """Several expansions per step follow the oracle's multi-expansion search
    (same visits and counts), with the list cache and ragged picks."""
    V, d = 6000, 96
    W = synth.make_w(V, d, synth.BF16, 880)
    H, _ = synth.make_queries(W, synth.BF16, 32, 881)
    g = O.hnsw_build(W, synth.BF16, 8, 40, 5)
    exact, _, _ = O.topk(W, synth.BF16, H, 50)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, synth.BF16, tmp)
        # ef = 600: more than 256 entries past the first unexpanded one, so the
        # picks are found eight flags per lane until the span shortens
        for k, ef in [(10, 10), (50, 64), (50, 200), (50, 600)]:
            what = "multi width=%d k=%d ef=%d" % (width, k, ef)
            ids, st, _ = _compare_hnsw(vie, ix, W, synth.BF16, g, H, k, ef, what, width=width)
            say("  %s recall@k=%.3f mean n_dist=%.0f n_expand=%.1f" %
                (what, parity.recall(ids, exact[:, :k]), st[:, 0].mean(), st[:, 1].mean()))


@pytest.mark.parametrize("team", [2, 4, 32, 64, 128, 256])
def test_hnsw_team_equals_one_workgroup(vie, team):
    """A team of workgroups per query (each scoring its share of the new
    nodes, all exchanging the keys that can enter the beam) walks the same
    path as one workgroup: ids, logits, stats and expansion records are
    bitwise those of team = 1, for the sequential and wide steps on bf16
    and int8 rows, and the team's search matches the oracle.  (All B x team
    workgroups must be resident at once: at most two 1024-thread workgroups
    per CU, so the batch shrinks as the team grows.)"""
    V, d = 6000, 96
    W = synth.make_w(V, d, synth.BF16, 1880)
    H, _ = synth.make_queries(W, synth.BF16, min(24, 256 // team), 1881)
    g = O.hnsw_build(W, synth.BF16, 8, 40, 5)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, synth.BF16, tmp)
    h = dev_tensor(vie, H, synth.BF16)
    oq, osc = O.quantize_rows(W, synth.BF16)
    q8, sc = vie.quantize_rows(ix._W_dev, synth.BF16)
    for int8 in (False, True):
        ix.attach_int8(q8, sc) if int8 else ix.attach_int8(None, None)
        for width in (1, 8, 64, 128):
            for k, ef in [(10, 10), (50, 200), (50, 600)]:
                what = "team=%d int8=%d width=%d k=%d ef=%d" % (team, int8, width, k, ef)
                say(what)
                one = ix.query(h, k, ef, stats=True, width=width, int8=int8, trace_cap=ef + 1024)
                many = ix.query(h, k, ef, stats=True, width=width, int8=int8, trace_cap=ef + 1024, team=team)
                torch.cuda.synchronize()
                for a, b, name in zip(one, many, ("ids", "logits", "stats", "trace")):
                    a, b = a.cpu().numpy(), b.cpu().numpy()
                    assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), "%s: %s differ" % (what, name)
        _compare_hnsw(vie, ix, W, synth.BF16, g, H, 50, 200, "team=%d int8=%d vs oracle" % (team, int8), width=8,
                      int8=(oq, osc) if int8 else None, team=team)
    ix.attach_int8(None, None)
    # one query after a batch: the arrival counters start again from zero
    a = ix.query(h[:1], 10, 50, team=team)
    b = ix.query(h[:1], 10, 50)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


@pytest.mark.parametrize("dtype,d", [(synth.BF16, 96), (synth.F32, 64)])
def test_hnsw_row_sharing_equals_independent(vie, dtype, d):
    """Queries that share fetched rows in groups (a row fetched for one query
    is scored for every query of its group, the others' scores published in
    the workspace) walk exactly the paths of independent workgroups: ids,
    logits, stats and expansion records bitwise equal to share = 1, for
    groups of 2, 4 and 16 with a partial last group, on stored and int8
    rows, across calls that reuse the workspace; and against the oracle."""
    V = 6000
    W = synth.make_w(V, d, dtype, 1900 + d)
    H, _ = synth.make_queries(W, dtype, 23, 1901 + d)
    g = O.hnsw_build(W, dtype, 8, 40, 5)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, dtype, tmp)
    h = dev_tensor(vie, H, dtype)
    oq, osc = O.quantize_rows(W, dtype)
    q8, sc = vie.quantize_rows(ix._W_dev, dtype)
    for int8 in (False, True):
        ix.attach_int8(q8, sc) if int8 else ix.attach_int8(None, None)
        for width in (1, 8, 64):
            for k, ef in [(10, 10), (50, 200), (50, 600)]:
                one = ix.query(h, k, ef, stats=True, width=width, int8=int8, trace_cap=ef + 1024)
                for share in (2, 4, 16):
                    what = "share=%d int8=%d width=%d k=%d ef=%d" % (share, int8, width, k, ef)
                    many = ix.query(h, k, ef, stats=True, width=width, int8=int8, trace_cap=ef + 1024, share=share)
                    torch.cuda.synchronize()
                    for a, b, name in zip(one, many, ("ids", "logits", "stats", "trace")):
                        a, b = a.cpu().numpy(), b.cpu().numpy()
                        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), "%s: %s differ" % (what, name)
            say("  share int8=%d width=%d equal to independent workgroups" % (int8, width))
        _compare_hnsw(vie, ix, W, dtype, g, H, 50, 200, "share=4 int8=%d vs oracle" % int8, width=8,
                      int8=(oq, osc) if int8 else None, share=4)
    ix.attach_int8(None, None)


def test_hnsw_lds_at_the_limit_is_refused_cleanly(vie):
    """Beams whose LDS carve-up lands within a couple of KB of the per-block
    limit (where the kernels' static variables no longer fit beside it):
    every call either runs or is refused with VIE_EUNSUPPORTED before any
    launch, never a failed launch."""
    V, d = 3000, 3072
    W = synth.make_w(V, d, synth.F32, 1910)
    H, _ = synth.make_queries(W, synth.F32, 2, 1911)
    g = O.hnsw_build(W, synth.F32, 32, 40, 5)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, synth.F32, tmp)
    h = dev_tensor(vie, H, synth.F32)
    seen = set()
    # LDS about 110968 + 18 ef bytes against 160 KB less a 3 KB reserve: the
    # sweep crosses near ef = 2766
    for ef in range(2700, 2860, 4):
        try:
            ids, _ = ix.query(h, 10, ef, width=128, team=2)
            torch.cuda.synchronize()
            assert (ids.cpu().numpy() >= 0).all()
            seen.add("ok")
        except vie.VieError as e:
            assert e.status == vie.EUNSUPPORTED, (ef, str(e))
            seen.add("refused")
    assert seen == {"ok", "refused"}, seen  # the sweep crosses the limit


def test_hnsw_team_too_large_is_refused(vie):
    """More team workgroups than the device holds at once: refused before
    any launch (a member would otherwise wait for one never scheduled)."""
    V, d = 3000, 64
    W = synth.make_w(V, d, synth.BF16, 1890)
    g = O.hnsw_build(W, synth.BF16, 8, 40, 5)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, synth.BF16, tmp)
    H, _ = synth.make_queries(W, synth.BF16, 4096, 1891)
    with pytest.raises(vie.VieError) as e:
        ix.query(dev_tensor(vie, H, synth.BF16), 10, 50, team=32)
    assert e.value.status == vie.EUNSUPPORTED


@pytest.mark.parametrize("case", ["first64", "overlap", "max", "width4", "none"])
def test_forced_tokens_match_oracle(vie, case):
    """Search plus forced-inclusion ids against the oracle's search joined
    with the same ids (each id once, by exact score, -1/-inf padding)."""
    V, d, k, ef = 5000, 64, 20, 40
    W = synth.make_w(V, d, synth.BF16, 990)
    H, _ = synth.make_queries(W, synth.BF16, 24, 991)
    g = O.hnsw_build(W, synth.BF16, 8, 40, 6)
    width = 4 if case == "width4" else 1
    if width == 1:
        oid, olg, ost, _ = O.hnsw_search(W, synth.BF16, g, H, k, ef, validate=False)
    else:
        oid, olg, ost = O.hnsw_search_multi(W, synth.BF16, g, H, k, ef, width, validate=False)
    rng = np.random.default_rng(7)
    if case in ("first64", "width4"):
        forced = np.arange(64, dtype=np.int32)
    elif case == "overlap":  # half of them are found by the search of query 0
        forced = np.unique(np.concatenate([oid[0, :10], rng.choice(V, 30, replace=False)])).astype(np.int32)
    elif case == "max":
        forced = rng.choice(V, 1024, replace=False).astype(np.int32)
    else:
        forced = np.zeros(0, np.int32)
    n = forced.size
    fid, flg = O.forced_merge(W, synth.BF16, H, oid, forced)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, synth.BF16, tmp)
        ids = torch.empty((len(H), k + n), dtype=torch.int32, device="cuda")
        lg = torch.empty((len(H), k + n), dtype=torch.float32, device="cuda")
        st = torch.empty((len(H), 2), dtype=torch.int32, device="cuda")
        ix.query_forced_into(dev_tensor(vie, H, synth.BF16), k, ef, torch.from_numpy(forced).cuda(), ids, lg, st,
                             width)
        torch.cuda.synchronize()
    ids, lg, st = ids.cpu().numpy(), lg.cpu().numpy(), st.cpu().numpy().astype(np.uint32)
    same = np.all(st == ost, axis=1)
    assert int((~same).sum()) == 0, case
    parity.check_logits(W, synth.BF16, H, ids, lg, "forced " + case)
    osk = parity.exact_scores(W, synth.BF16, H, oid)[:, -1]
    parity.check_id_sets(W, synth.BF16, H, ids, fid, osk, queries=np.nonzero(same)[0], what="forced " + case)
    for q in np.nonzero(same)[0]:
        assert set(forced.tolist()) <= set(ids[q].tolist()), case  # every forced id is present
        assert (ids[q] >= 0).sum() == (fid[q] >= 0).sum(), case     # the same number of distinct ids


@pytest.mark.parametrize("V,d,dtype", [(3000, 64, synth.BF16), (1000, 48, synth.F32), (500, 3072, synth.BF16),
                                       (777, 256, synth.F32)])
def test_int8_rows_bitwise(vie, V, d, dtype):
    W = synth.make_w(V, d, dtype, 400 + d)
    if dtype == synth.F32:
        W[::97] = 0.0  # rows of zeros: scale 0
    q, sc = vie.quantize_rows(dev_tensor(vie, W, dtype), dtype)
    torch.cuda.synchronize()
    oq, osc = O.quantize_rows(W, dtype)
    assert np.array_equal(q.cpu().numpy(), oq)
    assert np.array_equal(sc.cpu().numpy().view(np.uint32), osc.view(np.uint32))


@pytest.mark.parametrize("width", [1, 4, 8, 64])
def test_int8_search_matches_oracle(vie, width):
    """Layer 0 on int8 scores (integer dot, fp32 scale products) walks exactly
    the oracle's path; the re-ranked result matches within the tolerances."""
    V, d = 6000, 128
    W = synth.make_w(V, d, synth.BF16, 1234)
    H, _ = synth.make_queries(W, synth.BF16, 32, 1235)
    g = O.hnsw_build(W, synth.BF16, 8, 40, 8)
    oq, osc = O.quantize_rows(W, synth.BF16)
    exact, _, _ = O.topk(W, synth.BF16, H, 50)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, synth.BF16, tmp)
        q, sc = vie.quantize_rows(ix._W_dev, synth.BF16)
        ix.attach_int8(q, sc)
        for k, ef in [(10, 40), (50, 100), (50, 512)]:
            what = "int8 width=%d k=%d ef=%d" % (width, k, ef)
            ids, st, _ = _compare_hnsw(vie, ix, W, synth.BF16, g, H, k, ef, what, width=width, int8=(oq, osc))
            say("  %s recall@k=%.3f mean n_dist=%.0f" % (what, parity.recall(ids, exact[:, :k]), st[:, 0].mean()))


def test_hnsw_wide_beams_match_oracle(vie):
    """Beams of 2048 and 4096 entries (LDS above 64 KiB) follow the oracle's
    traversal exactly, and recall does not drop as the beam grows."""
    V, d = 20000, 64
    W = synth.make_w(V, d, synth.BF16, 555)
    H, _ = synth.make_queries(W, synth.BF16, 12, 556)
    g = O.hnsw_build(W, synth.BF16, 8, 40, 9)
    exact, _, _ = O.topk(W, synth.BF16, H, 50)
    rec = []
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, synth.BF16, tmp)
        for ef in (2048, 4096):
            ids, st, nd = _compare_hnsw(vie, ix, W, synth.BF16, g, H, 50, ef, "hnsw ef=%d" % ef)
            rec.append(parity.recall(ids, exact))
            say("  ef=%d recall@50=%.3f divergent=%d mean n_dist=%.0f" % (ef, rec[-1], nd, st[:, 0].mean()))
    assert rec[1] >= rec[0] - 1e-9


def test_hnsw_ef_at_least_v_is_exact(vie):
    W = synth.make_w(400, 12, synth.F32, 121)
    W = (W / np.linalg.norm(W, axis=1, keepdims=True)).astype(np.float32)
    g = O.hnsw_build(W, synth.F32, 5, 40, 21)
    H, _ = synth.make_queries(W, synth.F32, 16, 22)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, synth.F32, tmp)
        ids, lg = ix.query(dev_tensor(vie, H, synth.F32), 10, 400)
    torch.cuda.synchronize()
    oid, olg, osc = O.topk(W, synth.F32, H, 10)
    parity.check_id_sets(W, synth.F32, H, ids.cpu().numpy(), oid, osc[:, -1], what="ef>=V")
    parity.check_logits(W, synth.F32, H, ids.cpu().numpy(), lg.cpu().numpy(), "ef>=V")


def test_hnsw_small_graph_pads_missing_results(vie):
    # 6 nodes, k = 6: everything reachable is returned, the rest is -1 / -inf
    W = synth.make_w(6, 4, synth.F32, 3)
    g = O.hnsw_build(W, synth.F32, 2, 6, 1, M0=2, select="simple")
    H, _ = synth.make_queries(W, synth.F32, 3, 4)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, synth.F32, tmp)
        ids, lg = ix.query(dev_tensor(vie, H, synth.F32), 6, 6)
    oid, olg, _, _ = O.hnsw_search(W, synth.F32, g, H, 6, 6)
    assert np.array_equal(ids.cpu().numpy(), oid)
    assert np.array_equal(np.isneginf(lg.cpu().numpy()), np.isneginf(olg))


# ------------------------------------------- full-size workload shapes

def test_tiny_workload_full_size(vie):
    """|V| = 32768, d = 256 fp32, M = 16, efC = 100, ef = 64, k = 50, 256 queries:
    HNSW on the library-built graph against the oracle's search of that graph
    (sampled), the dense head against the exact top-k (sampled), recall@50."""
    wl = synth.WORKLOADS["tiny"]
    W = wl.make_w()
    H, _ = wl.make_queries(W)
    ix = vie.Index.build(W, wl.dtype, wl.M, wl.efC, seed=wl.seed_levels, n_threads=16)
    e, info = ix.export(), ix.info()
    g = O.Graph(wl.V, wl.d, wl.dtype, info["M"], info["M0"], wl.efC, wl.seed_levels, info["maxlevel"],
                info["entry"], e["levels"], e["adj0"], e["upper_off"], e["upper"])
    assert O.check_graph(g) == ""
    Wd = dev_tensor(vie, W, wl.dtype)
    ix.to_device(Wd)
    sample = np.arange(0, wl.Q, 8)
    ids, st, nd = _compare_hnsw(vie, ix, W, wl.dtype, g, H[sample], 50, 64, "tiny hnsw")
    hid, _ = ix.query(dev_tensor(vie, H, wl.dtype), 50, 64)
    head = vie.DenseHead(Wd, max_batch=1, max_k=50)
    did = np.stack([head(dev_tensor(vie, H[q:q + 1], wl.dtype), 50)[0].cpu().numpy()[0] for q in sample])
    oid, olg, osc = O.topk(W, wl.dtype, H[sample], 50)
    parity.check_id_sets(W, wl.dtype, H[sample], did, oid, osc[:, -1], what="tiny dense")
    say("tiny: recall@50 = %.4f, divergent = %d, mean n_dist = %.0f" %
        (parity.recall(hid.cpu().numpy()[sample], oid), nd, st[:, 0].mean()))


@pytest.mark.parametrize("name", ["qwen3-0.6b", "llama3.2-1b", "gemma3-270m", "llama3.2-3b"])
def test_dense_full_size_sampled(vie, name):
    wl = synth.WORKLOADS[name]
    say("dense full", name)
    W = wl.make_w()
    H, _ = wl.make_queries(W, Q=2)
    Wd = dev_tensor(vie, W, wl.dtype)
    head = vie.DenseHead(Wd, max_batch=1, max_k=max(wl.k))
    oid, olg, osc = O.topk(W, wl.dtype, H, max(wl.k))
    for k in wl.k:
        got = [head(dev_tensor(vie, H[q:q + 1], wl.dtype), k) for q in range(2)]
        ids = np.stack([g[0].cpu().numpy()[0] for g in got])
        lg = np.stack([g[1].cpu().numpy()[0] for g in got])
        parity.check_logits(W, wl.dtype, H, ids, lg, name)
        parity.check_id_sets(W, wl.dtype, H, ids, oid[:, :k], osc[:, k - 1], what=name)
    # a batch of 64 (matrix-core path) whose first two queries are the ones above
    HB, _ = wl.make_queries(W, Q=64)
    assert np.array_equal(HB[:2], H)
    bhead = vie.DenseHead(Wd, max_batch=64, max_k=max(wl.k))
    k = max(wl.k)
    ids, lg = bhead(dev_tensor(vie, HB, wl.dtype), k)
    ids, lg = ids.cpu().numpy()[:2], lg.cpu().numpy()[:2]
    parity.check_logits(W, wl.dtype, H, ids, lg, name + " B=64")
    parity.check_id_sets(W, wl.dtype, H, ids, oid[:, :k], osc[:, k - 1], what=name + " B=64")


@pytest.mark.parametrize("name", ["qwen3-0.6b", "llama3.2-1b", "gemma3-270m", "llama3.2-3b"])
def test_hnsw_row_shapes_of_each_workload(vie, name):
    """The HNSW kernel at each workload's row width and dtype (and, for Gemma,
    its hub rows) on a 12k-row slice with a quickly built graph."""
    wl = synth.WORKLOADS[name]
    say("hnsw shape", name)
    V = 12000
    W = synth.make_w(V, wl.d, wl.dtype, wl.seed_w, wl.hub_frac, seed_hub=wl.seed_hub)
    H, _ = synth.make_queries(W, wl.dtype, 24, wl.seed_q)
    ix = vie.Index.build(W, wl.dtype, 16, 40, seed=wl.seed_levels, n_threads=16)
    e, info = ix.export(), ix.info()
    g = O.Graph(V, wl.d, wl.dtype, info["M"], info["M0"], 40, wl.seed_levels, info["maxlevel"], info["entry"],
                e["levels"], e["adj0"], e["upper_off"], e["upper"])
    ix.to_device(dev_tensor(vie, W, wl.dtype))
    for k in wl.k:
        _compare_hnsw(vie, ix, W, wl.dtype, g, H, k, max(wl.ef), "%s k=%d" % (name, k))


@pytest.mark.parametrize("d,dtype", [(2048, synth.BF16), (3072, synth.BF16), (1500, synth.BF16), (384, synth.F32),
                                     (1000, synth.F32), (1008, synth.F32)])
def test_multi_and_int8_at_wide_rows(vie, d, dtype):
    """Several expansions per step and int8 layer-0 scores on rows wide
    enough for the 32- and 64-lane groups (bf16 rows of 2048 and 3072 values,
    a ragged 1500; fp32 rows of 384, 1000 and 1008), against the oracle's
    multi-expansion and int8 searches on the same graph; int8 rows whose
    width is not a multiple of 16 are refused."""
    say("multi/int8 wide rows", d, dtype)
    V = 6000
    W = synth.make_w(V, d, dtype, 700 + d)
    H, _ = synth.make_queries(W, dtype, 16, 701 + d)
    ix = vie.Index.build(W, dtype, 16, 40, seed=702 + d, n_threads=16)
    e, info = ix.export(), ix.info()
    g = O.Graph(V, d, dtype, info["M"], info["M0"], 40, 702 + d, info["maxlevel"], info["entry"],
                e["levels"], e["adj0"], e["upper_off"], e["upper"])
    ix.to_device(dev_tensor(vie, W, dtype))
    k, ef = 50, 128
    # one expansion per step (hnsw_kernel at the same widths; 3000-byte rows
    # load 8 bytes per lane chunk)
    _compare_hnsw(vie, ix, W, dtype, g, H, k, ef, "hnsw d=%d" % d)
    for width in (2, 4, 8):
        what = "multi d=%d width=%d" % (d, width)
        ids, st, _ = _compare_hnsw(vie, ix, W, dtype, g, H, k, ef, what, width=width)
        say("  %s mean n_dist=%.0f" % (what, st[:, 0].mean()))
    oq, osc = O.quantize_rows(W, dtype)
    q, sc = vie.quantize_rows(ix._W_dev, dtype)
    assert np.array_equal(q.cpu().numpy(), oq)
    if d % 16 != 0:
        # int8 layer-0 scores load 16-byte chunks of a row: refused on the host
        with pytest.raises(vie.VieError, match="divisible by 16"):
            ix.attach_int8(q, sc)
        return
    ix.attach_int8(q, sc)
    for width in (1, 8):
        what = "int8 d=%d width=%d" % (d, width)
        ids, st, _ = _compare_hnsw(vie, ix, W, dtype, g, H, k, ef, what, width=width, int8=(oq, osc))
        say("  %s mean n_dist=%.0f" % (what, st[:, 0].mean()))


@pytest.mark.parametrize("V,d,dtype", [(3001, 37, synth.BF16), (2500, 38, synth.BF16), (2000, 5, synth.F32),
                                       (2500, 36, synth.BF16)])
def test_hnsw_narrow_loads_match_oracle(vie, V, d, dtype):
    """Rows whose size is not a multiple of 16 bytes (74 bytes: 2-byte
    chunks; 76 and 20 bytes: 4-byte chunks; 72 bytes: 8-byte chunks), one
    and four expansions per step, against the oracle on its own graph."""
    say("hnsw narrow loads", V, d, dtype)
    W = synth.make_w(V, d, dtype, 300 + d)
    H, _ = synth.make_queries(W, dtype, 24, 301 + d)
    g = O.hnsw_build(W, dtype, 8, 40, 302 + d)
    with tempfile.TemporaryDirectory() as tmp:
        ix = _load_on_gpu(vie, g, W, dtype, tmp)
        for k, ef in [(10, 50), (50, 128)]:
            _compare_hnsw(vie, ix, W, dtype, g, H, k, ef, "hnsw d=%d k=%d ef=%d" % (d, k, ef))
            what = "multi d=%d k=%d ef=%d" % (d, k, ef)
            ids, st, _ = _compare_hnsw(vie, ix, W, dtype, g, H, k, ef, what, width=4)
            say("  %s mean n_dist=%.0f" % (what, st[:, 0].mean()))


@pytest.mark.parametrize("V,d,dtype", [(3000, 2048, synth.BF16), (3000, 3072, synth.BF16), (3001, 37, synth.BF16),
                                       (2000, 1000, synth.F32)])
def test_forced_tokens_at_other_row_widths(vie, V, d, dtype):
    """Forced-inclusion ids scored by 32- and 64-lane groups (bf16 rows of
    2048 and 3072 values, fp32 rows of 1000) and with 2-byte lane chunks
    (bf16 rows of 37 values), after one and four expansions per step."""
    say("forced widths", V, d, dtype)
    k, ef = 20, 40
    W = synth.make_w(V, d, dtype, 950 + d)
    H, _ = synth.make_queries(W, dtype, 16, 951 + d)
    ix = vie.Index.build(W, dtype, 8, 40, seed=952 + d, n_threads=16)
    e, info = ix.export(), ix.info()
    g = O.Graph(V, d, dtype, info["M"], info["M0"], 40, 952 + d, info["maxlevel"], info["entry"],
                e["levels"], e["adj0"], e["upper_off"], e["upper"])
    ix.to_device(dev_tensor(vie, W, dtype))
    for width in (1, 4):
        if width == 1:
            oid, olg, ost, _ = O.hnsw_search(W, dtype, g, H, k, ef, validate=False)
        else:
            oid, olg, ost = O.hnsw_search_multi(W, dtype, g, H, k, ef, width, validate=False)
        rng = np.random.default_rng(d + width)
        forced = np.unique(np.concatenate([oid[0, :10], rng.choice(V, 50, replace=False)])).astype(np.int32)
        n = forced.size
        fid, flg = O.forced_merge(W, dtype, H, oid, forced)
        ids = torch.empty((len(H), k + n), dtype=torch.int32, device="cuda")
        lg = torch.empty((len(H), k + n), dtype=torch.float32, device="cuda")
        st = torch.empty((len(H), 2), dtype=torch.int32, device="cuda")
        ix.query_forced_into(dev_tensor(vie, H, dtype), k, ef, torch.from_numpy(forced).cuda(), ids, lg, st, width)
        torch.cuda.synchronize()
        ids, lg, st = ids.cpu().numpy(), lg.cpu().numpy(), st.cpu().numpy().astype(np.uint32)
        what = "forced d=%d width=%d" % (d, width)
        same = np.all(st == ost, axis=1)
        assert int((~same).sum()) == 0, what
        parity.check_logits(W, dtype, H, ids, lg, what)
        osk = parity.exact_scores(W, dtype, H, oid)[:, -1]
        parity.check_id_sets(W, dtype, H, ids, fid, osk, queries=np.nonzero(same)[0], what=what)
        for q in np.nonzero(same)[0]:
            assert set(forced.tolist()) <= set(ids[q].tolist()), what
            assert (ids[q] >= 0).sum() == (fid[q] >= 0).sum(), what
        say("  %s n=%d divergent=%d" % (what, n, int((~same).sum())))


# ------------------------------------- configurations of the workloads

def _variants(vie, ix, W, dtype, g, H, k, ef, what, widths=(1, 8), int8=True):
    """The sequential search, the multi-expansion search and, for rows of a
    multiple of 16 values, the int8 walk, each against the oracle."""
    for width in widths:
        ids, st, _ = _compare_hnsw(vie, ix, W, dtype, g, H, k, ef, "%s width=%d" % (what, width), width=width)
        say("  %s width=%d mean n_dist=%.0f n_expand=%.1f" % (what, width, st[:, 0].mean(), st[:, 1].mean()))
    if int8 and W.shape[1] % 16 == 0:
        oq, osc = O.quantize_rows(W, dtype)
        q, sc = vie.quantize_rows(ix._W_dev, dtype)
        ix.attach_int8(q, sc)
        for width in widths:
            _compare_hnsw(vie, ix, W, dtype, g, H, k, ef, "%s int8 width=%d" % (what, width), width=width,
                          int8=(oq, osc))
        ix.attach_int8(None, None)


def test_repeat_runs_are_byte_identical(vie):
    """Every kernel family run twice on the same inputs writes the same
    bytes: the dense head on the vector path (B = 1, 4) and the matrix cores
    (B = 64), the row quantization, the sequential, wide, team and
    row-sharing searches on bf16 and int8 rows (ids, logits, counters and
    expansion records) and the scatter.  Waves and workgroups that raced
    over shared state would show up here as a difference."""
    V, d = 30000, 1024
    W = synth.make_w(V, d, synth.BF16, 2100)
    H, _ = synth.make_queries(W, synth.BF16, 64, 2101)
    Wd, Hd = dev_tensor(vie, W, synth.BF16), dev_tensor(vie, H, synth.BF16)

    def twice(what, fn):
        say("repeat", what)
        a = [t.cpu().numpy().copy() for t in fn()]
        b = [t.cpu().numpy().copy() for t in fn()]
        torch.cuda.synchronize()
        for x, y in zip(a, b):
            assert x.tobytes() == y.tobytes(), what
        return a

    dense = vie.DenseHead(Wd, max_batch=64, max_k=100)
    for B in (1, 4, 64):
        for k in (1, 50, 100):
            twice("dense B=%d k=%d" % (B, k), lambda: dense(Hd[:B], k))
    q8, sc = twice("quantize", lambda: vie.quantize_rows(Wd, synth.BF16))
    ix = vie.Index.build(W, synth.BF16, 16, 40, seed=2102, n_threads=16)
    ix.to_device(Wd)
    ix.attach_int8(torch.from_numpy(q8).cuda(), torch.from_numpy(sc).cuda())
    ef = 200
    for width, int8, team, share, B in [(1, False, 1, 1, 64), (8, False, 1, 1, 64), (64, False, 4, 1, 16),
                                        (128, False, 8, 1, 8), (32, True, 2, 1, 32), (8, False, 1, 4, 64),
                                        (8, True, 1, 4, 64)]:
        what = "hnsw width=%d int8=%d team=%d share=%d B=%d" % (width, int8, team, share, B)
        ids, lg, _, _ = twice(what, lambda: ix.query(Hd[:B], 50, ef, stats=True, width=width, int8=int8,
                                                     trace_cap=ef + 1024, team=team, share=share))
    ids_d, lg_d = torch.from_numpy(ids).cuda(), torch.from_numpy(lg).cuda()
    twice("scatter", lambda: (vie.scatter(ids_d, lg_d, V),))
    ix.attach_int8(None, None)


def test_hnsw_full_size_headline_configuration(vie):
    """The configuration the benchmark times, at full size: the
    Llama-3.2-3B-shaped head (128256 rows of 3072 bf16 values), its graph
    built by the library at M = 32, ef_construction = 200, one query per
    launch, 128 expansions per layer-0 step in a team of 128 workgroups,
    k = 50, ef = 2048; 8 queries on the stored rows and 4 on int8 rows, each
    against the oracle's search of the exported graph (exact counters and
    expansion records, ids and logits)."""
    wl = synth.WORKLOADS["llama3.2-3b"]
    W = wl.make_w()
    H, _ = wl.make_queries(W, Q=8)
    ix = vie.Index.build(W, wl.dtype, wl.M, wl.efC, seed=wl.seed_levels, n_threads=16)
    g = _library_graph(ix, W, wl.dtype, wl.efC, wl.seed_levels)
    say("llama3.2-3b full: maxlevel %d entry %d" % (g.maxlevel, g.entry))
    ix.to_device(dev_tensor(vie, W, wl.dtype))
    for q in range(8):
        _, st, _ = _compare_hnsw(vie, ix, W, wl.dtype, g, H[q:q + 1], 50, 2048, "headline q=%d" % q, width=128,
                                 team=128)
        say("  q=%d n_dist=%d n_expand=%d" % (q, st[0, 0], st[0, 1]))
    oq, osc = O.quantize_rows(W, wl.dtype)
    q8, sc = vie.quantize_rows(ix._W_dev, wl.dtype)
    ix.attach_int8(q8, sc)
    for q in range(4):
        _compare_hnsw(vie, ix, W, wl.dtype, g, H[q:q + 1], 50, 2048, "headline int8 q=%d" % q, width=128,
                      team=128, int8=(oq, osc))
    ix.attach_int8(None, None)


@pytest.mark.parametrize("dtype", [synth.BF16, synth.F32])
def test_hnsw_batches_of_256_and_more(vie, dtype):
    """300 queries in one launch (more workgroups than the device holds at
    once) in every search variant; each query still walks the oracle's
    path."""
    say("hnsw B=300", dtype)
    V, d, B = 8000, 256, 300
    W = synth.make_w(V, d, dtype, 1500)
    H, _ = synth.make_queries(W, dtype, B, 1501)
    ix = vie.Index.build(W, dtype, 16, 60, seed=1502, n_threads=16)
    g = _library_graph(ix, W, dtype, 60, 1502)
    ix.to_device(dev_tensor(vie, W, dtype))
    _variants(vie, ix, W, dtype, g, H, 50, 128, "B=300", widths=(1, 8, 32))


def test_hnsw_large_batches_with_wide_beams(vie):
    """260 queries whose beams take more than half of a CU's LDS (one
    workgroup per CU at a time); every variant still walks the oracle's
    path."""
    V, d, B = 8000, 128, 260
    W = synth.make_w(V, d, synth.BF16, 1700)
    H, _ = synth.make_queries(W, synth.BF16, B, 1701)
    ix = vie.Index.build(W, synth.BF16, 16, 60, seed=1702, n_threads=16)
    g = _library_graph(ix, W, synth.BF16, 60, 1702)
    ix.to_device(dev_tensor(vie, W, synth.BF16))
    _variants(vie, ix, W, synth.BF16, g, H, 50, 5000, "B=260 ef=5000", widths=(1, 8))


@pytest.mark.parametrize("d", [640, 1024, 2048, 3072])
def test_hnsw_degree_64_at_model_row_widths(vie, d):
    """M = 32 (layer-0 lists of M0 = 64, the degree of every model-shaped
    workload) at the row widths of the Gemma-, Qwen-, Llama-1B- and
    Llama-3B-shaped heads: the lists fill the per-lane prefetch exactly."""
    say("hnsw M0=64", d)
    V = 6000
    W = synth.make_w(V, d, synth.BF16, 1600 + d)
    H, _ = synth.make_queries(W, synth.BF16, 32, 1601 + d)
    ix = vie.Index.build(W, synth.BF16, 32, 100, seed=1602 + d, n_threads=16)
    g = _library_graph(ix, W, synth.BF16, 100, 1602 + d)
    assert g.M0 == 64 and (g.adj0 >= 0).sum(axis=1).max() == 64
    ix.to_device(dev_tensor(vie, W, synth.BF16))
    for k, ef in [(50, 128), (50, 512)]:
        _variants(vie, ix, W, synth.BF16, g, H, k, ef, "M0=64 d=%d ef=%d" % (d, ef), widths=(1, 8, 32))


@pytest.mark.parametrize("d", [256, 2048])
def test_hnsw_lists_longer_than_the_prefetch(vie, d):
    """Layer-0 lists of up to 128 ids (M0 = 128, more than a lane group
    prefetches: 64 ids for 16- and 32-lane groups) are claimed from HBM."""
    say("hnsw M0=128", d)
    V = 5000
    W = synth.make_w(V, d, synth.BF16, 1700 + d)
    H, _ = synth.make_queries(W, synth.BF16, 24, 1701 + d)
    ix = vie.Index.build(W, synth.BF16, 32, 160, seed=1702 + d, n_threads=16, M0=128)
    g = _library_graph(ix, W, synth.BF16, 160, 1702 + d)
    assert g.M0 == 128 and (g.adj0 >= 0).sum(axis=1).max() > 64
    ix.to_device(dev_tensor(vie, W, synth.BF16))
    _variants(vie, ix, W, synth.BF16, g, H, 50, 200, "M0=128 d=%d" % d, widths=(1, 4))


def test_hnsw_full_size_gemma_graph(vie):
    """The Gemma-3-270M-shaped head at full size (262144 rows of 640 bf16
    values with 10% hub rows: the largest visited bitmap, 32 KiB), its graph
    built by the library at M = 32, ef_construction = 200: 32 queries at
    ef = 128 and ef = 2048, sequential and 8 expansions per step, bf16 and
    int8 rows, each against the oracle's search of the exported graph."""
    wl = synth.WORKLOADS["gemma3-270m"]
    W = wl.make_w()
    H, _ = wl.make_queries(W, Q=32)
    ix = vie.Index.build(W, wl.dtype, wl.M, wl.efC, seed=wl.seed_levels, n_threads=16)
    g = _library_graph(ix, W, wl.dtype, wl.efC, wl.seed_levels)
    say("gemma full: maxlevel %d entry %d" % (g.maxlevel, g.entry))
    ix.to_device(dev_tensor(vie, W, wl.dtype))
    for ef in (128, 2048):
        _variants(vie, ix, W, wl.dtype, g, H, 50, ef, "gemma full ef=%d" % ef, widths=(1, 8, 32))
