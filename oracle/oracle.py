"""ctypes front end of the plain-C oracle (liboracle.so).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the package smoke check
and the benchmark's CPU-baseline leg, never by the product library.

Arrays: ``W`` is [V, d] fp32, or uint16 bf16 bit patterns when ``dtype`` is 1;
queries ``h`` are [B, d] in the same form.  Each function names the part of the
paper (Section 3) or of Malkov & Yashunin's HNSW algorithms that it follows; the
C source holds the details.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os

import numpy as np

from . import build as _build

F32, BF16 = 0, 1
_lib = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        path = _build.LIB if os.path.exists(_build.LIB) else _build.build(force=False)
        L = C.CDLL(path)
        vp, i64, i32, u64 = C.c_void_p, C.c_int64, C.c_int, C.c_uint64
        L.oracle_scores.argtypes = [vp, i32, i64, i32, vp, vp]
        L.oracle_topk.argtypes = [vp, i32, i64, i32, vp, i32, i32, vp, vp, vp]
        L.oracle_topk.restype = i32
        L.oracle_pair_scores.argtypes = [vp, i32, i64, i32, vp, i64, vp, vp, vp]
        L.oracle_pair_abs_scores.argtypes = [vp, i32, i64, i32, vp, i64, vp, vp, vp]
        L.oracle_scatter.argtypes = [vp, vp, i32, i32, i64, vp]
        L.oracle_levels.argtypes = [i64, i32, u64, vp]
        L.oracle_hnsw_build.argtypes = [vp, i32, i64, i32, i32, i32, i32, u64, i32]
        L.oracle_hnsw_build.restype = vp
        L.oracle_hnsw_build_levels.argtypes = [vp, i32, i64, i32, i32, i32, i32, vp, i32]
        L.oracle_hnsw_build_levels.restype = vp
        L.oracle_graph_free.argtypes = [vp]
        L.oracle_graph_info.argtypes = [vp, vp]
        L.oracle_graph_export.argtypes = [vp, vp, vp, vp, vp]
        L.oracle_graph_check.argtypes = [i64, i32, i32, i32, i32, vp, vp, vp, vp, i64, C.c_char_p, i32]
        L.oracle_graph_check.restype = i32
        L.oracle_hnsw_search.argtypes = [vp, i32, i64, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp,
                                         i32, i32, i32, vp, vp, vp, vp, vp, i32]
        L.oracle_hnsw_search.restype = i32
        L.oracle_hnsw_search_multi.argtypes = [vp, i32, i64, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp,
                                               i32, i32, i32, i32, vp, vp, vp, vp, i32]
        L.oracle_hnsw_search_multi.restype = i32
        L.oracle_forced_merge.argtypes = [vp, i32, i64, i32, vp, i32, i32, vp, i32, vp, vp, vp]
        L.oracle_forced_merge.restype = i32
        L.oracle_quantize_rows.argtypes = [vp, i32, i64, i32, vp, vp]
        L.oracle_knn_graph.argtypes = [vp, i32, i64, i32, i32, i32, vp, vp, vp]
        L.oracle_knn_graph.restype = i32
        L.oracle_hnsw_search_q.argtypes = [vp, i32, i64, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp,
                                           i32, i32, i32, i32, vp, vp, vp, vp, i32]
        L.oracle_hnsw_search_q.restype = i32
        L.oracle_w_fingerprint.argtypes = [vp, i32, i64, i32]
        L.oracle_w_fingerprint.restype = u64
        L.oracle_file_write.argtypes = [C.c_char_p, i32, i64, i32, i32, i32, i32, u64, i32, i32, i64, u64,
                                        vp, vp, vp, vp]
        L.oracle_file_write.restype = i32
        L.oracle_file_header.argtypes = [C.c_char_p, vp]
        L.oracle_file_header.restype = i32
        L.oracle_file_body.argtypes = [C.c_char_p, i64, i32, i32, i64, vp, vp, vp, vp]
        L.oracle_file_body.restype = i32
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


def _check_w(W: np.ndarray, dtype: int) -> np.ndarray:
    want = np.float32 if dtype == F32 else np.uint16
    if W.dtype != want or W.ndim != 2:
        raise TypeError("W must be a 2-D %s array" % np.dtype(want).name)
    return np.ascontiguousarray(W)


def _check_h(h: np.ndarray, dtype: int, d: int) -> np.ndarray:
    want = np.float32 if dtype == F32 else np.uint16
    h = np.ascontiguousarray(h, dtype=want)
    if h.ndim == 1:
        h = h[None, :]
    if h.shape[1] != d:
        raise ValueError("query width %d != d %d" % (h.shape[1], d))
    return h


# --- O1: exact head (Section 3, z = W_out h) --------------------------------

def scores(W: np.ndarray, dtype: int, h: np.ndarray) -> np.ndarray:
    """All exact float64 scores <w_i, h> of one query."""
    W = _check_w(W, dtype)
    h = _check_h(h, dtype, W.shape[1])
    out = np.empty(W.shape[0], dtype=np.float64)
    lib().oracle_scores(_p(W), dtype, W.shape[0], W.shape[1], _p(h), _p(out))
    return out


def topk(W: np.ndarray, dtype: int, h: np.ndarray, k: int):
    """Exact top-k by (score desc, id asc): ids [B,k] int32, logits [B,k] fp32,
    exact scores [B,k] float64."""
    W = _check_w(W, dtype)
    h = _check_h(h, dtype, W.shape[1])
    B = h.shape[0]
    ids = np.empty((B, k), np.int32)
    lg = np.empty((B, k), np.float32)
    sc = np.empty((B, k), np.float64)
    rc = lib().oracle_topk(_p(W), dtype, W.shape[0], W.shape[1], _p(h), B, k, _p(ids), _p(lg), _p(sc))
    if rc != 0:
        raise ValueError("oracle_topk: bad arguments")
    return ids, lg, sc


def pair_scores(W: np.ndarray, dtype: int, h: np.ndarray, qidx: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Exact float64 <w_ids[t], h[qidx[t]]> for a list of pairs (NaN for bad ids)."""
    W = _check_w(W, dtype)
    h = _check_h(h, dtype, W.shape[1])
    qidx = np.ascontiguousarray(qidx, np.int32).ravel()
    ids = np.ascontiguousarray(ids, np.int32).ravel()
    out = np.empty(ids.size, np.float64)
    lib().oracle_pair_scores(_p(W), dtype, W.shape[0], W.shape[1], _p(h), ids.size, _p(qidx), _p(ids),
                             _p(out))
    return out


def pair_abs_scores(W: np.ndarray, dtype: int, h: np.ndarray, qidx: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """sum_j |w_ids[t],j * h[qidx[t]],j| for a list of pairs (NaN for bad ids)."""
    W = _check_w(W, dtype)
    h = _check_h(h, dtype, W.shape[1])
    qidx = np.ascontiguousarray(qidx, np.int32).ravel()
    ids = np.ascontiguousarray(ids, np.int32).ravel()
    out = np.empty(ids.size, np.float64)
    lib().oracle_pair_abs_scores(_p(W), dtype, W.shape[0], W.shape[1], _p(h), ids.size, _p(qidx), _p(ids),
                                 _p(out))
    return out


# --- O4: scatter (Section 3) -------------------------------------------------

def scatter(ids: np.ndarray, logits: np.ndarray, V: int) -> np.ndarray:
    ids = np.ascontiguousarray(ids, np.int32)
    logits = np.ascontiguousarray(logits, np.float32)
    if ids.ndim == 1:
        ids, logits = ids[None], logits[None]
    B, k = ids.shape
    out = np.empty((B, V), np.float32)
    lib().oracle_scatter(_p(ids), _p(logits), B, k, V, _p(out))
    return out


# --- O2 / O3: HNSW ------------------------------------------------------------

@dataclasses.dataclass
class Graph:
    """Flat HNSW graph: the layout of the index file."""
    V: int
    d: int
    dtype: int
    M: int
    M0: int
    efC: int
    seed: int
    maxlevel: int
    entry: int
    levels: np.ndarray     # uint8 [V]
    adj0: np.ndarray       # int32 [V, M0], -1 padded
    upper_off: np.ndarray  # int32 [V]
    upper: np.ndarray      # int32 [nb, M]

    @property
    def nb(self) -> int:
        return int(self.upper.shape[0])


def levels(V: int, M: int, seed: int) -> np.ndarray:
    out = np.empty(V, np.uint8)
    lib().oracle_levels(V, M, seed, _p(out))
    return out


def hnsw_build(W: np.ndarray, dtype: int, M: int, efC: int, seed: int, M0: int | None = None,
               select: str = "heuristic", levels: np.ndarray | None = None) -> Graph:
    """HNSW over the rows of W, inner product similarity (MY18 Alg. 1 + 4).
    levels (uint8 [V]) replaces the seeded level draw when given."""
    W = _check_w(W, dtype)
    V, d = W.shape
    M0 = 2 * M if M0 is None else M0
    mode = 0 if select == "heuristic" else 1
    if levels is None:
        h = lib().oracle_hnsw_build(_p(W), dtype, V, d, M, M0, efC, seed, mode)
    else:
        lv = np.ascontiguousarray(levels, np.uint8)
        if lv.shape != (V,):
            raise ValueError("levels must hold one value per row")
        h = lib().oracle_hnsw_build_levels(_p(W), dtype, V, d, M, M0, efC, _p(lv), mode)
        seed = 0
    if not h:
        raise ValueError("oracle_hnsw_build failed")
    try:
        info = np.zeros(5, np.int64)
        lib().oracle_graph_info(h, _p(info))
        nb = int(info[2])
        lv = np.empty(V, np.uint8)
        adj0 = np.empty((V, M0), np.int32)
        uo = np.empty(V, np.int32)
        up = np.empty((max(nb, 0), M), np.int32)
        lib().oracle_graph_export(h, _p(lv), _p(adj0), _p(uo), _p(up) if nb else None)
    finally:
        lib().oracle_graph_free(h)
    return Graph(V, d, dtype, M, M0, efC, seed, int(info[0]), int(info[1]), lv, adj0, uo, up)


def check_graph(g: Graph) -> str:
    """'' if every invariant holds, else the first violation."""
    msg = C.create_string_buffer(256)
    up = np.ascontiguousarray(g.upper, np.int32)
    rc = lib().oracle_graph_check(g.V, g.M, g.M0, g.maxlevel, g.entry, _p(np.ascontiguousarray(g.levels)),
                                  _p(np.ascontiguousarray(g.adj0, np.int32)),
                                  _p(np.ascontiguousarray(g.upper_off, np.int32)),
                                  _p(up) if up.size else None, g.nb, msg, 256)
    return "" if rc == 0 else (msg.value.decode() or "invalid")


def _trace_buf(B: int, cap: int):
    return (np.full((B, cap), -1, np.int32), cap) if cap > 0 else (None, 0)


def hnsw_search(W: np.ndarray, dtype: int, g: Graph, h: np.ndarray, k: int, ef: int,
                validate: bool = True, trace_cap: int = 0):
    """K-NN-SEARCH (MY18 Alg. 5 over Alg. 2): ids [B,k], logits [B,k],
    stats [B,2] = (n_dist, n_expand), layer-0 start node [B]; with trace_cap
    > 0 also the expansions of each query in order, [B, trace_cap] int32 of
    (layer << 27) | (s << 26) | node (s = 1: first node of its step), -1
    past the last."""
    W = _check_w(W, dtype)
    h = _check_h(h, dtype, W.shape[1])
    if validate:
        err = check_graph(g)
        if err:
            raise ValueError("invalid graph: " + err)
    B = h.shape[0]
    ids = np.empty((B, k), np.int32)
    lg = np.empty((B, k), np.float32)
    st = np.empty((B, 2), np.uint32)
    l0 = np.empty(B, np.int32)
    tr, cap = _trace_buf(B, trace_cap)
    up = np.ascontiguousarray(g.upper, np.int32)
    rc = lib().oracle_hnsw_search(_p(W), dtype, W.shape[0], W.shape[1], g.M, g.M0, g.maxlevel, g.entry,
                                  _p(np.ascontiguousarray(g.levels)), _p(np.ascontiguousarray(g.adj0)),
                                  _p(np.ascontiguousarray(g.upper_off)), _p(up) if up.size else None,
                                  _p(h), B, k, ef, _p(ids), _p(lg), _p(st), _p(l0),
                                  _p(tr) if cap else None, cap)
    if rc != 0:
        raise ValueError("oracle_hnsw_search: bad arguments")
    return (ids, lg, st, l0, tr) if cap else (ids, lg, st, l0)


def hnsw_search_multi(W: np.ndarray, dtype: int, g: Graph, h: np.ndarray, k: int, ef: int,
                      expand_width: int, validate: bool = True, trace_cap: int = 0):
    """K-NN-SEARCH whose layer-0 step expands the expand_width best
    unexpanded beam entries at once: ids [B,k], logits [B,k], stats [B,2]
    (and the expansions, as hnsw_search, with trace_cap > 0)."""
    W = _check_w(W, dtype)
    h = _check_h(h, dtype, W.shape[1])
    if validate:
        err = check_graph(g)
        if err:
            raise ValueError("invalid graph: " + err)
    B = h.shape[0]
    ids = np.empty((B, k), np.int32)
    lg = np.empty((B, k), np.float32)
    st = np.empty((B, 2), np.uint32)
    tr, cap = _trace_buf(B, trace_cap)
    up = np.ascontiguousarray(g.upper, np.int32)
    rc = lib().oracle_hnsw_search_multi(_p(W), dtype, W.shape[0], W.shape[1], g.M, g.M0, g.maxlevel, g.entry,
                                        _p(np.ascontiguousarray(g.levels)), _p(np.ascontiguousarray(g.adj0)),
                                        _p(np.ascontiguousarray(g.upper_off)), _p(up) if up.size else None,
                                        _p(h), B, k, ef, expand_width, _p(ids), _p(lg), _p(st),
                                        _p(tr) if cap else None, cap)
    if rc != 0:
        raise ValueError("oracle_hnsw_search_multi: bad arguments")
    return (ids, lg, st, tr) if cap else (ids, lg, st)


def forced_merge(W: np.ndarray, dtype: int, h: np.ndarray, ids_in: np.ndarray, forced: np.ndarray):
    """Search results ids_in [B,k] joined with the forced ids (Section 3):
    ids [B,k+n], logits [B,k+n] by exact score, each id once, -1/-inf padded."""
    W = _check_w(W, dtype)
    h = _check_h(h, dtype, W.shape[1])
    ids_in = np.ascontiguousarray(np.atleast_2d(ids_in), np.int32)
    forced = np.ascontiguousarray(forced, np.int32).reshape(-1)
    B, k = ids_in.shape
    n = forced.size
    ids = np.empty((B, k + n), np.int32)
    lg = np.empty((B, k + n), np.float32)
    rc = lib().oracle_forced_merge(_p(W), dtype, W.shape[0], W.shape[1], _p(h), B, k, _p(ids_in), n,
                                   _p(forced) if n else None, _p(ids), _p(lg))
    if rc != 0:
        raise ValueError("oracle_forced_merge: bad arguments")
    return ids, lg


def quantize_rows(W: np.ndarray, dtype: int):
    """int8 rows [V,d] and fp32 scales [V] (per-row symmetric, O7)."""
    W = _check_w(W, dtype)
    V, d = W.shape
    q = np.empty((V, d), np.int8)
    sc = np.empty(V, np.float32)
    lib().oracle_quantize_rows(_p(W), dtype, V, d, _p(q), _p(sc))
    return q, sc


def hnsw_search_q(W: np.ndarray, dtype: int, g: Graph, qw: np.ndarray, qscale: np.ndarray, h: np.ndarray, k: int,
                  ef: int, expand_width: int = 1, validate: bool = True, trace_cap: int = 0):
    """K-NN-SEARCH with int8 layer-0 distances and an exact re-rank of the
    final beam: ids [B,k], logits [B,k], stats [B,2]."""
    W = _check_w(W, dtype)
    h = _check_h(h, dtype, W.shape[1])
    if validate:
        err = check_graph(g)
        if err:
            raise ValueError("invalid graph: " + err)
    qw = np.ascontiguousarray(qw, np.int8)
    qscale = np.ascontiguousarray(qscale, np.float32)
    B = h.shape[0]
    ids = np.empty((B, k), np.int32)
    lg = np.empty((B, k), np.float32)
    st = np.empty((B, 2), np.uint32)
    tr, cap = _trace_buf(B, trace_cap)
    up = np.ascontiguousarray(g.upper, np.int32)
    rc = lib().oracle_hnsw_search_q(_p(W), dtype, W.shape[0], W.shape[1], g.M, g.M0, g.maxlevel, g.entry,
                                    _p(np.ascontiguousarray(g.levels)), _p(np.ascontiguousarray(g.adj0)),
                                    _p(np.ascontiguousarray(g.upper_off)), _p(up) if up.size else None, _p(qw),
                                    _p(qscale), _p(h), B, k, ef, expand_width, _p(ids), _p(lg), _p(st),
                                    _p(tr) if cap else None, cap)
    if rc != 0:
        raise ValueError("oracle_hnsw_search_q: bad arguments")
    return (ids, lg, st, tr) if cap else (ids, lg, st)


def knn_graph(W: np.ndarray, dtype: int, K: int, M0: int, seed: int = 0, with_forward: bool = False):
    """Single-layer graph of the batch construction (O8) as a Graph (and the
    forward lists [V, M0] if with_forward)."""
    W = _check_w(W, dtype)
    V, d = W.shape
    adj0 = np.empty((V, M0), np.int32)
    fwd = np.empty((V, M0), np.int32)
    entry = C.c_int32(0)
    rc = lib().oracle_knn_graph(_p(W), dtype, V, d, K, M0, _p(adj0), C.byref(entry), _p(fwd))
    if rc != 0:
        raise ValueError("oracle_knn_graph: bad arguments")
    M = max(2, M0 // 2)
    g = Graph(V, d, dtype, M, M0, K, seed, 0, int(entry.value), np.zeros(V, np.uint8), adj0,
              -np.ones(V, np.int32), np.zeros((0, M), np.int32))
    return (g, fwd) if with_forward else g


def fingerprint(W: np.ndarray, dtype: int) -> int:
    W = _check_w(W, dtype)
    return int(lib().oracle_w_fingerprint(_p(W), dtype, W.shape[0], W.shape[1]))


def save_graph(g: Graph, path: str, W: np.ndarray) -> None:
    fp = fingerprint(W, g.dtype)
    up = np.ascontiguousarray(g.upper, np.int32)
    rc = lib().oracle_file_write(path.encode(), g.dtype, g.V, g.d, g.M, g.M0, g.efC, g.seed, g.maxlevel,
                                 g.entry, g.nb, fp, _p(np.ascontiguousarray(g.levels)),
                                 _p(np.ascontiguousarray(g.adj0)), _p(np.ascontiguousarray(g.upper_off)),
                                 _p(up) if up.size else None)
    if rc != 0:
        raise OSError("oracle_file_write failed: " + path)


def load_graph(path: str) -> tuple[Graph, int]:
    """Reads an index file; returns the graph and the stored W fingerprint."""
    hdr = np.zeros(12, np.int64)
    if lib().oracle_file_header(path.encode(), _p(hdr)) != 0:
        raise ValueError("not an index file: " + path)
    ver, dtype, V, d, M, M0, efC, seed, maxlevel, entry, nb, fp = (int(x) for x in hdr)
    if ver != 1:
        raise ValueError("unsupported index version %d" % ver)
    lv = np.empty(V, np.uint8)
    adj0 = np.empty((V, M0), np.int32)
    uo = np.empty(V, np.int32)
    up = np.empty((nb, M), np.int32)
    rc = lib().oracle_file_body(path.encode(), V, M, M0, nb, _p(lv), _p(adj0), _p(uo), _p(up) if nb else None)
    if rc != 0:
        raise ValueError("corrupt index file (%s): %s" % ("checksum" if rc == -2 else "short read", path))
    return Graph(V, d, dtype, M, M0, efC, seed & 0xFFFFFFFFFFFFFFFF, maxlevel, entry, lv, adj0, uo, up), \
        fp & 0xFFFFFFFFFFFFFFFF


# --- O5: recall (Section 4, "Index Accuracy", generalised from k = 2) --------

def recall(found: np.ndarray, exact: np.ndarray) -> np.ndarray:
    """Per-query |found ∩ exact| / k."""
    found = np.atleast_2d(found)
    exact = np.atleast_2d(exact)
    k = exact.shape[1]
    return np.array([len(set(f[f >= 0].tolist()) & set(e.tolist())) / k for f, e in zip(found, exact)])
