/*
 * oracle.c -- plain CPU reference for the vector-index output head.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
 * the benchmark's CPU-baseline leg may load this library.  The product library
 * never links, loads or calls it, and it shares no source with the product.
 *
 * What it computes (paper: "Accelerating LLM Inference via Vector Index Based
 * Output Embeddings", Section 3, and the HNSW paper it builds on, Malkov &
 * Yashunin, "Efficient and robust approximate nearest neighbor search using
 * HNSW graphs", cited as MY18 below):
 *
 *   O1  exact scores  s_i = <w_i, h>  (Section 3, z = W_out h) in float64 over
 *       the stored values, summed in index order j = 0..d-1, and the exact
 *       top-k ordered by (s desc, id asc); reported logits are fp32(s).
 *   O2  HNSW build over the rows of W_out with inner product as the similarity
 *       (Section 3): insertion following MY18 Algorithm 1, neighbour choice by
 *       the MY18 Algorithm 4 heuristic (no candidate extension, no kept pruned
 *       connections), distance  dist(a, b) = -<a, b>.
 *   O3  HNSW k-NN search following MY18 Algorithms 2 and 5: greedy descent with
 *       ef = 1 through the upper layers, then a beam of size max(ef, k) at
 *       layer 0 (Section 3: ef is the size of the dynamic candidate list).
 *   O4  scatter of the retrieved logits into a full-vocabulary row that is
 *       -inf everywhere else (Section 3, reconstruction of z).
 *   O5  graph invariants (degree caps per layer, no self loops or duplicates,
 *       nested levels, entry point at the top level).
 *
 * Readings where the papers leave a choice (each one is listed in the design
 * notes):
 *   - every comparison of two nodes orders by (dist, id): smaller id is nearer
 *     on equal distance; a full result set is only changed on strict
 *     improvement;
 *   - degree caps: M on layers >= 1 and M0 (normally 2M) on layer 0, which is
 *     what the memory formula |V|(4d + 8M) of Section 3 implies;
 *   - level of node i: floor(-ln(u_i) / ln M), u_i = ((splitmix64(seed ^ i)
 *     >> 11) + 1) * 2^-53 in (0, 1], capped at 16; rows are inserted in id
 *     order and the entry point changes only on a strictly higher level;
 *   - SELECT returns its input unchanged (sorted) when it holds <= m nodes;
 *   - a SEARCH call starts with a fresh visited set that holds its entry
 *     points; n_dist counts every distance evaluation of the query (the entry
 *     point once, then each newly visited node per layer) and n_expand counts
 *     every node whose neighbour list was scanned, over all layers.
 *
 * All floating point is float64.  Nothing here is blocked, fused or reordered
 * beyond what the definitions state; it is meant to be read against the
 * papers, not to be fast.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#define OR_F32 0
#define OR_BF16 1
#define OR_MAX_LEVEL 16

/* ------------------------------------------------------------------------ */
/* stored values                                                             */
/* ------------------------------------------------------------------------ */

/* Exact value of element idx of an fp32 array or of an array of bf16 bits. */
static double stored(const void *base, int dtype, int64_t idx)
{
    if (dtype == OR_F32)
        return (double)((const float *)base)[idx];
    uint32_t bits = (uint32_t)((const uint16_t *)base)[idx] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* <w_row, x> with x already widened to float64; plain sum in index order. */
static double dot_row(const void *W, int dtype, int d, int64_t row, const double *x)
{
    double s = 0.0;
    for (int j = 0; j < d; ++j)
        s += stored(W, dtype, row * (int64_t)d + j) * x[j];
    return s;
}

static void widen(const void *src, int dtype, int d, int64_t row, double *out)
{
    for (int j = 0; j < d; ++j)
        out[j] = stored(src, dtype, row * (int64_t)d + j);
}

/* ------------------------------------------------------------------------ */
/* O1: exact scores and exact top-k (Section 3: z = W_out h, z_i = <w_i, h>)  */
/* ------------------------------------------------------------------------ */

void oracle_scores(const void *W, int dtype, int64_t V, int d, const void *h, double *out)
{
    double *x = malloc(sizeof(double) * (size_t)d);
    widen(h, dtype, d, 0, x);
    for (int64_t i = 0; i < V; ++i)
        out[i] = dot_row(W, dtype, d, i, x);
    free(x);
}

typedef struct {
    double s;
    int32_t id;
} scored;

/* (s desc, id asc) */
static int by_score_desc(const void *a, const void *b)
{
    const scored *x = a, *y = b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->id > y->id) - (x->id < y->id);
}

/* Exact top-k of B queries.  ids [B][k], logits [B][k] (fp32 of the exact
 * score), scores_out [B][k] (optional, the exact float64 scores).
 * Returns 0, or -1 on bad arguments / allocation failure. */
int oracle_topk(const void *W, int dtype, int64_t V, int d, const void *h, int B, int k,
                int32_t *ids, float *logits, double *scores_out)
{
    if (V < 1 || d < 1 || B < 1 || k < 1 || k > V) return -1;
    scored *all = malloc(sizeof(scored) * (size_t)V);
    double *x = malloc(sizeof(double) * (size_t)d);
    if (!all || !x) { free(all); free(x); return -1; }
    for (int b = 0; b < B; ++b) {
        widen(h, dtype, d, b, x);
        for (int64_t i = 0; i < V; ++i) {
            all[i].s = dot_row(W, dtype, d, i, x);
            all[i].id = (int32_t)i;
        }
        qsort(all, (size_t)V, sizeof(scored), by_score_desc);
        for (int j = 0; j < k; ++j) {
            ids[(int64_t)b * k + j] = all[j].id;
            logits[(int64_t)b * k + j] = (float)all[j].s;
            if (scores_out) scores_out[(int64_t)b * k + j] = all[j].s;
        }
    }
    free(all);
    free(x);
    return 0;
}

/* Exact float64 score of a list of (query, id) pairs; used by tolerance checks
 * that need the score of an id that only one side returned. */
void oracle_pair_scores(const void *W, int dtype, int64_t V, int d, const void *h,
                        int64_t n, const int32_t *qidx, const int32_t *ids, double *out)
{
    double *x = malloc(sizeof(double) * (size_t)d);
    for (int64_t t = 0; t < n; ++t) {
        widen(h, dtype, d, qidx[t], x);
        out[t] = (ids[t] >= 0 && ids[t] < V) ? dot_row(W, dtype, d, ids[t], x) : NAN;
    }
    free(x);
}

/* Sum of |w_ij h_j| for a list of (query, id) pairs: the scale of the
 * rounding error of any fp32 evaluation of <w_i, h> (a length-d fp32 sum
 * errs by at most about d * 2^-24 times this, whatever its order). */
void oracle_pair_abs_scores(const void *W, int dtype, int64_t V, int d, const void *h, int64_t n,
                            const int32_t *qidx, const int32_t *ids, double *out)
{
    for (int64_t t = 0; t < n; ++t) {
        double s = 0.0;
        if (ids[t] >= 0 && ids[t] < V)
            for (int j = 0; j < d; ++j)
                s += fabs(stored(W, dtype, (int64_t)ids[t] * d + j) * stored(h, dtype, (int64_t)qidx[t] * d + j));
        out[t] = (ids[t] >= 0 && ids[t] < V) ? s : NAN;
    }
}

/* ------------------------------------------------------------------------ */
/* O4: scatter (Section 3: unretrieved entries are -inf)                     */
/* ------------------------------------------------------------------------ */

void oracle_scatter(const int32_t *ids, const float *logits, int B, int k, int64_t V, float *out)
{
    for (int b = 0; b < B; ++b) {
        float *row = out + (int64_t)b * V;
        for (int64_t i = 0; i < V; ++i)
            row[i] = -INFINITY;
        for (int j = 0; j < k; ++j) {
            int32_t id = ids[(int64_t)b * k + j];
            if (id >= 0 && id < V)
                row[id] = logits[(int64_t)b * k + j];
        }
    }
}

/* ------------------------------------------------------------------------ */
/* level assignment                                                          */
/* ------------------------------------------------------------------------ */

/* SplitMix64 finaliser (Steele, Lea & Flood, "Fast splittable pseudorandom
 * number generators", 2014). */
static uint64_t splitmix64(uint64_t x)
{
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* MY18: level = floor(-ln(unif(0..1)) * mL) with mL = 1 / ln M. */
static int node_level(uint64_t seed, int64_t i, int M)
{
    double u = (double)((splitmix64(seed ^ (uint64_t)i) >> 11) + 1) * (1.0 / 9007199254740992.0);
    double ml = 1.0 / log((double)M);
    int l = (int)floor(-log(u) * ml);
    return l > OR_MAX_LEVEL ? OR_MAX_LEVEL : l;
}

void oracle_levels(int64_t V, int M, uint64_t seed, uint8_t *out)
{
    for (int64_t i = 0; i < V; ++i)
        out[i] = (uint8_t)node_level(seed, i, M);
}

/* ------------------------------------------------------------------------ */
/* graph held by the oracle                                                  */
/* ------------------------------------------------------------------------ */

/* Every neighbour list is a block [count, id_0, ..., id_{cap}] with one spare
 * slot, so "append, then shrink if over the cap" can be written as stated. */
typedef struct {
    int64_t V;
    int M, M0, maxlevel;
    int32_t entry;
    uint8_t *level;  /* [V] */
    int32_t *l0;     /* [V][M0 + 2] */
    int64_t *upoff;  /* [V] offset of the level-1 block in up, -1 if level 0 */
    int32_t *up;     /* blocks of M + 2 */
} ograph;

static int32_t *olist(const ograph *g, int32_t u, int l)
{
    if (l == 0) return g->l0 + (int64_t)u * (g->M0 + 2);
    return g->up + g->upoff[u] + (int64_t)(l - 1) * (g->M + 2);
}

static int cap_of(const ograph *g, int l) { return l == 0 ? g->M0 : g->M; }

static void ograph_free(ograph *g)
{
    if (!g) return;
    free(g->level);
    free(g->l0);
    free(g->upoff);
    free(g->up);
    free(g);
}

static ograph *ograph_alloc(int64_t V, int M, int M0, const uint8_t *levels)
{
    ograph *g = calloc(1, sizeof *g);
    if (!g) return NULL;
    g->V = V;
    g->M = M;
    g->M0 = M0;
    g->level = malloc((size_t)V);
    g->l0 = calloc((size_t)V * (size_t)(M0 + 2), sizeof(int32_t));
    g->upoff = malloc(sizeof(int64_t) * (size_t)V);
    int64_t nblk = 0;
    for (int64_t i = 0; i < V; ++i) nblk += levels[i];
    g->up = calloc((size_t)(nblk > 0 ? nblk : 1) * (size_t)(M + 2), sizeof(int32_t));
    if (!g->level || !g->l0 || !g->upoff || !g->up) { ograph_free(g); return NULL; }
    int64_t off = 0;
    for (int64_t i = 0; i < V; ++i) {
        g->level[i] = levels[i];
        g->upoff[i] = levels[i] ? off : -1;
        off += (int64_t)levels[i] * (M + 2);
    }
    return g;
}

/* ------------------------------------------------------------------------ */
/* O3 building block: SEARCH-LAYER, MY18 Algorithm 2                         */
/* ------------------------------------------------------------------------ */

typedef struct {
    double dist;
    int32_t id;
} cand;

/* (dist, id) lexicographic: is a nearer than b? */
static int nearer(cand a, cand b)
{
    return a.dist < b.dist || (a.dist == b.dist && a.id < b.id);
}

static int by_dist_asc(const void *a, const void *b)
{
    const cand *x = a, *y = b;
    if (nearer(*x, *y)) return -1;
    if (nearer(*y, *x)) return 1;
    return 0;
}

typedef struct {
    const void *W;
    int dtype, d;
    int64_t V;
    uint32_t *seen; /* [V] visit tags */
    uint32_t tag;
    cand *C;        /* candidate set, capacity V */
    cand *R;        /* result set W of MY18, capacity ef + 1 */
    uint64_t n_dist, n_expand;
    /* int8 rows (O7), used only by beam_multi when approx is set */
    const int8_t *qw;
    const float *qscale;
    const int8_t *qh;
    float sh;
    /* optional record of the expansions of one query, in order: entry t is
     * (layer << 27) | (s << 26) | node for t < trace_cap, s = 1 for the first
     * node a step expands */
    int32_t *trace;
    int trace_cap;
} searcher;

/* Counts an expansion of node id on layer lc and records it (first: the
 * first node of its step). */
static void note_expand(searcher *s, int lc, int32_t id, int first)
{
    if (s->trace && s->n_expand < (uint64_t)s->trace_cap)
        s->trace[s->n_expand] = (int32_t)(((uint32_t)lc << 27) | ((uint32_t)(first != 0) << 26) | (uint32_t)id);
    s->n_expand++;
}

static double qdist(searcher *s, const double *q, int32_t id)
{
    s->n_dist++;
    return -dot_row(s->W, s->dtype, s->d, id, q);
}

/* O7: approximate distance from int8 rows: the integer dot product of the
 * quantized row and query (exact), converted to fp32 and multiplied by the
 * row scale, then by the query scale, each product rounded to fp32. */
static double qdist8(searcher *s, int32_t id)
{
    s->n_dist++;
    const int8_t *r = s->qw + (int64_t)id * s->d;
    int64_t acc = 0;
    for (int j = 0; j < s->d; ++j) acc += (int64_t)r[j] * (int64_t)s->qh[j];
    float a = (float)acc;
    a = a * s->qscale[id];
    a = a * s->sh;
    return -(double)a;
}

/* SEARCH-LAYER(q, ep, ef, lc): ep[0..nep) hold entry points with their
 * distances already evaluated.  The nearest ef elements are written to out
 * (unsorted); returns their number. */
static int search_layer(searcher *s, const ograph *g, const double *q, const cand *ep, int nep,
                        int ef, int lc, cand *out)
{
    if (++s->tag == 0) { /* tag wrap: clear and restart */
        memset(s->seen, 0, sizeof(uint32_t) * (size_t)s->V);
        s->tag = 1;
    }
    int nC = 0, nR = 0;
    for (int i = 0; i < nep; ++i) {
        s->seen[ep[i].id] = s->tag;      /* v <- ep */
        s->C[nC++] = ep[i];               /* C <- ep */
        s->R[nR++] = ep[i];               /* W <- ep */
    }
    while (nC > 0) {
        /* c <- extract nearest element from C */
        int ci = 0;
        for (int i = 1; i < nC; ++i)
            if (nearer(s->C[i], s->C[ci])) ci = i;
        cand c = s->C[ci];
        s->C[ci] = s->C[--nC];
        /* f <- get furthest element from W */
        int fi = 0;
        for (int i = 1; i < nR; ++i)
            if (nearer(s->R[fi], s->R[i])) fi = i;
        if (nearer(s->R[fi], c)) break; /* all elements of W are evaluated */
        note_expand(s, lc, c.id, 1);
        int32_t *lst = olist(g, c.id, lc);
        for (int j = 0; j < lst[0]; ++j) {
            int32_t e = lst[1 + j];
            if (s->seen[e] == s->tag) continue;
            s->seen[e] = s->tag;
            cand ce = { qdist(s, q, e), e };
            fi = 0;
            for (int i = 1; i < nR; ++i)
                if (nearer(s->R[fi], s->R[i])) fi = i;
            if (nR < ef || nearer(ce, s->R[fi])) {
                s->C[nC++] = ce;
                s->R[nR++] = ce;
                if (nR > ef) { /* remove furthest element from W */
                    fi = 0;
                    for (int i = 1; i < nR; ++i)
                        if (nearer(s->R[fi], s->R[i])) fi = i;
                    s->R[fi] = s->R[--nR];
                }
            }
        }
    }
    memcpy(out, s->R, sizeof(cand) * (size_t)nR);
    return nR;
}

/* ------------------------------------------------------------------------ */
/* O2: HNSW build, MY18 Algorithm 1 with the Algorithm 4 heuristic           */
/* ------------------------------------------------------------------------ */

/* SELECT-NEIGHBORS(q, C, m).  C is rewritten in place, sorted by (dist to q,
 * id); returns the number kept.  heuristic = 0 keeps the m nearest. */
static int select_neighbors(const void *W, int dtype, int d, cand *C, int n, int m, int heuristic,
                            double *xa)
{
    qsort(C, (size_t)n, sizeof(cand), by_dist_asc);
    if (n <= m) return n;
    if (!heuristic) return m;
    int kept = 0;
    for (int i = 0; i < n && kept < m; ++i) {
        int good = 1;
        widen(W, dtype, d, C[i].id, xa);
        for (int r = 0; r < kept; ++r) {
            double d_er = -dot_row(W, dtype, d, C[r].id, xa); /* dist(e, r) */
            if (!(C[i].dist < d_er)) { good = 0; break; }
        }
        if (good) C[kept++] = C[i];
    }
    return kept;
}

typedef struct {
    ograph *g;
    int efC;
    uint64_t seed;
    int dtype, d;
} obuilt;

/* Builds the graph over the V rows of W with the given node levels.
 * select_mode: 0 = heuristic (MY18 Algorithm 4), 1 = simple (m nearest).
 * Returns an opaque handle or NULL. */
static void *build_with_levels(const void *W, int dtype, int64_t V, int d, int M, int M0, int efC,
                               uint64_t seed, const uint8_t *lv, int select_mode)
{
    ograph *g = ograph_alloc(V, M, M0, lv);
    obuilt *ob = calloc(1, sizeof *ob);
    searcher s = { W, dtype, d, V, calloc((size_t)V, sizeof(uint32_t)), 0,
                   malloc(sizeof(cand) * (size_t)V), malloc(sizeof(cand) * (size_t)(efC + 2)), 0, 0, NULL, NULL, NULL, 0.0f, NULL, 0 };
    int capmax = efC + M0 + M + 4; /* search result, or a selection plus an over-full list */
    cand *Wc = malloc(sizeof(cand) * (size_t)capmax);
    cand *ep = malloc(sizeof(cand) * (size_t)capmax);
    cand *tmp = malloc(sizeof(cand) * (size_t)capmax);
    double *q = malloc(sizeof(double) * (size_t)d);
    double *xa = malloc(sizeof(double) * (size_t)d);
    double *xe = malloc(sizeof(double) * (size_t)d);
    if (!g || !ob || !s.seen || !s.C || !s.R || !Wc || !ep || !tmp || !q || !xa || !xe) {
        ograph_free(g);
        free(ob);
        g = NULL;
        ob = NULL;
        goto done;
    }
    ob->g = g;
    ob->efC = efC;
    ob->seed = seed;
    ob->dtype = dtype;
    ob->d = d;
    g->entry = 0;
    g->maxlevel = g->level[0];
    for (int64_t i = 1; i < V; ++i) {
        int l = g->level[i];
        widen(W, dtype, d, i, q);
        int nep = 1;
        ep[0].id = g->entry;
        ep[0].dist = -dot_row(W, dtype, d, g->entry, q);
        /* greedy descent through the layers above l */
        for (int lc = g->maxlevel; lc > l; --lc) {
            int n = search_layer(&s, g, q, ep, nep, 1, lc, Wc);
            int best = 0;
            for (int t = 1; t < n; ++t)
                if (nearer(Wc[t], Wc[best])) best = t;
            ep[0] = Wc[best];
            nep = 1;
        }
        for (int lc = (l < g->maxlevel ? l : g->maxlevel); lc >= 0; --lc) {
            int n = search_layer(&s, g, q, ep, nep, efC, lc, Wc);
            memcpy(tmp, Wc, sizeof(cand) * (size_t)n);
            int nn = select_neighbors(W, dtype, d, tmp, n, M, select_mode == 0, xa);
            int32_t *mine = olist(g, (int32_t)i, lc);
            mine[0] = nn;
            for (int t = 0; t < nn; ++t) mine[1 + t] = tmp[t].id;
            int cap = cap_of(g, lc);
            for (int t = 0; t < nn; ++t) {
                int32_t e = tmp[t].id;
                int32_t *el = olist(g, e, lc);
                el[1 + el[0]] = (int32_t)i; /* add connection e -> i */
                el[0]++;
                if (el[0] > cap) {          /* shrink connections of e */
                    widen(W, dtype, d, e, xe);
                    int ne = el[0];
                    for (int u = 0; u < ne; ++u) {
                        tmp[nn + u].id = el[1 + u];
                        tmp[nn + u].dist = -dot_row(W, dtype, d, el[1 + u], xe);
                    }
                    int ke = select_neighbors(W, dtype, d, tmp + nn, ne, cap, select_mode == 0, xa);
                    el[0] = ke;
                    for (int u = 0; u < ke; ++u) el[1 + u] = tmp[nn + u].id;
                }
            }
            memcpy(ep, Wc, sizeof(cand) * (size_t)n); /* ep <- W */
            nep = n;
        }
        if (l > g->maxlevel) {
            g->maxlevel = l;
            g->entry = (int32_t)i;
        }
    }
done:
    free(s.seen);
    free(s.C);
    free(s.R);
    free(Wc);
    free(ep);
    free(tmp);
    free(q);
    free(xa);
    free(xe);
    return ob;
}

/* The graph of MY18 Algorithm 1 with levels drawn as stated above. */
void *oracle_hnsw_build(const void *W, int dtype, int64_t V, int d, int M, int M0, int efC,
                        uint64_t seed, int select_mode)
{
    if (V < 1 || d < 1 || M < 2 || M0 < M || efC < 1) return NULL;
    uint8_t *lv = malloc((size_t)V);
    if (!lv) return NULL;
    oracle_levels(V, M, seed, lv);
    void *h = build_with_levels(W, dtype, V, d, M, M0, efC, seed, lv, select_mode);
    free(lv);
    return h;
}

/* The same insertion with caller-chosen levels (levels[i] <= 16), so that a
 * small hand-traced build can make the cases of Algorithm 1 happen. */
void *oracle_hnsw_build_levels(const void *W, int dtype, int64_t V, int d, int M, int M0, int efC,
                               const uint8_t *levels, int select_mode)
{
    if (V < 1 || d < 1 || M < 2 || M0 < M || efC < 1 || !levels) return NULL;
    for (int64_t i = 0; i < V; ++i)
        if (levels[i] > OR_MAX_LEVEL) return NULL;
    return build_with_levels(W, dtype, V, d, M, M0, efC, 0, levels, select_mode);
}

void oracle_graph_free(void *h)
{
    obuilt *ob = h;
    if (!ob) return;
    ograph_free(ob->g);
    free(ob);
}

/* info[0..4] = maxlevel, entry, number of upper blocks, M, M0 */
void oracle_graph_info(const void *h, int64_t *info)
{
    const ograph *g = ((const obuilt *)h)->g;
    int64_t nb = 0;
    for (int64_t i = 0; i < g->V; ++i) nb += g->level[i];
    info[0] = g->maxlevel;
    info[1] = g->entry;
    info[2] = nb;
    info[3] = g->M;
    info[4] = g->M0;
}

/* Flat exchange layout (also the layout of the index file):
 *   levels   uint8 [V]
 *   adj0     int32 [V][M0]   layer-0 lists in stored order, padded with -1
 *   upper_off int32 [V]      first upper block of the node, -1 at level 0
 *   upper    int32 [nb][M]   block upper_off[u] + l - 1 is the level-l list */
void oracle_graph_export(const void *h, uint8_t *levels, int32_t *adj0, int32_t *upper_off,
                         int32_t *upper)
{
    const ograph *g = ((const obuilt *)h)->g;
    int64_t blk = 0;
    for (int64_t u = 0; u < g->V; ++u) {
        levels[u] = g->level[u];
        int32_t *l = olist(g, (int32_t)u, 0);
        for (int j = 0; j < g->M0; ++j) adj0[u * g->M0 + j] = j < l[0] ? l[1 + j] : -1;
        upper_off[u] = g->level[u] ? (int32_t)blk : -1;
        for (int lc = 1; lc <= g->level[u]; ++lc, ++blk) {
            int32_t *ul = olist(g, (int32_t)u, lc);
            for (int j = 0; j < g->M; ++j) upper[blk * g->M + j] = j < ul[0] ? ul[1 + j] : -1;
        }
    }
}

/* Rebuilds the oracle's own graph form from the flat layout.  Lists end at the
 * first -1.  The caller validates the arrays with oracle_graph_check first. */
static ograph *from_flat(int64_t V, int M, int M0, int maxlevel, int32_t entry, const uint8_t *levels,
                         const int32_t *adj0, const int32_t *upper_off, const int32_t *upper)
{
    ograph *g = ograph_alloc(V, M, M0, levels);
    if (!g) return NULL;
    g->maxlevel = maxlevel;
    g->entry = entry;
    for (int64_t u = 0; u < V; ++u) {
        int32_t *l = olist(g, (int32_t)u, 0);
        int n = 0;
        while (n < M0 && adj0[u * M0 + n] >= 0) { l[1 + n] = adj0[u * M0 + n]; ++n; }
        l[0] = n;
        for (int lc = 1; lc <= levels[u]; ++lc) {
            int32_t *ul = olist(g, (int32_t)u, lc);
            const int32_t *src = upper + ((int64_t)upper_off[u] + lc - 1) * M;
            int m = 0;
            while (m < M && src[m] >= 0) { ul[1 + m] = src[m]; ++m; }
            ul[0] = m;
        }
    }
    return g;
}

/* ------------------------------------------------------------------------ */
/* O5: graph invariants                                                      */
/* ------------------------------------------------------------------------ */

static int check_list(const int32_t *lst, int cap, int64_t V, int32_t self, const uint8_t *levels,
                      int lc, char *msg, int msglen)
{
    int n = 0;
    while (n < cap && lst[n] >= 0) ++n;
    for (int j = n; j < cap; ++j)
        if (lst[j] != -1) { snprintf(msg, msglen, "node %d level %d: bad padding", self, lc); return -1; }
    for (int j = 0; j < n; ++j) {
        int32_t e = lst[j];
        if (e >= V) { snprintf(msg, msglen, "node %d level %d: id %d out of range", self, lc, e); return -1; }
        if (e == self) { snprintf(msg, msglen, "node %d level %d: self loop", self, lc); return -1; }
        if (levels[e] < lc) {
            snprintf(msg, msglen, "node %d level %d: neighbour %d has level %d", self, lc, e, levels[e]);
            return -1;
        }
        for (int t = 0; t < j; ++t)
            if (lst[t] == e) { snprintf(msg, msglen, "node %d level %d: duplicate %d", self, lc, e); return -1; }
    }
    return 0;
}

/* Returns 0 if the flat graph satisfies every invariant, else -1 with a
 * message.  nb is the number of upper blocks the arrays hold. */
int oracle_graph_check(int64_t V, int M, int M0, int maxlevel, int32_t entry, const uint8_t *levels,
                       const int32_t *adj0, const int32_t *upper_off, const int32_t *upper, int64_t nb,
                       char *msg, int msglen)
{
    msg[0] = 0;
    if (V < 1 || M < 1 || M0 < 1) { snprintf(msg, msglen, "bad sizes"); return -1; }
    if (entry < 0 || entry >= V) { snprintf(msg, msglen, "entry out of range"); return -1; }
    int top = 0;
    int64_t blocks = 0;
    for (int64_t u = 0; u < V; ++u) {
        if (levels[u] > OR_MAX_LEVEL) { snprintf(msg, msglen, "node %ld: level too high", (long)u); return -1; }
        if (levels[u] > top) top = levels[u];
        if (levels[u] == 0 && upper_off[u] != -1) {
            snprintf(msg, msglen, "node %ld: level 0 with upper lists", (long)u);
            return -1;
        }
        if (levels[u] > 0 && upper_off[u] != blocks) {
            snprintf(msg, msglen, "node %ld: upper block %d, expected %ld", (long)u, upper_off[u], (long)blocks);
            return -1;
        }
        blocks += levels[u];
    }
    if (blocks != nb) { snprintf(msg, msglen, "block count %ld != %ld", (long)blocks, (long)nb); return -1; }
    if (top != maxlevel) { snprintf(msg, msglen, "maxlevel %d != top level %d", maxlevel, top); return -1; }
    if (levels[entry] != maxlevel) { snprintf(msg, msglen, "entry not on the top level"); return -1; }
    for (int64_t u = 0; u < V; ++u) {
        if (check_list(adj0 + u * M0, M0, V, (int32_t)u, levels, 0, msg, msglen)) return -1;
        for (int lc = 1; lc <= levels[u]; ++lc)
            if (check_list(upper + ((int64_t)upper_off[u] + lc - 1) * M, M, V, (int32_t)u, levels, lc, msg,
                           msglen))
                return -1;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* O3: K-NN-SEARCH, MY18 Algorithm 5                                         */
/* ------------------------------------------------------------------------ */

/* B queries h [B][d] on the flat graph.  ids/logits [B][k] (ids -1 and logits
 * -inf past the number found); stats [B][2] = n_dist, n_expand (optional);
 * l0_entry [B] = the node the layer-0 search started from (optional).
 * Returns 0, or -1 on bad arguments. */
int oracle_hnsw_search(const void *W, int dtype, int64_t V, int d, int M, int M0, int maxlevel,
                       int32_t entry, const uint8_t *levels, const int32_t *adj0, const int32_t *upper_off,
                       const int32_t *upper, const void *h, int B, int k, int ef, int32_t *ids,
                       float *logits, uint32_t *stats, int32_t *l0_entry, int32_t *trace, int trace_cap)
{
    if (V < 1 || d < 1 || B < 1 || k < 1 || k > V || ef < 1 || entry < 0 || entry >= V) return -1;
    ograph *g = from_flat(V, M, M0, maxlevel, entry, levels, adj0, upper_off, upper);
    int efe = ef > k ? ef : k; /* ef < k is read as ef = k */
    searcher s = { W, dtype, d, V, calloc((size_t)V, sizeof(uint32_t)), 0, malloc(sizeof(cand) * (size_t)V),
                   malloc(sizeof(cand) * (size_t)(efe + 2)), 0, 0, NULL, NULL, NULL, 0.0f, NULL, 0 };
    cand *out = malloc(sizeof(cand) * (size_t)(efe + 2));
    double *q = malloc(sizeof(double) * (size_t)d);
    int rc = 0;
    if (!g || !s.seen || !s.C || !s.R || !out || !q) { rc = -1; goto done; }
    for (int b = 0; b < B; ++b) {
        s.n_dist = s.n_expand = 0;
        s.trace = trace ? trace + (int64_t)b * trace_cap : NULL;
        s.trace_cap = trace_cap;
        widen(h, dtype, d, b, q);
        cand ep = { qdist(&s, q, entry), entry };
        for (int lc = maxlevel; lc >= 1; --lc) {
            int n = search_layer(&s, g, q, &ep, 1, 1, lc, out);
            int best = 0;
            for (int t = 1; t < n; ++t)
                if (nearer(out[t], out[best])) best = t;
            ep = out[best];
        }
        if (l0_entry) l0_entry[b] = ep.id;
        int n = search_layer(&s, g, q, &ep, 1, efe, 0, out);
        qsort(out, (size_t)n, sizeof(cand), by_dist_asc);
        for (int j = 0; j < k; ++j) {
            ids[(int64_t)b * k + j] = j < n ? out[j].id : -1;
            logits[(int64_t)b * k + j] = j < n ? (float)(-out[j].dist) : -INFINITY;
        }
        if (stats) {
            stats[2 * b] = (uint32_t)s.n_dist;
            stats[2 * b + 1] = (uint32_t)s.n_expand;
        }
    }
done:
    ograph_free(g);
    free(s.seen);
    free(s.C);
    free(s.R);
    free(out);
    free(q);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* O3': layer-0 search expanding several beam entries per step               */
/* ------------------------------------------------------------------------ */

/* A variant of SEARCH-LAYER for wide hardware (it is not in either paper; the
 * library's batched traversal follows it).  The result set R is kept sorted
 * by (dist, id) with an "expanded" flag per entry.  Each step takes the P
 * best unexpanded entries of R and marks them expanded; their lists are
 * scanned in that order, each list in stored order, and every neighbour not
 * visited yet is marked visited and its distance evaluated.  All of them are
 * then inserted into R, which keeps its ef nearest.  The search ends when
 * every entry of R is expanded.  With P = 1 this visits, scores and expands
 * the same nodes as SEARCH-LAYER: an entry dropped from R is worse than all
 * of R and would only have been popped to end the search. */
typedef struct {
    cand c;
    int expanded;
} bentry;

static int by_bentry(const void *a, const void *b)
{
    return by_dist_asc(&((const bentry *)a)->c, &((const bentry *)b)->c);
}

static int beam_multi(searcher *s, const ograph *g, const double *q, cand ep, int ef, int P, int approx,
                      cand *out)
{
    if (++s->tag == 0) {
        memset(s->seen, 0, sizeof(uint32_t) * (size_t)s->V);
        s->tag = 1;
    }
    const int cap = ef + P * g->M0 + 1;
    bentry *R = malloc(sizeof(bentry) * (size_t)cap);
    int *pick = malloc(sizeof(int) * (size_t)P);
    if (!R || !pick) {
        free(R);
        free(pick);
        return -1;
    }
    int nR = 1;
    R[0].c = ep;
    R[0].expanded = 0;
    s->seen[ep.id] = s->tag;
    for (;;) {
        int np = 0;
        for (int i = 0; i < nR && np < P; ++i)
            if (!R[i].expanded) pick[np++] = i;
        if (np == 0) break;
        int n = nR;
        for (int t = 0; t < np; ++t) {
            R[pick[t]].expanded = 1;
            note_expand(s, 0, R[pick[t]].c.id, t == 0);
            const int32_t *lst = olist(g, R[pick[t]].c.id, 0);
            for (int j = 0; j < lst[0]; ++j) {
                const int32_t e = lst[1 + j];
                if (s->seen[e] == s->tag) continue;
                s->seen[e] = s->tag;
                R[n].c.dist = approx ? qdist8(s, e) : qdist(s, q, e);
                R[n].c.id = e;
                R[n].expanded = 0;
                ++n;
            }
        }
        qsort(R, (size_t)n, sizeof(bentry), by_bentry);
        nR = n < ef ? n : ef;
    }
    for (int i = 0; i < nR; ++i) out[i] = R[i].c;
    free(R);
    free(pick);
    return nR;
}

/* K-NN-SEARCH with the layer-0 step above (expand_width = P >= 1); the upper
 * layers are the greedy descent of MY18 Algorithm 5.  Same outputs and
 * return value as oracle_hnsw_search. */
int oracle_hnsw_search_multi(const void *W, int dtype, int64_t V, int d, int M, int M0, int maxlevel,
                             int32_t entry, const uint8_t *levels, const int32_t *adj0, const int32_t *upper_off,
                             const int32_t *upper, const void *h, int B, int k, int ef, int expand_width,
                             int32_t *ids, float *logits, uint32_t *stats, int32_t *trace, int trace_cap)
{
    if (V < 1 || d < 1 || B < 1 || k < 1 || k > V || ef < 1 || entry < 0 || entry >= V || expand_width < 1)
        return -1;
    ograph *g = from_flat(V, M, M0, maxlevel, entry, levels, adj0, upper_off, upper);
    int efe = ef > k ? ef : k;
    searcher s = { W, dtype, d, V, calloc((size_t)V, sizeof(uint32_t)), 0, malloc(sizeof(cand) * (size_t)V),
                   malloc(sizeof(cand) * (size_t)(efe + 2)), 0, 0, NULL, NULL, NULL, 0.0f, NULL, 0 };
    cand *out = malloc(sizeof(cand) * (size_t)(efe + 2));
    double *q = malloc(sizeof(double) * (size_t)d);
    int rc = 0;
    if (!g || !s.seen || !s.C || !s.R || !out || !q) { rc = -1; goto done; }
    for (int b = 0; b < B; ++b) {
        s.n_dist = s.n_expand = 0;
        s.trace = trace ? trace + (int64_t)b * trace_cap : NULL;
        s.trace_cap = trace_cap;
        widen(h, dtype, d, b, q);
        cand ep = { qdist(&s, q, entry), entry };
        for (int lc = maxlevel; lc >= 1; --lc) {
            int n = search_layer(&s, g, q, &ep, 1, 1, lc, out);
            int best = 0;
            for (int t = 1; t < n; ++t)
                if (nearer(out[t], out[best])) best = t;
            ep = out[best];
        }
        int n = beam_multi(&s, g, q, ep, efe, expand_width, 0, out);
        if (n < 0) { rc = -1; goto done; }
        for (int j = 0; j < k; ++j) {
            ids[(int64_t)b * k + j] = j < n ? out[j].id : -1;
            logits[(int64_t)b * k + j] = j < n ? (float)(-out[j].dist) : -INFINITY;
        }
        if (stats) {
            stats[2 * b] = (uint32_t)s.n_dist;
            stats[2 * b + 1] = (uint32_t)s.n_expand;
        }
    }
done:
    ograph_free(g);
    free(s.seen);
    free(s.C);
    free(s.R);
    free(out);
    free(q);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* O8: batch construction of a single-layer graph                            */
/* ------------------------------------------------------------------------ */

/* The library's GPU build (a batch construction in the spirit of CAGRA,
 * which Section 3 considered; GPU indices are the future work of Section 5).
 * Our definition:
 *   1. cand(i): the K nodes nearest to i (dist = -<w_i, w_j>, j != i),
 *      ordered by (dist, id);
 *   2. fwd(i) = SELECT(i, cand(i), M0) with the MY18 Algorithm 4 heuristic;
 *   3. rev(j): every i with j in fwd(i);
 *   4. the list of j is fwd(j) followed by the nodes of rev(j) that are not
 *      in fwd(j), ordered by (dist to j, id), cut at M0 entries (reverse
 *      edges fill the slots the heuristic left free, nearest first);
 *   5. one layer; the entry point is the row of largest squared norm (ties:
 *      smaller id).
 * adj0 [V][M0] (-1 padded) and *entry are written, and fwd(i) to fwd_out
 * [V][M0] (-1 padded) if it is not NULL.  Returns 0 or -1. */
int oracle_knn_graph(const void *W, int dtype, int64_t V, int d, int K, int M0, int32_t *adj0, int32_t *entry,
                     int32_t *fwd_out)
{
    if (V < 2 || d < 1 || K < 1 || K > V - 1 || M0 < 1) return -1;
    cand *all = malloc(sizeof(cand) * (size_t)V);
    cand *c = malloc(sizeof(cand) * (size_t)(V + M0));
    int32_t *fwd = malloc(sizeof(int32_t) * (size_t)V * M0);
    int *nf = calloc((size_t)V, sizeof(int));
    int *nr = calloc((size_t)V, sizeof(int));
    double *q = malloc(sizeof(double) * (size_t)d), *xa = malloc(sizeof(double) * (size_t)d);
    int rc = 0;
    if (!all || !c || !fwd || !nf || !nr || !q || !xa) { rc = -1; goto done; }
    /* 1 + 2 */
    for (int64_t i = 0; i < V; ++i) {
        widen(W, dtype, d, i, q);
        int n = 0;
        for (int64_t j = 0; j < V; ++j)
            if (j != i) {
                all[n].dist = -dot_row(W, dtype, d, j, q);
                all[n].id = (int32_t)j;
                ++n;
            }
        qsort(all, (size_t)n, sizeof(cand), by_dist_asc);
        const int kept = select_neighbors(W, dtype, d, all, K, M0, 1, xa);
        nf[i] = kept;
        for (int t = 0; t < kept; ++t) fwd[i * M0 + t] = all[t].id;
        for (int t = 0; t < kept; ++t) nr[all[t].id]++;
        if (fwd_out)
            for (int t = 0; t < M0; ++t) fwd_out[i * M0 + t] = t < kept ? all[t].id : -1;
    }
    /* 3 + 4: reverse lists (i ascending), then the final lists */
    int64_t *roff = malloc(sizeof(int64_t) * (size_t)(V + 1));
    int32_t *rev = NULL;
    if (!roff) { rc = -1; goto done; }
    roff[0] = 0;
    for (int64_t j = 0; j < V; ++j) roff[j + 1] = roff[j] + nr[j];
    rev = malloc(sizeof(int32_t) * (size_t)(roff[V] > 0 ? roff[V] : 1));
    if (!rev) { free(roff); rc = -1; goto done; }
    memset(nr, 0, sizeof(int) * (size_t)V);
    for (int64_t i = 0; i < V; ++i)
        for (int t = 0; t < nf[i]; ++t) {
            const int32_t j = fwd[i * M0 + t];
            rev[roff[j] + nr[j]++] = (int32_t)i;
        }
    for (int64_t j = 0; j < V; ++j) {
        const int f = nf[j];
        int n = 0;
        for (int t = 0; t < f; ++t) c[n++].id = fwd[j * M0 + t];
        widen(W, dtype, d, j, q);
        for (int t = 0; t < nr[j]; ++t) {
            const int32_t u = rev[roff[j] + t];
            int dup = 0;
            for (int x = 0; x < f && !dup; ++x) dup = fwd[j * M0 + x] == u;
            if (!dup) {
                c[n].id = u;
                c[n].dist = -dot_row(W, dtype, d, u, q);
                ++n;
            }
        }
        qsort(c + f, (size_t)(n - f), sizeof(cand), by_dist_asc);
        for (int t = 0; t < M0; ++t) adj0[j * M0 + t] = t < n ? c[t].id : -1;
    }
    free(roff);
    free(rev);
    /* 5 */
    double best = -1.0;
    for (int64_t i = 0; i < V; ++i) {
        widen(W, dtype, d, i, q);
        double s2 = 0.0;
        for (int j = 0; j < d; ++j) s2 += q[j] * q[j];
        if (s2 > best) {
            best = s2;
            *entry = (int32_t)i;
        }
    }
done:
    free(all);
    free(c);
    free(fwd);
    free(nf);
    free(nr);
    free(q);
    free(xa);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* O7: int8 rows for the traversal, exact re-rank of the beam                */
/* ------------------------------------------------------------------------ */

/* Quantized data types are the paper's stated future work (Section 5).  Our
 * definition, per vector (a row of W_out or a query) of stored values x:
 * scale = fp32(max_j |x_j| / 127) (an fp32 division of the fp32 maximum) and
 * q_j = rint(fp32(x_j / scale)) clamped to [-127, 127] (round half to even);
 * a vector of zeros has scale 0 and q = 0. */
static float quantize_vec(const void *base, int dtype, int d, int64_t row, int8_t *q)
{
    float mx = 0.0f;
    for (int j = 0; j < d; ++j) {
        const float v = fabsf((float)stored(base, dtype, row * d + j));
        if (v > mx) mx = v;
    }
    const float scale = mx / 127.0f;
    for (int j = 0; j < d; ++j) {
        if (scale == 0.0f) {
            q[j] = 0;
            continue;
        }
        float r = rintf((float)stored(base, dtype, row * d + j) / scale);
        if (r > 127.0f) r = 127.0f;
        if (r < -127.0f) r = -127.0f;
        q[j] = (int8_t)r;
    }
    return scale;
}

void oracle_quantize_rows(const void *W, int dtype, int64_t V, int d, int8_t *q, float *scale)
{
    for (int64_t i = 0; i < V; ++i) scale[i] = quantize_vec(W, dtype, d, i, q + i * d);
}

/* K-NN-SEARCH whose layer-0 step (expand_width P, as O3') scores nodes with
 * qdist8 over the int8 rows qw / qscale (from oracle_quantize_rows) and the
 * query quantized the same way; the upper layers use exact distances.  The
 * layer-0 entry point is scored again with qdist8 (one more evaluation).  The
 * final result set is then ranked by exact score and its first k returned
 * with fp32 exact logits (the re-rank is not counted in n_dist). */
int oracle_hnsw_search_q(const void *W, int dtype, int64_t V, int d, int M, int M0, int maxlevel, int32_t entry,
                         const uint8_t *levels, const int32_t *adj0, const int32_t *upper_off, const int32_t *upper,
                         const int8_t *qw, const float *qscale, const void *h, int B, int k, int ef,
                         int expand_width, int32_t *ids, float *logits, uint32_t *stats, int32_t *trace,
                         int trace_cap)
{
    if (V < 1 || d < 1 || B < 1 || k < 1 || k > V || ef < 1 || entry < 0 || entry >= V || expand_width < 1)
        return -1;
    ograph *g = from_flat(V, M, M0, maxlevel, entry, levels, adj0, upper_off, upper);
    int efe = ef > k ? ef : k;
    searcher s = { W, dtype, d, V, calloc((size_t)V, sizeof(uint32_t)), 0, malloc(sizeof(cand) * (size_t)V),
                   malloc(sizeof(cand) * (size_t)(efe + 2)), 0, 0, qw, qscale, NULL, 0.0f, NULL, 0 };
    cand *out = malloc(sizeof(cand) * (size_t)(efe + 2));
    scored *ex = malloc(sizeof(scored) * (size_t)(efe + 2));
    double *q = malloc(sizeof(double) * (size_t)d);
    int8_t *qh = malloc((size_t)d);
    int rc = 0;
    if (!g || !s.seen || !s.C || !s.R || !out || !ex || !q || !qh) { rc = -1; goto done; }
    s.qh = qh;
    for (int b = 0; b < B; ++b) {
        s.n_dist = s.n_expand = 0;
        s.trace = trace ? trace + (int64_t)b * trace_cap : NULL;
        s.trace_cap = trace_cap;
        widen(h, dtype, d, b, q);
        s.sh = quantize_vec(h, dtype, d, b, qh);
        cand ep = { qdist(&s, q, entry), entry };
        for (int lc = maxlevel; lc >= 1; --lc) {
            int n = search_layer(&s, g, q, &ep, 1, 1, lc, out);
            int best = 0;
            for (int t = 1; t < n; ++t)
                if (nearer(out[t], out[best])) best = t;
            ep = out[best];
        }
        ep.dist = qdist8(&s, ep.id);
        int n = beam_multi(&s, g, q, ep, efe, expand_width, 1, out);
        if (n < 0) { rc = -1; goto done; }
        for (int t = 0; t < n; ++t) {
            ex[t].id = out[t].id;
            ex[t].s = dot_row(W, dtype, d, out[t].id, q);
        }
        qsort(ex, (size_t)n, sizeof(scored), by_score_desc);
        for (int j = 0; j < k; ++j) {
            ids[(int64_t)b * k + j] = j < n ? ex[j].id : -1;
            logits[(int64_t)b * k + j] = j < n ? (float)ex[j].s : -INFINITY;
        }
        if (stats) {
            stats[2 * b] = (uint32_t)s.n_dist;
            stats[2 * b + 1] = (uint32_t)s.n_expand;
        }
    }
done:
    ograph_free(g);
    free(s.seen);
    free(s.C);
    free(s.R);
    free(out);
    free(ex);
    free(q);
    free(qh);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* O6: forced-inclusion tokens (Section 3)                                   */
/* ------------------------------------------------------------------------ */

/* Section 3 computes the logits of a fixed set of tokens (special tokens,
 * punctuation, structural words) explicitly, so that they are never missing
 * from the reconstructed logits.  For query b: the union of the search
 * result ids_in[b][0..k) (entries < 0 ignored) and the forced ids, each id
 * once, every logit fp32 of its exact fp64 score, ordered by (score desc,
 * id asc); out_ids / out_logits [B][k + n] are padded with -1 / -inf.
 * Returns 0, or -1 on bad arguments. */
int oracle_forced_merge(const void *W, int dtype, int64_t V, int d, const void *h, int B, int k,
                        const int32_t *ids_in, int n, const int32_t *forced, int32_t *out_ids, float *out_logits)
{
    if (V < 1 || d < 1 || B < 1 || k < 0 || n < 0) return -1;
    for (int i = 0; i < n; ++i)
        if (forced[i] < 0 || forced[i] >= V) return -1;
    const int w = k + n;
    scored *c = malloc(sizeof(scored) * (size_t)(w > 0 ? w : 1));
    double *q = malloc(sizeof(double) * (size_t)d);
    if (!c || !q) {
        free(c);
        free(q);
        return -1;
    }
    for (int b = 0; b < B; ++b) {
        widen(h, dtype, d, b, q);
        int m = 0;
        for (int j = 0; j < k + n; ++j) {
            const int32_t id = j < k ? ids_in[(int64_t)b * k + j] : forced[j - k];
            if (id < 0) continue;
            int dup = 0;
            for (int t = 0; t < m && !dup; ++t) dup = c[t].id == id;
            if (dup) continue;
            c[m].id = id;
            c[m].s = dot_row(W, dtype, d, id, q);
            ++m;
        }
        qsort(c, (size_t)m, sizeof(scored), by_score_desc);
        for (int j = 0; j < w; ++j) {
            out_ids[(int64_t)b * w + j] = j < m ? c[j].id : -1;
            out_logits[(int64_t)b * w + j] = j < m ? (float)c[j].s : -INFINITY;
        }
    }
    free(c);
    free(q);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* index file (the on-disk form of the precomputed index of Section 3)      */
/* ------------------------------------------------------------------------ */

/* Layout, little endian:
 *   0   char[8]  "VIEHNSW1"
 *   8   u32      version (1)
 *   12  u32      dtype (0 fp32, 1 bf16)
 *   16  i64      V
 *   24  i32      d
 *   28  i32      M
 *   32  i32      M0
 *   36  i32      ef_construction
 *   40  u64      seed
 *   48  i32      maxlevel
 *   52  i32      entry
 *   56  i64      number of upper blocks
 *   64  u64      fingerprint of W
 *   72  zero padding to 128
 *   128 levels u8[V], zero padding to a multiple of 8
 *       adj0 i32[V][M0], upper_off i32[V], upper i32[nb][M]
 *       u64 FNV-1a-64 checksum of every preceding byte
 * Fingerprint of W: FNV-1a-64 over V (8 bytes), d (4), dtype (4), then the
 * bytes of rows 0, s, 2s, ... (< V) with s = max(1, V / 1024), then of row
 * V - 1. */

#define FNV_OFF 0xcbf29ce484222325ull
#define FNV_PRIME 0x100000001b3ull

static uint64_t fnv(uint64_t hsh, const void *p, size_t n)
{
    const unsigned char *c = p;
    for (size_t i = 0; i < n; ++i) {
        hsh ^= c[i];
        hsh *= FNV_PRIME;
    }
    return hsh;
}

uint64_t oracle_w_fingerprint(const void *W, int dtype, int64_t V, int d)
{
    uint64_t hsh = FNV_OFF;
    int32_t d32 = d;
    uint32_t dt = (uint32_t)dtype;
    hsh = fnv(hsh, &V, 8);
    hsh = fnv(hsh, &d32, 4);
    hsh = fnv(hsh, &dt, 4);
    size_t rb = (size_t)d * (dtype == OR_F32 ? 4 : 2);
    int64_t step = V / 1024 > 1 ? V / 1024 : 1;
    for (int64_t i = 0; i < V; i += step)
        hsh = fnv(hsh, (const char *)W + (size_t)i * rb, rb);
    hsh = fnv(hsh, (const char *)W + (size_t)(V - 1) * rb, rb);
    return hsh;
}

typedef struct {
    FILE *f;
    uint64_t h;
    int err;
} wstream;

static void put(wstream *w, const void *p, size_t n)
{
    if (w->err) return;
    if (fwrite(p, 1, n, w->f) != n) w->err = 1;
    w->h = fnv(w->h, p, n);
}

/* Writes the flat graph to path.  Returns 0 or -1. */
int oracle_file_write(const char *path, int dtype, int64_t V, int d, int M, int M0, int efC, uint64_t seed,
                      int maxlevel, int32_t entry, int64_t nb, uint64_t fingerprint, const uint8_t *levels,
                      const int32_t *adj0, const int32_t *upper_off, const int32_t *upper)
{
    FILE *f = fopen(path, "wb");
    if (!f) return -1;
    wstream w = { f, FNV_OFF, 0 };
    unsigned char hdr[128];
    memset(hdr, 0, sizeof hdr);
    uint32_t ver = 1, dt = (uint32_t)dtype;
    int32_t d32 = d, M32 = M, M032 = M0, e32 = efC, ml = maxlevel, en = entry;
    memcpy(hdr + 0, "VIEHNSW1", 8);
    memcpy(hdr + 8, &ver, 4);
    memcpy(hdr + 12, &dt, 4);
    memcpy(hdr + 16, &V, 8);
    memcpy(hdr + 24, &d32, 4);
    memcpy(hdr + 28, &M32, 4);
    memcpy(hdr + 32, &M032, 4);
    memcpy(hdr + 36, &e32, 4);
    memcpy(hdr + 40, &seed, 8);
    memcpy(hdr + 48, &ml, 4);
    memcpy(hdr + 52, &en, 4);
    memcpy(hdr + 56, &nb, 8);
    memcpy(hdr + 64, &fingerprint, 8);
    put(&w, hdr, sizeof hdr);
    put(&w, levels, (size_t)V);
    static const unsigned char zeros[8] = { 0 };
    put(&w, zeros, (size_t)((8 - V % 8) % 8));
    put(&w, adj0, sizeof(int32_t) * (size_t)V * (size_t)M0);
    put(&w, upper_off, sizeof(int32_t) * (size_t)V);
    put(&w, upper, sizeof(int32_t) * (size_t)nb * (size_t)M);
    uint64_t cs = w.h;
    if (!w.err && fwrite(&cs, 1, 8, f) != 8) w.err = 1;
    if (fclose(f) != 0) w.err = 1;
    return w.err ? -1 : 0;
}

/* Reads the header: hdr[0..11] = version, dtype, V, d, M, M0, efC, seed,
 * maxlevel, entry, nb, fingerprint.  Returns 0, or -1 if the file cannot be
 * read or the magic is wrong. */
int oracle_file_header(const char *path, int64_t *hdr)
{
    FILE *f = fopen(path, "rb");
    if (!f) return -1;
    unsigned char b[128];
    size_t got = fread(b, 1, sizeof b, f);
    fclose(f);
    if (got != sizeof b || memcmp(b, "VIEHNSW1", 8) != 0) return -1;
    uint32_t u32;
    int32_t i32;
    int64_t i64;
    uint64_t u64;
    memcpy(&u32, b + 8, 4); hdr[0] = u32;
    memcpy(&u32, b + 12, 4); hdr[1] = u32;
    memcpy(&i64, b + 16, 8); hdr[2] = i64;
    memcpy(&i32, b + 24, 4); hdr[3] = i32;
    memcpy(&i32, b + 28, 4); hdr[4] = i32;
    memcpy(&i32, b + 32, 4); hdr[5] = i32;
    memcpy(&i32, b + 36, 4); hdr[6] = i32;
    memcpy(&u64, b + 40, 8); hdr[7] = (int64_t)u64;
    memcpy(&i32, b + 48, 4); hdr[8] = i32;
    memcpy(&i32, b + 52, 4); hdr[9] = i32;
    memcpy(&i64, b + 56, 8); hdr[10] = i64;
    memcpy(&u64, b + 64, 8); hdr[11] = (int64_t)u64;
    return 0;
}

/* Reads the arrays (sized from the header) and verifies the checksum.
 * Returns 0, -1 on a read error, -2 on a checksum mismatch. */
int oracle_file_body(const char *path, int64_t V, int M, int M0, int64_t nb, uint8_t *levels, int32_t *adj0,
                     int32_t *upper_off, int32_t *upper)
{
    FILE *f = fopen(path, "rb");
    if (!f) return -1;
    uint64_t h = FNV_OFF;
    unsigned char hdr[128], pad[8];
    size_t np = (size_t)((8 - V % 8) % 8);
    int ok = fread(hdr, 1, 128, f) == 128;
    h = fnv(h, hdr, 128);
    ok = ok && fread(levels, 1, (size_t)V, f) == (size_t)V;
    if (ok) h = fnv(h, levels, (size_t)V);
    ok = ok && fread(pad, 1, np, f) == np;
    if (ok) h = fnv(h, pad, np);
    size_t n0 = (size_t)V * (size_t)M0;
    ok = ok && fread(adj0, sizeof(int32_t), n0, f) == n0;
    if (ok) h = fnv(h, adj0, n0 * 4);
    ok = ok && fread(upper_off, sizeof(int32_t), (size_t)V, f) == (size_t)V;
    if (ok) h = fnv(h, upper_off, (size_t)V * 4);
    size_t nu = (size_t)nb * (size_t)M;
    ok = ok && fread(upper, sizeof(int32_t), nu, f) == nu;
    if (ok) h = fnv(h, upper, nu * 4);
    uint64_t cs = 0;
    ok = ok && fread(&cs, 1, 8, f) == 8;
    fclose(f);
    if (!ok) return -1;
    return cs == h ? 0 : -2;
}
