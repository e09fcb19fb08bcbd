// CPU construction of the HNSW index over the rows of W_out.
//
// Section 3 of the paper builds the graph offline over the rows of the output
// embedding with inner product as the similarity and ships it with the
// checkpoint; construction time is traded for index quality.  Insertion
// follows Malkov & Yashunin Algorithm 1 (rows inserted in id order; entry
// points of a layer are the result set of the layer above), neighbour choice
// follows their Algorithm 4 heuristic without candidate extension or kept
// pruned connections.  Distances are dist(a, b) = -<a, b> and every tie
// between two nodes is broken by the smaller id.  A single-thread build
// accumulates them in float64 (the products of stored fp32/bf16 values are
// exact there), so it makes the same decisions as a plain float64 reference;
// a multi-thread build, whose result depends on the schedule anyway, uses
// fp32 SIMD dot products (AVX-512 BF16 / FMA when the CPU has them).  The level of node
// i is floor(-ln(u_i) / ln M), u_i = ((splitmix64(seed ^ i) >> 11) + 1) 2^-53.
//
// With several threads, nodes are taken in id order from a shared counter and
// inserted concurrently (per-node locks guard the neighbour lists; a node that
// raises the top level holds the global lock for its whole insertion), so the
// graph depends on the schedule.  With one thread it is deterministic.
#include <immintrin.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <memory>
#include <mutex>
#include <thread>
#include <vector>

#include "index.hpp"

namespace vie {

int node_level(uint64_t seed, int64_t i, int M)
{
    uint64_t z = (seed ^ (uint64_t)i) + 0x9E3779B97F4A7C15ull;  // SplitMix64
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    const double u = (double)((z >> 11) + 1) * (1.0 / 9007199254740992.0);
    const int l = (int)std::floor(-std::log(u) * (1.0 / std::log((double)M)));
    return l > kMaxLevel ? kMaxLevel : l;
}

namespace {

struct Cand {
    double dist;
    int32_t id;
};
inline bool nearer(const Cand &a, const Cand &b) { return a.dist < b.dist || (a.dist == b.dist && a.id < b.id); }
struct NearerFirst {  // std heap comparator: top = nearest
    bool operator()(const Cand &a, const Cand &b) const { return nearer(b, a); }
};
struct FurtherFirst {  // top = furthest
    bool operator()(const Cand &a, const Cand &b) const { return nearer(a, b); }
};

// ---- <stored row, float64 vector> ------------------------------------------

double dot_scalar(const void *W, int dtype, int d, int64_t row, const double *q)
{
    double s = 0.0;
    if (dtype == VIE_F32) {
        const float *w = static_cast<const float *>(W) + row * d;
        for (int j = 0; j < d; ++j) s += (double)w[j] * q[j];
    } else {
        const uint16_t *w = static_cast<const uint16_t *>(W) + row * d;
        for (int j = 0; j < d; ++j) {
            uint32_t b = (uint32_t)w[j] << 16;
            float f;
            std::memcpy(&f, &b, 4);
            s += (double)f * q[j];
        }
    }
    return s;
}

__attribute__((target("avx2,fma"))) double dot_avx2(const void *W, int dtype, int d, int64_t row, const double *q)
{
    __m256d a0 = _mm256_setzero_pd(), a1 = _mm256_setzero_pd();
    int j = 0;
    if (dtype == VIE_F32) {
        const float *w = static_cast<const float *>(W) + row * d;
        for (; j + 8 <= d; j += 8) {
            __m256 f = _mm256_loadu_ps(w + j);
            a0 = _mm256_fmadd_pd(_mm256_cvtps_pd(_mm256_castps256_ps128(f)), _mm256_loadu_pd(q + j), a0);
            a1 = _mm256_fmadd_pd(_mm256_cvtps_pd(_mm256_extractf128_ps(f, 1)), _mm256_loadu_pd(q + j + 4), a1);
        }
        double s[4];
        _mm256_storeu_pd(s, _mm256_add_pd(a0, a1));
        double t = (s[0] + s[1]) + (s[2] + s[3]);
        for (; j < d; ++j) t += (double)w[j] * q[j];
        return t;
    }
    const uint16_t *w = static_cast<const uint16_t *>(W) + row * d;
    for (; j + 8 <= d; j += 8) {
        __m256i x = _mm256_slli_epi32(_mm256_cvtepu16_epi32(_mm_loadu_si128((const __m128i *)(w + j))), 16);
        __m256 f = _mm256_castsi256_ps(x);
        a0 = _mm256_fmadd_pd(_mm256_cvtps_pd(_mm256_castps256_ps128(f)), _mm256_loadu_pd(q + j), a0);
        a1 = _mm256_fmadd_pd(_mm256_cvtps_pd(_mm256_extractf128_ps(f, 1)), _mm256_loadu_pd(q + j + 4), a1);
    }
    double s[4];
    _mm256_storeu_pd(s, _mm256_add_pd(a0, a1));
    double t = (s[0] + s[1]) + (s[2] + s[3]);
    for (; j < d; ++j) {
        uint32_t b = (uint32_t)w[j] << 16;
        float f;
        std::memcpy(&f, &b, 4);
        t += (double)f * q[j];
    }
    return t;
}

void widen_row(const void *W, int dtype, int d, int64_t row, double *out)
{
    if (dtype == VIE_F32) {
        const float *w = static_cast<const float *>(W) + row * d;
        for (int j = 0; j < d; ++j) out[j] = w[j];
    } else {
        const uint16_t *w = static_cast<const uint16_t *>(W) + row * d;
        for (int j = 0; j < d; ++j) {
            uint32_t b = (uint32_t)w[j] << 16;
            float f;
            std::memcpy(&f, &b, 4);
            out[j] = f;
        }
    }
}

// ---- fast <stored row a, stored row b> in fp32 (multi-thread builds) --------

float fdot_scalar(const void *W, int dtype, int d, int64_t a, int64_t b)
{
    float s = 0.0f;
    if (dtype == VIE_F32) {
        const float *x = static_cast<const float *>(W) + a * d, *y = static_cast<const float *>(W) + b * d;
        for (int j = 0; j < d; ++j) s += x[j] * y[j];
    } else {
        const uint16_t *x = static_cast<const uint16_t *>(W) + a * d, *y = static_cast<const uint16_t *>(W) + b * d;
        for (int j = 0; j < d; ++j) {
            uint32_t u = (uint32_t)x[j] << 16, v = (uint32_t)y[j] << 16;
            float fu, fv;
            std::memcpy(&fu, &u, 4);
            std::memcpy(&fv, &v, 4);
            s += fu * fv;
        }
    }
    return s;
}

__attribute__((target("avx512f,avx512bf16"))) float fdot_avx512(const void *W, int dtype, int d, int64_t a,
                                                                 int64_t b)
{
    __m512 acc0 = _mm512_setzero_ps(), acc1 = _mm512_setzero_ps();
    int j = 0;
    float t = 0.0f;
    if (dtype == VIE_F32) {
        const float *x = static_cast<const float *>(W) + a * d, *y = static_cast<const float *>(W) + b * d;
        for (; j + 32 <= d; j += 32) {
            acc0 = _mm512_fmadd_ps(_mm512_loadu_ps(x + j), _mm512_loadu_ps(y + j), acc0);
            acc1 = _mm512_fmadd_ps(_mm512_loadu_ps(x + j + 16), _mm512_loadu_ps(y + j + 16), acc1);
        }
        for (; j < d; ++j) t += x[j] * y[j];
    } else {
        const uint16_t *x = static_cast<const uint16_t *>(W) + a * d, *y = static_cast<const uint16_t *>(W) + b * d;
        for (; j + 64 <= d; j += 64) {
            acc0 = _mm512_dpbf16_ps(acc0, (__m512bh)_mm512_loadu_si512(x + j), (__m512bh)_mm512_loadu_si512(y + j));
            acc1 = _mm512_dpbf16_ps(acc1, (__m512bh)_mm512_loadu_si512(x + j + 32),
                                    (__m512bh)_mm512_loadu_si512(y + j + 32));
        }
        for (; j < d; ++j) {
            uint32_t u = (uint32_t)x[j] << 16, v = (uint32_t)y[j] << 16;
            float fu, fv;
            std::memcpy(&fu, &u, 4);
            std::memcpy(&fv, &v, 4);
            t += fu * fv;
        }
    }
    return _mm512_reduce_add_ps(_mm512_add_ps(acc0, acc1)) + t;
}

// ---- shared build state ------------------------------------------------------

struct Build {
    const void *W;
    int dtype, d;
    int64_t V;
    int M, M0, efC;
    bool heuristic;
    size_t row_bytes;
    bool exact;  // float64 distances (single thread) or fp32 SIMD
    double (*dot)(const void *, int, int, int64_t, const double *);
    float (*fdot)(const void *, int, int, int64_t, int64_t);
    std::vector<uint8_t> level;
    // Lists are blocks [count, id_0 .. id_cap] (one spare slot for the
    // append-then-shrink step).
    std::vector<int32_t> l0;       // [V][M0 + 2]
    std::vector<int64_t> upoff;    // [V] offset of the level-1 block in up
    std::vector<int32_t> up;       // blocks of M + 2
    std::unique_ptr<std::mutex[]> locks;
    std::mutex global;
    std::atomic<int32_t> entry{0};
    std::atomic<int> maxlevel{0};

    int cap(int l) const { return l == 0 ? M0 : M; }
    int32_t *list(int32_t u, int l)
    {
        return l == 0 ? &l0[(size_t)u * (M0 + 2)] : &up[(size_t)upoff[u] + (size_t)(l - 1) * (M + 2)];
    }
    void prefetch_row(int32_t u) const
    {
        const char *p = static_cast<const char *>(W) + (size_t)u * row_bytes;
        for (size_t o = 0; o < row_bytes && o < 512; o += 64) __builtin_prefetch(p + o);
    }
};

// A node whose distances to others are being evaluated: its row, widened
// to float64 once when the build is exact.
struct Probe {
    int32_t row = -1;
    std::vector<double> wide;
};

// Per-thread search state.
struct Worker {
    Build &b;
    std::vector<uint32_t> seen;
    uint32_t tag = 0;
    Probe q, xe;
    std::vector<int32_t> nbuf;
    std::vector<Cand> res, sel, tmp;

    explicit Worker(Build &bb) : b(bb), seen(bb.V, 0), nbuf(std::max(bb.M0, bb.M) + 2)
    {
        if (b.exact) {
            q.wide.resize(b.d);
            xe.wide.resize(b.d);
        }
    }

    void set(Probe &p, int32_t row)
    {
        p.row = row;
        if (b.exact) widen_row(b.W, b.dtype, b.d, row, p.wide.data());
    }

    double dist(const Probe &p, int32_t id)
    {
        return b.exact ? -b.dot(b.W, b.dtype, b.d, id, p.wide.data()) : -(double)b.fdot(b.W, b.dtype, b.d, p.row, id);
    }

    // Snapshot of the level-l list of u under its lock.
    int read_list(int32_t u, int l)
    {
        std::lock_guard<std::mutex> g(b.locks[u]);
        const int32_t *lst = b.list(u, l);
        const int n = lst[0];
        std::memcpy(nbuf.data(), lst + 1, sizeof(int32_t) * n);
        return n;
    }

    // SEARCH-LAYER (Malkov & Yashunin Algorithm 2) with candidate set C as a
    // min-heap and result set W as a max-heap, both ordered by (dist, id).
    // The result (unsorted) is left in res.  `self` (the node being inserted)
    // counts as already visited: with concurrent inserts another thread may
    // have linked it into a list this search reads, and a node must never
    // become its own neighbour.  Sequentially it is never reachable here.
    void search_layer(const std::vector<Cand> &ep, int ef, int lc, int32_t self)
    {
        if (++tag == 0) {
            std::fill(seen.begin(), seen.end(), 0u);
            tag = 1;
        }
        seen[self] = tag;
        std::vector<Cand> C;
        C.reserve(4 * ef + 16);
        res.clear();
        for (const Cand &e : ep) {
            seen[e.id] = tag;
            C.push_back(e);
            std::push_heap(C.begin(), C.end(), NearerFirst());
            res.push_back(e);
            std::push_heap(res.begin(), res.end(), FurtherFirst());
        }
        while (!C.empty()) {
            const Cand c = C.front();
            if (nearer(res.front(), c)) break;
            std::pop_heap(C.begin(), C.end(), NearerFirst());
            C.pop_back();
            const int n = read_list(c.id, lc);
            for (int j = 0; j < n; ++j)
                if (seen[nbuf[j]] != tag) b.prefetch_row(nbuf[j]);
            for (int j = 0; j < n; ++j) {
                const int32_t e = nbuf[j];
                if (seen[e] == tag) continue;
                seen[e] = tag;
                const Cand ce{dist(q, e), e};
                if ((int)res.size() < ef || nearer(ce, res.front())) {
                    C.push_back(ce);
                    std::push_heap(C.begin(), C.end(), NearerFirst());
                    res.push_back(ce);
                    std::push_heap(res.begin(), res.end(), FurtherFirst());
                    if ((int)res.size() > ef) {
                        std::pop_heap(res.begin(), res.end(), FurtherFirst());
                        res.pop_back();
                    }
                }
            }
        }
    }

    // SELECT-NEIGHBORS (Algorithm 4 heuristic, or the m nearest): c is
    // sorted by (dist, id) and cut to the kept nodes.  Keeps e when it is
    // nearer to the base than to every node kept before it.
    void select(std::vector<Cand> &c, int m)
    {
        std::sort(c.begin(), c.end(), nearer);
        if ((int)c.size() <= m) return;
        if (!b.heuristic) {
            c.resize(m);
            return;
        }
        size_t kept = 0;
        for (size_t i = 0; i < c.size() && (int)kept < m; ++i) {
            set(xe, c[i].id);
            bool good = true;
            for (size_t r = 0; r < kept; ++r)
                if (!(c[i].dist < dist(xe, c[r].id))) {
                    good = false;
                    break;
                }
            if (good) c[kept++] = c[i];
        }
        c.resize(kept);
    }

    void insert(int32_t i)
    {
        const int l = b.level[i];
        std::unique_lock<std::mutex> top(b.global);
        const int L = b.maxlevel.load();
        const int32_t ep0 = b.entry.load();
        if (l <= L) top.unlock();  // keep the global lock only when raising the top level
        set(q, i);
        std::vector<Cand> ep{{dist(q, ep0), ep0}};
        for (int lc = L; lc > l; --lc) {
            search_layer(ep, 1, lc, i);
            ep.assign(1, *std::min_element(res.begin(), res.end(), nearer));
        }
        for (int lc = std::min(l, L); lc >= 0; --lc) {
            search_layer(ep, b.efC, lc, i);
            sel = res;
            select(sel, b.M);
            {
                std::lock_guard<std::mutex> g(b.locks[i]);
                int32_t *mine = b.list(i, lc);
                mine[0] = (int32_t)sel.size();
                for (size_t t = 0; t < sel.size(); ++t) mine[1 + t] = sel[t].id;
            }
            const int cap = b.cap(lc);
            for (const Cand &s : sel) {
                const int32_t e = s.id;
                std::lock_guard<std::mutex> g(b.locks[e]);
                int32_t *el = b.list(e, lc);
                // a concurrent insertion of e may have listed i already
                bool present = false;
                for (int u = 0; u < el[0]; ++u) present |= el[1 + u] == i;
                if (present) continue;
                el[1 + el[0]] = i;
                el[0]++;
                if (el[0] > cap) {
                    set(xe, e);
                    tmp.resize(el[0]);
                    for (int u = 0; u < el[0]; ++u) tmp[u] = Cand{dist(xe, el[1 + u]), el[1 + u]};
                    select(tmp, cap);  // distances to e are in tmp; select() reuses xe
                    el[0] = (int32_t)tmp.size();
                    for (size_t u = 0; u < tmp.size(); ++u) el[1 + u] = tmp[u].id;
                }
            }
            ep = res;  // entry points of the next layer: the whole result set
        }
        if (l > L) {
            b.entry.store(i);
            b.maxlevel.store(l);
        }
    }
};

}  // namespace

vie_status build_graph(const void *W, int dtype, int64_t V, int d, const vie_build_params &p, Graph &g)
{
    Build b;
    b.W = W;
    b.dtype = dtype;
    b.d = d;
    b.V = V;
    b.M = p.M;
    b.M0 = p.M0 ? p.M0 : 2 * p.M;
    b.efC = p.ef_construction;
    b.heuristic = p.select == 0;
    b.row_bytes = (size_t)d * elem_bytes(dtype);
    b.dot = __builtin_cpu_supports("avx2") && __builtin_cpu_supports("fma") ? dot_avx2 : dot_scalar;
    b.fdot = __builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bf16") ? fdot_avx512 : fdot_scalar;
    int64_t nb = 0;
    try {
        b.level.resize(V);
        b.upoff.resize(V);
        for (int64_t i = 0; i < V; ++i) {
            b.level[i] = (uint8_t)node_level(p.seed, i, p.M);
            b.upoff[i] = b.level[i] ? nb * (b.M + 2) : -1;
            nb += b.level[i];
        }
        b.l0.assign((size_t)V * (b.M0 + 2), 0);
        b.up.assign((size_t)std::max<int64_t>(nb, 1) * (b.M + 2), 0);
        b.locks.reset(new std::mutex[V]);
    } catch (...) {
        return fail(VIE_ENOMEM, "cannot allocate the build state for V = %lld", (long long)V);
    }
    b.entry = 0;
    b.maxlevel = b.level[0];

    unsigned nt = p.n_threads > 0 ? (unsigned)p.n_threads : std::max(1u, std::thread::hardware_concurrency());
    if ((int64_t)nt > V) nt = (unsigned)std::max<int64_t>(1, V);
    b.exact = nt == 1;
    std::atomic<int64_t> next{1};
    std::atomic<bool> oom{false};
    auto run = [&]() {
        try {
            Worker w(b);
            for (;;) {
                const int64_t i = next.fetch_add(1);
                if (i >= V) break;
                w.insert((int32_t)i);
            }
        } catch (...) {
            oom = true;
            next = V;
        }
    };
    if (nt == 1) {
        run();
    } else {
        std::vector<std::thread> pool;
        for (unsigned t = 0; t < nt; ++t) pool.emplace_back(run);
        for (auto &t : pool) t.join();
    }
    if (oom) return fail(VIE_ENOMEM, "allocation failed during the build");

    g.V = V;
    g.d = d;
    g.dtype = dtype;
    g.M = b.M;
    g.M0 = b.M0;
    g.efC = b.efC;
    g.seed = p.seed;
    g.maxlevel = b.maxlevel;
    g.entry = b.entry;
    g.fingerprint = w_fingerprint(W, dtype, V, d);
    g.levels = b.level;
    g.adj0.assign((size_t)V * b.M0, -1);
    g.upper_off.assign(V, -1);
    g.upper.assign((size_t)nb * b.M, -1);
    int64_t blk = 0;
    for (int64_t u = 0; u < V; ++u) {
        const int32_t *l = b.list((int32_t)u, 0);
        std::memcpy(&g.adj0[(size_t)u * b.M0], l + 1, sizeof(int32_t) * l[0]);
        if (b.level[u]) g.upper_off[u] = (int32_t)blk;
        for (int lc = 1; lc <= b.level[u]; ++lc, ++blk) {
            const int32_t *ul = b.list((int32_t)u, lc);
            std::memcpy(&g.upper[(size_t)blk * b.M], ul + 1, sizeof(int32_t) * ul[0]);
        }
    }
    return VIE_OK;
}

}  // namespace vie
