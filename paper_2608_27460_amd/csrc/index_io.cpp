// Index file form, W fingerprint and structural validation of a graph.
//
// The paper precomputes the index offline and ships it with the checkpoint
// (Section 3); this file is that artefact.  The layout is specified in vie.h.
#include <cerrno>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "index.hpp"

namespace vie {

namespace {

constexpr uint64_t kFnvOffset = 0xcbf29ce484222325ull;
constexpr uint64_t kFnvPrime = 0x100000001b3ull;

uint64_t fnv1a(uint64_t h, const void *p, size_t n)
{
    const unsigned char *c = static_cast<const unsigned char *>(p);
    for (size_t i = 0; i < n; ++i) {
        h ^= c[i];
        h *= kFnvPrime;
    }
    return h;
}

struct Header {
    char magic[8];
    uint32_t version;
    uint32_t dtype;
    int64_t V;
    int32_t d, M, M0, efC;
    uint64_t seed;
    int32_t maxlevel, entry;
    int64_t nb;
    uint64_t fingerprint;
    unsigned char pad[56];
};
static_assert(sizeof(Header) == 128, "index header is 128 bytes");

size_t level_pad(int64_t V) { return (size_t)((8 - V % 8) % 8); }

}  // namespace

uint64_t w_fingerprint(const void *W, int dtype, int64_t V, int d)
{
    uint64_t h = kFnvOffset;
    int32_t d32 = d;
    uint32_t dt = (uint32_t)dtype;
    h = fnv1a(h, &V, 8);
    h = fnv1a(h, &d32, 4);
    h = fnv1a(h, &dt, 4);
    const size_t row = (size_t)d * elem_bytes(dtype);
    const char *base = static_cast<const char *>(W);
    const int64_t step = V / 1024 > 1 ? V / 1024 : 1;
    for (int64_t i = 0; i < V; i += step) h = fnv1a(h, base + (size_t)i * row, row);
    return fnv1a(h, base + (size_t)(V - 1) * row, row);
}

uint64_t w_fingerprint_rows(const void *rows, int dtype, int64_t V, int d, int64_t n_rows)
{
    uint64_t h = kFnvOffset;
    int32_t d32 = d;
    uint32_t dt = (uint32_t)dtype;
    h = fnv1a(h, &V, 8);
    h = fnv1a(h, &d32, 4);
    h = fnv1a(h, &dt, 4);
    const size_t row = (size_t)d * elem_bytes(dtype);
    for (int64_t t = 0; t < n_rows; ++t) h = fnv1a(h, static_cast<const char *>(rows) + (size_t)t * row, row);
    return h;
}

vie_status validate_graph(const Graph &g)
{
    if (g.V < 1 || g.V >= (int64_t(1) << 31)) return fail(VIE_EFORMAT, "V = %lld out of range", (long long)g.V);
    if (g.d < 1 || g.d > kMaxD) return fail(VIE_EFORMAT, "d = %d out of range", g.d);
    if (g.dtype != VIE_F32 && g.dtype != VIE_BF16) return fail(VIE_EFORMAT, "unknown dtype %d", g.dtype);
    if (g.M < 2 || g.M > kMaxM || g.M0 < g.M || g.M0 > kMaxM0)
        return fail(VIE_EFORMAT, "degree caps M = %d, M0 = %d out of range", g.M, g.M0);
    if ((int64_t)g.levels.size() != g.V || (int64_t)g.adj0.size() != g.V * g.M0 ||
        (int64_t)g.upper_off.size() != g.V || g.upper.size() % g.M != 0)
        return fail(VIE_EFORMAT, "array sizes do not match V, M, M0");
    if (g.entry < 0 || g.entry >= g.V) return fail(VIE_EFORMAT, "entry %d out of range", g.entry);
    int top = 0;
    int64_t blocks = 0;
    for (int64_t u = 0; u < g.V; ++u) {
        const int lv = g.levels[u];
        if (lv > kMaxLevel) return fail(VIE_EFORMAT, "node %lld: level %d above %d", (long long)u, lv, kMaxLevel);
        top = lv > top ? lv : top;
        if (lv == 0 ? g.upper_off[u] != -1 : g.upper_off[u] != blocks)
            return fail(VIE_EFORMAT, "node %lld: upper block offset %d", (long long)u, g.upper_off[u]);
        blocks += lv;
    }
    if (blocks != g.nb()) return fail(VIE_EFORMAT, "%lld upper blocks, levels need %lld", (long long)g.nb(),
                                      (long long)blocks);
    if (top != g.maxlevel) return fail(VIE_EFORMAT, "maxlevel %d but the top level is %d", g.maxlevel, top);
    if (g.levels[g.entry] != g.maxlevel) return fail(VIE_EFORMAT, "entry %d is not on the top level", g.entry);
    std::vector<uint32_t> mark(g.V, 0);
    uint32_t stamp = 0;
    auto check = [&](const int32_t *lst, int cap, int64_t u, int lc) -> vie_status {
        ++stamp;
        int n = 0;
        while (n < cap && lst[n] >= 0) ++n;
        for (int j = n; j < cap; ++j)
            if (lst[j] != -1) return fail(VIE_EFORMAT, "node %lld level %d: bad padding", (long long)u, lc);
        for (int j = 0; j < n; ++j) {
            const int32_t e = lst[j];
            if (e >= g.V) return fail(VIE_EFORMAT, "node %lld level %d: id %d out of range", (long long)u, lc, e);
            if (e == u) return fail(VIE_EFORMAT, "node %lld level %d: self loop", (long long)u, lc);
            if (g.levels[e] < lc)
                return fail(VIE_EFORMAT, "node %lld level %d: neighbour %d only reaches level %d", (long long)u,
                            lc, e, g.levels[e]);
            if (mark[e] == stamp) return fail(VIE_EFORMAT, "node %lld level %d: duplicate %d", (long long)u, lc, e);
            mark[e] = stamp;
        }
        return VIE_OK;
    };
    for (int64_t u = 0; u < g.V; ++u) {
        if (vie_status s = check(&g.adj0[u * g.M0], g.M0, u, 0)) return s;
        for (int lc = 1; lc <= g.levels[u]; ++lc)
            if (vie_status s = check(&g.upper[((int64_t)g.upper_off[u] + lc - 1) * g.M], g.M, u, lc)) return s;
    }
    return VIE_OK;
}

vie_status save_graph(const Graph &g, const char *path)
{
    Header h;
    std::memset(&h, 0, sizeof h);
    std::memcpy(h.magic, "VIEHNSW1", 8);
    h.version = 1;
    h.dtype = (uint32_t)g.dtype;
    h.V = g.V;
    h.d = g.d;
    h.M = g.M;
    h.M0 = g.M0;
    h.efC = g.efC;
    h.seed = g.seed;
    h.maxlevel = g.maxlevel;
    h.entry = g.entry;
    h.nb = g.nb();
    h.fingerprint = g.fingerprint;
    FILE *f = std::fopen(path, "wb");
    if (!f) return fail(VIE_EIO, "cannot open %s for writing: %s", path, std::strerror(errno));
    uint64_t cs = kFnvOffset;
    bool ok = true;
    auto put = [&](const void *p, size_t n) {
        if (!ok || n == 0) return;
        ok = std::fwrite(p, 1, n, f) == n;
        cs = fnv1a(cs, p, n);
    };
    const unsigned char zeros[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    put(&h, sizeof h);
    put(g.levels.data(), g.levels.size());
    put(zeros, level_pad(g.V));
    put(g.adj0.data(), g.adj0.size() * 4);
    put(g.upper_off.data(), g.upper_off.size() * 4);
    put(g.upper.data(), g.upper.size() * 4);
    if (ok) ok = std::fwrite(&cs, 1, 8, f) == 8;
    if (std::fclose(f) != 0) ok = false;
    if (!ok) return fail(VIE_EIO, "write to %s failed", path);
    return VIE_OK;
}

vie_status load_graph(const char *path, Graph &g)
{
    FILE *f = std::fopen(path, "rb");
    if (!f) return fail(VIE_EIO, "cannot open %s: %s", path, std::strerror(errno));
    Header h;
    uint64_t cs = kFnvOffset;
    bool ok = std::fread(&h, 1, sizeof h, f) == sizeof h;
    auto get = [&](void *p, size_t n) {
        if (!ok || n == 0) return;
        ok = std::fread(p, 1, n, f) == n;
        if (ok) cs = fnv1a(cs, p, n);
    };
    if (!ok) {
        std::fclose(f);
        return fail(VIE_EFORMAT, "%s: shorter than the header", path);
    }
    cs = fnv1a(cs, &h, sizeof h);
    if (std::memcmp(h.magic, "VIEHNSW1", 8) != 0) {
        std::fclose(f);
        return fail(VIE_EFORMAT, "%s: not an index file", path);
    }
    if (h.version != 1) {
        std::fclose(f);
        return fail(VIE_EFORMAT, "%s: version %u not supported", path, h.version);
    }
    if (h.V < 1 || h.V >= (int64_t(1) << 31) || h.M < 2 || h.M > kMaxM || h.M0 < h.M || h.M0 > kMaxM0 ||
        h.nb < 0 || h.nb > h.V * kMaxLevel || h.d < 1 || h.d > kMaxD) {
        std::fclose(f);
        return fail(VIE_EFORMAT, "%s: header sizes out of range", path);
    }
    g.V = h.V;
    g.d = h.d;
    g.dtype = (int32_t)h.dtype;
    g.M = h.M;
    g.M0 = h.M0;
    g.efC = h.efC;
    g.seed = h.seed;
    g.maxlevel = h.maxlevel;
    g.entry = h.entry;
    g.fingerprint = h.fingerprint;
    try {
        g.levels.resize(h.V);
        g.adj0.resize((size_t)h.V * h.M0);
        g.upper_off.resize(h.V);
        g.upper.resize((size_t)h.nb * h.M);
    } catch (...) {
        std::fclose(f);
        return fail(VIE_ENOMEM, "%s: cannot allocate the graph", path);
    }
    unsigned char pad[8];
    get(g.levels.data(), g.levels.size());
    get(pad, level_pad(h.V));
    get(g.adj0.data(), g.adj0.size() * 4);
    get(g.upper_off.data(), g.upper_off.size() * 4);
    get(g.upper.data(), g.upper.size() * 4);
    uint64_t stored = 0;
    if (ok) ok = std::fread(&stored, 1, 8, f) == 8;
    std::fclose(f);
    if (!ok) return fail(VIE_EFORMAT, "%s: truncated", path);
    if (stored != cs) return fail(VIE_EFORMAT, "%s: checksum mismatch", path);
    return validate_graph(g);
}

}  // namespace vie
