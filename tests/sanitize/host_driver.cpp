// Drives the host half of libvie under the host compiler's sanitizers: the
// CPU builder (one and several threads, both neighbour-selection rules),
// the index file (save, load, fingerprint check, corrupt and truncated
// files), export, info, and the argument and state checks of the query
// calls.  Linked with device_stubs.cpp, whose HIP stand-ins fail every
// allocation, so vie_index_to_device must report VIE_ENOMEM and leak
// nothing.  Exits 0 when every check holds.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "vie.h"

#define CHECK(c)                                                                                    \
    do {                                                                                            \
        if (!(c)) {                                                                                 \
            std::fprintf(stderr, "line %d: %s failed (last error: %s)\n", __LINE__, #c, vie_last_error()); \
            return 1;                                                                               \
        }                                                                                           \
    } while (0)

namespace {
uint64_t next(uint64_t &s)
{
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// V x d rows, values uniform in [-1, 1): fp32, or bf16 as the upper half
// of the fp32 bits
std::vector<uint8_t> make_rows(int64_t V, int d, vie_dtype dt, uint64_t seed)
{
    const size_t es = dt == VIE_F32 ? 4 : 2;
    std::vector<uint8_t> w((size_t)V * d * es);
    for (int64_t i = 0; i < V * d; ++i) {
        const float f = (float)((double)(next(seed) >> 11) * 0x1.0p-52 - 1.0);
        uint32_t b;
        std::memcpy(&b, &f, 4);
        if (dt == VIE_F32) std::memcpy(&w[i * 4], &b, 4);
        else {
            const uint16_t h = (uint16_t)(b >> 16);
            std::memcpy(&w[i * 2], &h, 2);
        }
    }
    return w;
}

std::vector<uint8_t> read_file(const std::string &p)
{
    std::vector<uint8_t> b;
    if (FILE *f = std::fopen(p.c_str(), "rb")) {
        uint8_t buf[4096];
        size_t n;
        while ((n = std::fread(buf, 1, sizeof buf, f)) > 0) b.insert(b.end(), buf, buf + n);
        std::fclose(f);
    }
    return b;
}

bool write_file(const std::string &p, const uint8_t *b, size_t n)
{
    FILE *f = std::fopen(p.c_str(), "wb");
    if (!f) return false;
    const bool ok = std::fwrite(b, 1, n, f) == n;
    return std::fclose(f) == 0 && ok;
}

struct Export {
    std::vector<uint8_t> levels;
    std::vector<int32_t> adj0, upper_off, upper;
};

int export_all(const vie_index *ix, Export &e)
{
    vie_index_desc ds;
    CHECK(vie_index_info(ix, &ds) == VIE_OK);
    e.levels.resize(ds.V);
    e.adj0.resize((size_t)ds.V * ds.M0);
    e.upper_off.resize(ds.V);
    e.upper.resize((size_t)ds.n_upper_blocks * ds.M + 1);
    CHECK(vie_index_export(ix, e.levels.data(), e.adj0.data(), e.upper_off.data(), e.upper.data()) == VIE_OK);
    return 0;
}

int one_case(const std::string &dir, vie_dtype dt, int threads, int select)
{
    const int64_t V = 700;
    const int d = 32;
    const std::vector<uint8_t> W = make_rows(V, d, dt, 11 + threads + 2 * select);
    vie_build_params p = {8, 0, 40, threads, 5, select};
    vie_index *ix = nullptr;
    CHECK(vie_index_build(W.data(), dt, V, d, &p, &ix) == VIE_OK && ix);
    vie_index_desc ds;
    CHECK(vie_index_info(ix, &ds) == VIE_OK);
    CHECK(ds.V == V && ds.d == d && ds.M == 8 && ds.M0 == 16 && ds.on_device == 0 && ds.device == -1);
    Export a, b;
    CHECK(export_all(ix, a) == 0);

    const std::string path = dir + "/g.vie";
    CHECK(vie_index_save(ix, path.c_str()) == VIE_OK);
    vie_index *ld = nullptr;
    CHECK(vie_index_load(path.c_str(), W.data(), &ld) == VIE_OK && ld);
    CHECK(export_all(ld, b) == 0);
    CHECK(a.levels == b.levels && a.adj0 == b.adj0 && a.upper_off == b.upper_off && a.upper == b.upper);
    vie_index_free(ld);

    // another W_out: the fingerprint no longer matches
    const std::vector<uint8_t> W2 = make_rows(V, d, dt, 99);
    ld = nullptr;
    CHECK(vie_index_load(path.c_str(), W2.data(), &ld) == VIE_EFORMAT && !ld);

    // a flipped byte in the body, then the file cut short at several points
    std::vector<uint8_t> f = read_file(path);
    CHECK(f.size() > 256);
    const std::string bad = dir + "/bad.vie";
    std::vector<uint8_t> g = f;
    g[g.size() / 2] ^= 0x40;
    CHECK(write_file(bad, g.data(), g.size()));
    CHECK(vie_index_load(bad.c_str(), nullptr, &ld) == VIE_EFORMAT && !ld);
    for (size_t cut : {(size_t)0, (size_t)7, (size_t)64, f.size() / 3, f.size() - 1}) {
        CHECK(write_file(bad, f.data(), cut));
        CHECK(vie_index_load(bad.c_str(), nullptr, &ld) == VIE_EFORMAT && !ld);
    }
    CHECK(vie_index_load((dir + "/missing.vie").c_str(), nullptr, &ld) == VIE_EIO && !ld);

    // the device copy cannot be allocated: VIE_ENOMEM, the index unchanged
    int dummy = 0;
    CHECK(vie_index_to_device(ix, &dummy, nullptr) == VIE_ENOMEM);
    CHECK(vie_index_info(ix, &ds) == VIE_OK && ds.on_device == 0);
    int32_t ids[4];
    float lg[4];
    CHECK(vie_query(ix, &dummy, 1, 4, 8, ids, lg, nullptr, nullptr) == VIE_ESTATE);
    vie_index_free(ix);
    return 0;
}

int argument_checks()
{
    const std::vector<uint8_t> W = make_rows(50, 8, VIE_F32, 3);
    vie_index *ix = nullptr;
    vie_build_params p = {8, 0, 20, 1, 1, 0};
    CHECK(vie_index_build(nullptr, VIE_F32, 50, 8, &p, &ix) == VIE_EINVAL && !ix);
    CHECK(vie_index_build(W.data(), VIE_F32, 0, 8, &p, &ix) == VIE_EINVAL && !ix);
    CHECK(vie_index_build(W.data(), VIE_F32, 50, 0, &p, &ix) == VIE_EINVAL && !ix);
    CHECK(vie_index_build(W.data(), VIE_F32, 50, 8, nullptr, &ix) == VIE_EINVAL && !ix);
    vie_build_params q = p;
    q.M = 1;
    CHECK(vie_index_build(W.data(), VIE_F32, 50, 8, &q, &ix) == VIE_EINVAL && !ix);
    q = p;
    q.M0 = 4;  // below M
    CHECK(vie_index_build(W.data(), VIE_F32, 50, 8, &q, &ix) == VIE_EINVAL && !ix);
    q = p;
    q.ef_construction = 0;
    CHECK(vie_index_build(W.data(), VIE_F32, 50, 8, &q, &ix) == VIE_EINVAL && !ix);
    CHECK(vie_index_build(W.data(), (vie_dtype)9, 50, 8, &p, &ix) == VIE_EINVAL && !ix);
    CHECK(vie_index_save(nullptr, "x") == VIE_EINVAL);
    CHECK(vie_index_load(nullptr, nullptr, &ix) == VIE_EINVAL && !ix);
    CHECK(vie_index_info(nullptr, nullptr) == VIE_EINVAL);
    vie_index_free(nullptr);
    for (int s = 0; s <= 7; ++s) CHECK(vie_status_string((vie_status)s) != nullptr);
    return 0;
}
}  // namespace

int main(int argc, char **argv)
{
    if (argc != 2) {
        std::fprintf(stderr, "usage: host_driver <scratch directory>\n");
        return 2;
    }
    if (argument_checks()) return 1;
    for (vie_dtype dt : {VIE_F32, VIE_BF16})
        for (int threads : {1, 4})
            for (int select : {0, 1})
                if (one_case(argv[1], dt, threads, select)) {
                    std::fprintf(stderr, "case dtype %d threads %d select %d\n", (int)dt, threads, select);
                    return 1;
                }
    std::printf("host driver: all checks passed\n");
    return 0;
}
