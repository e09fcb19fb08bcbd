// Internal declarations of libvie: the host-side index, its file form, the
// CPU graph builder and the kernel launchers.  Nothing here is part of the
// public C ABI (include/vie.h).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "vie.h"

namespace vie {

constexpr int kMaxLevel = 16;     // level cap of the level draw
constexpr int kMaxM = 128;        // cap on M (upper layers)
constexpr int kMaxM0 = 256;       // cap on M0 (layer 0)
constexpr int kMaxK = 1024;       // largest k of any query
constexpr int kMaxEf = 8192;      // largest beam of the HNSW kernel (LDS permitting)
constexpr int kMaxD = 8192;       // largest row width
constexpr int kMaxGpuBuildK = 128;  // candidates per node of the GPU batch build
constexpr int kMaxTeam = 256;     // workgroups that may search one query together
constexpr int kMaxShare = 16;     // queries per row-sharing group

inline int elem_bytes(int dtype) { return dtype == VIE_F32 ? 4 : 2; }

// Host form of an HNSW graph; the arrays use the file layout (vie.h).
struct Graph {
    int64_t V = 0;
    int32_t d = 0;
    int32_t dtype = 0;
    int32_t M = 0, M0 = 0, efC = 0;
    uint64_t seed = 0;
    int32_t maxlevel = 0;
    int32_t entry = 0;
    uint64_t fingerprint = 0;
    std::vector<uint8_t> levels;     // [V]
    std::vector<int32_t> adj0;       // [V][M0]
    std::vector<int32_t> upper_off;  // [V]
    std::vector<int32_t> upper;      // [nb][M]
    int64_t nb() const { return M > 0 ? (int64_t)upper.size() / M : 0; }
};

// Device copy of the graph plus the borrowed W_out.
struct DeviceGraph {
    int device = -1;
    const void *W = nullptr;
    int32_t *adj0 = nullptr;
    int32_t *upper_off = nullptr;
    int32_t *upper = nullptr;
    const int8_t *q8 = nullptr;     // borrowed int8 rows [V][d] (vie_index_attach_int8)
    const float *q8scale = nullptr; // borrowed row scales [V]
};

// Thread-local error detail returned by vie_last_error().
void set_error(const char *fmt, ...) __attribute__((format(printf, 1, 2)));
vie_status fail(vie_status s, const char *fmt, ...) __attribute__((format(printf, 2, 3)));

uint64_t w_fingerprint(const void *W, int dtype, int64_t V, int d);
// The same fingerprint from the rows it samples (rows 0, s, 2s, ... below V,
// then row V - 1, with s = max(1, V / 1024)), packed in that order.
uint64_t w_fingerprint_rows(const void *rows, int dtype, int64_t V, int d, int64_t n_rows);
int node_level(uint64_t seed, int64_t i, int M);

vie_status build_graph(const void *W, int dtype, int64_t V, int d, const vie_build_params &p, Graph &g);
vie_status save_graph(const Graph &g, const char *path);
vie_status load_graph(const char *path, Graph &g);
vie_status validate_graph(const Graph &g);

// ---- kernel launchers (kernels.hip) -----------------------------------

struct HnswLaunch {
    const void *W;
    int dtype;
    int64_t V;
    int d;
    const int32_t *adj0;
    int M0;
    const int32_t *upper_off;
    const int32_t *upper;
    int M;
    int maxlevel;
    int32_t entry;
    const void *h;
    int B, k, ef_eff;
    int width;  // beam entries expanded per layer-0 step (1 = the sequential algorithm)
    int ldo;    // row stride of ids / logits (k, or k + forced tokens)
    const int8_t *q8 = nullptr;      // int8 rows for layer-0 scores (nullptr: exact rows)
    const float *q8scale = nullptr;
    int32_t *ids;
    float *logits;
    uint32_t *stats;
    int32_t *trace = nullptr;  // [B][trace_cap] expansion record (nullptr: none)
    int trace_cap = 0;
    int team = 1;              // workgroups per query (1: one)
    void *team_ws = nullptr;   // team exchange workspace (hnsw_team_workspace_bytes)
    int share = 1;             // queries per row-sharing group (1: none)
    void *share_ws = nullptr;  // row-sharing workspace (hnsw_share_workspace_bytes)
};
size_t hnsw_team_workspace_bytes(const HnswLaunch &a);
size_t hnsw_share_workspace_bytes(int B, int64_t V, int d, int dtype, bool q8, int share);
// Launchers return VIE_OK, VIE_EUNSUPPORTED for a shape they cannot serve, or
// VIE_EHIP for a failed launch; the detail goes to set_error().
vie_status launch_hnsw_search(const HnswLaunch &a, hipStream_t s);
size_t hnsw_lds_bytes(int64_t V, int d, int dtype, int ef_eff, int M0, int M);
constexpr int kMaxForced = 1024;  // forced-inclusion tokens per query
vie_status launch_quantize_rows(const void *W, int dtype, int64_t V, int d, int8_t *q, float *scale, hipStream_t s);
vie_status launch_forced(const HnswLaunch &a, const int32_t *forced, int n, hipStream_t s);
size_t hnsw_lds_limit();

size_t dense_workspace_bytes(int64_t V, int d, int B, int k);
// The library's static per-GPU workspace of the dense head (kernels.hip):
// its size, and its device address on the current device.
size_t dense_scratch_bytes();
vie_status dense_scratch(void **out);
vie_status launch_dense_topk(const void *W, int dtype, int64_t V, int d, const void *h, int B, int k,
                             int32_t *ids, float *logits, void *ws, hipStream_t s);

// Batch construction of a single-layer graph on the GPU (knn_build.hip):
// exact K nearest rows by inner product, the Algorithm 4 heuristic with cap
// M0, reverse edges in the free slots, entry = the largest squared norm.
// Fills the host graph and its device copy (dg.W = W_dev).
vie_status build_knn_graph_gpu(const void *W_dev, int dtype, int64_t V, int d, int K, int M0, int64_t chunk_rows,
                               hipStream_t s, Graph &g, DeviceGraph &dg);

vie_status launch_scatter(const int32_t *ids, const float *logits, int B, int k, int64_t V, float *out,
                          hipStream_t s);

}  // namespace vie
