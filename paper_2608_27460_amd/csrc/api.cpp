// C ABI of libvie (include/vie.h): argument checking, error reporting, index
// ownership and dispatch to the CPU builder and the HIP kernels.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "index.hpp"
#include "vie.h"

struct vie_index {
    vie::Graph g;
    vie::DeviceGraph dev;
    // A GPU-built index keeps its layer-0 lists on the device only until a
    // host-side call needs them (save, export, moving the index); the first
    // such call copies them into g.adj0.
    bool adj0_device_only = false;
    std::mutex host_mu;
};

namespace vie {

namespace {
thread_local std::string g_last_error;
}

void set_error(const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
}

vie_status fail(vie_status s, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

namespace {

vie_status hip_fail(hipError_t e, const char *what)
{
    return fail(VIE_EHIP, "HIP error in %s: %s", what, hipGetErrorString(e));
}

vie_status check_dims(int64_t V, int32_t d, int32_t dtype)
{
    if (V < 1 || V >= (int64_t(1) << 31)) return fail(VIE_EINVAL, "V = %lld out of range", (long long)V);
    if (d < 1 || d > kMaxD) return fail(VIE_EINVAL, "d = %d out of range [1, %d]", d, kMaxD);
    if (dtype != VIE_F32 && dtype != VIE_BF16) return fail(VIE_EINVAL, "unknown dtype %d", dtype);
    return VIE_OK;
}

vie_status check_k(int32_t k, int64_t V, int32_t B)
{
    if (B < 1 || B > 65535) return fail(VIE_EINVAL, "B = %d out of range [1, 65535]", B);
    if (k < 1 || k > kMaxK || k > V) return fail(VIE_EINVAL, "k = %d out of range [1, min(V, %d)]", k, kMaxK);
    return VIE_OK;
}

// The host copy of a GPU-built index's layer-0 lists (see vie_index).
vie_status fetch_host_adjacency(vie_index *ix)
{
    std::lock_guard<std::mutex> lock(ix->host_mu);
    if (!ix->adj0_device_only) return VIE_OK;
    Graph &g = ix->g;
    std::vector<int32_t> adj((size_t)g.V * g.M0);
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e == hipSuccess) e = hipSetDevice(ix->dev.device);
    if (e == hipSuccess) e = hipMemcpy(adj.data(), ix->dev.adj0, adj.size() * 4, hipMemcpyDeviceToHost);
    (void)hipSetDevice(cur);
    if (e != hipSuccess) return hip_fail(e, "copying the graph to the host");
    g.adj0.swap(adj);
    ix->adj0_device_only = false;
    return VIE_OK;
}

void free_device(DeviceGraph &d)
{
    if (d.device >= 0) {
        int cur = 0;
        (void)hipGetDevice(&cur);
        (void)hipSetDevice(d.device);
        (void)hipFree(d.adj0);
        (void)hipFree(d.upper_off);
        (void)hipFree(d.upper);
        (void)hipSetDevice(cur);
    }
    d = DeviceGraph();
}

}  // namespace
}  // namespace vie

using namespace vie;

extern "C" {

const char *vie_status_string(vie_status s)
{
    switch (s) {
    case VIE_OK: return "ok";
    case VIE_EINVAL: return "invalid argument";
    case VIE_ENOMEM: return "out of memory";
    case VIE_EHIP: return "HIP runtime error";
    case VIE_EIO: return "I/O error";
    case VIE_EFORMAT: return "bad index file";
    case VIE_ESTATE: return "index not ready on this device";
    case VIE_EUNSUPPORTED: return "unsupported shape";
    }
    return "unknown status";
}

const char *vie_last_error(void) { return g_last_error.c_str(); }

int32_t vie_version(void) { return 10000; }

vie_status vie_index_build(const void *W_host, vie_dtype dtype, int64_t V, int32_t d, const vie_build_params *p,
                           vie_index **out)
{
    g_last_error.clear();
    if (!W_host || !p || !out) return fail(VIE_EINVAL, "NULL argument");
    *out = nullptr;
    if (vie_status s = check_dims(V, d, dtype)) return s;
    const int M0 = p->M0 ? p->M0 : 2 * p->M;
    if (p->M < 2 || p->M > kMaxM) return fail(VIE_EINVAL, "M = %d out of range [2, %d]", p->M, kMaxM);
    if (M0 < p->M || M0 > kMaxM0) return fail(VIE_EINVAL, "M0 = %d out of range [M, %d]", M0, kMaxM0);
    if (p->ef_construction < 1) return fail(VIE_EINVAL, "ef_construction = %d < 1", p->ef_construction);
    if (p->n_threads < 0) return fail(VIE_EINVAL, "n_threads = %d < 0", p->n_threads);
    if (p->select != 0 && p->select != 1) return fail(VIE_EINVAL, "select = %d is neither 0 nor 1", p->select);
    vie_index *ix = new (std::nothrow) vie_index;
    if (!ix) return fail(VIE_ENOMEM, "cannot allocate the index");
    if (vie_status s = build_graph(W_host, dtype, V, d, *p, ix->g)) {
        delete ix;
        return s;
    }
    *out = ix;
    return VIE_OK;
}

vie_status vie_index_build_gpu(const void *W_dev, vie_dtype dtype, int64_t V, int32_t d,
                               const vie_gpu_build_params *p, void *hip_stream, vie_index **out)
{
    g_last_error.clear();
    if (!W_dev || !p || !out) return fail(VIE_EINVAL, "NULL argument");
    *out = nullptr;
    if (vie_status s = check_dims(V, d, dtype)) return s;
    if (V < 2) return fail(VIE_EINVAL, "V = %lld: the batch graph needs two rows", (long long)V);
    if (p->K < 1 || p->K > kMaxGpuBuildK || p->K > V - 1)
        return fail(VIE_EINVAL, "K = %d out of range [1, min(V - 1, %d)]", p->K, kMaxGpuBuildK);
    if (p->M0 < 2 || p->M0 > kMaxM0) return fail(VIE_EINVAL, "M0 = %d out of range [2, %d]", p->M0, kMaxM0);
    if (p->chunk_rows < 0) return fail(VIE_EINVAL, "chunk_rows = %lld < 0", (long long)p->chunk_rows);
    const int row_bytes = d * elem_bytes(dtype);
    if (row_bytes % 16 || (uintptr_t)W_dev % 16)
        return fail(VIE_EUNSUPPORTED, "GPU build needs 16-byte aligned rows (d = %d of dtype %d)", d, (int)dtype);
    vie_index *ix = new (std::nothrow) vie_index;
    if (!ix) return fail(VIE_ENOMEM, "cannot allocate the index");
    if (vie_status s = build_knn_graph_gpu(W_dev, dtype, V, d, p->K, p->M0, p->chunk_rows,
                                           static_cast<hipStream_t>(hip_stream), ix->g, ix->dev)) {
        delete ix;
        return s;
    }
    ix->adj0_device_only = true;
    *out = ix;
    return VIE_OK;
}

vie_status vie_index_save(const vie_index *ix, const char *path)
{
    g_last_error.clear();
    if (!ix || !path) return fail(VIE_EINVAL, "NULL argument");
    if (vie_status s = fetch_host_adjacency(const_cast<vie_index *>(ix))) return s;
    return save_graph(ix->g, path);
}

vie_status vie_index_load(const char *path, const void *W_host, vie_index **out)
{
    g_last_error.clear();
    if (!path || !out) return fail(VIE_EINVAL, "NULL argument");
    *out = nullptr;
    vie_index *ix = new (std::nothrow) vie_index;
    if (!ix) return fail(VIE_ENOMEM, "cannot allocate the index");
    if (vie_status s = load_graph(path, ix->g)) {
        delete ix;
        return s;
    }
    if (W_host && w_fingerprint(W_host, ix->g.dtype, ix->g.V, ix->g.d) != ix->g.fingerprint) {
        delete ix;
        return fail(VIE_EFORMAT, "%s was built for another W_out (fingerprint mismatch)", path);
    }
    *out = ix;
    return VIE_OK;
}

vie_status vie_index_to_device(vie_index *ix, const void *W_dev, void *hip_stream)
{
    g_last_error.clear();
    if (!ix || !W_dev) return fail(VIE_EINVAL, "NULL argument");
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (vie_status s = fetch_host_adjacency(ix)) return s;
    free_device(ix->dev);
    const Graph &g = ix->g;
    DeviceGraph d;
    d.device = dev;
    const size_t b0 = g.adj0.size() * 4, b1 = g.upper_off.size() * 4, b2 = std::max<size_t>(g.upper.size() * 4, 4);
    if (hipMalloc(&d.adj0, b0) != hipSuccess || hipMalloc(&d.upper_off, b1) != hipSuccess ||
        hipMalloc(&d.upper, b2) != hipSuccess) {
        free_device(d);
        (void)hipGetLastError();
        return fail(VIE_ENOMEM, "cannot allocate %zu bytes of device graph", b0 + b1 + b2);
    }
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    e = hipMemcpyAsync(d.adj0, g.adj0.data(), b0, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(d.upper_off, g.upper_off.data(), b1, hipMemcpyHostToDevice, s);
    if (e == hipSuccess && !g.upper.empty())
        e = hipMemcpyAsync(d.upper, g.upper.data(), g.upper.size() * 4, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        free_device(d);
        return hip_fail(e, "graph upload");
    }
    d.W = W_dev;
    ix->dev = d;
    return VIE_OK;
}

vie_status vie_index_info(const vie_index *ix, vie_index_desc *out)
{
    g_last_error.clear();
    if (!ix || !out) return fail(VIE_EINVAL, "NULL argument");
    const Graph &g = ix->g;
    out->V = g.V;
    out->d = g.d;
    out->dtype = g.dtype;
    out->M = g.M;
    out->M0 = g.M0;
    out->ef_construction = g.efC;
    out->maxlevel = g.maxlevel;
    out->entry = g.entry;
    out->n_upper_blocks = g.nb();
    out->seed = g.seed;
    out->w_fingerprint = g.fingerprint;
    out->on_device = ix->dev.device >= 0;
    out->device = ix->dev.device;
    return VIE_OK;
}

vie_status vie_index_export(const vie_index *ix, uint8_t *levels, int32_t *adj0, int32_t *upper_off,
                            int32_t *upper)
{
    g_last_error.clear();
    if (!ix) return fail(VIE_EINVAL, "NULL index");
    if (vie_status s = fetch_host_adjacency(const_cast<vie_index *>(ix))) return s;
    const Graph &g = ix->g;
    if (levels) std::memcpy(levels, g.levels.data(), g.levels.size());
    if (adj0) std::memcpy(adj0, g.adj0.data(), g.adj0.size() * 4);
    if (upper_off) std::memcpy(upper_off, g.upper_off.data(), g.upper_off.size() * 4);
    if (upper && !g.upper.empty()) std::memcpy(upper, g.upper.data(), g.upper.size() * 4);
    return VIE_OK;
}

void vie_index_free(vie_index *ix)
{
    if (!ix) return;
    free_device(ix->dev);
    delete ix;
}

namespace {
vie_status query_impl(const vie_index *ix, const void *h_dev, int32_t B, int32_t k, int32_t ef,
                      const vie_search_params *params, const int32_t *forced_dev, int32_t n_forced,
                      int32_t *ids_dev, float *logits_dev, uint32_t *stats_dev, void *hip_stream);

vie_status check_params(const vie_search_params *params)
{
    if (!params) return VIE_OK;
    if (params->expand_width < 1 || params->expand_width > 128)
        return fail(VIE_EINVAL, "expand_width = %d outside 1..128", params->expand_width);
    if (params->int8_rows != 0 && params->int8_rows != 1)
        return fail(VIE_EINVAL, "int8_rows = %d is neither 0 nor 1", params->int8_rows);
    if (params->trace_dev && params->trace_cap < 1)
        return fail(VIE_EINVAL, "trace_cap = %d < 1 with a trace buffer", params->trace_cap);
    if (params->team < 0 || params->team > kMaxTeam || (params->team & (params->team - 1)))
        return fail(VIE_EINVAL, "team = %d is neither 0 nor a power of two up to %d", params->team, kMaxTeam);
    if (params->share < 0 || params->share > kMaxShare || (params->share & (params->share - 1)))
        return fail(VIE_EINVAL, "share = %d is neither 0 nor a power of two up to %d", params->share, kMaxShare);
    if (params->team > 1 && params->share > 1) return fail(VIE_EINVAL, "team and share cannot be combined");
    const bool ws = params->team > 1 || params->share > 1;
    if (ws && !params->workspace_dev) return fail(VIE_EINVAL, "a team or row-sharing search needs workspace_dev");
    if (ws && (uintptr_t)params->workspace_dev % 256) return fail(VIE_EINVAL, "workspace_dev is not 256-byte aligned");
    return VIE_OK;
}

int team_of(const vie_search_params *params) { return params && params->team > 1 ? params->team : 1; }
int share_of(const vie_search_params *params) { return params && params->share > 1 ? params->share : 1; }
}  // namespace

vie_status vie_query_workspace(const vie_index *ix, int32_t B, int32_t k, int32_t ef,
                               const vie_search_params *params, size_t *bytes)
{
    g_last_error.clear();
    if (!ix || !params || !bytes) return fail(VIE_EINVAL, "NULL argument");
    if (params->expand_width < 1 || params->expand_width > 128)
        return fail(VIE_EINVAL, "expand_width = %d outside 1..128", params->expand_width);
    if (params->team < 0 || params->team > kMaxTeam || (params->team & (params->team - 1)))
        return fail(VIE_EINVAL, "team = %d is neither 0 nor a power of two up to %d", params->team, kMaxTeam);
    if (params->share < 0 || params->share > kMaxShare || (params->share & (params->share - 1)))
        return fail(VIE_EINVAL, "share = %d is neither 0 nor a power of two up to %d", params->share, kMaxShare);
    if (vie_status s = check_k(k, ix->g.V, B)) return s;
    if (ef < 1) return fail(VIE_EINVAL, "ef = %d < 1", ef);
    HnswLaunch a{};
    a.B = B;
    a.M0 = ix->g.M0;
    a.width = params->expand_width;
    a.ef_eff = ef > k ? ef : k;
    a.team = team_of(params);
    *bytes = hnsw_team_workspace_bytes(a) + hnsw_share_workspace_bytes(B, ix->g.V, ix->g.d, ix->g.dtype,
                                                                        params->int8_rows != 0, share_of(params));
    return VIE_OK;
}

vie_status vie_quantize_rows(const void *W_dev, vie_dtype dtype, int64_t V, int32_t d, int8_t *q_dev,
                             float *scale_dev, void *hip_stream)
{
    g_last_error.clear();
    if (!W_dev || !q_dev || !scale_dev) return fail(VIE_EINVAL, "NULL argument");
    if (dtype != VIE_F32 && dtype != VIE_BF16) return fail(VIE_EINVAL, "dtype %d", (int)dtype);
    if (V < 1 || V >= ((int64_t)1 << 31)) return fail(VIE_EINVAL, "V = %lld", (long long)V);
    if (d < 1 || d > kMaxD) return fail(VIE_EINVAL, "d = %d", d);
    return launch_quantize_rows(W_dev, dtype, V, d, q_dev, scale_dev, static_cast<hipStream_t>(hip_stream));
}

vie_status vie_index_attach_int8(vie_index *ix, const int8_t *q_dev, const float *scale_dev)
{
    g_last_error.clear();
    if (!ix) return fail(VIE_EINVAL, "NULL argument");
    if ((q_dev == nullptr) != (scale_dev == nullptr)) return fail(VIE_EINVAL, "NULL argument");
    if (ix->dev.device < 0) return fail(VIE_ESTATE, "index is not on a device (call vie_index_to_device)");
    if (q_dev && ix->g.d % 16 != 0) return fail(VIE_EUNSUPPORTED, "int8 rows need d divisible by 16");
    ix->dev.q8 = q_dev;
    ix->dev.q8scale = scale_dev;
    return VIE_OK;
}

vie_status vie_query(const vie_index *ix, const void *h_dev, int32_t B, int32_t k, int32_t ef, int32_t *ids_dev,
                     float *logits_dev, uint32_t *stats_dev, void *hip_stream)
{
    g_last_error.clear();
    return query_impl(ix, h_dev, B, k, ef, nullptr, nullptr, 0, ids_dev, logits_dev, stats_dev, hip_stream);
}

vie_status vie_query_ex(const vie_index *ix, const void *h_dev, int32_t B, int32_t k, int32_t ef,
                        const vie_search_params *params, int32_t *ids_dev, float *logits_dev, uint32_t *stats_dev,
                        void *hip_stream)
{
    g_last_error.clear();
    if (!params) return fail(VIE_EINVAL, "NULL argument");
    if (vie_status r = check_params(params)) return r;
    return query_impl(ix, h_dev, B, k, ef, params, nullptr, 0, ids_dev, logits_dev, stats_dev, hip_stream);
}

vie_status vie_query_forced(const vie_index *ix, const void *h_dev, int32_t B, int32_t k, int32_t ef,
                            const vie_search_params *params, const int32_t *forced_dev, int32_t n_forced,
                            int32_t *ids_dev, float *logits_dev, uint32_t *stats_dev, void *hip_stream)
{
    g_last_error.clear();
    if (vie_status r = check_params(params)) return r;
    if (n_forced < 0 || n_forced > kMaxForced)
        return fail(VIE_EINVAL, "n_forced = %d outside 0..%d", n_forced, kMaxForced);
    if (n_forced > 0 && !forced_dev) return fail(VIE_EINVAL, "NULL argument");
    return query_impl(ix, h_dev, B, k, ef, params, forced_dev, n_forced, ids_dev, logits_dev, stats_dev, hip_stream);
}

namespace {
// params NULL: one expansion per step on the stored rows, no trace.
vie_status query_impl(const vie_index *ix, const void *h_dev, int32_t B, int32_t k, int32_t ef,
                      const vie_search_params *params, const int32_t *forced_dev, int32_t n_forced,
                      int32_t *ids_dev, float *logits_dev, uint32_t *stats_dev, void *hip_stream)
{
    if (!ix || !h_dev || !ids_dev || !logits_dev) return fail(VIE_EINVAL, "NULL argument");
    const Graph &g = ix->g;
    const int width = params ? params->expand_width : 1;
    const bool int8_rows = params && params->int8_rows != 0;
    int32_t *trace = params ? params->trace_dev : nullptr;
    if (trace && g.V >= (int64_t(1) << 26))
        return fail(VIE_EUNSUPPORTED, "an expansion trace needs V < 2^26 (V = %lld)", (long long)g.V);
    if (vie_status s = check_k(k, g.V, B)) return s;
    if (ef < 1) return fail(VIE_EINVAL, "ef = %d < 1", ef);
    const int ef_eff = ef > k ? ef : k;
    if (ef_eff > kMaxEf) return fail(VIE_EUNSUPPORTED, "max(ef, k) = %d above %d", ef_eff, kMaxEf);
    if (ix->dev.device < 0) return fail(VIE_ESTATE, "index is not on a device (call vie_index_to_device)");
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (ix->dev.device != dev)
        return fail(VIE_ESTATE, "index lives on device %d, current device is %d", ix->dev.device, dev);
    HnswLaunch a;
    a.W = ix->dev.W;
    a.dtype = g.dtype;
    a.V = g.V;
    a.d = g.d;
    a.adj0 = ix->dev.adj0;
    a.M0 = g.M0;
    a.upper_off = ix->dev.upper_off;
    a.upper = ix->dev.upper;
    a.M = g.M;
    a.maxlevel = g.maxlevel;
    a.entry = g.entry;
    a.h = h_dev;
    a.B = B;
    a.k = k;
    a.ef_eff = ef_eff;
    a.ids = ids_dev;
    a.logits = logits_dev;
    a.stats = stats_dev;
    a.width = width;
    a.ldo = k + n_forced;
    a.trace = trace;
    a.trace_cap = trace ? params->trace_cap : 0;
    a.team = team_of(params);
    if (a.team > 1) {
        const size_t need = hnsw_team_workspace_bytes(a);
        if (params->workspace_bytes < need)
            return fail(VIE_EINVAL, "workspace holds %zu bytes, a team of %d needs %zu", params->workspace_bytes,
                        a.team, need);
        a.team_ws = params->workspace_dev;
    }
    if (int8_rows) {
        if (!ix->dev.q8) return fail(VIE_ESTATE, "no int8 rows attached (call vie_index_attach_int8)");
        a.q8 = ix->dev.q8;
        a.q8scale = ix->dev.q8scale;
    }
    a.share = share_of(params);
    if (a.share > 1) {
        const size_t need = hnsw_share_workspace_bytes(a.B, a.V, a.d, a.dtype, a.q8 != nullptr, a.share);
        if (params->workspace_bytes < need)
            return fail(VIE_EINVAL, "workspace holds %zu bytes, row sharing in groups of %d needs %zu",
                        params->workspace_bytes, a.share, need);
        a.share_ws = params->workspace_dev;
    }
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    if (vie_status r = launch_hnsw_search(a, st)) return r;
    return n_forced > 0 ? launch_forced(a, forced_dev, n_forced, st) : VIE_OK;
}
}  // namespace

vie_status vie_dense_topk_workspace(int64_t V, int32_t d, int32_t B, int32_t k, size_t *bytes)
{
    g_last_error.clear();
    if (!bytes) return fail(VIE_EINVAL, "NULL argument");
    if (vie_status s = check_dims(V, d, VIE_F32)) return s;
    if (vie_status s = check_k(k, V, B)) return s;
    *bytes = dense_workspace_bytes(V, d, B, k);
    return VIE_OK;
}

vie_status vie_dense_topk(const void *W_dev, vie_dtype dtype, int64_t V, int32_t d, const void *h_dev, int32_t B,
                          int32_t k, int32_t *ids_dev, float *logits_dev, void *ws, size_t ws_bytes,
                          void *hip_stream)
{
    g_last_error.clear();
    if (!W_dev || !h_dev || !ids_dev || !logits_dev || !ws) return fail(VIE_EINVAL, "NULL argument");
    if (vie_status s = check_dims(V, d, dtype)) return s;
    if (vie_status s = check_k(k, V, B)) return s;
    if ((uintptr_t)ws % 256) return fail(VIE_EINVAL, "workspace is not 256-byte aligned");
    const size_t need = dense_workspace_bytes(V, d, B, k);
    if (ws_bytes < need) return fail(VIE_EINVAL, "workspace holds %zu bytes, needs %zu", ws_bytes, need);
    return launch_dense_topk(W_dev, dtype, V, d, h_dev, B, k, ids_dev, logits_dev, ws,
                             static_cast<hipStream_t>(hip_stream));
}

vie_status vie_dense_topk_noalloc(const void *W_dev, vie_dtype dtype, int64_t V, int32_t d, const void *h_dev,
                                  int32_t B, int32_t k, int32_t *ids_dev, float *logits_dev, void *hip_stream)
{
    g_last_error.clear();
    if (!W_dev || !h_dev || !ids_dev || !logits_dev) return fail(VIE_EINVAL, "NULL argument");
    if (vie_status s = check_dims(V, d, dtype)) return s;
    if (vie_status s = check_k(k, V, B)) return s;
    const size_t need = dense_workspace_bytes(V, d, B, k);
    if (need > dense_scratch_bytes())
        return fail(VIE_EUNSUPPORTED, "V = %lld, B = %d needs %zu bytes of workspace; the static one holds %zu",
                    (long long)V, B, need, dense_scratch_bytes());
    void *ws = nullptr;
    if (vie_status s = dense_scratch(&ws)) return s;
    return launch_dense_topk(W_dev, dtype, V, d, h_dev, B, k, ids_dev, logits_dev, ws,
                             static_cast<hipStream_t>(hip_stream));
}

vie_status vie_scatter(const int32_t *ids_dev, const float *logits_dev, int32_t B, int32_t k, int64_t V,
                       float *out_dev, void *hip_stream)
{
    g_last_error.clear();
    if (!ids_dev || !logits_dev || !out_dev) return fail(VIE_EINVAL, "NULL argument");
    if (V < 1 || V >= (int64_t(1) << 31)) return fail(VIE_EINVAL, "V = %lld out of range", (long long)V);
    if (B < 1 || B > 65535) return fail(VIE_EINVAL, "B = %d out of range [1, 65535]", B);
    if (k < 1 || k > kMaxK) return fail(VIE_EINVAL, "k = %d out of range [1, %d]", k, kMaxK);
    return launch_scatter(ids_dev, logits_dev, B, k, V, out_dev, static_cast<hipStream_t>(hip_stream));
}

}  // extern "C"
