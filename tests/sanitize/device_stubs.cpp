// Stand-ins for the device half of libvie (kernels.hip, knn_build.hip) and
// for the few HIP runtime calls the host half makes, so that the host half
// (api.cpp, builder.cpp, index_io.cpp) can be built with the host compiler's
// sanitizers and run without a GPU.  The runtime stand-ins report device 0
// and fail every allocation with hipErrorOutOfMemory, which drives the
// library's out-of-memory paths; every launcher refuses with
// VIE_EUNSUPPORTED.  Test infrastructure only.
#include "index.hpp"

extern "C" {
hipError_t hipGetDevice(int *dev)
{
    *dev = 0;
    return hipSuccess;
}
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipMalloc(void **p, size_t)
{
    *p = nullptr;
    return hipErrorOutOfMemory;
}
hipError_t hipFree(void *) { return hipSuccess; }
hipError_t hipMemcpy(void *, const void *, size_t, hipMemcpyKind) { return hipErrorNoDevice; }
hipError_t hipMemcpyAsync(void *, const void *, size_t, hipMemcpyKind, hipStream_t) { return hipErrorNoDevice; }
hipError_t hipStreamSynchronize(hipStream_t) { return hipErrorNoDevice; }
hipError_t hipGetLastError(void) { return hipSuccess; }
const char *hipGetErrorString(hipError_t e) { return e == hipErrorOutOfMemory ? "out of memory" : "no device"; }
}

namespace vie {
namespace {
vie_status no_device() { return fail(VIE_EUNSUPPORTED, "built without device code"); }
}  // namespace

size_t hnsw_team_workspace_bytes(const HnswLaunch &) { return 0; }
size_t hnsw_share_workspace_bytes(int, int64_t, int, int, bool, int) { return 0; }
vie_status launch_hnsw_search(const HnswLaunch &, hipStream_t) { return no_device(); }
vie_status launch_quantize_rows(const void *, int, int64_t, int, int8_t *, float *, hipStream_t) { return no_device(); }
vie_status launch_forced(const HnswLaunch &, const int32_t *, int, hipStream_t) { return no_device(); }
size_t dense_workspace_bytes(int64_t, int, int, int) { return 0; }
size_t dense_scratch_bytes() { return 0; }
vie_status dense_scratch(void **out)
{
    *out = nullptr;
    return no_device();
}
vie_status launch_dense_topk(const void *, int, int64_t, int, const void *, int, int, int32_t *, float *, void *,
                             hipStream_t)
{
    return no_device();
}
vie_status build_knn_graph_gpu(const void *, int, int64_t, int, int, int, int64_t, hipStream_t, Graph &, DeviceGraph &)
{
    return no_device();
}
vie_status launch_scatter(const int32_t *, const float *, int, int, int64_t, float *, hipStream_t) { return no_device(); }
}  // namespace vie
