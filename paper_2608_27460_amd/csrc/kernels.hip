// gfx950 (CDNA4) kernels of the vector-index output head.
//
//   scatter_kernel       Section 3: full-vocabulary logits, -inf except the
//                        retrieved ids.
//   dense_stream_kernel, exact head z = W_out h fused with top-k (Section 3;
//   dense_slab_kernel,   the dense baseline of Section 4.1): slab logits on
//   dense_mfma_kernel,   the vector ALUs (one to a few queries) or the
//   dense_merge_kernel   matrix cores (batches), then the top k from the
//                        slabs' candidate lists.
//   hnsw_kernel          HNSW k-NN search (Sections 2-3; Malkov & Yashunin
//                        Algorithms 2 and 5), one workgroup per query.
//   hnsw_multi_kernel    the same search expanding up to 128 beam entries
//                        per layer-0 step, optionally on int8 rows, in a
//                        team of up to 256 workgroups per query that divide
//                        each step's row scoring, or with the rows a launch's
//                        queries fetch shared within groups of queries
//                        (Section 5's open problems: sequential traversal,
//                        quantization).
//   team_clear_kernel,   set-up of a team search (published counts zeroed)
//   share_*_kernel       and of row sharing (workspace cleared once, epoch,
//                        queries copied).
//   quantize_kernel      per-row scaled int8 copy of W_out (and of a
//                        launch's queries for row sharing).
//   forced_kernel        search result joined with explicitly scored ids
//                        (Section 3's forced-inclusion tokens).
//
// Ordering: candidates are the 64-bit keys of keys.hpp (larger logit first,
// smaller id first on equal logits).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <mutex>

#include "index.hpp"
#include "keys.hpp"

namespace vie {

namespace {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// dot products of stored rows with a query held in LDS
// ---------------------------------------------------------------------------

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int VEC> struct Vec;
template <> struct Vec<16> { typedef u32x4 T; };
template <> struct Vec<8> { typedef u32x2 T; };
template <> struct Vec<4> { typedef uint32_t T; };
template <> struct Vec<2> { typedef uint16_t T; };

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }

// Accumulator of a dot product.  A product of two bf16 values is exact in
// fp32 and the sums are fp32; a product of two fp32 values is exact in fp64
// and the sums are fp64, rounded to fp32 once at the end, so fp32 rows give
// the exact score to within the fp32 rounding of the result.
template <bool BF16> struct AccOf { typedef float T; };
template <> struct AccOf<false> { typedef double T; };

__device__ __forceinline__ float dot_word(uint32_t w, uint32_t h, float acc)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w), __builtin_bit_cast(bf16x2_t, h), acc,
                                           false);
}
__device__ __forceinline__ double dot_word(uint32_t w, uint32_t h, double acc)
{
    return fma((double)__uint_as_float(w), (double)__uint_as_float(h), acc);
}

template <int VEC, bool BF16>
__device__ __forceinline__ typename AccOf<BF16>::T dot_vec(typename Vec<VEC>::T w, typename Vec<VEC>::T h,
                                                           typename AccOf<BF16>::T acc)
{
    if constexpr (VEC == 16) {
        acc = dot_word(w.x, h.x, acc);
        acc = dot_word(w.y, h.y, acc);
        acc = dot_word(w.z, h.z, acc);
        acc = dot_word(w.w, h.w, acc);
    } else if constexpr (VEC == 8) {
        acc = dot_word(w.x, h.x, acc);
        acc = dot_word(w.y, h.y, acc);
    } else if constexpr (VEC == 4) {
        acc = dot_word(w, h, acc);
    } else {  // one bf16 (rows of an odd number of bf16 values)
        static_assert(BF16, "2-byte chunks hold bf16 values");
        acc = fmaf(__uint_as_float((uint32_t)w << 16), __uint_as_float((uint32_t)h << 16), acc);
    }
    return acc;
}

// One DPP move within each row of 16 lanes (CTRL: a quad_perm, row mirror
// or half-row mirror pattern; every source lane lies in the same row).
template <int CTRL> __device__ __forceinline__ float dpp_move(float v)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
template <int CTRL> __device__ __forceinline__ int dpp_move(int v)
{
    return __builtin_amdgcn_mov_dpp(v, CTRL, 0xF, 0xF, true);
}
template <int CTRL> __device__ __forceinline__ double dpp_move(double v)
{
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)u, CTRL, 0xF, 0xF, true);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, true);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// The value held by lane (lane ^ s), s = 1, 2, 4, 8, 16 or 32, without an
// LDS round trip: DPP within rows of 16 lanes (quad permutes for 1 and 2,
// row shifts up and down for 4, a row rotation by 8 for 8) and the permlane
// swaps across rows (16, 32).  Every lane of the wave must be active.  s is
// a compile-time constant wherever these are called (unrolled loops), so the
// switch folds away.
__device__ __forceinline__ uint32_t xor_lane(uint32_t v, int s)
{
    const int lane = threadIdx.x & (kWave - 1);
    switch (s) {
    case 1: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, true);   // quad_perm [1, 0, 3, 2]
    case 2: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, true);   // quad_perm [2, 3, 0, 1]
    case 4: {
        const uint32_t up = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x104, 0xF, 0xF, true);  // row_shl:4
        const uint32_t dn = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x114, 0xF, 0xF, true);  // row_shr:4
        return (lane & 4) ? dn : up;
    }
    case 8: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, true);  // row_ror:8
    case 16: {
        const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return (lane & 16) ? r[0] : r[1];
    }
    case 32: {
        const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        return (lane & 32) ? r[0] : r[1];
    }
    default: return (uint32_t)__shfl_xor((int)v, s, kWave);
    }
}
__device__ __forceinline__ uint64_t xor_lane(uint64_t v, int s)
{
    return ((uint64_t)xor_lane((uint32_t)(v >> 32), s) << 32) | xor_lane((uint32_t)v, s);
}

// Inclusive prefix sum over the 64 lanes of a wave by DPP: shifts right by
// 1, 2, 4 and 8 within each row of 16 lanes (lanes shifted in read zero),
// then lane 15 of each row added into rows 1 and 3 and lane 31 into rows 2
// and 3.  Every lane of the wave must be active.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x)
{
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, true);   // row_shr:1
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, true);   // row_shr:2
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, true);   // row_shr:4
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, true);   // row_shr:8
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false);  // row_bcast:15
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false);  // row_bcast:31
    return x;
}

// Minimum and maximum over the 64 lanes of a wave (strides written out, so
// that xor_lane's switch folds away).  Every lane of the wave must be active.
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v)
{
    v = min(v, xor_lane(v, 32));
    v = min(v, xor_lane(v, 16));
    v = min(v, xor_lane(v, 8));
    v = min(v, xor_lane(v, 4));
    v = min(v, xor_lane(v, 2));
    return min(v, xor_lane(v, 1));
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v)
{
    v = max(v, xor_lane(v, 32));
    v = max(v, xor_lane(v, 16));
    v = max(v, xor_lane(v, 8));
    v = max(v, xor_lane(v, 4));
    v = max(v, xor_lane(v, 2));
    return max(v, xor_lane(v, 1));
}

// xor_lane for 32- and 64-bit values of any type (float, int, double).
template <typename T> __device__ __forceinline__ T xor_lane_as(T v, int s)
{
    if constexpr (sizeof(T) == 8)
        return __builtin_bit_cast(T, xor_lane(__builtin_bit_cast(uint64_t, v), s));
    else
        return __builtin_bit_cast(T, xor_lane(__builtin_bit_cast(uint32_t, v), s));
}

// Sum over the G lanes of an aligned group (G = 16, 32 or 64), the same
// bits in every lane of the group: within a row of 16 lanes by DPP (lane ^ 1
// and lane ^ 2 by quad permutes, then the half-row and row mirrors, each
// pairing a lane with one of the other half), across rows by permlane swaps
// (the partner lanes of a 32- or 64-lane group lie inside the group).
// Each step adds two values in either order, so every lane rounds alike.
template <int G, typename T> __device__ __forceinline__ T group_sum(T v)
{
    static_assert(G == 16 || G == 32 || G == 64, "groups of 16, 32 or 64 lanes");
    v += dpp_move<0xB1>(v);   // quad_perm [1, 0, 3, 2]
    v += dpp_move<0x4E>(v);   // quad_perm [2, 3, 0, 1]
    v += dpp_move<0x141>(v);  // row_half_mirror
    v += dpp_move<0x140>(v);  // row_mirror
    if constexpr (G >= 32) v += xor_lane_as(v, 16);
    if constexpr (G >= 64) v += xor_lane_as(v, 32);
    return v;
}

// ---------------------------------------------------------------------------
// scatter
// ---------------------------------------------------------------------------

constexpr int kScatterTile = 4096;
constexpr int kScatterThreads = 256;

__global__ __launch_bounds__(kScatterThreads) void scatter_kernel(const int32_t *__restrict__ ids,
                                                                  const float *__restrict__ logits, int k,
                                                                  int64_t V, float *__restrict__ out)
{
    __shared__ float tile[kScatterTile];
    const int b = blockIdx.y;
    const int64_t t0 = (int64_t)blockIdx.x * kScatterTile;
    const int n = (int)min<int64_t>(kScatterTile, V - t0);
    for (int i = threadIdx.x; i < kScatterTile; i += kScatterThreads) tile[i] = -__builtin_inff();
    __syncthreads();
    for (int j = threadIdx.x; j < k; j += kScatterThreads) {
        const int64_t id = ids[(int64_t)b * k + j];
        if (id >= t0 && id < t0 + n) tile[id - t0] = logits[(int64_t)b * k + j];
    }
    __syncthreads();
    float *o = out + (int64_t)b * V + t0;
    // scalar head up to 16-byte alignment, float4 body, scalar tail
    const int head = (int)(((16 - ((uintptr_t)o & 15)) & 15) / 4);
    const int h = head < n ? head : n;
    if (threadIdx.x < h) o[threadIdx.x] = tile[threadIdx.x];
    const int body = (n - h) / 4;
    f32x4 *o4 = reinterpret_cast<f32x4 *>(o + h);
    for (int i = threadIdx.x; i < body; i += kScatterThreads) {
        const int e = h + 4 * i;
        const f32x4 v = {tile[e], tile[e + 1], tile[e + 2], tile[e + 3]};
        __builtin_nontemporal_store(v, o4 + i);
    }
    for (int e = h + 4 * body + threadIdx.x; e < n; e += kScatterThreads) o[e] = tile[e];
}

// ---------------------------------------------------------------------------
// dense head: GEMV + top-k
// ---------------------------------------------------------------------------
//
// Two launches on the caller's stream.
//
// Slab kernels (dense_stream_kernel for one or two queries over 16-byte
// aligned rows, dense_slab_kernel otherwise): workgroup w owns a contiguous
// slab of rows and streams it once with 16-byte (or narrower) non-temporal
// loads, accumulates in fp32 and reduces over the wave.  The slab writes its
// logits to the workspace and, per query, its kTopR largest keys.
//
// dense_merge_kernel: one workgroup per query.  Any T at or below the k-th
// largest slab maximum is a lower bound of the k-th largest key overall (k
// distinct elements are >= T), so every key of the answer is >= T, and only
// the slabs whose maximum is >= T can hold one.  T is the k-th largest
// maximum (a sorting network for k <= 64, else a radix select over the
// maxima, 8 bits per pass from the first bit where they differ).  A
// qualifying slab whose kTopR-th key is below T holds no key >= T outside
// its list, so the answer normally comes from the lists alone, read in one
// round trip; only slabs with kTopR or more keys >= T are read again from
// the workspace.  The candidates (typically little more than k) are ordered
// by rank.  The kernel boundary between the two launches is the only
// cross-workgroup synchronisation: no atomics across workgroups, no fences
// (a release fence per workgroup, needed for a last-workgroup merge inside
// one launch, made the slab kernel several times slower on MI355X).

// Tuning knobs (compile-time; defaults measured on MI355X).
#ifndef VIE_DENSE_UNROLL
#define VIE_DENSE_UNROLL 1
#endif
#ifndef VIE_DENSE_ROWS
#define VIE_DENSE_ROWS 4
#endif
#ifndef VIE_DENSE_WGS
#define VIE_DENSE_WGS 1024
#endif
#ifndef VIE_DENSE_THREADS
#define VIE_DENSE_THREADS 512
#endif

constexpr int kDenseThreads = VIE_DENSE_THREADS;
constexpr int kDenseWaves = kDenseThreads / kWave;
constexpr int kDenseMaxWgs = VIE_DENSE_WGS;
constexpr int kDenseMaxNB = 8;        // queries per pass
constexpr int kDenseMaxRows = 16384;  // rows per workgroup
constexpr size_t kDenseLdsBudget = 96 * 1024;
constexpr int kMergeThreads = 1024;
constexpr int kMergeGather = 4096;    // gathered keys held in LDS
static_assert(kDenseMaxWgs <= kMergeThreads, "the merge gives every slab maximum a thread");

// Sums N values per lane over the 64 lanes of a wave.  The first log2(N)
// steps halve the set each lane carries (lanes trade the half they give
// away), the rest are plain xor steps; afterwards lane l holds the total of
// value index l >> (6 - log2 N).
template <int N, typename T>
__device__ __forceinline__ T wave_sum_multi(T (&v)[N], int lane)
{
#pragma unroll
    for (int n = N, o = 32; n > 1; n >>= 1, o >>= 1) {
        const bool upper = lane & o;
#pragma unroll
        for (int i = 0; i < n / 2; ++i) {
            const T give = upper ? v[i] : v[i + n / 2];
            const T keep = upper ? v[i + n / 2] : v[i];
            v[i] = keep + xor_lane_as(give, o);
        }
    }
    T a = v[0];
#pragma unroll
    for (int o = 32 / N; o >= 1; o >>= 1) a += xor_lane_as(a, o);
    return a;
}

template <int N> struct Log2 { static constexpr int value = 1 + Log2<N / 2>::value; };
template <> struct Log2<1> { static constexpr int value = 0; };

// Per-slab candidate lists: the kTopR largest keys of a slab, in descending
// order, 0 for "none" (no element has key 0: the id half of a key is never
// zero).  Four keys per slab let the merge take the top k from the lists
// alone unless some slab holds four or more keys above the threshold.
constexpr int kTopR = 4;

// Inserts key into the descending list b (selects only: branches here make
// the compiler keep the list in scratch).
__device__ __forceinline__ void topr_insert(uint64_t key, uint64_t (&b)[kTopR])
{
#pragma unroll
    for (int i = 0; i < kTopR; ++i) {
        const bool gt = key > b[i];
        const uint64_t hi = gt ? key : b[i];
        key = gt ? b[i] : key;
        b[i] = hi;
    }
}

// b := the kTopR largest of the descending lists b and o.  Taking the larger
// of b[i] and o[kTopR - 1 - i] keeps the kTopR largest of the union as a
// bitonic sequence, which two half-cleaner stages order.
__device__ __forceinline__ void topr_merge(const uint64_t (&o)[kTopR], uint64_t (&b)[kTopR])
{
#pragma unroll
    for (int i = 0; i < kTopR; ++i) b[i] = o[kTopR - 1 - i] > b[i] ? o[kTopR - 1 - i] : b[i];
#pragma unroll
    for (int st = kTopR / 2; st >= 1; st >>= 1)
#pragma unroll
        for (int i = 0; i < kTopR; ++i)
            if ((i & st) == 0) {
                const uint64_t x = b[i], y = b[i + st];
                b[i] = x > y ? x : y;
                b[i + st] = x > y ? y : x;
            }
}

// The kTopR largest over the lanes whose index differs in the bits of
// `span` (xor steps from span down to FROM); every such lane ends with them.
template <int SPAN, int FROM = 1>
__device__ __forceinline__ void topr_reduce(uint64_t (&b)[kTopR])
{
#pragma unroll
    for (int o = SPAN; o >= FROM; o >>= 1) {
        uint64_t t[kTopR];
#pragma unroll
        for (int i = 0; i < kTopR; ++i) t[i] = xor_lane(b[i], o);
        topr_merge(t, b);
    }
}

__device__ __forceinline__ void store_topr(uint64_t *dst, const uint64_t (&b)[kTopR])
{
    u32x4 *p = reinterpret_cast<u32x4 *>(dst);
    p[0] = u32x4{(uint32_t)b[0], (uint32_t)(b[0] >> 32), (uint32_t)b[1], (uint32_t)(b[1] >> 32)};
    p[1] = u32x4{(uint32_t)b[2], (uint32_t)(b[2] >> 32), (uint32_t)b[3], (uint32_t)(b[3] >> 32)};
}

// End of a vector-path slab: its logits (z, [nq][zpitch] in LDS) go to the
// workspace, coalesced, and wave q finds the kTopR largest keys of query q.
template <int NT>
__device__ __forceinline__ void slab_epilogue(const float *z, int zpitch, int nq, int nrows, int64_t r0, int64_t V,
                                              float *__restrict__ zout, uint64_t *__restrict__ tops)
{
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    for (int q = 0; q < nq; ++q) {
        const float *zq = z + q * zpitch;
        float *oq = zout + (int64_t)q * V + r0;
        for (int i = tid; i < nrows; i += NT) oq[i] = zq[i];
    }
    for (int q = wave; q < nq; q += NT / kWave) {
        const float *zq = z + q * zpitch;
        uint64_t b[kTopR] = {0ull, 0ull, 0ull, 0ull};
        for (int i = lane; i < nrows; i += kWave) topr_insert(make_key(zq[i], (int32_t)(r0 + i)), b);
        topr_reduce<kWave / 2>(b);
        if (lane == 0) store_topr(tops + ((int64_t)q * gridDim.x + blockIdx.x) * kTopR, b);
    }
}

// (occupancy hints: the fp32 variants of one and four queries had spilled
// registers at eight and four waves per SIMD; measured per call on MI355X,
// 100000 x 4096 fp32 at B = 1 280 -> 265 us, 128256 x 3072 fp32 at B = 4
// 426 -> 407 us)
template <int VEC, bool BF16, int NB>
__global__ __launch_bounds__(kDenseThreads) __attribute__((amdgpu_waves_per_eu(NB == 1 ? (BF16 ? 8 : 6) : !BF16 && NB == 4 ? (VEC == 16 ? 2 : 3) : 4))) void
dense_slab_kernel(const char *__restrict__ W, int64_t V, int row_bytes, const char *__restrict__ hq, int nq,
                  int rows_per_wg, float *__restrict__ zout, uint64_t *__restrict__ tops)
{
    extern __shared__ __align__(16) char smem[];
    constexpr int U = NB >= 8 ? 2 : VIE_DENSE_ROWS;  // rows in flight per wave
    constexpr int NV = NB * U;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int hbytes = (row_bytes + 15) & ~15;
    char *hs = smem;                                                   // [NB][hbytes]
    float *z = reinterpret_cast<float *>(smem + (size_t)NB * hbytes);  // [NB][rows_per_wg]

    // queries into LDS (bytewise: rows need not be 4-byte aligned), zero padded
    for (int i = tid; i < NB * hbytes; i += kDenseThreads) {
        const int q = i / hbytes, c = i - q * hbytes;
        hs[i] = (q < nq && c < row_bytes) ? hq[(int64_t)q * row_bytes + c] : 0;
    }
    __syncthreads();

    const int64_t r0 = (int64_t)blockIdx.x * rows_per_wg;
    const int nrows = (int)max<int64_t>(0, min<int64_t>(rows_per_wg, V - r0));
    const int nchunk = row_bytes / VEC;
    typedef typename Vec<VEC>::T TV;
    for (int rb = wave * U; rb < nrows; rb += kDenseWaves * U) {
        const TV *wr[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            wr[u] = reinterpret_cast<const TV *>(W + (r0 + min(rb + u, nrows - 1)) * (int64_t)row_bytes);
        typename AccOf<BF16>::T acc[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) acc[v] = 0;
#pragma unroll VIE_DENSE_UNROLL
        for (int c = lane; c < nchunk; c += kWave) {
            TV wv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) wv[u] = __builtin_nontemporal_load(wr[u] + c);
#pragma unroll
            for (int q = 0; q < NB; ++q) {
                const TV hv = reinterpret_cast<const TV *>(hs + q * hbytes)[c];
#pragma unroll
                for (int u = 0; u < U; ++u) acc[q * U + u] = dot_vec<VEC, BF16>(wv[u], hv, acc[q * U + u]);
            }
        }
        const float total = (float)wave_sum_multi<NV>(acc, lane);
        constexpr int lg = 6 - Log2<NV>::value;
        if ((lane & ((1 << lg) - 1)) == 0) {
            const int v = lane >> lg, q = v / U, u = v % U;
            if (rb + u < nrows) z[q * rows_per_wg + rb + u] = total;
        }
    }
    __syncthreads();

    slab_epilogue<kDenseThreads>(z, rows_per_wg, nq, nrows, r0, V, zout, tops);
}

// One or two queries over 16-byte aligned rows.  A lane's chunks of the
// queries stay in registers for the whole kernel (no LDS reads in the loop),
// the first row loads are issued before the queries are read, and each wave
// issues the loads of its next row group before it reduces the current one,
// so the load stream does not drain between groups.  A row of CPL 16-byte
// chunks per lane (the last ones predicated off where the row is shorter);
// a group is U rows.  Sums are formed in the same order as in
// dense_slab_kernel, so both give identical logits.
#ifndef VIE_STREAM_ROWS2
#define VIE_STREAM_ROWS2 4  // rows per group when a row is two chunks per lane (a power of two)
#endif
template <int CPL> struct StreamRows { static constexpr int value = CPL >= 4 ? 1 : CPL == 2 ? VIE_STREAM_ROWS2 : 4 / CPL; };

// Occupancy hints: rows of 12 chunks per lane at two waves per SIMD, fp32
// rows of 2 to 8 chunks at three, so that no single-query variant spills
// registers (measured on MI355X: with 8 chunks at four waves the fp32 variant
// spilled and streamed a 128256 x 2048 fp32 head at 57% of the HBM peak,
// against 83% without the spill).

template <bool BF16, int NB, int CPL>
__global__ __launch_bounds__(kDenseThreads) __attribute__((amdgpu_waves_per_eu(CPL >= 12 ? 2 : !BF16 && CPL >= 2 ? 3 : !BF16 ? 4 : NB == 1 && CPL <= 2 && CPL * StreamRows<CPL>::value <= 4 ? 8 : 4))) void
dense_stream_kernel(const char *__restrict__ W, int64_t V, int row_bytes, const char *__restrict__ hq, int nq,
                    int rows_per_wg, float *__restrict__ zout, uint64_t *__restrict__ tops)
{
    constexpr int U = StreamRows<CPL>::value;
    constexpr int NV = NB * U;
    static_assert((NV & (NV - 1)) == 0 && NV <= kWave, "the wave reduction sums a power of two of values");
    extern __shared__ __align__(16) char smem[];
    float *z = reinterpret_cast<float *>(smem);  // [NB][rows_per_wg]
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int nchunk = row_bytes / 16;
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_wg;
    const int nrows = (int)max<int64_t>(0, min<int64_t>(rows_per_wg, V - r0));
    const int ngroups = (nrows + U - 1) / U;
    const u32x4 zero = {0u, 0u, 0u, 0u};
    bool live[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) live[j] = lane + kWave * j < nchunk;

    u32x4 a[U][CPL], b[U][CPL];
    auto load_group = [&](int gi, u32x4(&buf)[U][CPL]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const u32x4 *w = reinterpret_cast<const u32x4 *>(W + (r0 + min(gi * U + u, nrows - 1)) * (int64_t)row_bytes);
#pragma unroll
            for (int j = 0; j < CPL; ++j) buf[u][j] = live[j] ? __builtin_nontemporal_load(w + lane + kWave * j) : zero;
        }
    };
    int g = wave;
    if (g < ngroups) load_group(g, a);
    u32x4 hv[NB][CPL];
#pragma unroll
    for (int q = 0; q < NB; ++q)
#pragma unroll
        for (int j = 0; j < CPL; ++j)
            hv[q][j] = live[j] && q < nq
                           ? reinterpret_cast<const u32x4 *>(hq + (int64_t)q * row_bytes)[lane + kWave * j]
                           : zero;

    auto reduce_group = [&](int gi, const u32x4(&buf)[U][CPL]) {
        typename AccOf<BF16>::T acc[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) acc[v] = 0;
#pragma unroll
        for (int j = 0; j < CPL; ++j)
#pragma unroll
            for (int q = 0; q < NB; ++q)
#pragma unroll
                for (int u = 0; u < U; ++u) acc[q * U + u] = dot_vec<16, BF16>(buf[u][j], hv[q][j], acc[q * U + u]);
        const float total = (float)wave_sum_multi<NV>(acc, lane);
        constexpr int lg = 6 - Log2<NV>::value;
        if ((lane & ((1 << lg) - 1)) == 0) {
            const int v = lane >> lg, q = v / U, u = v % U;
            if (gi * U + u < nrows) z[q * rows_per_wg + gi * U + u] = total;
        }
    };
    for (; g < ngroups; g += 2 * kDenseWaves) {
        const int g1 = g + kDenseWaves, g2 = g1 + kDenseWaves;
        if (g1 < ngroups) load_group(g1, b);
        reduce_group(g, a);
        if (g2 < ngroups) load_group(g2, a);
        if (g1 < ngroups) reduce_group(g1, b);
    }
    __syncthreads();
    slab_epilogue<kDenseThreads>(z, rows_per_wg, nq, nrows, r0, V, zout, tops);
}

constexpr int kGatherBatch = 8;  // row loads in flight per thread while gathering
constexpr int kMergeBuckets = 256;     // histogram of the slab maxima
constexpr int kMergeBucketShift = 18;  // order-space width of a bucket (log2)
constexpr int kMergeWaves = kMergeThreads / kWave;

// Sorts one key per lane of a wave, largest first (bitonic network over xor
// partners).
__device__ __forceinline__ uint64_t wave_sort_desc(uint64_t key, int lane)
{
#pragma unroll
    for (int size = 2; size <= kWave; size <<= 1)
#pragma unroll
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            const uint64_t other = xor_lane(key, stride);
            const bool keep_max = ((lane & stride) == 0) == ((lane & size) == 0);
            key = keep_max ? (other > key ? other : key) : (other < key ? other : key);
        }
    return key;
}

// Sorts a bitonic sequence held one key per lane, largest first.
__device__ __forceinline__ uint64_t wave_bitonic_merge_desc(uint64_t key, int lane)
{
#pragma unroll
    for (int stride = kWave / 2; stride > 0; stride >>= 1) {
        const uint64_t other = xor_lane(key, stride);
        key = (lane & stride) == 0 ? (other > key ? other : key) : (other < key ? other : key);
    }
    return key;
}

// The key of lane 63 - lane.
__device__ __forceinline__ uint64_t lane_reverse(uint64_t v, int lane)
{
    const int src = kWave - 1 - lane;
    return ((uint64_t)(uint32_t)__shfl((int)(uint32_t)(v >> 32), src) << 32) | (uint32_t)__shfl((int)(uint32_t)v, src);
}

// Adds the keys >= T of rows [row0, row0 + nrows) (clamped to V) of zq to
// gat; the whole workgroup takes part, kGatherBatch loads in flight per
// thread.  Element i is row i % rows_per of listed slab i / rows_per.
__device__ __forceinline__ void gather_slabs(const float *__restrict__ zq, int64_t V, const int *slabs, int nslab,
                                             int rows_per, uint64_t T, uint64_t *gat, uint32_t *s_n)
{
    const int tid = threadIdx.x;
    const int total = nslab * rows_per;
    const int step_c = kMergeThreads / rows_per, step_r = kMergeThreads % rows_per;
    for (int base = 0; base < total; base += kMergeThreads * kGatherBatch) {
        float z[kGatherBatch];
        int64_t row[kGatherBatch];
        int c = (base + tid) / rows_per, rr = (base + tid) - c * rows_per;
#pragma unroll
        for (int j = 0; j < kGatherBatch; ++j) {
            row[j] = -1;
            z[j] = 0.0f;
            if (c < nslab) {
                const int64_t r = (int64_t)slabs[c] * rows_per + rr;
                if (r < V) {
                    row[j] = r;
                    z[j] = zq[r];
                }
            }
            c += step_c;
            rr += step_r;
            if (rr >= rows_per) {
                rr -= rows_per;
                ++c;
            }
        }
#pragma unroll
        for (int j = 0; j < kGatherBatch; ++j) {
            if (row[j] >= 0) {
                const uint64_t key = make_key(z[j], (int32_t)row[j]);
                if (key >= T) {
                    const uint32_t slot = atomicAdd(s_n, 1u);
                    if (slot < (uint32_t)kMergeGather) gat[slot] = key;
                }
            }
        }
    }
}

__global__ __launch_bounds__(kMergeThreads) void dense_merge_kernel(const float *__restrict__ zbuf,
                                                                     const uint64_t *__restrict__ tops, int64_t V,
                                                                     int rows_per_wg, int nwg, int k,
                                                                     int32_t *__restrict__ ids,
                                                                     float *__restrict__ logits)
{
    __shared__ uint32_t hist[256];
    __shared__ uint64_t gat[kMergeGather];
    __shared__ uint64_t lists[kMergeWaves][kWave];
    __shared__ int cand[kMergeThreads], scan[kMergeThreads];
    __shared__ uint32_t s_nc, s_n, s_nscan, s_want, s_count, s_bucket;
    __shared__ uint32_t s_wmax[kMergeWaves];
    __shared__ unsigned long long s_prefix, s_and, s_or, s_T;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave, q = blockIdx.x;
    const float *zq = zbuf + (int64_t)q * V;

    // the slab's list of its kTopR largest keys, in one round trip
    uint64_t key[kTopR] = {0ull, 0ull, 0ull, 0ull};
    if (tid < nwg) {
        const u32x4 *p = reinterpret_cast<const u32x4 *>(tops + ((int64_t)q * nwg + tid) * kTopR);
        const u32x4 v0 = p[0], v1 = p[1];
        key[0] = ((uint64_t)v0.y << 32) | v0.x;
        key[1] = ((uint64_t)v0.w << 32) | v0.z;
        key[2] = ((uint64_t)v1.y << 32) | v1.x;
        key[3] = ((uint64_t)v1.w << 32) | v1.z;
    }
    const uint64_t m = key[0];  // the slab's maximum
    if (tid == 0) {
        s_nc = 0;
        s_n = 0;
        s_nscan = 0;
        s_and = ~0ull;
        s_or = 0ull;
        s_T = 0ull;
        s_bucket = kMergeBuckets;
    }
    if (tid < kMergeBuckets) hist[tid] = 0u;
    // 1. T, a lower bound of the k-th largest slab maximum.  First one pass:
    //    a histogram of the maxima by their distance below the largest one
    //    in the order space of the logits, 2^kMergeBucketShift per bucket
    //    (1/32 of a binade for positive logits); T is the lower edge of the
    //    bucket in which the count from the top reaches k.  The slabs above
    //    T are then k or a few more.
    const uint32_t mo = (uint32_t)(m >> 32);
    {
        uint32_t w = mo;
        // (strides written out: a loop here is left rolled, and xor_lane's
        // stride switch would then run as branches)
        w = max(w, xor_lane(w, 32));
        w = max(w, xor_lane(w, 16));
        w = max(w, xor_lane(w, 8));
        w = max(w, xor_lane(w, 4));
        w = max(w, xor_lane(w, 2));
        w = max(w, xor_lane(w, 1));
        if (lane == 0) s_wmax[wave] = w;
        __syncthreads();  // also publishes the zeroed histogram and counters
        uint32_t top = s_wmax[0];
#pragma unroll
        for (int x = 1; x < kMergeWaves; ++x) top = max(top, s_wmax[x]);
        const uint32_t dist = (top - mo) >> kMergeBucketShift;
        if (tid < nwg && dist < (uint32_t)kMergeBuckets) atomicAdd(&hist[dist], 1u);
        __syncthreads();
        if (tid < kWave) {  // wave 0: the bucket where the count from the top reaches k
            constexpr int per = kMergeBuckets / kWave;
            uint32_t c[per], sum = 0;
#pragma unroll
            for (int j = 0; j < per; ++j) {
                c[j] = hist[per * lane + j];
                sum += c[j];
            }
            const uint32_t incl = wave_incl_scan(sum);
            uint32_t above = incl - sum;
#pragma unroll
            for (int j = 0; j < per; ++j) {
                if (above < (uint32_t)k && (uint32_t)k <= above + c[j]) {
                    const uint64_t span = (uint64_t)(per * lane + j + 1) << kMergeBucketShift;
                    s_bucket = per * lane + j;
                    s_T = (uint64_t)top + 1 > span ? ((uint64_t)top + 1 - span) << 32 : 0ull;
                }
                above += c[j];
            }
        }
        __syncthreads();
    }
    if (s_bucket < (uint32_t)kMergeBuckets) {
        // T from the histogram
    } else if (k <= kWave && nwg >= k) {
        // 1. T = the k-th largest slab maximum, exactly: every wave sorts its
        //    64 maxima, then pairs of sorted lists merge (keeping the larger
        //    64) in four rounds until wave 0 holds the largest 64.
        uint64_t srt = wave_sort_desc(m, lane);
#pragma unroll
        for (int span = 1; span < kMergeWaves; span <<= 1) {
            if ((wave & (2 * span - 1)) == span) lists[wave][lane] = srt;
            __syncthreads();
            if ((wave & (2 * span - 1)) == 0) {
                const uint64_t other = lists[wave + span][kWave - 1 - lane];
                srt = wave_bitonic_merge_desc(other > srt ? other : srt, lane);
            }
        }
        const uint64_t t = __shfl(srt, k - 1, kWave);
        if (tid == 0) s_T = t;
    } else if (nwg >= k) {
        // 1'. any k: T by radix select over the maxima, 8 bits per pass from
        //     the first bit where they differ, until the bucket of the k-th
        //     largest is taken whole (so exactly k slabs have maximum >= T)
        __syncthreads();
        uint64_t a = tid < nwg ? m : ~0ull, o = m;
#pragma unroll
        for (int x = 32; x >= 1; x >>= 1) {
            a &= __shfl_xor(a, x, kWave);
            o |= __shfl_xor(o, x, kWave);
        }
        if (lane == 0) {
            atomicAnd(&s_and, (unsigned long long)a);
            atomicOr(&s_or, (unsigned long long)o);
        }
        __syncthreads();
        const uint64_t diff = s_and ^ s_or;
        uint64_t prefix = s_and;
        if (diff != 0ull) {
            // bits >= hi are known (in prefix); each pass decides bits [lo, hi)
            int hi = 64 - __clzll((long long)diff);
            prefix &= hi >= 64 ? 0ull : (~0ull << hi);
            uint32_t want = (uint32_t)k;
            for (;;) {
                const int lo = hi > 8 ? hi - 8 : 0;
                const uint64_t known = hi >= 64 ? 0ull : (~0ull << hi);
                const uint64_t dmask = (1ull << (hi - lo)) - 1ull;
                if (tid < 256) hist[tid] = 0u;
                __syncthreads();
                if (tid < nwg && (m & known) == prefix) atomicAdd(&hist[(m >> lo) & dmask], 1u);
                __syncthreads();
                if (tid < kWave) {  // wave 0: the bucket holding the want-th largest
                    uint32_t c[4], sum = 0;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        c[j] = hist[255 - 4 * lane - j];
                        sum += c[j];
                    }
                    const uint32_t incl = wave_incl_scan(sum);
                    uint32_t above = incl - sum;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if (above < want && want <= above + c[j]) {
                            s_prefix = prefix | ((uint64_t)(255 - 4 * lane - j) << lo);
                            s_want = want - above;
                            s_count = c[j];
                        }
                        above += c[j];
                    }
                }
                __syncthreads();
                prefix = s_prefix;
                want = s_want;
                if (s_count == want || lo == 0) break;  // uniform: shared values after a barrier
                hi = lo;
            }
        }
        if (tid == 0) s_T = prefix;
    }
    // (fewer slabs than k: T = 0, every slab qualifies)
    __syncthreads();
    {
        // 2. every key >= T lies in a slab whose maximum is >= T.  A slab
        //    whose last listed key is below T has all its keys >= T in its
        //    list; the others (four or more keys >= T) are read again.
        const uint64_t T = s_T;
        if (tid < nwg && m >= T) {
            cand[atomicAdd(&s_nc, 1u)] = tid;
            if (key[kTopR - 1] >= T) {
                scan[atomicAdd(&s_nscan, 1u)] = tid;
            } else {
#pragma unroll
                for (int i = 0; i < kTopR; ++i)
                    if (key[i] >= T) {
                        const uint32_t slot = atomicAdd(&s_n, 1u);
                        if (slot < (uint32_t)kMergeGather) gat[slot] = key[i];
                    }
            }
        }
        __syncthreads();
        if (s_nscan) gather_slabs(zq, V, scan, (int)s_nscan, rows_per_wg, T, gat, &s_n);
    }
    __syncthreads();
    const uint64_t T = s_T;
    const int nc = (int)s_nc;
    const int n = (int)s_n;

    if (n <= kWave) {
        // 3. one wave sorts the (typically little more than k) keys >= T
        if (tid < kWave) {
            const uint64_t key = wave_sort_desc(tid < n ? gat[tid] : 0ull, lane);
            if (tid < k && tid < n) {
                ids[(int64_t)q * k + tid] = key_id(key);
                logits[(int64_t)q * k + tid] = key_logit(key);
            }
        }
        return;
    }
    if (n <= kMergeGather) {
        // 3'. more keys: order by rank, key t lands at its rank if that is below k
        for (int t = tid; t < n; t += kMergeThreads) {
            const uint64_t key = gat[t];
            int rank = 0;
            for (int j = 0; j < n; ++j) rank += gat[j] > key;
            if (rank < k) {
                ids[(int64_t)q * k + rank] = key_id(key);
                logits[(int64_t)q * k + rank] = key_logit(key);
            }
        }
        return;
    }
    // 3''. too many keys >= T (e.g. many equal logits): the k-th largest of
    //      the candidate slabs by bisection on the key, then order by rank
    //      among the ones above it (a slow path for degenerate inputs only).
    __shared__ unsigned long long s_cnt;
    uint64_t lo = T, hi = ~0ull;  // invariant: count(>= lo) >= k, count(>= hi + 1) < k
    while (lo < hi) {
        // lo < mid <= hi, so every round shrinks [lo, hi]; written so that
        // nothing wraps when the interval is the whole key space (T = 0)
        const uint64_t mid = hi - (hi - lo) / 2;
        if (tid == 0) s_cnt = 0;
        __syncthreads();
        unsigned long long c = 0;
        for (int i = tid; i < nc * rows_per_wg; i += kMergeThreads) {
            const int cc = i / rows_per_wg;
            const int64_t row = (int64_t)cand[cc] * rows_per_wg + (i - cc * rows_per_wg);
            if (row < V && make_key(zq[row], (int32_t)row) >= mid) ++c;
        }
        atomicAdd(&s_cnt, c);
        __syncthreads();
        if (s_cnt >= (unsigned long long)k) lo = mid; else hi = mid - 1;
        __syncthreads();
    }
    if (tid == 0) s_n = 0;
    __syncthreads();
    for (int i = tid; i < nc * rows_per_wg; i += kMergeThreads) {
        const int c = i / rows_per_wg;
        const int64_t row = (int64_t)cand[c] * rows_per_wg + (i - c * rows_per_wg);
        if (row < V) {
            const uint64_t key = make_key(zq[row], (int32_t)row);
            if (key >= lo) {
                const uint32_t slot = atomicAdd(&s_n, 1u);
                if (slot < (uint32_t)kMergeGather) gat[slot] = key;
            }
        }
    }
    __syncthreads();
    const int n2 = min((int)s_n, k);  // exactly k keys are >= lo
    for (int t = tid; t < n2; t += kMergeThreads) {
        const uint64_t key = gat[t];
        int rank = 0;
        for (int j = 0; j < n2; ++j) rank += gat[j] > key;
        ids[(int64_t)q * k + rank] = key_id(key);
        logits[(int64_t)q * k + rank] = key_logit(key);
    }
}

// ---------------------------------------------------------------------------
// dense head, batched bf16: skinny GEMM on the matrix cores
// ---------------------------------------------------------------------------
//
// For several queries at once the slab logits come from
// v_mfma_f32_16x16x32_bf16 (16 rows of W_out times 16 queries per
// instruction, fp32 accumulation).  Workgroup w owns a slab of rows; each of
// its four waves takes 32 rows at a time against all the queries of the pass
// (NQT 16-query tiles) and walks the row width in stages of KC columns.
//
// The operand layout of the instruction wants 16 different rows per load,
// which scatters a wave's accesses over 16 rows (64 bytes of each); loaded
// that way straight into the operand registers, a 128256 x 3072 bf16 W_out
// streamed at 3.7-4.8 TB/s per call on MI355X (64 to 4 queries), against
// 5.0-6.1 TB/s staged.  So each wave stages its rows through its own slice of
// LDS: a stage is read with non-temporal loads that cover whole contiguous
// row segments (the next one or two stages are loaded while the current one
// is multiplied), written to LDS and read back in operand layout: lane
// (r, g) = (lane % 16, lane / 16) takes columns 32 t + 8 g .. + 7 of step t
// for its row r and the same columns of its query.  The queries' columns of
// a stage are staged in LDS once for the four waves (read with the row
// stage, one stage ahead), which keeps the registers for loads in flight.
// The slab's logits (16-byte stores) and its kTopR largest keys per query go
// to the workspace in the layout of the single-query path, and
// dense_merge_kernel selects the top k.
//
// Staged rows are padded by 32 bytes.  A 16-byte LDS read of 64 lanes takes
// four cycles on gfx950 when no bank is over-used; measured with the LDS
// counters, the operand read (16 rows, four 16-byte pieces each) takes four
// cycles when the row pitch is 32 bytes more than a multiple of 64 and eight
// cycles (half of them bank conflicts) when it is 16 or 48 more, while the
// stage writes take eight cycles at any of these pitches.

#ifndef VIE_MFMA_MIN_B
#define VIE_MFMA_MIN_B 3
#endif
#ifndef VIE_MFMA_MAX_WGS
#define VIE_MFMA_MAX_WGS 1024
#endif
// Stage width (columns) and W stages loaded ahead, per pass size (up to
// 16, 32 or 64 queries); defaults measured on MI355X.
#ifndef VIE_MFMA_KC1
#define VIE_MFMA_KC1 256
#endif
#ifndef VIE_MFMA_LA1
#define VIE_MFMA_LA1 1
#endif
#ifndef VIE_MFMA_KC2
#define VIE_MFMA_KC2 128
#endif
#ifndef VIE_MFMA_LA2
#define VIE_MFMA_LA2 2
#endif
#ifndef VIE_MFMA_KC4
#define VIE_MFMA_KC4 128
#endif
#ifndef VIE_MFMA_LA4
#define VIE_MFMA_LA4 1
#endif

constexpr int kMfmaWaves = 4;
constexpr int kMfmaThreads = kMfmaWaves * kWave;
constexpr int kMfmaMaxNB = 64;                    // queries per pass
constexpr int kMfmaMinB = VIE_MFMA_MIN_B;
constexpr int kMfmaMaxWgs = VIE_MFMA_MAX_WGS;
constexpr int kMfmaRowsPerWave = 32;              // two 16-row tiles
constexpr int kMfmaRowsPerIter = kMfmaWaves * kMfmaRowsPerWave;
static_assert(kMfmaMaxWgs <= kMergeThreads, "the merge gives every slab maximum a thread");

#ifndef VIE_MFMA_PAD
#define VIE_MFMA_PAD 32
#endif
constexpr int mfma_pitch(int KC) { return KC * 2 + VIE_MFMA_PAD; }  // LDS bytes per staged row (padded)
constexpr size_t mfma_lds(int NQT, int KC)
{
    return (size_t)(kMfmaWaves * kMfmaRowsPerWave + 16 * NQT) * mfma_pitch(KC);
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
}

template <int NQT, int KC, int LA>
__global__ __launch_bounds__(kMfmaThreads) __attribute__((amdgpu_waves_per_eu(2))) void dense_mfma_kernel(const uint16_t *__restrict__ W, int64_t V, int d,
                                                                   const uint16_t *__restrict__ hq, int nq,
                                                                   int rows_per_wg, float *__restrict__ zout,
                                                                   uint64_t *__restrict__ tops)
{
    extern __shared__ __align__(16) char smem[];
    __shared__ uint64_t s_top[16 * NQT][kMfmaWaves][kTopR];
    constexpr int kPitch = mfma_pitch(KC);
    constexpr int kSteps = KC / 32;                     // MFMA steps per stage
    constexpr int kLanesPerRow = KC / 8;                // 16-byte pieces per staged row
    constexpr int kRowsPerLoad = kWave / kLanesPerRow;
    constexpr int kLoads = kMfmaRowsPerWave / kRowsPerLoad;  // W stage loads per lane
    constexpr int kHLoads = 16 * NQT * kLanesPerRow / kMfmaThreads;  // query stage loads per thread
    static_assert(kRowsPerLoad >= 1 && kMfmaRowsPerWave % kRowsPerLoad == 0, "stage shape");
    static_assert(kHLoads >= 1 && (16 * NQT * kLanesPerRow) % kMfmaThreads == 0, "query stage shape");
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int r = lane & 15, g = lane >> 4;
    char *slice = smem + (size_t)wave * kMfmaRowsPerWave * kPitch;
    char *hsl = smem + (size_t)kMfmaWaves * kMfmaRowsPerWave * kPitch;  // [16 NQT][kPitch]
    const int64_t r0 = (int64_t)blockIdx.x * rows_per_wg;
    const int nrows = (int)max<int64_t>(0, min<int64_t>(rows_per_wg, V - r0));
    const int nstage = (d + KC - 1) / KC;
    const u32x4 zero = {0u, 0u, 0u, 0u};
    // slab starts are multiples of 128 rows, so with V % 4 == 0 every group
    // of four rows of a query's logits is 16-byte aligned
    const bool zvec = (V & 3) == 0 && ((uintptr_t)zout & 15) == 0;
    // W staging: load j of a lane covers row kRowsPerLoad j + srow, 16 bytes
    // at column scol of the stage
    const int srow = lane / kLanesPerRow, scol = 8 * (lane % kLanesPerRow);

    // query staging: load j of a thread covers query row L / kLanesPerRow
    // (padding rows repeat the last query), column hcol[j]
    const uint16_t *hrowp[kHLoads];
    int hoff[kHLoads], hcol[kHLoads];
#pragma unroll
    for (int j = 0; j < kHLoads; ++j) {
        const int L = j * kMfmaThreads + tid;
        const int row = L / kLanesPerRow;
        hcol[j] = 8 * (L % kLanesPerRow);
        hrowp[j] = hq + (int64_t)min(row, nq - 1) * d;
        hoff[j] = row * kPitch + hcol[j] * 2;
    }

    uint64_t best[NQT][kTopR];
#pragma unroll
    for (int n = 0; n < NQT; ++n)
#pragma unroll
        for (int i = 0; i < kTopR; ++i) best[n][i] = 0ull;

    // Every wave runs the same number of iterations (the workgroup barriers
    // need it); rows past the slab are clamped and discarded.  W stages run
    // LA ahead: stage st's loads sit in buffer st % LA (the loop is unrolled
    // over the buffers, so no in-flight load is ever copied); the query stage
    // runs one ahead.  Every stage issues the same loads with no branch
    // around them, in the order they are consumed (columns past the row are
    // clamped to its last piece and replaced by zeros when staged; the loads
    // of stages past the end re-read a query piece, which stays in L2), with
    // scheduling barriers keeping that order: the compiler then counts the
    // loads in flight exactly and waits only for the stage being staged, not
    // for the ones still ahead.
    for (int rb0 = 0; rb0 < nrows; rb0 += kMfmaRowsPerIter) {
        const int rb = rb0 + wave * kMfmaRowsPerWave;
        const uint16_t *wrow[kLoads];
#pragma unroll
        for (int j = 0; j < kLoads; ++j)
            wrow[j] = W + (r0 + min(rb + kRowsPerLoad * j + srow, nrows - 1)) * (int64_t)d;
        u32x4 pre[LA][kLoads];
        u32x4 hpre[kHLoads];
#pragma unroll
        for (int b = 0; b < LA; ++b) {
#pragma unroll
            for (int j = 0; j < kLoads; ++j)
                pre[b][j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(
                    b < nstage ? wrow[j] + min(b * KC + scol, d - 8) : hrowp[0]));
            __builtin_amdgcn_sched_barrier(0);  // keep the issue order
            if (b == 0) {
#pragma unroll
                for (int j = 0; j < kHLoads; ++j)
                    hpre[j] = *reinterpret_cast<const u32x4 *>(hrowp[j] + min(hcol[j], d - 8));
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        f32x4 acc[2][NQT];
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int n = 0; n < NQT; ++n) acc[m][n] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

        for (int st0 = 0; st0 < nstage; st0 += LA) {
#pragma unroll
            for (int b = 0; b < LA; ++b) {
                const int st = st0 + b;
                if (st >= nstage) break;  // uniform across the workgroup
                const int c0 = st * KC;
                __syncthreads();  // every wave is done with the previous query stage
                // this stage into LDS, then the loads of stage st + 1 (queries)
                // and st + LA (W)
                const bool win = c0 + scol + 8 <= d;
#pragma unroll
                for (int j = 0; j < kLoads; ++j)
                    *reinterpret_cast<u32x4 *>(slice + (kRowsPerLoad * j + srow) * kPitch + scol * 2) =
                        win ? pre[b][j] : zero;
#pragma unroll
                for (int j = 0; j < kHLoads; ++j)
                    *reinterpret_cast<u32x4 *>(hsl + hoff[j]) = c0 + hcol[j] + 8 <= d ? hpre[j] : zero;
#pragma unroll
                for (int j = 0; j < kHLoads; ++j)
                    hpre[j] = *reinterpret_cast<const u32x4 *>(hrowp[j] + min(c0 + KC + hcol[j], d - 8));
                __builtin_amdgcn_sched_barrier(0);
                const bool ahead = st + LA < nstage;
#pragma unroll
                for (int j = 0; j < kLoads; ++j)
                    pre[b][j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(
                        ahead ? wrow[j] + min(c0 + LA * KC + scol, d - 8) : hrowp[0]));
                __syncthreads();  // the query stage is complete
#pragma unroll
                for (int t = 0; t < kSteps; ++t) {
                    u32x4 a[2];
#pragma unroll
                    for (int m = 0; m < 2; ++m)
                        a[m] = *reinterpret_cast<const u32x4 *>(slice + (m * 16 + r) * kPitch + (32 * t + 8 * g) * 2);
#pragma unroll
                    for (int n = 0; n < NQT; ++n) {
                        const u32x4 bv =
                            *reinterpret_cast<const u32x4 *>(hsl + (n * 16 + r) * kPitch + (32 * t + 8 * g) * 2);
#pragma unroll
                        for (int m = 0; m < 2; ++m) acc[m][n] = mfma_bf16(a[m], bv, acc[m][n]);
                    }
                }
                __builtin_amdgcn_wave_barrier();
            }
        }
        // lane (r, g) holds rows 4 g + i of each 16-row tile for query 16 n + r:
        // one 16-byte store where the four rows exist and are 16-byte aligned
        // (non-temporal from 32 queries on; measured: a 16-query pass is
        // faster with ordinary stores, a 32-query pass with non-temporal ones)
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int n = 0; n < NQT; ++n) {
                const int q = n * 16 + r;
                const int lr = rb + m * 16 + 4 * g;
                if (q < nq) {
                    float *zp = zout + (int64_t)q * V + r0 + lr;
                    if (zvec && lr + 3 < nrows) {
                        if constexpr (NQT == 1)
                            *reinterpret_cast<f32x4 *>(zp) = acc[m][n];
                        else
                            __builtin_nontemporal_store(acc[m][n], reinterpret_cast<f32x4 *>(zp));
                    } else
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (lr + i < nrows) zp[i] = acc[m][n][i];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        if (lr + i < nrows) topr_insert(make_key(acc[m][n][i], (int32_t)(r0 + lr + i)), best[n]);
                }
            }
    }
    // per query: the kTopR largest over the four lane groups, then over the waves
#pragma unroll
    for (int n = 0; n < NQT; ++n) {
        topr_reduce<32, 16>(best[n]);
        if (g == 0)
#pragma unroll
            for (int i = 0; i < kTopR; ++i) s_top[n * 16 + r][wave][i] = best[n][i];
    }
    __syncthreads();
    if (tid < nq) {
        uint64_t b[kTopR], o[kTopR];
#pragma unroll
        for (int i = 0; i < kTopR; ++i) b[i] = s_top[tid][0][i];
        for (int w = 1; w < kMfmaWaves; ++w) {
#pragma unroll
            for (int i = 0; i < kTopR; ++i) o[i] = s_top[tid][w][i];
            topr_merge(o, b);
        }
        store_topr(tops + ((int64_t)tid * gridDim.x + blockIdx.x) * kTopR, b);
    }
}

// ---------------------------------------------------------------------------
// int8 rows
// ---------------------------------------------------------------------------
//
// Quantized storage is the paper's future work (Section 5).  Per vector (a
// row of W_out, or a query inside the search): scale = max |x| / 127 as an
// fp32 division, q = rint(x / scale) (fp32 division, ties to even) clamped to
// [-127, 127]; a vector of zeros has scale 0 and q = 0.  One wave per row.

constexpr int kQuantWaves = 4;

template <bool BF16>
__device__ __forceinline__ float stored_at(const void *base, int64_t i)
{
    if constexpr (BF16) return __uint_as_float((uint32_t) static_cast<const uint16_t *>(base)[i] << 16);
    else return static_cast<const float *>(base)[i];
}

__device__ __forceinline__ int8_t quantize_one(float x, float scale)
{
    if (scale == 0.0f) return 0;
    const float r = rintf(__fdiv_rn(x, scale));
    return (int8_t)fminf(fmaxf(r, -127.0f), 127.0f);
}

template <bool BF16>
__global__ __launch_bounds__(kQuantWaves *kWave) void quantize_kernel(const void *__restrict__ W, int64_t V, int d,
                                                                      int8_t *__restrict__ q,
                                                                      float *__restrict__ scale)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t row = (int64_t)blockIdx.x * kQuantWaves + threadIdx.x / kWave;
    if (row >= V) return;
    float mx = 0.0f;
    for (int j = lane; j < d; j += kWave) mx = fmaxf(mx, fabsf(stored_at<BF16>(W, row * d + j)));
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
    const float sc = __fdiv_rn(mx, 127.0f);
    for (int j = lane; j < d; j += kWave) q[row * d + j] = quantize_one(stored_at<BF16>(W, row * d + j), sc);
    if (lane == 0) scale[row] = sc;
}

// ---------------------------------------------------------------------------
// HNSW search, one workgroup per query
// ---------------------------------------------------------------------------
//
// Exact restatement of K-NN-SEARCH over SEARCH-LAYER: greedy descent (result
// set of 1) through layers maxlevel..1, then a sorted beam of ef_eff keys on
// layer 0.  Each step expands the best unexpanded beam entry: its neighbour
// list is read by one thread per slot, unseen ids are claimed in the LDS
// visited bitmap, and their rows are dotted with h by G-lane groups (every
// chunk of a row is loaded before the first is used, so one memory round
// trip covers all the new rows of a step).  New keys that cannot enter a full
// beam are dropped; the rest are ordered and merged in (the beam keeps the
// best ef_eff).  The search ends when every beam entry is expanded.  This
// visits, scores and expands exactly the nodes the sequential algorithm
// does: a node evicted from the result set is worse than all of it and would
// only be popped to stop the search.  So the distance and expansion counts
// match it.
//
// Latency hiding that keeps those semantics: the next step expands either
// the entry that is now second best among the unexpanded ones, or the best
// node this step inserts, and which one is known as soon as the rows are
// scored.  Both layer-0 lists are fetched into registers during this step's
// row loads (the second with spare threads, each new node's by the group
// that scores its row), and the threads holding the winner's list claim its
// neighbours for the next step while the others merge the beam.  The beam is
// double buffered (merge from one buffer into the other).

struct HnswShared {
    unsigned long long best;
    uint32_t nnew, nkeep;
    uint32_t first, second, nbeam;
    int32_t pfa_id, pfb_id;  // nodes whose layer-0 lists sit in pfa[] / pfb[]
    // hnsw_kernel's layer-0 loop: per step parity
    unsigned long long bestp[2];
    uint32_t nnewp[2], nkeepp[2], firstp[2];
    // hnsw_multi_kernel in a team: new nodes scored by the other members,
    // and a wait that gave up
    uint32_t nother;
    int team_err;
    uint32_t nfetch;  // hnsw_multi_kernel sharing rows: new nodes whose row is fetched
    // hnsw_multi_kernel: the bound below which kept keys cannot enter the beam
    uint32_t fmin, fmax, fsel, fcount, fn, ftau;
};

// A team: `size` workgroups (a power of two) search one query together
// (workgroup q * size + m is member m of query q).  Every member keeps the
// whole search state and takes every decision itself; each scores only the
// new nodes n with n mod size == m and passes its kept keys to the others through `keys`
// ([query][3][member][slot] with `slot` entries each) and their number
// through `tags` ([query][3][member], zero before the launch): at its e-th
// exchange (from 1) a member publishes (e << 32) | count.  Everything the
// members pass each other is written with device-scope stores (written
// through to the device's coherence point) and read with device-scope loads,
// and a member waits for its own stores to complete before it publishes the
// count, so no cache needs to be written back or invalidated.
struct TeamArgs {
    int size;
    int slot;
    uint64_t *keys;
    uint64_t *tags;
};

// Waits of a team member at an exchange are bounded (about two seconds):
// members are launched only when all of them fit on the device at once, so
// a wait that runs out means the members were not resident together, and
// the search reports it in its results instead of waiting on.
constexpr uint32_t kTeamSpin = 1u << 21;

// Row sharing: the queries of one launch form groups of `size` (query q is
// member q % size of group q / size).  A workgroup that fetches a row scores
// it for every query of its group, with the same instructions the owner's
// workgroup would use, and publishes the others' scores in `table`
// ([query][V] words (epoch << 32) | ord(score)); a query that claims a node
// whose word carries this launch's epoch takes the score from it and reads
// no row.  `hq` holds the launch's queries in the kernel's layout (rows of
// hbytes, zero padded), `hq8` / `hscale` their int8 form for int8 walks.
struct ShareArgs {
    int size;
    int B;
    uint64_t *table;
    const uint32_t *epoch;
    const char *hq;
    const int8_t *hq8;
    const float *hscale;
};

// p rounded up to 16 bytes past base (base 16-byte aligned), by pointer
// arithmetic only: a pointer into LDS keeps its address space, so the
// compiler emits LDS instructions for it (a round trip through an integer
// would make every access a generic one, which also waits on global loads).
template <typename T> __device__ __forceinline__ T *align16_past(char *base, char *p)
{
    return reinterpret_cast<T *>(base + (((p - base) + 15) & ~(ptrdiff_t)15));
}

__device__ __forceinline__ void clear_bits(uint32_t *vis, int words)
{
    for (int i = threadIdx.x; i < words; i += blockDim.x) vis[i] = 0u;
}

// Returns true if id was not yet marked (and marks it).
__device__ __forceinline__ bool claim(uint32_t *vis, int32_t id)
{
    const uint32_t bit = 1u << (id & 31);
    return (atomicOr(&vis[id >> 5], bit) & bit) == 0u;
}

// 64-bit value of lane l (l uniform across the wave).
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}

// Row chunks per lane held in registers (fp32 rows: 4, which avoids the
// register spills 8 causes there).
template <bool BF16> struct RowCpl { static constexpr int value = BF16 ? 8 : 4; };

// <row, h> by the G lanes of a group (lane gl of the group covers chunks gl,
// gl + G, ...): up to RowCpl chunks per lane are loaded before any is used,
// chunks past the row's end read as zeros.  Every lane of the group returns
// the sum.
template <int VEC, bool BF16, int G>
__device__ __forceinline__ void row_issue(const char *__restrict__ W, int64_t row, int row_bytes, int gl,
                                          typename Vec<VEC>::T (&buf)[RowCpl<BF16>::value])
{
    typedef typename Vec<VEC>::T T;
    const T *w = reinterpret_cast<const T *>(W + row * (int64_t)row_bytes);
    const int nchunk = row_bytes / VEC;
#pragma unroll
    for (int i = 0; i < RowCpl<BF16>::value; ++i) {
        const int c = gl + i * G;
        buf[i] = c < nchunk ? w[c] : T{};
    }
}

// The second half of row_dot: the query's chunks are read from LDS in
// batches of four before any of them is used (their index clamped to the
// row, so no branch; a clamped chunk meets a zero row chunk), dotted with the row chunks
// in buf (and any chunks beyond RowCpl per lane), then summed over the group.
template <int VEC, bool BF16, int G>
__device__ __forceinline__ float row_finish(const char *__restrict__ W, int64_t row, int row_bytes, const char *hs,
                                            int gl, const typename Vec<VEC>::T (&buf)[RowCpl<BF16>::value])
{
    typedef typename Vec<VEC>::T T;
    const T *w = reinterpret_cast<const T *>(W + row * (int64_t)row_bytes);
    const T *h = reinterpret_cast<const T *>(hs);
    const int nchunk = row_bytes / VEC;
    constexpr int CPL = RowCpl<BF16>::value;
    constexpr int HB = CPL < 2 ? CPL : 2;  // query chunks per batch of reads (register budget)
    typename AccOf<BF16>::T acc = 0;
#pragma unroll
    for (int i0 = 0; i0 < CPL; i0 += HB) {
        T hv[HB];
#pragma unroll
        for (int i = 0; i < HB; ++i) hv[i] = h[min(gl + (i0 + i) * G, nchunk - 1)];
#pragma unroll
        for (int i = 0; i < HB; ++i) acc = dot_vec<VEC, BF16>(buf[i0 + i], hv[i], acc);
    }
    for (int c = gl + CPL * G; c < nchunk; c += G) acc = dot_vec<VEC, BF16>(w[c], h[c], acc);
    return (float)group_sum<G>(acc);
}

template <int VEC, bool BF16, int G>
__device__ __forceinline__ float row_dot(const char *__restrict__ W, int64_t row, int row_bytes, const char *hs,
                                         int gl)
{
    typename Vec<VEC>::T buf[RowCpl<BF16>::value];
    row_issue<VEC, BF16, G>(W, row, row_bytes, gl, buf);
    return row_finish<VEC, BF16, G>(W, row, row_bytes, hs, gl, buf);
}

// Scores the entry point, then SEARCH-LAYER with a result set of one
// (greedy) through layers maxlevel..1; returns the key of the layer-0 entry
// point.  cid holds at least M ids; counts go to n_dist / n_expand.
// Records expansion number n (node id on layer lc; first: the first node
// its step expands) in the query's trace row.
__device__ __forceinline__ void note_expand(int32_t *trace, int cap, uint32_t n, int lc, int32_t id, bool first)
{
    if (trace && n < (uint32_t)cap)
        trace[n] = (int32_t)(((uint32_t)lc << 27) | ((uint32_t)first << 26) | (uint32_t)id);
}

template <int NT, int VEC, bool BF16, int G>
__device__ uint64_t descend_upper(const char *__restrict__ W, int64_t V, int row_bytes,
                                  const int32_t *__restrict__ upper_off, const int32_t *__restrict__ upper, int M,
                                  int maxlevel, int32_t entry, const char *hs, int32_t *cid, uint32_t *vis,
                                  HnswShared &sh, uint32_t &n_dist, uint32_t &n_expand, int32_t *trace,
                                  int trace_cap)
{
    constexpr int kGroups = NT / G;
    const int tid = threadIdx.x, gl = tid % G, grp = tid / G;
    const int vwords = (int)((V + 31) / 32);
    if (grp == 0) {
        const float s = row_dot<VEC, BF16, G>(W, entry, row_bytes, hs, gl);
        if (gl == 0) sh.best = make_key(s, entry);
    }
    __syncthreads();
    uint64_t cur = sh.best;
    n_dist = 1;
    for (int lc = maxlevel; lc >= 1; --lc) {
        clear_bits(vis, vwords);
        __syncthreads();
        if (tid == 0) vis[key_id(cur) >> 5] |= 1u << (key_id(cur) & 31);
        for (;;) {
            const int32_t c = key_id(cur);
            if (tid == 0) {
                sh.nnew = 0;
                note_expand(trace, trace_cap, n_expand, lc, c, true);
            }
            __syncthreads();
            ++n_expand;
            const int32_t *lst = upper + ((int64_t)upper_off[c] + lc - 1) * M;
            for (int t = tid; t < M; t += NT) {
                const int32_t e = lst[t];
                if (e >= 0 && claim(vis, e)) cid[atomicAdd(&sh.nnew, 1u)] = e;
            }
            __syncthreads();
            const int nn = (int)sh.nnew;
            for (int j = grp; j < nn; j += kGroups) {
                const float s = row_dot<VEC, BF16, G>(W, cid[j], row_bytes, hs, gl);
                if (gl == 0) atomicMax(&sh.best, (unsigned long long)make_key(s, cid[j]));
            }
            __syncthreads();
            n_dist += nn;
            const uint64_t best = sh.best;
            __syncthreads();
            if (best <= cur) break;
            cur = best;
        }
    }
    return cur;
}

constexpr int kPfbPerLane = 4;       // a new node's list is prefetched when M0 <= 4 * G
constexpr int kHnswThreads = 1024;  // threads per search workgroup

template <int NT, int VEC, bool BF16, int G>
__global__ __launch_bounds__(NT) void hnsw_kernel(
    const char *__restrict__ W, int64_t V, int row_bytes, const int32_t *__restrict__ adj0, int M0,
    const int32_t *__restrict__ upper_off, const int32_t *__restrict__ upper, int M, int maxlevel, int32_t entry,
    const char *__restrict__ hq, int k, int ef, int32_t *__restrict__ ids, float *__restrict__ logits, int ldo,
    uint32_t *__restrict__ stats, int32_t *__restrict__ trace_all, int trace_cap)
{
    extern __shared__ __align__(16) char smem[];
    __shared__ HnswShared sh;
    constexpr int kGroups = NT / G;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int q = blockIdx.x;
    int32_t *trace = trace_all ? trace_all + (int64_t)q * trace_cap : nullptr;
    const int hbytes = (row_bytes + 15) & ~15;
    const int vwords = (int)((V + 31) / 32);
    const int maxdeg = M0 > M ? M0 : M;
    // list entries prefetched per lane: enough for M0 = 64 at every group
    // width (16-lane groups: 4, 32: 2, 64: 1), which spares registers in the
    // wider groups; longer lists take the unprefetched claim
    constexpr int PF = G >= 64 ? 1 : G >= 32 ? 2 : kPfbPerLane;
    const bool pfb_on = M0 <= PF * G;
    // LDS carve-up (sizes mirror hnsw_lds_bytes)
    char *p = smem;
    char *hs = p;
    p += hbytes;
    uint64_t *beam = reinterpret_cast<uint64_t *>(p);
    p += (size_t)ef * 8;
    uint64_t *beam2 = reinterpret_cast<uint64_t *>(p);
    p += (size_t)ef * 8;
    uint64_t *ckey = reinterpret_cast<uint64_t *>(p);
    p += (size_t)maxdeg * 8;
    int32_t *cid = reinterpret_cast<int32_t *>(p);
    p += (size_t)maxdeg * 4;
    uint8_t *flag = reinterpret_cast<uint8_t *>(p);
    p += (size_t)ef;
    uint8_t *flag2 = reinterpret_cast<uint8_t *>(p);
    p += (size_t)ef;
    uint32_t *vis = align16_past<uint32_t>(smem, p);

    const char *h = hq + (int64_t)q * row_bytes;
    for (int i = tid; i < hbytes; i += NT) hs[i] = i < row_bytes ? h[i] : 0;
    if (tid == 0) sh.best = 0;
    __syncthreads();

    const int gl = tid % G;
    const int grp = tid / G;
    uint32_t n_dist = 0, n_expand = 0;

    uint64_t cur = descend_upper<NT, VEC, BF16, G>(W, V, row_bytes, upper_off, upper, M, maxlevel, entry, hs, cid,
                                                   vis, sh, n_dist, n_expand, trace, trace_cap);

    // layer 0: beam of ef keys, sorted descending, with expanded flags,
    // double buffered (beam/flag -> beam2/flag2 -> beam/flag ...).  Two
    // workgroup barriers per expansion.  Step t: (score) the rows of the
    // nodes claimed for step t are scored while the list of the second-best
    // unexpanded entry is fetched into registers; (merge) the kept keys are
    // merged into the other buffer while the node expanded at step t + 1 --
    // the better of the best kept key and that second entry, both known at
    // this point -- has its list claimed by the threads that hold it in
    // registers.  Counters used across the two phases are double buffered by
    // the parity of t and reset by thread 0 only in a phase where no other
    // thread reads or updates them.
    clear_bits(vis, vwords);
    __syncthreads();
    if (tid == 0) {
        vis[key_id(cur) >> 5] |= 1u << (key_id(cur) & 31);
        note_expand(trace, trace_cap, n_expand, 0, key_id(cur), true);
        beam[0] = cur;
        flag[0] = 1;  // expanded at step 0
        sh.nbeam = 1;
        sh.firstp[0] = 0;
        sh.firstp[1] = 0xFFFFFFFFu;
        sh.nnewp[0] = sh.nnewp[1] = 0;
        sh.nkeepp[0] = sh.nkeepp[1] = 0;
        sh.bestp[0] = sh.bestp[1] = 0ull;
    }
    __syncthreads();
    {
        // claim the layer-0 entry point's neighbours for step 0
        const int32_t c = key_id(cur);
        for (int t = tid; t < M0; t += NT) {
            const int32_t e = adj0[(int64_t)c * M0 + t];
            if (e >= 0 && claim(vis, e)) cid[atomicAdd(&sh.nnewp[0], 1u)] = e;
        }
    }
    __syncthreads();
    for (int step = 0;; ++step) {
        const int par = step & 1;
        // ---- score ----
        const uint32_t first = sh.firstp[par], nbeam = sh.nbeam;
        const int nn = (int)sh.nnewp[par];
        ++n_expand;
        n_dist += nn;
        if (tid == 0) sh.firstp[par ^ 1] = 0xFFFFFFFFu;  // last read in the previous step's score phase
        // the first row of this group (and its list) starts loading before
        // the scan below, which then runs under the load latency
        typedef typename Vec<VEC>::T TV;
        TV rbuf[RowCpl<BF16>::value];
        int32_t l0[PF];
#pragma unroll
        for (int u = 0; u < PF; ++u) l0[u] = -1;
        const int32_t e0 = grp < nn ? cid[grp] : -1;
        // (an opaque copy of the lane index: the per-lane addresses are then
        // formed here, not held in registers across the whole loop)
        int glv = gl;
        __asm__ volatile("" : "+v"(glv));
        if (e0 >= 0) {
            if (pfb_on) {
#pragma unroll
                for (int u = 0; u < PF; ++u) {
                    const int t = glv + u * G;
                    l0[u] = t < M0 ? adj0[(int64_t)e0 * M0 + t] : -1;
                }
            }
            row_issue<VEC, BF16, G>(W, e0, row_bytes, glv, rbuf);
        }
        // the second-best unexpanded entry: every wave scans the flags itself
        uint32_t second = 0xFFFFFFFFu;
        for (int i0 = (int)first + 1; i0 < (int)nbeam; i0 += kWave) {
            const int i = i0 + lane;
            const uint64_t ball = __ballot(i < (int)nbeam && !flag[i]);
            if (ball) {
                second = (uint32_t)(i0 + __ffsll((long long)ball) - 1);
                break;
            }
        }
        const int32_t ida = second < nbeam ? key_id(beam[second]) : -1;
        // spare threads fetch the second entry's list while the rows load
        int32_t pfv = -1;
        const int pft = tid - (NT - M0);  // the last M0 threads
        if (ida >= 0 && pft >= 0) pfv = adj0[(int64_t)ida * M0 + pft];
        const uint64_t worst = nbeam == (uint32_t)ef ? beam[nbeam - 1] : 0ull;
        uint64_t gbest = 0ull;  // best key this group scored, and its node's list
        int32_t glist[PF];
        if (e0 >= 0) {
            const float s = row_finish<VEC, BF16, G>(W, e0, row_bytes, hs, gl, rbuf);
            const uint64_t key = make_key(s, e0);
            if (gl == 0 && key > worst) ckey[atomicAdd(&sh.nkeepp[par], 1u)] = key;
            gbest = key;
#pragma unroll
            for (int u = 0; u < PF; ++u) glist[u] = l0[u];
        }
        for (int j = grp + kGroups; j < nn; j += kGroups) {
            const int32_t e = cid[j];
            int32_t l[PF];
            if (pfb_on) {
#pragma unroll
                for (int u = 0; u < PF; ++u) {
                    const int t = gl + u * G;
                    l[u] = t < M0 ? adj0[(int64_t)e * M0 + t] : -1;
                }
            }
            const float s = row_dot<VEC, BF16, G>(W, e, row_bytes, hs, gl);
            const uint64_t key = make_key(s, e);
            if (gl == 0 && key > worst) ckey[atomicAdd(&sh.nkeepp[par], 1u)] = key;
            if (key > gbest) {
                gbest = key;
#pragma unroll
                for (int u = 0; u < PF; ++u) glist[u] = l[u];
            }
        }
        if (gl == 0 && gbest > worst) atomicMax(&sh.bestp[par], (unsigned long long)gbest);
        __syncthreads();
        // ---- merge, and the claim of the next step ----
        const uint64_t bestnew = sh.bestp[par];
        const int nk = (int)sh.nkeepp[par];
        const uint64_t second_key = ida >= 0 ? beam[second] : 0ull;
        const uint64_t next = bestnew > second_key ? bestnew : second_key;  // expanded at step + 1
        if (next != 0ull) {
            if (next == second_key) {
                if (pft >= 0 && pfv >= 0 && claim(vis, pfv)) cid[atomicAdd(&sh.nnewp[par ^ 1], 1u)] = pfv;
            } else if (pfb_on) {
                if (gbest == bestnew) {
#pragma unroll
                    for (int u = 0; u < PF; ++u) {
                        const int t = gl + u * G;
                        if (t < M0 && glist[u] >= 0 && claim(vis, glist[u]))
                            cid[atomicAdd(&sh.nnewp[par ^ 1], 1u)] = glist[u];
                    }
                }
            } else {
                const int32_t c = key_id(next);
                for (int t = tid; t < M0; t += NT) {
                    const int32_t e = adj0[(int64_t)c * M0 + t];
                    if (e >= 0 && claim(vis, e)) cid[atomicAdd(&sh.nnewp[par ^ 1], 1u)] = e;
                }
            }
        }
        // merge the beam (nbeam, sorted) and the kept keys (nk, unordered,
        // distinct) into beam2, keeping the best ef: a kept key lands at
        // (kept keys above it) + (beam keys above it), a beam key at its
        // index + (kept keys above it).  The next expanded entry is marked.
        const int total = min((int)nbeam + nk, ef);
        for (int j = tid; j < nk; j += NT) {
            const uint64_t key = ckey[j];
            int above = 0;
            for (int t = 0; t < nk; ++t) above += ckey[t] > key;
            int lo = 0, hi = (int)nbeam;  // count beam keys > key
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (beam[mid] > key) lo = mid + 1; else hi = mid;
            }
            const int pos = lo + above;
            if (pos < total) {
                beam2[pos] = key;
                flag2[pos] = key == next;
                if (key == next) sh.firstp[par ^ 1] = (uint32_t)pos;
            }
        }
        // the beam keys on the other half of the workgroup, in parallel with the kept keys
        for (int i = (tid + NT / 2) % NT; i < (int)nbeam; i += NT) {
            const uint64_t key = beam[i];
            int above = 0;
            for (int t = 0; t < nk; ++t) above += ckey[t] > key;
            const int pos = i + above;
            if (pos < total) {
                beam2[pos] = key;
                flag2[pos] = flag[i] | (key == next);
                if (key == next) sh.firstp[par ^ 1] = (uint32_t)pos;
            }
        }
        if (tid == 0) {
            if (next != 0ull) note_expand(trace, trace_cap, n_expand, 0, key_id(next), true);  // step + 1
            sh.nbeam = (uint32_t)total;
            sh.nnewp[par] = 0;     // read at the top of this step only
            sh.nkeepp[par ^ 1] = 0;  // last used in the previous step
            sh.bestp[par ^ 1] = 0ull;
        }
        __syncthreads();
        uint64_t *tb = beam;
        beam = beam2;
        beam2 = tb;
        uint8_t *tf = flag;
        flag = flag2;
        flag2 = tf;
        if (next == 0ull) break;
    }

    const int nb = (int)sh.nbeam;
    for (int t = tid; t < k; t += NT) {
        ids[(int64_t)q * ldo + t] = t < nb ? key_id(beam[t]) : -1;
        logits[(int64_t)q * ldo + t] = t < nb ? key_logit(beam[t]) : -__builtin_inff();
    }
    if (stats && tid == 0) {
        stats[2 * q] = n_dist;
        stats[2 * q + 1] = n_expand;
    }
}

// ---------------------------------------------------------------------------
// HNSW search, several expansions per step
// ---------------------------------------------------------------------------
//
// The batched traversal: every step expands the `width` best unexpanded beam
// entries at once (their lists are claimed together, all the new rows are
// scored in one pass, and the new keys are merged in as above).  It follows
// the oracle's multi-expansion search exactly (width 1 is the sequential
// algorithm), trading a few more distance evaluations for width times fewer
// dependent steps.
//
// A step: wave 0 finds the picks (ballots over the expanded flags, from the
// best unexpanded entry on) and publishes them in LDS behind one barrier;
// the threads that claim a pick's list mark it expanded; the new rows are
// scored two per group at a time; the keys that can enter the beam are
// sorted into runs of 128 and ranked, and beam and kept keys are merged into
// the other beam buffer.  Lists: the groups that score the best `width` new
// rows keep those rows' lists in a small LDS cache (one workgroup per query
// only), so the next step reads most of its lists there; the rest come from
// HBM.
//
// A team (TeamArgs) runs this on several workgroups per query that divide
// only the scoring and pass each other the kept keys every step; row sharing
// (ShareArgs) lets the queries of a group reuse each other's scores.  Both
// leave every decision, and so the traversal, exactly as above.

constexpr int kMaxWidth = 128;      // widest expansion step
// Kept keys a wide step drops below the beam's reach before ranking them
// (only when a step keeps more than this many keys and has this many list
// slots: the histogram and the per-edge beam counts take 2 KB of the
// claimed-id array).
constexpr int kKeepFilterMin = 512;
constexpr int kPickNarrowSpan = 256;  // picks scan: one flag per lane up to this many entries past the first
constexpr int kMultiHeld = 2;       // rows per group whose lists a group can cache
constexpr int kClaimBatch = 4;      // list entries a thread claims together

// <row a, h> and <row b, h> (b < 0: only a) with both rows' chunks loaded
// before either is used (chunks past the row's end read as zeros), the
// query's chunks read from LDS two at a time before use (index clamped to
// the row), and both sums taken over the group as in group_sum.
template <int VEC, bool BF16, int G>
__device__ __forceinline__ void row_dot2(const char *__restrict__ W, int64_t ra, int64_t rb, int row_bytes,
                                         const char *hs, int gl, float &sa, float &sb)
{
    typedef typename Vec<VEC>::T T;
    const T *wa = reinterpret_cast<const T *>(W + ra * (int64_t)row_bytes);
    const T *wb = reinterpret_cast<const T *>(W + (rb >= 0 ? rb : ra) * (int64_t)row_bytes);
    const T *h = reinterpret_cast<const T *>(hs);
    const int nchunk = row_bytes / VEC;
    constexpr int CPL = RowCpl<BF16>::value;
    T ba[CPL], bb[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        const int c = gl + i * G;
        ba[i] = c < nchunk ? wa[c] : T{};
        bb[i] = c < nchunk && rb >= 0 ? wb[c] : T{};
    }
    constexpr int HB = 1;
    typename AccOf<BF16>::T xa = 0, xb = 0;
#pragma unroll
    for (int i0 = 0; i0 < CPL; i0 += HB) {
        T hv[HB];
#pragma unroll
        for (int i = 0; i < HB; ++i) hv[i] = h[min(gl + (i0 + i) * G, nchunk - 1)];
#pragma unroll
        for (int i = 0; i < HB; ++i) {
            xa = dot_vec<VEC, BF16>(ba[i0 + i], hv[i], xa);
            xb = dot_vec<VEC, BF16>(bb[i0 + i], hv[i], xb);
        }
    }
    for (int c = gl + CPL * G; c < nchunk; c += G) {
        xa = dot_vec<VEC, BF16>(wa[c], h[c], xa);
        if (rb >= 0) xb = dot_vec<VEC, BF16>(wb[c], h[c], xb);
    }
    sa = (float)group_sum<G>(xa);
    sb = (float)group_sum<G>(xb);
}

__device__ __forceinline__ int sdot16(u32x4 w, u32x4 h, int acc)
{
    acc = __builtin_amdgcn_sdot4((int)w.x, (int)h.x, acc, false);
    acc = __builtin_amdgcn_sdot4((int)w.y, (int)h.y, acc, false);
    acc = __builtin_amdgcn_sdot4((int)w.z, (int)h.z, acc, false);
    return __builtin_amdgcn_sdot4((int)w.w, (int)h.w, acc, false);
}

// Integer <q_a, hq> and <q_b, hq> over int8 rows of d bytes (d % 16 == 0;
// b < 0: only a), loaded and summed as in row_dot2.
template <int G>
__device__ __forceinline__ void row_dot2_q8(const int8_t *__restrict__ Q, int64_t ra, int64_t rb, int d,
                                            const int8_t *hq, int gl, int &ia, int &ib)
{
    const u32x4 *qa = reinterpret_cast<const u32x4 *>(Q + ra * (int64_t)d);
    const u32x4 *qb = reinterpret_cast<const u32x4 *>(Q + (rb >= 0 ? rb : ra) * (int64_t)d);
    const u32x4 *h = reinterpret_cast<const u32x4 *>(hq);
    const int nchunk = d / 16;
    constexpr int CPL = 4;  // int8 rows are at most half a stored row: G lanes cover them in 4 chunks
    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 ba[CPL], bb[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        const int c = gl + i * G;
        ba[i] = c < nchunk ? qa[c] : zero;
        bb[i] = c < nchunk && rb >= 0 ? qb[c] : zero;
    }
    int xa = 0, xb = 0;
#pragma unroll
    for (int i0 = 0; i0 < CPL; i0 += 2) {
        u32x4 hv[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) hv[i] = h[min(gl + (i0 + i) * G, nchunk - 1)];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            xa = sdot16(ba[i0 + i], hv[i], xa);
            xb = sdot16(bb[i0 + i], hv[i], xb);
        }
    }
    for (int c = gl + CPL * G; c < nchunk; c += G) {
        xa = sdot16(qa[c], h[c], xa);
        if (rb >= 0) xb = sdot16(qb[c], h[c], xb);
    }
    ia = group_sum<G>(xa);
    ib = group_sum<G>(xb);
}

// row_dot2 for every query of a group (queries m = 0 .. qg - 1 at
// hgroup + m * hbytes, in the kernel's query layout): the two rows' chunks
// are loaded once, and each query's sums are taken with exactly row_dot2's
// sequence of operations, so a query's scores are the bits its own
// row_dot2 would give.  f(m, score_a, score_b) receives them in order.
template <int VEC, bool BF16, int G, typename F>
__device__ __forceinline__ void row_dot2_group(const char *__restrict__ W, int64_t ra, int64_t rb, int row_bytes,
                                               const char *__restrict__ hgroup, int hbytes, int qg, int gl, F f)
{
    typedef typename Vec<VEC>::T T;
    const T *wa = reinterpret_cast<const T *>(W + ra * (int64_t)row_bytes);
    const T *wb = reinterpret_cast<const T *>(W + (rb >= 0 ? rb : ra) * (int64_t)row_bytes);
    const int nchunk = row_bytes / VEC;
    constexpr int CPL = RowCpl<BF16>::value;
    T ba[CPL], bb[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        const int c = gl + i * G;
        ba[i] = c < nchunk ? wa[c] : T{};
        bb[i] = c < nchunk && rb >= 0 ? wb[c] : T{};
    }
    for (int m = 0; m < qg; ++m) {
        const T *h = reinterpret_cast<const T *>(hgroup + (int64_t)m * hbytes);
        typename AccOf<BF16>::T xa = 0, xb = 0;
#pragma unroll
        for (int i0 = 0; i0 < CPL; ++i0) {
            const T hv = h[min(gl + i0 * G, nchunk - 1)];
            xa = dot_vec<VEC, BF16>(ba[i0], hv, xa);
            xb = dot_vec<VEC, BF16>(bb[i0], hv, xb);
        }
        for (int c = gl + CPL * G; c < nchunk; c += G) {
            xa = dot_vec<VEC, BF16>(wa[c], h[c], xa);
            if (rb >= 0) xb = dot_vec<VEC, BF16>(wb[c], h[c], xb);
        }
        f(m, (float)group_sum<G>(xa), (float)group_sum<G>(xb));
    }
}

// row_dot2_q8 for every query of a group (int8 queries m at hgroup + m * d):
// f(m, dot_a, dot_b) with the integer dots.
template <int G, typename F>
__device__ __forceinline__ void row_dot2_q8_group(const int8_t *__restrict__ Q, int64_t ra, int64_t rb, int d,
                                                  const int8_t *__restrict__ hgroup, int qg, int gl, F f)
{
    const u32x4 *qa = reinterpret_cast<const u32x4 *>(Q + ra * (int64_t)d);
    const u32x4 *qb = reinterpret_cast<const u32x4 *>(Q + (rb >= 0 ? rb : ra) * (int64_t)d);
    const int nchunk = d / 16;
    constexpr int CPL = 4;
    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 ba[CPL], bb[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        const int c = gl + i * G;
        ba[i] = c < nchunk ? qa[c] : zero;
        bb[i] = c < nchunk && rb >= 0 ? qb[c] : zero;
    }
    for (int m = 0; m < qg; ++m) {
        const u32x4 *h = reinterpret_cast<const u32x4 *>(hgroup + (int64_t)m * d);
        int xa = 0, xb = 0;
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
            const u32x4 hv = h[min(gl + i * G, nchunk - 1)];
            xa = sdot16(ba[i], hv, xa);
            xb = sdot16(bb[i], hv, xb);
        }
        for (int c = gl + CPL * G; c < nchunk; c += G) {
            xa = sdot16(qa[c], h[c], xa);
            if (rb >= 0) xb = sdot16(qb[c], h[c], xb);
        }
        f(m, group_sum<G>(xa), group_sum<G>(xb));
    }
}

// Layer-0 score from int8 rows: fp32(integer dot) * row scale * query scale,
// each product rounded to fp32 (no fused operations).
__device__ __forceinline__ float q8_score(int acc, float row_scale, float query_scale)
{
    const float a = __fmul_rn((float)acc, row_scale);
    return __fmul_rn(a, query_scale);
}

template <int NT, int VEC, bool BF16, int G, bool Q8, bool SHARE>
__global__ __launch_bounds__(NT) void hnsw_multi_kernel(
    const char *__restrict__ W, int64_t V, int row_bytes, const int32_t *__restrict__ adj0, int M0,
    const int32_t *__restrict__ upper_off, const int32_t *__restrict__ upper, int M, int maxlevel, int32_t entry,
    const char *__restrict__ hq, int k, int ef, int width, int32_t *__restrict__ ids, float *__restrict__ logits, int ldo,
    uint32_t *__restrict__ stats, const int8_t *__restrict__ q8, const float *__restrict__ q8scale,
    int32_t *__restrict__ trace_all, int trace_cap, TeamArgs team, ShareArgs share)
{
    extern __shared__ __align__(16) char smem[];
    __shared__ HnswShared sh;
    __shared__ int32_t lc_id[kMaxWidth];  // nodes whose lists sit in the cache
    __shared__ int32_t s_pick[kMaxWidth];  // this step's picks (beam positions)
    __shared__ int32_t s_np, s_after;
    __shared__ uint32_t s_hmax;           // Q8: bits of max |h|
    __shared__ uint32_t s_xoff[kMaxTeam + 1];  // team exchange: where each member's keys go
    constexpr int kGroups = NT / G;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int T = team.size;              // 1: one workgroup per query
    const int q = blockIdx.x / T, mem = blockIdx.x - q * T;
    uint32_t exchanges = 0;               // team exchanges so far
    const int hbytes = (row_bytes + 15) & ~15;
    const int vwords = (int)((V + 31) / 32);
    const int cap = width * M0;  // most nodes claimed in one step
    // cache slots a flag byte can name (slot + 1 in its upper seven bits)
    const int hints = width < 127 ? width : 127;
    // t / M0 for t < 2^15 (M0 <= 256) as a multiply-high by this magic number
    const uint32_t m0_magic = (uint32_t)(((1ull << 32) + (uint32_t)M0 - 1u) / (uint32_t)M0);
    const int nid = cap > M ? cap : M;
    // list entries a group keeps per lane (as in hnsw_kernel: enough for
    // M0 = 64 at every group width)
    constexpr int PF = G >= 64 ? 1 : G >= 32 ? 2 : kPfbPerLane;
    const bool cache_on = M0 <= PF * G && T == 1;  // a member scores only its share of the rows
    const int d = row_bytes / (BF16 ? 2 : 4);
    const int d8 = Q8 ? (d + 15) & ~15 : 0;
    // LDS carve-up (sizes mirror hnsw_multi_lds_bytes)
    char *p = smem;
    char *hs = p;
    p += hbytes;
    uint64_t *beam = reinterpret_cast<uint64_t *>(p);
    p += (size_t)ef * 8;
    uint64_t *beam2 = reinterpret_cast<uint64_t *>(p);
    p += (size_t)ef * 8;
    uint64_t *ckey = reinterpret_cast<uint64_t *>(p);  // padded to whole 128-key runs
    p += (size_t)((cap + 2 * kWave - 1) & ~(2 * kWave - 1)) * 8;
    int32_t *cid = reinterpret_cast<int32_t *>(p);
    p += (size_t)nid * 4;
    int32_t *lcache = reinterpret_cast<int32_t *>(p);  // (none in a team)
    p += T == 1 ? (size_t)cap * 4 : 0;
    int32_t *fid = reinterpret_cast<int32_t *>(p);  // sharing rows: the new nodes whose rows are fetched
    p += SHARE ? (size_t)cap * 4 : 0;
    // flag arrays 8-byte aligned and padded to 8 bytes: the picks scan reads
    // them eight flags per lane
    const int efp = (ef + 7) & ~7;
    p = smem + (((p - smem) + 7) & ~(ptrdiff_t)7);
    uint8_t *flag = reinterpret_cast<uint8_t *>(p);
    p += (size_t)efp;
    uint8_t *flag2 = reinterpret_cast<uint8_t *>(p);
    p += (size_t)efp;
    int8_t *hq8 = align16_past<int8_t>(smem, p);  // Q8: the int8 query
    p = reinterpret_cast<char *>(hq8) + d8;
    // sharing rows: the group's queries (int8 rows of d8 bytes for Q8, else
    // rows of hbytes)
    const int gbytes = Q8 ? d8 : hbytes;
    char *hgrp = reinterpret_cast<char *>(align16_past<int8_t>(smem, p));
    p = hgrp + (SHARE ? (size_t)share.size * gbytes : 0);
    uint32_t *vis = align16_past<uint32_t>(smem, p);

    const char *h = hq + (int64_t)q * row_bytes;
    for (int i = tid; i < hbytes; i += NT) hs[i] = i < row_bytes ? h[i] : 0;
    if (tid == 0) {
        sh.best = 0;
        s_hmax = 0;
        sh.nother = 0;
        sh.team_err = 0;
        sh.nfetch = 0;
    }
    if (tid < kMaxWidth) lc_id[tid] = -1;
    __syncthreads();
    float hscale = 0.0f;
    if constexpr (Q8) {  // the query quantized like the rows
        for (int j = tid; j < d; j += NT) atomicMax(&s_hmax, __float_as_uint(fabsf(stored_at<BF16>(hs, j))));
        __syncthreads();
        hscale = __fdiv_rn(__uint_as_float(s_hmax), 127.0f);
        for (int j = tid; j < d8; j += NT) hq8[j] = j < d ? quantize_one(stored_at<BF16>(hs, j), hscale) : 0;
        __syncthreads();
    }

    const int gl = tid % G;
    const int grp = tid / G;
    uint32_t n_dist = 0, n_expand = 0;
    uint32_t n_other = 0;  // in a team: this thread's claims of nodes another member scores
    int32_t *trace = trace_all && mem == 0 ? trace_all + (int64_t)q * trace_cap : nullptr;
    // sharing rows: this query's group (queries gq0 .. gq0 + qg - 1) and the launch's epoch
    const int gq0 = SHARE ? q - q % share.size : q;
    const int qg = SHARE ? min(share.size, share.B - gq0) : 1;
    const uint32_t epoch = SHARE ? *share.epoch : 0u;
    if constexpr (SHARE) {  // the group's queries into LDS, 16 bytes per thread at a time
        const u32x4 *src = reinterpret_cast<const u32x4 *>(Q8 ? reinterpret_cast<const char *>(share.hq8) + (int64_t)gq0 * d8
                                                               : share.hq + (int64_t)gq0 * hbytes);
        u32x4 *dst = reinterpret_cast<u32x4 *>(hgrp);
        for (int i = tid; i < qg * gbytes / 16; i += NT) dst[i] = src[i];
        __syncthreads();
    }
    uint64_t cur = descend_upper<NT, VEC, BF16, G>(W, V, row_bytes, upper_off, upper, M, maxlevel, entry, hs, cid,
                                                   vis, sh, n_dist, n_expand, trace, trace_cap);

    // A team exchange: this member's `mine` keys (already in its slot of
    // area `area`) meet the other members' keys, appended to dst after the
    // `*n` already there.  Steps alternate between areas 0 and 1: a member
    // can only be one exchange ahead of the slowest, so it never overwrites
    // keys still being read.
    auto exchange = [&](int area, uint32_t mine, uint64_t *dst, uint32_t *n) {
        const int64_t base = ((int64_t)q * 3 + area) * T;
        const uint32_t tag = ++exchanges;
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_waitcnt(0);  // this wave's key stores are complete
        __syncthreads();
        if (tid == 0)
            __hip_atomic_store(team.tags + base + mem, ((uint64_t)tag << 32) | mine, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        // wave 0: lane l waits (bounded) for the counts of members l, l + 64,
        // ..., then the running sums say where each member's keys go
        constexpr int kPerLane = (kMaxTeam + kWave - 1) / kWave;
        if (tid < kWave) {
            uint32_t c[kPerLane];
            uint32_t need = 0u;  // bit i: the count of member lane + 64 i is still awaited
#pragma unroll
            for (int i = 0; i < kPerLane; ++i) {
                c[i] = 0u;
                const int o = lane + i * kWave;
                if (o < T && o != mem) need |= 1u << i;
            }
            uint32_t spins = 0;
            while (need) {
#pragma unroll
                for (int i = 0; i < kPerLane; ++i)
                    if (need & (1u << i)) {
                        const uint64_t w = __hip_atomic_load(team.tags + base + lane + i * kWave, __ATOMIC_RELAXED,
                                                             __HIP_MEMORY_SCOPE_AGENT);
                        if ((uint32_t)(w >> 32) == tag) {
                            c[i] = (uint32_t)w;
                            need &= ~(1u << i);
                        }
                    }
                if (!need) break;
                if (++spins > kTeamSpin) {
                    sh.team_err = 1;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
            uint32_t carry = 0u;
#pragma unroll
            for (int i = 0; i < kPerLane; ++i) {
                const uint32_t incl = wave_incl_scan(c[i]) + carry;
                const int o = lane + i * kWave;
                if (o < T) s_xoff[o + 1] = incl;
                carry = (uint32_t)__shfl((int)incl, kWave - 1, kWave);
            }
            if (lane == 0) s_xoff[0] = 0;
        }
        __syncthreads();
        if (sh.team_err) return;
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        const int total = (int)s_xoff[T];
        for (int j = tid; j < total; j += NT) {
            int o = 0;  // the member whose keys hold entry j: the last with s_xoff[o] <= j
            for (int step = kMaxTeam / 2; step > 0; step >>= 1)
                if (o + step < T && (int)s_xoff[o + step] <= j) o += step;
            const uint64_t *ok = team.keys + (base + o) * team.slot;
            dst[mine + j] = __hip_atomic_load(ok + (j - (int)s_xoff[o]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (tid == 0) *n = mine + (uint32_t)total;
        __syncthreads();
    };

    if constexpr (Q8) {  // the layer-0 entry point scored again on its int8 row
        if (grp == 0) {
            int ia, ib;
            row_dot2_q8<G>(q8, key_id(cur), -1, d, hq8, gl, ia, ib);
            if (gl == 0) sh.best = make_key(q8_score(ia, q8scale[key_id(cur)], hscale), key_id(cur));
        }
        __syncthreads();
        cur = sh.best;
        ++n_dist;
    }
    clear_bits(vis, vwords);
    __syncthreads();
    if (tid == 0) {
        vis[key_id(cur) >> 5] |= 1u << (key_id(cur) & 31);
        beam[0] = cur;
        flag[0] = 0;
        sh.nbeam = 1;
        sh.first = 0;
        sh.nnew = 0;
    }
    __syncthreads();
    for (;;) {
        const uint32_t first = sh.first, nbeam = sh.nbeam;
        if (first >= nbeam) break;  // no unexpanded entry (first is ~0 then)
        // the picks: up to width unexpanded entries from `first` on, in beam
        // order, and the next unexpanded entry after them, found by wave 0
        // (ballots over the expanded bits) and published in LDS
        if (tid < kWave) {
            int np = 0;
            bool found_after = false;
            if (lane == 0) s_after = -1;
            if ((int)nbeam - (int)first <= kPickNarrowSpan) {
                // a short span: one flag per lane, 64 entries per round
                for (int i0 = (int)first; i0 < (int)nbeam && !found_after; i0 += kWave) {
                    const int i = i0 + lane;
                    const bool un = i < (int)nbeam && !(flag[i] & 1);
                    const uint64_t ball = __ballot(un);
                    const int rank = np + (int)__builtin_amdgcn_mbcnt_hi(
                                              (uint32_t)(ball >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)ball, 0u));
                    if (un && rank < width) s_pick[rank] = i;
                    if (un && rank == width) s_after = i;
                    found_after = np + __popcll(ball) > width;
                    np = min(width, np + __popcll(ball));
                }
            } else {
                // eight flags per lane (512 entries per round): bit 8 b of a
                // lane's mask is set when entry 8 lane + b is unexpanded and in
                // [first, nbeam); a lane's entries take the ranks after those of
                // the lanes below it
                for (int b0 = (int)first & ~7; b0 < (int)nbeam && !found_after; b0 += 8 * kWave) {
                    const int i = b0 + 8 * lane;
                    uint64_t m = 0ull;
                    if (i < (int)nbeam) {
                        m = ~*reinterpret_cast<const uint64_t *>(flag + i) & 0x0101010101010101ull;
                        const int lo = (int)first - i, hi = (int)nbeam - i;
                        if (lo >= 8) m = 0ull;
                        else if (lo > 0) m &= ~0ull << (8 * lo);
                        if (hi < 8) m &= (1ull << (8 * hi)) - 1ull;
                    }
                    const uint32_t cnt = (uint32_t)__popcll(m);
                    const uint32_t incl = wave_incl_scan(cnt);
                    int rank = np + (int)(incl - cnt);
                    for (uint64_t mm = m; mm != 0ull && rank <= width; mm &= mm - 1ull, ++rank) {
                        const int idx = i + (__ffsll((long long)mm) - 1) / 8;
                        if (rank < width) s_pick[rank] = idx;
                        else s_after = idx;
                    }
                    const int total = __builtin_amdgcn_readlane((int)incl, kWave - 1);
                    found_after = np + total > width;
                    np = min(width, np + total);
                }
            }
            if (lane == 0) {
                s_np = np;
                sh.nkeep = 0;  // last read before the previous merge
            }
        }
        __syncthreads();
        const int np = s_np;
        if (np == 0) break;
        if (tid == 0 && trace) {
            for (int t = 0; t < np; ++t) note_expand(trace, trace_cap, n_expand + t, 0, key_id(beam[s_pick[t]]), t == 0);
        }
        n_expand += np;
        // claim the unseen neighbours of the picks (node t / M0, slot t % M0);
        // a pick's list comes from the cache slot its flag names while the
        // cache still holds that node's list, else from HBM.  The first slot
        // of each pick marks it expanded (the other bits of its flag stay).
        // A thread loads its kClaimBatch list entries, marks the picks it
        // meets expanded, issues all its bitmap claims (an OR of zero where
        // there is no entry), then appends its new nodes: no claim waits
        // behind another.
        const int ncl = np * M0;
        for (int t0 = tid; t0 < ncl; t0 += kClaimBatch * NT) {
            int32_t ev[kClaimBatch];
#pragma unroll
            for (int u = 0; u < kClaimBatch; ++u) {
                const int t = min(t0 + u * NT, ncl - 1);
                const int j = (int)__umulhi((uint32_t)t, m0_magic), slot = t - j * M0;
                const int pj = s_pick[j];
                const int32_t c = key_id(beam[pj]);
                const int hint = (int)(flag[pj] >> 1) - 1;
                const int src = hint >= 0 && lc_id[hint] == c ? hint : -1;
                // two guarded loads, not one through a selected pointer (that
                // would be a generic load, which waits on both memory counters)
                const int32_t ec = src >= 0 ? lcache[max(src, 0) * M0 + slot] : -1;
                const int32_t eg = src < 0 ? adj0[(int64_t)c * M0 + slot] : -1;
                ev[u] = t0 + u * NT < ncl ? (src >= 0 ? ec : eg) : -1;
            }
#pragma unroll
            for (int u = 0; u < kClaimBatch; ++u) {
                const int t = t0 + u * NT;
                const int j = (int)__umulhi((uint32_t)t, m0_magic);
                if (t < ncl && t == j * M0) flag[s_pick[j]] |= 1;
            }
            uint32_t old[kClaimBatch];
#pragma unroll
            for (int u = 0; u < kClaimBatch; ++u)
                old[u] = atomicOr(&vis[max(ev[u], 0) >> 5], ev[u] >= 0 ? 1u << (ev[u] & 31) : 0u);
#pragma unroll
            for (int u = 0; u < kClaimBatch; ++u)
                if (ev[u] >= 0 && !(old[u] & (1u << (ev[u] & 31)))) {
                    if ((ev[u] & (T - 1)) == mem) cid[atomicAdd(&sh.nnew, 1u)] = ev[u];
                    else ++n_other;
                }
        }
        __syncthreads();
        const int nn = (int)sh.nnew;  // this member's share of the new nodes
        n_dist += nn;
        const int area = (int)(exchanges & 1);
        uint64_t *xk = T > 1 ? team.keys + (((int64_t)q * 3 + area) * T + mem) * team.slot : nullptr;
        const uint64_t worst = nbeam == (uint32_t)ef ? beam[nbeam - 1] : 0ull;
        // sharing rows: a new node whose score another query of the group
        // published in this launch is kept or dropped on that score; the
        // others go to the fetch list
        const int32_t *lst = cid;
        int nl = nn;
        if constexpr (SHARE) {
            for (int j = tid; j < nn; j += NT) {
                const int32_t e = cid[j];
                const uint64_t w = __hip_atomic_load(share.table + (int64_t)q * V + e, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT);
                if ((uint32_t)(w >> 32) == epoch) {
                    const uint64_t key = (w << 32) | (uint64_t)(~(uint32_t)e);
                    if (key > worst) ckey[atomicAdd(&sh.nkeep, 1u)] = key;
                } else {
                    fid[atomicAdd(&sh.nfetch, 1u)] = e;
                }
            }
            __syncthreads();
            lst = fid;
            nl = (int)sh.nfetch;
        }
        // score the new rows, two per group at a time; keep the keys that
        // can enter the beam, and the lists of a group's first rows
        uint64_t rk[kMultiHeld];
        int32_t rl[kMultiHeld][PF];
#pragma unroll
        for (int r = 0; r < kMultiHeld; ++r) rk[r] = 0ull;
        int r = 0;
        for (int j = grp; j < nl; j += 2 * kGroups, r += 2) {
            const int32_t ea = lst[j];
            const int32_t eb = j + kGroups < nl ? lst[j + kGroups] : -1;
            int32_t la[PF], lb[PF];
            if (cache_on && r < kMultiHeld) {
#pragma unroll
                for (int u = 0; u < PF; ++u) {
                    const int t = gl + u * G;
                    la[u] = t < M0 ? adj0[(int64_t)ea * M0 + t] : -1;
                    lb[u] = t < M0 && eb >= 0 ? adj0[(int64_t)eb * M0 + t] : -1;
                }
            }
            float sa, sb;
            if constexpr (SHARE) {
                // every query of the group against the two rows; the others'
                // scores published (one lane per row)
                auto publish = [&](int m, float xa, float xb) {
                    if (m == q - gq0) {
                        sa = xa;
                        sb = xb;
                    } else if (gl == 0) {
                        uint64_t *tm = share.table + (int64_t)(gq0 + m) * V;
                        __hip_atomic_store(tm + ea, ((uint64_t)epoch << 32) | f2ord(xa), __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                        if (eb >= 0)
                            __hip_atomic_store(tm + eb, ((uint64_t)epoch << 32) | f2ord(xb), __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                    }
                };
                if constexpr (Q8) {
                    const float ca = q8scale[ea], cb = eb >= 0 ? q8scale[eb] : 0.0f;
                    row_dot2_q8_group<G>(q8, ea, eb, d, reinterpret_cast<const int8_t *>(hgrp), qg, gl,
                                         [&](int m, int ia, int ib) {
                                             const float hsc = share.hscale[gq0 + m];
                                             publish(m, q8_score(ia, ca, hsc), q8_score(ib, cb, hsc));
                                         });
                } else {
                    row_dot2_group<VEC, BF16, G>(W, ea, eb, row_bytes, hgrp, hbytes, qg, gl, publish);
                }
            } else if constexpr (Q8) {
                const float ca = q8scale[ea], cb = eb >= 0 ? q8scale[eb] : 0.0f;
                int ia, ib;
                row_dot2_q8<G>(q8, ea, eb, d, hq8, gl, ia, ib);
                sa = q8_score(ia, ca, hscale);
                sb = q8_score(ib, cb, hscale);
            } else {
                row_dot2<VEC, BF16, G>(W, ea, eb, row_bytes, hs, gl, sa, sb);
            }
            const uint64_t ka = make_key(sa, ea), kb = eb >= 0 ? make_key(sb, eb) : 0ull;
            if (gl == 0 && ka > worst) {
                const uint32_t slot = atomicAdd(&sh.nkeep, 1u);
                ckey[slot] = ka;
                if (xk) __hip_atomic_store(xk + slot, ka, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            if (gl == 0 && eb >= 0 && kb > worst) {
                const uint32_t slot = atomicAdd(&sh.nkeep, 1u);
                ckey[slot] = kb;
                if (xk) __hip_atomic_store(xk + slot, kb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
#pragma unroll
            for (int x = 0; x + 1 < kMultiHeld; x += 2)
                if (x == r) {
                    rk[x] = ka > worst ? ka : 0ull;
                    rk[x + 1] = kb > worst ? kb : 0ull;
#pragma unroll
                    for (int u = 0; u < PF; ++u) {
                        rl[x][u] = la[u];
                        rl[x + 1][u] = lb[u];
                    }
                }
        }
        if (tid == 0) {
            sh.first = 0xFFFFFFFFu;  // every thread read it before the claim barrier
            sh.ftau = 0u;
        }
        __syncthreads();
        if (T > 1) {  // the kept keys of the other members join this member's
            exchange(area, sh.nkeep, ckey, &sh.nkeep);
            if (sh.team_err) break;
        }
        int nk = (int)sh.nkeep;
        // A step that keeps many more keys than the beam can take (the first
        // steps of a wide walk, while the beam fills) drops the kept keys that
        // cannot enter it before they are sorted and ranked.  A histogram of
        // the kept keys' score bits (256 buckets over their range) and, per
        // bucket edge, the beam entries at or above it suggest the highest
        // edge with at least ef keys of the beam and the kept keys at or above
        // it.  The kept keys at or above that edge are gathered and counted
        // exactly; only if they and the beam entries at or above the edge are
        // at least ef do they replace the kept keys: every key dropped then has
        // ef larger keys, so the merge would drop it anyway and the new beam
        // is the same.  The histogram, the per-edge beam counts and the
        // gathered keys use the claimed-id array, which is free between the
        // scoring and the merge.
        static_assert(NT >= 256, "a thread per histogram bucket");
        if (cap >= kKeepFilterMin && nk > kKeepFilterMin && (int)nbeam + nk > ef) {  // uniform
            uint32_t *hist = reinterpret_cast<uint32_t *>(cid);            // [256]
            uint32_t *bcount = hist + 256;                                 // [256], by descending bucket
            uint64_t *keep2 = reinterpret_cast<uint64_t *>(hist + 256);    // gathered keys (after bcount is read)
            const uint32_t room = (uint32_t)(cap - 256) / 2;
            if (tid == 0) {
                sh.fmin = 0xFFFFFFFFu;
                sh.fmax = 0u;
                sh.fsel = 256u;
                sh.fn = 0u;
            }
            for (int t = tid; t < 256; t += NT) hist[t] = 0u;
            __syncthreads();
            uint32_t mn = 0xFFFFFFFFu, mx = 0u;
            for (int j = tid; j < nk; j += NT) {
                const uint32_t sbits = (uint32_t)(ckey[j] >> 32);
                mn = min(mn, sbits);
                mx = max(mx, sbits);
            }
            mn = wave_min_u32(mn);
            mx = wave_max_u32(mx);
            if (lane == 0) {
                atomicMin(&sh.fmin, mn);
                atomicMax(&sh.fmax, mx);
            }
            __syncthreads();
            const uint32_t lo = sh.fmin;
            const uint32_t span = sh.fmax - lo;
            const float scale = 256.0f / ((float)span + 1.0f);
            for (int j = tid; j < nk; j += NT) {
                const uint32_t sbits = (uint32_t)(ckey[j] >> 32);
                atomicAdd(&hist[min(255u, (uint32_t)((float)(sbits - lo) * scale))], 1u);
            }
            // edge of bucket b: lo + b (span + 1) / 256 (an exact count is
            // taken below, so the edges need not match the buckets exactly)
            auto edge = [&](int b) { return lo + (uint32_t)(((uint64_t)b * ((uint64_t)span + 1)) >> 8); };
            if (tid < 256) {
                const uint64_t thr = (uint64_t)edge(255 - tid) << 32;
                const int bst = 1 << (31 - __builtin_clz(nbeam));  // nbeam >= 1
                int c = 0;  // beam entries at or above the edge of bucket 255 - tid
                for (int step = bst; step > 0; step >>= 1)
                    if (c + step <= (int)nbeam && beam[c + step - 1] >= thr) c += step;
                bcount[tid] = (uint32_t)c;
            }
            __syncthreads();
            if (tid < kWave) {  // wave 0: the highest bucket whose edge reaches ef keys
                uint32_t v[4], sum = 0;
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    v[u] = hist[255 - (4 * lane + u)];
                    sum += v[u];
                }
                uint32_t run = wave_incl_scan(sum) - sum;  // kept keys in the buckets above this lane's
                int sel = 256;
                uint32_t nb = 0;
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    run += v[u];
                    if (sel == 256 && run + bcount[4 * lane + u] >= (uint32_t)ef) {
                        sel = 4 * lane + u;
                        nb = bcount[4 * lane + u];
                    }
                }
                const uint64_t any = __ballot(sel < 256);
                if (any != 0ull && lane == __ffsll((long long)any) - 1) {
                    sh.fsel = (uint32_t)sel;
                    sh.fcount = nb;  // beam entries at or above the chosen edge
                }
            }
            __syncthreads();
            if (sh.fsel < 256u) {  // uniform
                const uint32_t t = edge(255 - (int)sh.fsel);
                for (int j = tid; j < nk; j += NT) {
                    const uint64_t key = ckey[j];
                    if ((uint32_t)(key >> 32) >= t) {
                        const uint32_t slot = atomicAdd(&sh.fn, 1u);
                        if (slot < room) keep2[slot] = key;
                    }
                }
                __syncthreads();
                const uint32_t ng = sh.fn;
                if (ng <= room && ng < (uint32_t)nk && ng + sh.fcount >= (uint32_t)ef) {  // uniform
                    if (tid == 0) sh.ftau = t;  // kept keys with score bits below it were dropped
                    nk = (int)ng;
                    for (int j = tid; j < nk; j += NT) ckey[j] = keep2[j];
                    __syncthreads();
                }
            }
        }
        // with more than 64 kept keys, each wave sorts runs of 128 of them
        // (two sorted halves of 64, the second reversed so that the pair is
        // bitonic, half-cleaned and merged in registers), so that a key's rank
        // among the kept keys is a sum of binary searches.  (Runs of 256, four
        // halves per wave, measured slower: the sort outweighs the searches.)
        constexpr int kRun = 2 * kWave;
        const int nrun = (nk + kRun - 1) / kRun;
        if (nk > kWave) {
            for (int r = tid / kWave; r < nrun; r += NT / kWave) {
                const int j0 = r * kRun + lane, j1 = j0 + kWave;
                // the last run is padded with zero keys (below every real key)
                const uint64_t a = wave_sort_desc(j0 < nk ? ckey[j0] : 0ull, lane);
                const uint64_t br = lane_reverse(wave_sort_desc(j1 < nk ? ckey[j1] : 0ull, lane), lane);
                ckey[j0] = wave_bitonic_merge_desc(a > br ? a : br, lane);
                ckey[j1] = wave_bitonic_merge_desc(a > br ? br : a, lane);
            }
            __syncthreads();
        }
        auto kept_above = [&](uint64_t key) -> int {  // kept keys larger than key
            int above = 0;
            if (nk <= kWave) {
                for (int t = 0; t < nk; ++t) above += ckey[t] > key;
                return above;
            }
            // fixed-step searches of the 128-key runs, four runs at a time so
            // that their LDS loads overlap
            int r = 0;
            for (; r + 4 <= nrun; r += 4) {
                const uint64_t *a = ckey + r * kRun;
                int p0 = 0, p1 = 0, p2 = 0, p3 = 0;
#pragma unroll
                for (int step = kRun / 2; step > 0; step >>= 1) {
                    p0 += a[p0 + step - 1] > key ? step : 0;
                    p1 += a[kRun + p1 + step - 1] > key ? step : 0;
                    p2 += a[2 * kRun + p2 + step - 1] > key ? step : 0;
                    p3 += a[3 * kRun + p3 + step - 1] > key ? step : 0;
                }
                above += p0 + (a[p0] > key) + p1 + (a[kRun + p1] > key) + p2 + (a[2 * kRun + p2] > key) + p3 +
                         (a[3 * kRun + p3] > key);
            }
            for (; r < nrun; ++r) {
                const uint64_t *a = ckey + r * kRun;
                int p = 0;
#pragma unroll
                for (int step = kRun / 2; step > 0; step >>= 1) p += a[p + step - 1] > key ? step : 0;
                above += p + (a[p] > key);
            }
            return above;
        };
        // the lists of the best `width` new nodes into the cache, by rank
        if (cache_on) {
#pragma unroll
            for (int x = 0; x < kMultiHeld; ++x)
                if (rk[x] != 0ull && (uint32_t)(rk[x] >> 32) >= sh.ftau) {
                    const int above = kept_above(rk[x]);
                    if (above < hints) {
#pragma unroll
                        for (int u = 0; u < PF; ++u) {
                            const int t = gl + u * G;
                            if (t < M0) lcache[above * M0 + t] = rl[x][u];
                        }
                        if (gl == 0) lc_id[above] = key_id(rk[x]);
                    }
                }
        }
        // merge the beam and the kept keys (as in the sequential kernel); the
        // picks are marked expanded, and the new first unexpanded entry is
        // the best kept key or the entry after the picks
        // (the claimed ids are spent: cid[r] receives the beam position of
        // the kept key of rank r, non-decreasing in r, so that a beam entry's
        // count of larger kept keys is one binary search)
        const int total = min((int)nbeam + nk, ef);
        const int bstep = 1 << (31 - __builtin_clz(nbeam));  // nbeam >= 1
        for (int j = tid; j < nk; j += NT) {
            const uint64_t key = ckey[j];
            int lo = 0;  // beam entries larger than key
            for (int step = bstep; step > 0; step >>= 1)
                if (lo + step <= (int)nbeam && beam[lo + step - 1] > key) lo += step;
            const int above = kept_above(key);
            cid[above] = lo;
            const int pos = lo + above;
            if (pos < total) {
                beam2[pos] = key;
                // unexpanded; the best `width` kept keys name the cache slot
                // that may hold their list
                flag2[pos] = above < hints ? (uint8_t)((above + 1) << 1) : (uint8_t)0;
                if (above == 0) atomicMin(&sh.first, (uint32_t)pos);
            }
        }
        __syncthreads();
        const int after = s_after;
        const int kstep = nk > 0 ? 1 << (31 - __builtin_clz(nk)) : 0;
        for (int i = tid; i < (int)nbeam; i += NT) {
            const uint64_t key = beam[i];
            int lo = 0;  // kept keys whose beam position is <= i lie above beam[i]
            for (int step = kstep; step > 0; step >>= 1)
                if (lo + step <= nk && cid[lo + step - 1] <= i) lo += step;
            const int pos = i + lo;
            if (pos < total) {
                beam2[pos] = key;
                flag2[pos] = flag[i] & 1;  // older cache slots are stale
                if (i == after) atomicMin(&sh.first, (uint32_t)pos);
            }
        }
        if (tid == 0) {
            sh.nbeam = (uint32_t)total;
            sh.nnew = 0;  // read after the claim barrier only
            sh.nfetch = 0;
        }
        __syncthreads();
        uint64_t *tb = beam;
        beam = beam2;
        beam2 = tb;
        uint8_t *tf = flag;
        flag = flag2;
        flag2 = tf;
    }

    if (T > 1) {  // the other members' new nodes count as distance evaluations too (one add per wave)
        const uint32_t incl = wave_incl_scan(n_other);
        if (lane == kWave - 1) atomicAdd(&sh.nother, incl);
        __syncthreads();
        n_dist += sh.nother;
    }
    const int nb = (int)sh.nbeam;
    if (sh.team_err) {  // a team wait ran out: the results say so
        if (mem == 0) {
            for (int t = tid; t < k; t += NT) {
                ids[(int64_t)q * ldo + t] = -1;
                logits[(int64_t)q * ldo + t] = __builtin_nanf("");
            }
            if (stats && tid == 0) stats[2 * q] = stats[2 * q + 1] = 0xFFFFFFFFu;
        }
        return;
    }
    if constexpr (Q8) {
        // exact re-rank of the final beam: exact keys into beam2, then by
        // rank; in a team each member scores the entries of its share and
        // the first member gathers all of them
        if (T == 1) {
            for (int j = grp; j < nb; j += kGroups) {
                const int32_t e = key_id(beam[j]);
                const float sc = row_dot<VEC, BF16, G>(W, e, row_bytes, hs, gl);
                if (gl == 0) beam2[j] = make_key(sc, e);
            }
        } else {
            if (tid == 0) sh.nkeep = 0;
            __syncthreads();
            uint64_t *xr = team.keys + (((int64_t)q * 3 + 2) * T + mem) * team.slot;
            for (int j = grp; j < nb; j += kGroups) {
                const int32_t e = key_id(beam[j]);
                if ((e & (T - 1)) != mem) continue;
                const float sc = row_dot<VEC, BF16, G>(W, e, row_bytes, hs, gl);
                if (gl == 0) {
                    const uint32_t slot = atomicAdd(&sh.nkeep, 1u);
                    beam2[slot] = make_key(sc, e);
                    __hip_atomic_store(xr + slot, make_key(sc, e), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            __syncthreads();
            exchange(2, sh.nkeep, beam2, &sh.nkeep);
            if (mem != 0) return;
            if (sh.team_err) {
                for (int t = tid; t < k; t += NT) {
                    ids[(int64_t)q * ldo + t] = -1;
                    logits[(int64_t)q * ldo + t] = __builtin_nanf("");
                }
                if (stats && tid == 0) stats[2 * q] = stats[2 * q + 1] = 0xFFFFFFFFu;
                return;
            }
        }
        __syncthreads();
        // rank the exact keys: each wave sorts runs of 64, a key's rank is
        // the sum of its binary-search positions in the runs (stopped once
        // it reaches k)
        const int nrun = (nb + kWave - 1) / kWave;
        for (int r = tid / kWave; r < nrun; r += NT / kWave) {
            const int j = r * kWave + lane;
            const uint64_t key = wave_sort_desc(j < nb ? beam2[j] : 0ull, lane);
            if (j < nb) beam2[j] = key;  // the run's real keys are its largest
        }
        __syncthreads();
        for (int t = tid; t < nb; t += NT) {
            const uint64_t key = beam2[t];
            int rank = 0;
            for (int r = 0; r < nrun && rank < k; ++r) {
                const uint64_t *run = beam2 + r * kWave;
                int lo = 0, hi = min(kWave, nb - r * kWave);
                while (lo < hi) {
                    const int mid = (lo + hi) >> 1;
                    if (run[mid] > key) lo = mid + 1; else hi = mid;
                }
                rank += lo;
            }
            if (rank < k) {
                ids[(int64_t)q * ldo + rank] = key_id(key);
                logits[(int64_t)q * ldo + rank] = key_logit(key);
            }
        }
        for (int t = nb + tid; t < k; t += NT) {
            ids[(int64_t)q * ldo + t] = -1;
            logits[(int64_t)q * ldo + t] = -__builtin_inff();
        }
    } else {
        if (mem != 0) return;
        for (int t = tid; t < k; t += NT) {
            ids[(int64_t)q * ldo + t] = t < nb ? key_id(beam[t]) : -1;
            logits[(int64_t)q * ldo + t] = t < nb ? key_logit(beam[t]) : -__builtin_inff();
        }
    }
    if (stats && tid == 0) {
        stats[2 * q] = n_dist;
        stats[2 * q + 1] = n_expand;
    }
}

// ---------------------------------------------------------------------------
// forced-inclusion tokens (Section 3)
// ---------------------------------------------------------------------------
//
// One workgroup per query: the search result (the first k entries of the
// query's output row) and the logits of the forced ids, computed exactly
// like the search's (G-lane row dots, fp32), are joined with each id once
// and written back over the row (k + n entries) by rank, padded with -1 /
// -inf.  The row is read into LDS before anything is written.

constexpr int kForcedThreads = 256;

template <int VEC, bool BF16, int G>
__global__ __launch_bounds__(kForcedThreads) void forced_kernel(const char *__restrict__ W, int64_t V, int row_bytes,
                                                                const char *__restrict__ hq,
                                                                const int32_t *__restrict__ forced, int n, int k,
                                                                int32_t *__restrict__ ids, float *__restrict__ logits)
{
    extern __shared__ __align__(16) char smem[];
    __shared__ uint32_t s_m;
    constexpr int kGroups = kForcedThreads / G;
    const int tid = threadIdx.x, q = blockIdx.x;
    const int w = k + n;
    const int hbytes = (row_bytes + 15) & ~15;
    char *hs = smem;
    int32_t *sid = reinterpret_cast<int32_t *>(smem + hbytes);        // [k] search ids
    uint64_t *keys = reinterpret_cast<uint64_t *>(smem + hbytes + (((size_t)k * 4 + 7) & ~(size_t)7));  // [k + n]
    const char *h = hq + (int64_t)q * row_bytes;
    for (int i = tid; i < hbytes; i += kForcedThreads) hs[i] = i < row_bytes ? h[i] : 0;
    if (tid == 0) s_m = 0;
    __syncthreads();
    for (int j = tid; j < k; j += kForcedThreads) {
        const int32_t id = ids[(int64_t)q * w + j];
        sid[j] = id;
        if (id >= 0) keys[atomicAdd(&s_m, 1u)] = make_key(logits[(int64_t)q * w + j], id);
    }
    __syncthreads();
    const int gl = tid % G, grp = tid / G;
    for (int i = grp; i < n; i += kGroups) {
        const int32_t f = forced[i];
        if (f < 0 || f >= V) continue;
        bool dup = false;
        for (int j = 0; j < k; ++j) dup |= sid[j] == f;
        const float sc = row_dot<VEC, BF16, G>(W, f, row_bytes, hs, gl);
        if (!dup && gl == 0) keys[atomicAdd(&s_m, 1u)] = make_key(sc, f);
    }
    __syncthreads();
    const int m = (int)s_m;
    for (int t = tid; t < m; t += kForcedThreads) {
        const uint64_t key = keys[t];
        int rank = 0;
        for (int j = 0; j < m; ++j) rank += keys[j] > key;
        ids[(int64_t)q * w + rank] = key_id(key);
        logits[(int64_t)q * w + rank] = key_logit(key);
    }
    for (int t = m + tid; t < w; t += kForcedThreads) {
        ids[(int64_t)q * w + t] = -1;
        logits[(int64_t)q * w + t] = -__builtin_inff();
    }
}

// Widest load (bytes) that divides the row and keeps W aligned.
int pick_vec(int row_bytes, const void *W)
{
    const uintptr_t al = (uintptr_t)W;
    for (int v = 16; v >= 4; v >>= 1)
        if (row_bytes % v == 0 && al % v == 0) return v;
    return 2;
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

namespace {
vie_status launched(hipError_t e, const char *what)
{
    if (e == hipSuccess) return VIE_OK;
    return fail(VIE_EHIP, "%s: %s", what, hipGetErrorString(e));
}
}  // namespace

vie_status launch_scatter(const int32_t *ids, const float *logits, int B, int k, int64_t V, float *out,
                          hipStream_t s)
{
    dim3 grid((unsigned)((V + kScatterTile - 1) / kScatterTile), (unsigned)B);
    scatter_kernel<<<grid, kScatterThreads, 0, s>>>(ids, logits, k, V, out);
    return launched(hipGetLastError(), "scatter launch");
}

namespace {

// Grid size of the dense head: at most kDenseMaxWgs workgroups.
int dense_grid(int64_t V)
{
    const int64_t nwg = V < kDenseMaxWgs ? V : kDenseMaxWgs;
    return nwg < 1 ? 1 : (int)nwg;
}

struct DensePlan {
    int nwg, rpw, nbmax;
};

size_t dense_lds(int nb, int row_bytes, int rows_per_wg)
{
    const size_t hbytes = (size_t)((row_bytes + 15) & ~15);
    return (size_t)nb * (hbytes + (size_t)rows_per_wg * 4);
}

// Slab size, grid and queries per pass; a slab's logits and the queries of
// one pass must fit the LDS budget.
bool dense_plan(int64_t V, int row_bytes, DensePlan &p)
{
    const int nwg = dense_grid(V);
    const int rpw = (int)((V + nwg - 1) / nwg);
    if (rpw > kDenseMaxRows) return false;
    int nb = kDenseMaxNB;
    while (nb > 1 && dense_lds(nb, row_bytes, rpw) > kDenseLdsBudget) nb >>= 1;
    if (dense_lds(nb, row_bytes, rpw) > kDenseLdsBudget) return false;
    p.nwg = (int)((V + rpw - 1) / rpw);
    p.rpw = rpw;
    p.nbmax = nb;
    return true;
}

// Chunks of 16 bytes per lane per row for the streaming kernel (0: not served).
int stream_cpl(int row_bytes, int nb)
{
    const int c = (row_bytes / 16 + kWave - 1) / kWave;
    const int cpl = c <= 1 ? 1 : c <= 2 ? 2 : c <= 4 ? 4 : c <= 8 ? 8 : c <= 12 ? 12 : 0;
    return nb == 2 && cpl > 4 ? 0 : cpl;
}

template <bool BF16, int NB, int CPL>
hipError_t stream_launch(const void *W, int64_t V, int row_bytes, const char *h, int nq, int k, const DensePlan &p,
                         float *zbuf, uint64_t *tops, int32_t *ids, float *logits, hipStream_t s)
{
    const size_t lds = (size_t)NB * p.rpw * 4;
    auto kern = dense_stream_kernel<BF16, NB, CPL>;
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    kern<<<p.nwg, kDenseThreads, lds, s>>>(static_cast<const char *>(W), V, row_bytes, h, nq, p.rpw, zbuf, tops);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dense_merge_kernel<<<nq, kMergeThreads, 0, s>>>(zbuf, tops, V, p.rpw, p.nwg, k, ids, logits);
    return hipGetLastError();
}

template <bool BF16>
hipError_t stream_launch_cpl(int cpl, int nb, const void *W, int64_t V, int row_bytes, const char *h, int nq, int k,
                             const DensePlan &p, float *zbuf, uint64_t *tops, int32_t *ids, float *logits,
                             hipStream_t s)
{
    if (nb == 1) {
        switch (cpl) {
        case 1: return stream_launch<BF16, 1, 1>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
        case 2: return stream_launch<BF16, 1, 2>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
        case 4: return stream_launch<BF16, 1, 4>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
        case 8: return stream_launch<BF16, 1, 8>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
        default: return stream_launch<BF16, 1, 12>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
        }
    }
    switch (cpl) {
    case 1: return stream_launch<BF16, 2, 1>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
    case 2: return stream_launch<BF16, 2, 2>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
    default: return stream_launch<BF16, 2, 4>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
    }
}

template <int VEC, bool BF16, int NB>
hipError_t dense_launch(const void *W, int64_t V, int row_bytes, const char *h, int nq, int k, const DensePlan &p,
                        float *zbuf, uint64_t *tops, int32_t *ids, float *logits, hipStream_t s)
{
    const size_t lds = dense_lds(NB, row_bytes, p.rpw);
    auto kern = dense_slab_kernel<VEC, BF16, NB>;
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    kern<<<p.nwg, kDenseThreads, lds, s>>>(static_cast<const char *>(W), V, row_bytes, h, nq, p.rpw, zbuf, tops);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dense_merge_kernel<<<nq, kMergeThreads, 0, s>>>(zbuf, tops, V, p.rpw, p.nwg, k, ids, logits);
    return hipGetLastError();
}

template <int VEC, bool BF16>
hipError_t dense_launch_nb(int nb, const void *W, int64_t V, int row_bytes, const char *h, int nq, int k,
                           const DensePlan &p, float *zbuf, uint64_t *tops, int32_t *ids, float *logits,
                           hipStream_t s)
{
    switch (nb) {
    case 1: return dense_launch<VEC, BF16, 1>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
    case 2: return dense_launch<VEC, BF16, 2>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
    case 4: return dense_launch<VEC, BF16, 4>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
    default: return dense_launch<VEC, BF16, 8>(W, V, row_bytes, h, nq, k, p, zbuf, tops, ids, logits, s);
    }
}

}  // namespace

namespace {

// Matrix-core plan: slabs of whole workgroup iterations, at most
// kDenseMaxWgs of them (the merge gives every slab maximum a thread).
DensePlan mfma_plan(int64_t V)
{
    const int64_t iters = (V + kMfmaRowsPerIter - 1) / kMfmaRowsPerIter;
    const int64_t per = (iters + kMfmaMaxWgs - 1) / kMfmaMaxWgs;
    DensePlan p;
    p.rpw = (int)(per * kMfmaRowsPerIter);
    p.nwg = (int)((V + p.rpw - 1) / p.rpw);
    p.nbmax = kMfmaMaxNB;
    return p;
}

bool use_mfma(int dtype, int d, int B, const void *W, const void *h)
{
    return dtype == VIE_BF16 && B >= kMfmaMinB && d % 8 == 0 && (uintptr_t)W % 16 == 0 && (uintptr_t)h % 16 == 0;
}

// Queries per pass of either path.
int dense_pass(int B) { return B >= kMfmaMinB ? kMfmaMaxNB : kDenseMaxNB; }

template <int NQT, int KC, int LA>
hipError_t mfma_launch(const void *W, int64_t V, int d, const char *h, int nq, int k, const DensePlan &p,
                       float *zbuf, uint64_t *tops, int32_t *ids, float *logits, hipStream_t s)
{
    auto kern = dense_mfma_kernel<NQT, KC, LA>;
    constexpr size_t lds = mfma_lds(NQT, KC);
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    kern<<<p.nwg, kMfmaThreads, lds, s>>>(static_cast<const uint16_t *>(W), V, d,
                                           reinterpret_cast<const uint16_t *>(h), nq, p.rpw, zbuf, tops);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dense_merge_kernel<<<nq, kMergeThreads, 0, s>>>(zbuf, tops, V, p.rpw, p.nwg, k, ids, logits);
    return hipGetLastError();
}

}  // namespace

// Workspace: the logits [nb][V] fp32 (256-byte padded), then the kTopR
// largest keys of every slab [nb][slabs][kTopR] u64, nb = the queries of one
// pass (at most 8 on the vector path, 64 on the matrix-core path, never more
// than B).
size_t dense_workspace_bytes(int64_t V, int d, int B, int k)
{
    (void)d;
    (void)k;
    const int pass = dense_pass(B);
    const int nb = B < pass ? B : pass;
    const int slabs = std::max(dense_grid(V), mfma_plan(V).nwg);
    return (((size_t)nb * V * 4 + 255) & ~(size_t)255) + (size_t)nb * slabs * 8 * kTopR;
}

vie_status launch_dense_topk(const void *W, int dtype, int64_t V, int d, const void *h, int B, int k, int32_t *ids,
                             float *logits, void *ws, hipStream_t s)
{
    const int row_bytes = d * elem_bytes(dtype);
    DensePlan p;
    if (!dense_plan(V, row_bytes, p))
        return fail(VIE_EUNSUPPORTED, "dense top-k: V = %lld rows of %d bytes exceed one pass's slab", (long long)V,
                    row_bytes);
    const int pass = dense_pass(B);
    const int nbw = B < pass ? B : pass;
    float *zbuf = static_cast<float *>(ws);
    uint64_t *tops = reinterpret_cast<uint64_t *>(static_cast<char *>(ws) +
                                                   (((size_t)nbw * V * 4 + 255) & ~(size_t)255));
    const char *hb = static_cast<const char *>(h);
    if (use_mfma(dtype, d, B, W, h)) {
        const DensePlan mp = mfma_plan(V);
        for (int q0 = 0; q0 < B; q0 += kMfmaMaxNB) {
            const int nq = B - q0 < kMfmaMaxNB ? B - q0 : kMfmaMaxNB;
            const char *hp = hb + (int64_t)q0 * row_bytes;
            int32_t *ip = ids + (int64_t)q0 * k;
            float *lp = logits + (int64_t)q0 * k;
            hipError_t e =
                nq <= 16   ? mfma_launch<1, VIE_MFMA_KC1, VIE_MFMA_LA1>(W, V, d, hp, nq, k, mp, zbuf, tops, ip, lp, s)
                : nq <= 32 ? mfma_launch<2, VIE_MFMA_KC2, VIE_MFMA_LA2>(W, V, d, hp, nq, k, mp, zbuf, tops, ip, lp, s)
                           : mfma_launch<4, VIE_MFMA_KC4, VIE_MFMA_LA4>(W, V, d, hp, nq, k, mp, zbuf, tops, ip, lp, s);
            if (e != hipSuccess) return launched(e, "dense top-k (matrix cores) launch");
        }
        return VIE_OK;
    }
    const int vec = pick_vec(row_bytes, W);
    const bool bf = dtype == VIE_BF16;
    for (int q0 = 0; q0 < B; q0 += p.nbmax) {
        const int nq = B - q0 < p.nbmax ? B - q0 : p.nbmax;
        const int nb = nq == 1 ? 1 : nq == 2 ? 2 : nq <= 4 ? 4 : 8;
        const char *hp = hb + (int64_t)q0 * row_bytes;
        int32_t *ip = ids + (int64_t)q0 * k;
        float *lp = logits + (int64_t)q0 * k;
        hipError_t e;
        const int cpl = stream_cpl(row_bytes, nb);
        if (vec == 16 && nb <= 2 && cpl && (uintptr_t)hp % 16 == 0)
            e = bf ? stream_launch_cpl<true>(cpl, nb, W, V, row_bytes, hp, nq, k, p, zbuf, tops, ip, lp, s)
                   : stream_launch_cpl<false>(cpl, nb, W, V, row_bytes, hp, nq, k, p, zbuf, tops, ip, lp, s);
        else if (vec == 16)
            e = bf ? dense_launch_nb<16, true>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, tops, ip, lp, s)
                   : dense_launch_nb<16, false>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, tops, ip, lp, s);
        else if (vec == 8)
            e = bf ? dense_launch_nb<8, true>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, tops, ip, lp, s)
                   : dense_launch_nb<8, false>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, tops, ip, lp, s);
        else if (vec == 4)
            e = bf ? dense_launch_nb<4, true>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, tops, ip, lp, s)
                   : dense_launch_nb<4, false>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, tops, ip, lp, s);
        else
            e = dense_launch_nb<2, true>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, tops, ip, lp, s);
        if (e != hipSuccess) return launched(e, "dense top-k launch");
    }
    return VIE_OK;
}

// ---------------------------------------------------------------------------
// the dense head's workspace for callers that cannot allocate
// ---------------------------------------------------------------------------
//
// One array per GPU, held by the loaded library until the process ends.  On
// the host its name is a stand-in, not a device address: host code passes
// only the address hipGetSymbolAddress returns on each device.  Calls that
// use it on one GPU share it and must not overlap in time.

constexpr size_t kScratchBytes = size_t(16) << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kScratchDevices];  // device address of scratch, per device (set on first use)
}  // namespace

size_t dense_scratch_bytes() { return kScratchBytes; }

vie_status dense_scratch(void **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(VIE_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kScratchDevices)
        return fail(VIE_EUNSUPPORTED, "device %d: the static workspace serves devices 0..%d", dev,
                    kScratchDevices - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(VIE_EHIP, "hipGetSymbolAddress of the static workspace: %s", hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return VIE_OK;
}

size_t hnsw_lds_bytes(int64_t V, int d, int dtype, int ef_eff, int M0, int M)
{
    const int row_bytes = d * elem_bytes(dtype);
    const size_t hbytes = (size_t)((row_bytes + 15) & ~15);
    const size_t maxdeg = (size_t)(M0 > M ? M0 : M);
    size_t n = hbytes + (size_t)ef_eff * 8 * 2 + maxdeg * (8 + 4) + (size_t)ef_eff * 2;
    n = (n + 15) & ~(size_t)15;
    return n + (size_t)((V + 31) / 32) * 4;
}

size_t hnsw_multi_lds_bytes(int64_t V, int d, int dtype, int ef_eff, int M0, int M, int width, bool q8, int team,
                            int share)
{
    const int row_bytes = d * elem_bytes(dtype);
    const size_t hbytes = (size_t)((row_bytes + 15) & ~15);
    const size_t cap = (size_t)width * M0, nid = cap > (size_t)M ? cap : (size_t)M;
    const size_t capk = (cap + 127) & ~(size_t)127;
    size_t n = hbytes + (size_t)ef_eff * 8 * 2 + capk * 8 + nid * 4 + (team == 1 ? cap * 4 : 0) +
               (share > 1 ? cap * 4 : 0);
    n = ((n + 7) & ~(size_t)7) + 2 * (((size_t)ef_eff + 7) & ~(size_t)7);  // 8-aligned flag arrays
    n = (n + 15) & ~(size_t)15;
    if (q8) n += (size_t)((d + 15) & ~15);
    if (share > 1) n += (size_t)share * (q8 ? (size_t)((d + 15) & ~15) : hbytes);  // the group's queries
    return n + (size_t)((V + 31) / 32) * 4;
}

// LDS a search workgroup may take for its dynamic carve-up: the device's
// per-block limit less a reserve for the kernels' static variables (2.2 KB
// in hnsw_multi_kernel: shared counters, picks, cache ids and the offsets of
// up to kMaxTeam members' keys).
size_t hnsw_lds_limit()
{
    constexpr int kStaticReserve = 3072;
    static_assert((kMaxTeam + 1) * 4 + 1280 <= kStaticReserve, "team offsets fit the static reserve");
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 64 * 1024 - kStaticReserve;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= kStaticReserve)
        return 64 * 1024 - kStaticReserve;
    return (size_t)(v - kStaticReserve);
}

namespace {
__global__ void team_clear_kernel(uint64_t *__restrict__ tags, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) tags[i] = 0ull;
}

// Keys a member passes at one exchange: the most new nodes of a step, or a
// whole beam (the final re-rank).
int team_slot(const HnswLaunch &a) { return std::max(a.width * a.M0, a.ef_eff); }

size_t round256(size_t n) { return (n + 255) & ~(size_t)255; }

// The team workspace: keys [B][3][team][slot] u64, then the published
// counts [B][3][team] u64, each 256-byte aligned.
TeamArgs team_layout(void *ws, int B, int team, int slot)
{
    char *p = static_cast<char *>(ws);
    TeamArgs t;
    t.size = team;
    t.slot = slot;
    t.keys = reinterpret_cast<uint64_t *>(p);
    p += round256((size_t)B * 3 * team * slot * 8);
    t.tags = reinterpret_cast<uint64_t *>(p);
    return t;
}
}  // namespace

size_t hnsw_team_workspace_bytes(const HnswLaunch &a)
{
    if (a.team <= 1) return 0;
    const int slot = team_slot(a);
    return round256((size_t)a.B * 3 * a.team * slot * 8) + round256((size_t)a.B * 3 * a.team * 8);
}

namespace {
constexpr uint64_t kShareMagic = 0x5645534841524531ull;  // marks a row-sharing workspace as cleared

// The row-sharing workspace: a 256-byte header (magic word, epoch), the
// queries in the kernel's layout [B][hbytes], their int8 form [B][d] and
// scales [B] (int8 walks), then the score table [B][V] u64, each part
// 256-byte aligned.
struct ShareLayout {
    uint64_t *magic;
    uint32_t *epoch;
    char *hq;
    int8_t *hq8;
    float *hscale;
    uint64_t *table;
    size_t clear_bytes;  // from hq to the end
};

ShareLayout share_layout(void *ws, const HnswLaunch &a)
{
    char *p = static_cast<char *>(ws);
    ShareLayout l;
    l.magic = reinterpret_cast<uint64_t *>(p);
    l.epoch = reinterpret_cast<uint32_t *>(p + 8);
    p += 256;
    const size_t hbytes = (size_t)((a.d * elem_bytes(a.dtype) + 15) & ~15);
    l.hq = p;
    p += round256((size_t)a.B * hbytes);
    l.hq8 = reinterpret_cast<int8_t *>(p);
    p += a.q8 ? round256((size_t)a.B * a.d) : 0;
    l.hscale = reinterpret_cast<float *>(p);
    p += a.q8 ? round256((size_t)a.B * 4) : 0;
    l.table = reinterpret_cast<uint64_t *>(p);
    p += round256((size_t)a.B * a.V * 8);
    l.clear_bytes = (size_t)(p - l.hq);
    return l;
}

// Zeroes the workspace (past the header) unless its magic word says a
// previous call did; every workgroup reads the word first.
__global__ void share_clear_kernel(const uint64_t *__restrict__ magic, uint4 *__restrict__ body, size_t n16)
{
    if (*magic == kShareMagic) return;
    const uint4 z = {0u, 0u, 0u, 0u};
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
        body[i] = z;
}

// One thread: marks the workspace cleared and moves to the next epoch (an
// epoch that wraps to 0 starts again at 1 and drops the mark, so that the
// next call clears the table).
__global__ void share_epoch_kernel(uint64_t *__restrict__ magic, uint32_t *__restrict__ epoch)
{
    uint32_t e = *magic == kShareMagic ? *epoch + 1u : 1u;
    uint64_t m = kShareMagic;
    if (e == 0u) {
        e = 1u;
        m = 0ull;
    }
    *epoch = e;
    *magic = m;
}

// The queries in the kernel's layout (rows of hbytes, zero padded).
__global__ void share_copy_kernel(const char *__restrict__ h, int row_bytes, int hbytes, char *__restrict__ hq)
{
    const int64_t b = blockIdx.x;
    for (int i = threadIdx.x; i < hbytes; i += blockDim.x) hq[b * hbytes + i] = i < row_bytes ? h[b * row_bytes + i] : 0;
}

// The kernels that prepare a row-sharing search, on stream s.
hipError_t share_prepare(const HnswLaunch &a, const ShareLayout &l, hipStream_t s)
{
    const size_t n16 = l.clear_bytes / 16;
    share_clear_kernel<<<1024, 256, 0, s>>>(l.magic, reinterpret_cast<uint4 *>(l.hq), n16);
    share_epoch_kernel<<<1, 1, 0, s>>>(l.magic, l.epoch);
    const int row_bytes = a.d * elem_bytes(a.dtype);
    share_copy_kernel<<<a.B, 256, 0, s>>>(static_cast<const char *>(a.h), row_bytes, (row_bytes + 15) & ~15, l.hq);
    if (a.q8) {
        const int grid = (a.B + kQuantWaves - 1) / kQuantWaves;
        if (a.dtype == VIE_BF16)
            quantize_kernel<true><<<grid, kQuantWaves * kWave, 0, s>>>(a.h, a.B, a.d, l.hq8, l.hscale);
        else
            quantize_kernel<false><<<grid, kQuantWaves * kWave, 0, s>>>(a.h, a.B, a.d, l.hq8, l.hscale);
    }
    return hipGetLastError();
}
}  // namespace

size_t hnsw_share_workspace_bytes(int B, int64_t V, int d, int dtype, bool q8, int share)
{
    if (share <= 1) return 0;
    const size_t hbytes = (size_t)((d * elem_bytes(dtype) + 15) & ~15);
    return 256 + round256((size_t)B * hbytes) + (q8 ? round256((size_t)B * d) + round256((size_t)B * 4) : 0) +
           round256((size_t)B * V * 8);
}

namespace {
template <int NT, int VEC, bool BF16, int G>
hipError_t hnsw_launch(const HnswLaunch &a, size_t lds, hipStream_t s)
{
    if (a.width > 1 || a.q8 || a.team > 1 || a.share > 1) {
        auto kern = a.share > 1 ? (a.q8 ? hnsw_multi_kernel<NT, VEC, BF16, G, true, true>
                                        : hnsw_multi_kernel<NT, VEC, BF16, G, false, true>)
                                : (a.q8 ? hnsw_multi_kernel<NT, VEC, BF16, G, true, false>
                                        : hnsw_multi_kernel<NT, VEC, BF16, G, false, false>);
        if (lds > 64 * 1024) {
            hipError_t e =
                hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            if (e != hipSuccess) return e;
        }
        TeamArgs team{1, 0, nullptr, nullptr};
        if (a.team > 1) {
            // every member of every query must be resident at once
            int per = 0, dev = 0, cus = 0;
            hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kern, NT, lds);
            if (e == hipSuccess) e = hipGetDevice(&dev);
            if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
            if (e != hipSuccess) return e;
            if ((int64_t)per * cus < (int64_t)a.B * a.team) return hipErrorCooperativeLaunchTooLarge;
            team = team_layout(a.team_ws, a.B, a.team, team_slot(a));
            const int ntag = a.B * 3 * a.team;
            team_clear_kernel<<<(ntag + 255) / 256, 256, 0, s>>>(team.tags, ntag);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        ShareArgs share{1, a.B, nullptr, nullptr, nullptr, nullptr, nullptr};
        if (a.share > 1) {
            const ShareLayout l = share_layout(a.share_ws, a);
            hipError_t e = share_prepare(a, l, s);
            if (e != hipSuccess) return e;
            share = ShareArgs{a.share, a.B, l.table, l.epoch, l.hq, l.hq8, l.hscale};
        }
        kern<<<a.B * team.size, NT, lds, s>>>(static_cast<const char *>(a.W), a.V, a.d * elem_bytes(a.dtype), a.adj0,
                                               a.M0, a.upper_off, a.upper, a.M, a.maxlevel, a.entry,
                                               static_cast<const char *>(a.h), a.k, a.ef_eff, a.width, a.ids,
                                               a.logits, a.ldo, a.stats, a.q8, a.q8scale, a.trace, a.trace_cap,
                                               team, share);
        return hipGetLastError();
    }
    auto kern = hnsw_kernel<NT, VEC, BF16, G>;
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    kern<<<a.B, NT, lds, s>>>(static_cast<const char *>(a.W), a.V, a.d * elem_bytes(a.dtype), a.adj0, a.M0,
                               a.upper_off, a.upper, a.M, a.maxlevel, a.entry, static_cast<const char *>(a.h), a.k,
                               a.ef_eff, a.ids, a.logits, a.ldo, a.stats, a.trace, a.trace_cap);
    return hipGetLastError();
}

// Lanes per row: the fewest (16, 32 or 64) that cover a row in the
// register-held chunks per lane, so as many rows as possible load at once.
// Workgroup size: 1024 threads (the most rows in flight for one query) for
// small batches; 256 when the batch alone fills the GPU.
template <int VEC, bool BF16>
hipError_t hnsw_launch_g(const HnswLaunch &a, size_t lds, hipStream_t s)
{
    const int nchunk = a.d * elem_bytes(a.dtype) / VEC;
    constexpr int CPL = RowCpl<BF16>::value;
    // 1024-thread workgroups at every batch size: measured against 256-thread
    // ones for batches of 256 and 1024 queries they were as fast or faster
    // in every configuration (a 256-thread workgroup whose LDS fills half a
    // CU leaves it four or eight waves)
    if (nchunk <= 16 * CPL) return hnsw_launch<kHnswThreads, VEC, BF16, 16>(a, lds, s);
    if (nchunk <= 32 * CPL) return hnsw_launch<kHnswThreads, VEC, BF16, 32>(a, lds, s);
    return hnsw_launch<kHnswThreads, VEC, BF16, 64>(a, lds, s);
}
}  // namespace

namespace {
template <int VEC, bool BF16>
hipError_t forced_launch_g(const HnswLaunch &a, const int32_t *forced, int n, size_t lds, hipStream_t s)
{
    const int row_bytes = a.d * elem_bytes(a.dtype);
    const int nchunk = row_bytes / VEC;
    constexpr int CPL = RowCpl<BF16>::value;
    const char *W = static_cast<const char *>(a.W);
    const char *h = static_cast<const char *>(a.h);
    if (nchunk <= 16 * CPL)
        forced_kernel<VEC, BF16, 16><<<a.B, kForcedThreads, lds, s>>>(W, a.V, row_bytes, h, forced, n, a.k, a.ids,
                                                                        a.logits);
    else if (nchunk <= 32 * CPL)
        forced_kernel<VEC, BF16, 32><<<a.B, kForcedThreads, lds, s>>>(W, a.V, row_bytes, h, forced, n, a.k, a.ids,
                                                                        a.logits);
    else
        forced_kernel<VEC, BF16, 64><<<a.B, kForcedThreads, lds, s>>>(W, a.V, row_bytes, h, forced, n, a.k, a.ids,
                                                                        a.logits);
    return hipGetLastError();
}
}  // namespace

vie_status launch_forced(const HnswLaunch &a, const int32_t *forced, int n, hipStream_t s)
{
    const int row_bytes = a.d * elem_bytes(a.dtype);
    const size_t lds = (size_t)((row_bytes + 15) & ~15) + (((size_t)a.k * 4 + 7) & ~(size_t)7) +
                       (size_t)(a.k + n) * 8;
    if (lds > 64 * 1024) return fail(VIE_EUNSUPPORTED, "forced tokens: k + n too large for one workgroup");
    const int vec = pick_vec(row_bytes, a.W);
    const bool bf = a.dtype == VIE_BF16;
    hipError_t e;
    if (vec == 16) e = bf ? forced_launch_g<16, true>(a, forced, n, lds, s) : forced_launch_g<16, false>(a, forced, n, lds, s);
    else if (vec == 8) e = bf ? forced_launch_g<8, true>(a, forced, n, lds, s) : forced_launch_g<8, false>(a, forced, n, lds, s);
    else if (vec == 4) e = bf ? forced_launch_g<4, true>(a, forced, n, lds, s) : forced_launch_g<4, false>(a, forced, n, lds, s);
    else e = forced_launch_g<2, true>(a, forced, n, lds, s);
    return launched(e, "forced-token launch");
}

vie_status launch_quantize_rows(const void *W, int dtype, int64_t V, int d, int8_t *q, float *scale, hipStream_t s)
{
    const unsigned grid = (unsigned)((V + kQuantWaves - 1) / kQuantWaves);
    if (dtype == VIE_BF16) quantize_kernel<true><<<grid, kQuantWaves * kWave, 0, s>>>(W, V, d, q, scale);
    else quantize_kernel<false><<<grid, kQuantWaves * kWave, 0, s>>>(W, V, d, q, scale);
    return launched(hipGetLastError(), "row quantization launch");
}

vie_status launch_hnsw_search(const HnswLaunch &a, hipStream_t s)
{
    if (a.width < 1 || a.width > kMaxWidth)
        return fail(VIE_EUNSUPPORTED, "HNSW search: expansion width %d outside 1..%d", a.width, kMaxWidth);
    if (a.team < 1 || a.team > kMaxTeam || (a.team & (a.team - 1)))
        return fail(VIE_EUNSUPPORTED, "HNSW search: team of %d workgroups is not a power of two in 1..%d", a.team,
                    kMaxTeam);
    if (a.team > 1 && !a.team_ws) return fail(VIE_EINVAL, "a team search needs its workspace");
    if (a.share < 1 || a.share > kMaxShare || (a.share & (a.share - 1)))
        return fail(VIE_EUNSUPPORTED, "HNSW search: row-sharing groups of %d queries (not a power of two up to %d)",
                    a.share, kMaxShare);
    if (a.share > 1 && (a.team > 1 || !a.share_ws))
        return fail(VIE_EINVAL, "row sharing needs its workspace and one workgroup per query");
    const bool multi = a.width > 1 || a.q8 || a.team > 1 || a.share > 1;
    const size_t lds = multi ? hnsw_multi_lds_bytes(a.V, a.d, a.dtype, a.ef_eff, a.M0, a.M, a.width, a.q8, a.team, a.share)
                             : hnsw_lds_bytes(a.V, a.d, a.dtype, a.ef_eff, a.M0, a.M);
    const size_t lim = hnsw_lds_limit();
    if (lds > lim)
        return fail(VIE_EUNSUPPORTED, "HNSW search needs %zu bytes of LDS per workgroup; the device allows %zu", lds,
                    lim);
    if (a.M0 > 256 || a.M > 256) return fail(VIE_EUNSUPPORTED, "HNSW search: degree caps above 256");
    if (a.q8 && a.d % 16 != 0) return fail(VIE_EUNSUPPORTED, "int8 rows need d divisible by 16 (d = %d)", a.d);
    const int row_bytes = a.d * elem_bytes(a.dtype);
    const int vec = pick_vec(row_bytes, a.W);
    const bool bf = a.dtype == VIE_BF16;
    hipError_t e;
    if (vec == 16) e = bf ? hnsw_launch_g<16, true>(a, lds, s) : hnsw_launch_g<16, false>(a, lds, s);
    else if (vec == 8) e = bf ? hnsw_launch_g<8, true>(a, lds, s) : hnsw_launch_g<8, false>(a, lds, s);
    else if (vec == 4) e = bf ? hnsw_launch_g<4, true>(a, lds, s) : hnsw_launch_g<4, false>(a, lds, s);
    else e = hnsw_launch_g<2, true>(a, lds, s);
    if (e == hipErrorCooperativeLaunchTooLarge)
        return fail(VIE_EUNSUPPORTED, "a team of %d workgroups for each of %d queries does not fit on the device at once",
                    a.team, a.B);
    return launched(e, "HNSW search launch");
}

}  // namespace vie
