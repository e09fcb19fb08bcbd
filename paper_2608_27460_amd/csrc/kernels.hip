// gfx950 (CDNA4) kernels of the vector-index output head.
//
//   scatter_kernel     Section 3: full-vocabulary logits, -inf except the
//                      retrieved ids.
//   dense_topk_kernel  exact head z = W_out h fused with top-k (Section 3;
//                      the dense baseline of Section 4.1).
//   hnsw_kernel        HNSW k-NN search (Sections 2-3; Malkov & Yashunin
//                      Algorithms 2 and 5), one workgroup per query.
//
// Ordering: a candidate is the 64-bit key (ord(logit) << 32) | ~id, where
// ord() maps fp32 to an unsigned integer of the same order.  A larger key is
// a better candidate: larger logit first, smaller id first on equal logits.
// That is the (dist, id) order of the search with dist = -logit.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "index.hpp"

namespace vie {

namespace {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// keys
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t f2ord(float f)
{
    const uint32_t u = __float_as_uint(f == 0.0f ? 0.0f : f);  // -0 -> +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float ord2f(uint32_t o)
{
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

__device__ __forceinline__ uint64_t make_key(float logit, int32_t id)
{
    return ((uint64_t)f2ord(logit) << 32) | (uint64_t)(~(uint32_t)id);
}

__device__ __forceinline__ int32_t key_id(uint64_t k) { return (int32_t)(~(uint32_t)k); }
__device__ __forceinline__ float key_logit(uint64_t k) { return ord2f((uint32_t)(k >> 32)); }

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

__device__ __forceinline__ float dot_word(uint32_t w, uint32_t h, float acc, bool bf16)
{
    if (bf16)
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w), __builtin_bit_cast(bf16x2_t, h),
                                               acc, false);
    return fmaf(__uint_as_float(w), __uint_as_float(h), acc);
}

template <int VEC, bool BF16>
__device__ __forceinline__ float dot_vec(typename Vec<VEC>::T w, typename Vec<VEC>::T h, float acc)
{
    if constexpr (VEC == 16) {
        acc = dot_word(w.x, h.x, acc, BF16);
        acc = dot_word(w.y, h.y, acc, BF16);
        acc = dot_word(w.z, h.z, acc, BF16);
        acc = dot_word(w.w, h.w, acc, BF16);
    } else if constexpr (VEC == 8) {
        acc = dot_word(w.x, h.x, acc, BF16);
        acc = dot_word(w.y, h.y, acc, BF16);
    } else if constexpr (VEC == 4) {
        acc = dot_word(w, h, acc, BF16);
    } else {  // one bf16
        acc = fmaf(__uint_as_float((uint32_t)w << 16), __uint_as_float((uint32_t)h << 16), acc);
    }
    return acc;
}

// Partial dot of row `row` (row_bytes bytes at W) by the G lanes of a group:
// lane `gl` covers chunks gl, gl + G, ... of VEC bytes.  Reduced over the
// group with xor shuffles; every lane of the group returns the full sum.
template <int VEC, bool BF16, int G, bool STREAM = false>
__device__ __forceinline__ float group_row_dot(const char *__restrict__ W, int64_t row, int row_bytes,
                                               const char *hs, int gl)
{
    typedef typename Vec<VEC>::T T;
    const T *w = reinterpret_cast<const T *>(W + row * (int64_t)row_bytes);
    const T *h = reinterpret_cast<const T *>(hs);
    const int nchunk = row_bytes / VEC;
    float acc = 0.0f;
#pragma unroll 4
    for (int c = gl; c < nchunk; c += G)
        acc = dot_vec<VEC, BF16>(STREAM ? __builtin_nontemporal_load(w + c) : w[c], h[c], acc);
#pragma unroll
    for (int m = G / 2; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, G);
    return acc;
}

// ---------------------------------------------------------------------------
// block-wide helpers
// ---------------------------------------------------------------------------

// Inclusive prefix sum of v over the block (NT threads, NT / 64 waves).
template <int NT>
__device__ __forceinline__ uint32_t block_inclusive_scan(uint32_t v, uint32_t *s_wave)
{
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t t = __shfl_up(v, o, kWave);
        if (lane >= o) v += t;
    }
    if (lane == kWave - 1) s_wave[wave] = v;
    __syncthreads();
    uint32_t base = 0;
    for (int w = 0; w < wave; ++w) base += s_wave[w];
    __syncthreads();
    return v + base;
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
// dense_slab_kernel: workgroup w owns a contiguous slab of rows and streams it
// once.  Each wave takes U rows at a time; its 64 lanes read them with
// VEC-byte loads (U loads in flight per lane), accumulate in fp32 and reduce
// over the wave.  The slab writes its logits to the workspace and its
// largest key.
//
// dense_merge_kernel: one workgroup per query.  Any T at or below the k-th
// largest slab maximum is a lower bound of the k-th largest key overall (k
// distinct elements are >= T), so every key of the answer is >= T, and only
// the slabs whose maximum is >= T can hold one.  T comes from one radix pass
// over the maxima; the kernel gathers those slabs' keys >= T (typically
// little more than k) and orders them by rank.  The kernel boundary between the two launches is the only
// cross-workgroup synchronisation: no atomics across workgroups, no fences.

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
template <int N>
__device__ __forceinline__ float wave_sum_multi(float (&v)[N], int lane)
{
#pragma unroll
    for (int n = N, o = 32; n > 1; n >>= 1, o >>= 1) {
        const bool upper = lane & o;
#pragma unroll
        for (int i = 0; i < n / 2; ++i) {
            const float give = upper ? v[i] : v[i + n / 2];
            const float keep = upper ? v[i + n / 2] : v[i];
            v[i] = keep + __shfl_xor(give, o, kWave);
        }
    }
    float a = v[0];
#pragma unroll
    for (int o = 32 / N; o >= 1; o >>= 1) a += __shfl_xor(a, o, kWave);
    return a;
}

template <int N> struct Log2 { static constexpr int value = 1 + Log2<N / 2>::value; };
template <> struct Log2<1> { static constexpr int value = 0; };

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint64_t t = __shfl_xor(v, o, kWave);
        v = t > v ? t : v;
    }
    return v;
}

template <int VEC, bool BF16, int NB>
__global__ __launch_bounds__(kDenseThreads) __attribute__((amdgpu_waves_per_eu(NB == 1 ? 8 : 4))) void
dense_slab_kernel(const char *__restrict__ W, int64_t V, int row_bytes, const char *__restrict__ hq, int nq,
                  int rows_per_wg, float *__restrict__ zout, uint64_t *__restrict__ maxes)
{
    extern __shared__ __align__(16) char smem[];
    __shared__ unsigned long long s_max[kDenseMaxNB];
    constexpr int U = NB >= 8 ? 2 : VIE_DENSE_ROWS;  // rows in flight per wave
    constexpr int NV = NB * U;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int nwg = gridDim.x;
    const int hbytes = (row_bytes + 15) & ~15;
    char *hs = smem;                                                   // [NB][hbytes]
    float *z = reinterpret_cast<float *>(smem + (size_t)NB * hbytes);  // [NB][rows_per_wg]

    // queries into LDS (bytewise: rows need not be 4-byte aligned), zero padded
    for (int i = tid; i < NB * hbytes; i += kDenseThreads) {
        const int q = i / hbytes, c = i - q * hbytes;
        hs[i] = (q < nq && c < row_bytes) ? hq[(int64_t)q * row_bytes + c] : 0;
    }
    if (tid < kDenseMaxNB) s_max[tid] = 0ull;
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
        float acc[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) acc[v] = 0.0f;
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
        const float total = wave_sum_multi<NV>(acc, lane);
        constexpr int lg = 6 - Log2<NV>::value;
        if ((lane & ((1 << lg) - 1)) == 0) {
            const int v = lane >> lg, q = v / U, u = v % U;
            if (rb + u < nrows) z[q * rows_per_wg + rb + u] = total;
        }
    }
    __syncthreads();

    // the slab's logits (coalesced) and its largest key, per query
    for (int q = 0; q < nq; ++q) {
        const float *zq = z + q * rows_per_wg;
        float *oq = zout + (int64_t)q * V + r0;
        uint64_t best = 0ull;
        for (int i = tid; i < nrows; i += kDenseThreads) {
            oq[i] = zq[i];
            const uint64_t key = make_key(zq[i], (int32_t)(r0 + i));
            best = key > best ? key : best;
        }
        best = wave_max_u64(best);
        if (lane == 0) atomicMax(&s_max[q], (unsigned long long)best);
    }
    __syncthreads();
    if (tid < nq) maxes[(int64_t)tid * nwg + blockIdx.x] = s_max[tid];
}

__global__ __launch_bounds__(kMergeThreads) void dense_merge_kernel(const float *__restrict__ zbuf,
                                                                     const uint64_t *__restrict__ maxes, int64_t V,
                                                                     int rows_per_wg, int nwg, int k,
                                                                     int32_t *__restrict__ ids,
                                                                     float *__restrict__ logits)
{
    __shared__ uint32_t hist[256];
    __shared__ uint64_t gat[kMergeGather];
    __shared__ int cand[kMergeThreads];
    __shared__ uint32_t s_nc, s_n;
    __shared__ unsigned long long s_T, s_and, s_or;
    const int tid = threadIdx.x, q = blockIdx.x;
    const float *zq = zbuf + (int64_t)q * V;

    // 1. slab maxima and a lower bound T of their k-th largest: one radix
    //    pass on the first 8 bits where the maxima differ; T is the lower
    //    edge of the bucket that holds the k-th largest.  The slabs whose
    //    maximum is >= T are the only ones that can hold an answer (fewer
    //    than k slabs: T = 0, every slab).
    const uint64_t m = tid < nwg ? maxes[(int64_t)q * nwg + tid] : 0ull;
    if (tid < 256) hist[tid] = 0u;
    if (tid == 0) {
        s_nc = 0;
        s_n = 0;
        s_T = 0ull;
        s_and = ~0ull;
        s_or = 0ull;
    }
    __syncthreads();
    if (nwg >= k) {
        uint64_t a = tid < nwg ? m : ~0ull, o = m;
#pragma unroll
        for (int x = 32; x >= 1; x >>= 1) {
            a &= __shfl_xor(a, x, kWave);
            o |= __shfl_xor(o, x, kWave);
        }
        if ((tid & (kWave - 1)) == 0) {
            atomicAnd(&s_and, (unsigned long long)a);
            atomicOr(&s_or, (unsigned long long)o);
        }
        __syncthreads();
        const uint64_t common = s_and, diff = s_and ^ s_or;  // diff != 0: maxima are distinct
        const int top = 63 - __clzll((long long)diff);
        const int sh = top >= 7 ? top - 7 : 0;
        if (tid < nwg) atomicAdd(&hist[(m >> sh) & 255u], 1u);
        __syncthreads();
        if (tid < kWave) {  // wave 0: the bucket holding the k-th largest
            const int lane = tid;
            uint32_t c[4], sum = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                c[j] = hist[255 - 4 * lane - j];
                sum += c[j];
            }
            uint32_t incl = sum;
#pragma unroll
            for (int x = 1; x < kWave; x <<= 1) {
                const uint32_t t = __shfl_up(incl, x, kWave);
                if (lane >= x) incl += t;
            }
            uint32_t above = incl - sum;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (above < (uint32_t)k && (uint32_t)k <= above + c[j]) {
                    const uint64_t hi = sh + 8 >= 64 ? 0ull : (common & (~0ull << (sh + 8)));
                    s_T = hi | ((uint64_t)(255 - 4 * lane - j) << sh);
                }
                above += c[j];
            }
        }
        __syncthreads();
    }
    const uint64_t T = s_T;
    if (tid < nwg && m >= T) cand[atomicAdd(&s_nc, 1u)] = tid;
    __syncthreads();
    const int nc = (int)s_nc;

    // 2. gather the keys >= T of those slabs
    for (int i = tid; i < nc * rows_per_wg; i += kMergeThreads) {
        const int c = i / rows_per_wg;
        const int64_t row = (int64_t)cand[c] * rows_per_wg + (i - c * rows_per_wg);
        if (row < V) {
            const uint64_t key = make_key(zq[row], (int32_t)row);
            if (key >= T) {
                const uint32_t slot = atomicAdd(&s_n, 1u);
                if (slot < (uint32_t)kMergeGather) gat[slot] = key;
            }
        }
    }
    __syncthreads();
    const int n = (int)s_n;

    if (n <= kMergeGather) {
        // 3. order by rank: key t lands at its rank if that is below k
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
    // 3'. too many keys >= T (e.g. many equal logits): the k-th largest of
    //     the gathered range by bisection on the key, then order by rank
    //     among the ones above it (a slow path for degenerate inputs only).
    __shared__ unsigned long long s_cnt;
    uint64_t lo = T, hi = ~0ull;  // invariant: count(>= lo) >= k, count(>= hi + 1) < k
    while (lo < hi) {
        const uint64_t mid = lo + (hi - lo + 1) / 2;
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
// node this step inserts.  Both layer-0 lists are fetched during this step's
// row loads (the second with spare threads, each new node's by the group
// that scores its row), so the next step finds its list in LDS.  The beam is
// double buffered (merge from one buffer into the other).

struct HnswShared {
    unsigned long long best;
    uint32_t nnew, nkeep;
    uint32_t first, second, nbeam;
    int32_t pfa_id, pfb_id;  // nodes whose layer-0 lists sit in pfa[] / pfb[]
};

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

// Row chunks per lane held in registers (fp32 rows: 4, which avoids the
// register spills 8 causes there).
template <bool BF16> struct RowCpl { static constexpr int value = BF16 ? 8 : 4; };

// <row, h> by the G lanes of a group (lane gl of the group covers chunks gl,
// gl + G, ...): up to RowCpl chunks per lane are loaded before any is used.
// Every lane of the group returns the sum.
template <int VEC, bool BF16, int G>
__device__ __forceinline__ float row_dot(const char *__restrict__ W, int64_t row, int row_bytes, const char *hs,
                                         int gl)
{
    typedef typename Vec<VEC>::T T;
    const T *w = reinterpret_cast<const T *>(W + row * (int64_t)row_bytes);
    const T *h = reinterpret_cast<const T *>(hs);
    const int nchunk = row_bytes / VEC;
    constexpr int CPL = RowCpl<BF16>::value;
    T buf[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        const int c = gl + i * G;
        if (c < nchunk) buf[i] = w[c];
    }
    float acc = 0.0f;
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        const int c = gl + i * G;
        if (c < nchunk) acc = dot_vec<VEC, BF16>(buf[i], h[c], acc);
    }
    for (int c = gl + CPL * G; c < nchunk; c += G) acc = dot_vec<VEC, BF16>(w[c], h[c], acc);
#pragma unroll
    for (int m = G / 2; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, G);
    return acc;
}

constexpr int kPfbPerLane = 4;       // a new node's list is prefetched when M0 <= 4 * G
constexpr int kHnswWideBatch = 256;  // batches below this get 1024-thread workgroups

template <int NT, int VEC, bool BF16, int G>
__global__ __launch_bounds__(NT) void hnsw_kernel(
    const char *__restrict__ W, int64_t V, int row_bytes, const int32_t *__restrict__ adj0, int M0,
    const int32_t *__restrict__ upper_off, const int32_t *__restrict__ upper, int M, int maxlevel, int32_t entry,
    const char *__restrict__ hq, int k, int ef, int32_t *__restrict__ ids, float *__restrict__ logits,
    uint32_t *__restrict__ stats)
{
    extern __shared__ __align__(16) char smem[];
    __shared__ HnswShared sh;
    constexpr int kGroups = NT / G;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int q = blockIdx.x;
    const int hbytes = (row_bytes + 15) & ~15;
    const int vwords = (int)((V + 31) / 32);
    const int maxdeg = M0 > M ? M0 : M;
    const bool pfb_on = M0 <= kPfbPerLane * G;
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
    uint64_t *csort = reinterpret_cast<uint64_t *>(p);
    p += (size_t)maxdeg * 8;
    int32_t *cid = reinterpret_cast<int32_t *>(p);
    p += (size_t)maxdeg * 4;
    int32_t *pfa = reinterpret_cast<int32_t *>(p);
    p += (size_t)M0 * 4;
    int32_t *pfb = reinterpret_cast<int32_t *>(p);
    p += (size_t)M0 * 4;
    uint8_t *flag = reinterpret_cast<uint8_t *>(p);
    p += (size_t)ef;
    uint8_t *flag2 = reinterpret_cast<uint8_t *>(p);
    p += (size_t)ef;
    uint32_t *vis = reinterpret_cast<uint32_t *>(((uintptr_t)p + 15) & ~(uintptr_t)15);

    const char *h = hq + (int64_t)q * row_bytes;
    for (int i = tid; i < hbytes; i += NT) hs[i] = i < row_bytes ? h[i] : 0;
    if (tid == 0) {
        sh.best = 0;
        sh.pfa_id = -1;
        sh.pfb_id = -1;
    }
    __syncthreads();

    const int gl = tid % G;
    const int grp = tid / G;
    uint32_t n_dist = 0, n_expand = 0;

    // score the entry point
    if (grp == 0) {
        const float s = row_dot<VEC, BF16, G>(W, entry, row_bytes, hs, gl);
        if (gl == 0) sh.best = make_key(s, entry);
    }
    __syncthreads();
    uint64_t cur = sh.best;
    n_dist = 1;

    // upper layers: SEARCH-LAYER with a result set of one (greedy)
    for (int lc = maxlevel; lc >= 1; --lc) {
        clear_bits(vis, vwords);
        __syncthreads();
        if (tid == 0) vis[key_id(cur) >> 5] |= 1u << (key_id(cur) & 31);
        for (;;) {
            const int32_t c = key_id(cur);
            if (tid == 0) sh.nnew = 0;
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

    // layer 0: beam of ef keys, sorted descending, with expanded flags,
    // double buffered (beam/flag -> beam2/flag2 -> beam/flag ...)
    clear_bits(vis, vwords);
    __syncthreads();
    if (tid == 0) {
        vis[key_id(cur) >> 5] |= 1u << (key_id(cur) & 31);
        beam[0] = cur;
        flag[0] = 0;
        sh.nbeam = 1;
        sh.first = 0;
    }
    __syncthreads();
    for (;;) {
        const uint32_t first = sh.first, nbeam = sh.nbeam;
        if (first >= nbeam) break;
        const int32_t c = key_id(beam[first]);
        const int32_t *lst = sh.pfa_id == c ? pfa : (sh.pfb_id == c ? pfb : nullptr);
        __syncthreads();
        if (tid == 0) {
            flag[first] = 1;
            sh.nnew = 0;
            sh.nkeep = 0;
            sh.second = 0xFFFFFFFFu;
            sh.best = 0;
        }
        ++n_expand;
        __syncthreads();
        // claim the unseen neighbours; find the next unexpanded entry after first
        for (int t = tid; t < M0; t += NT) {
            const int32_t e = lst ? lst[t] : adj0[(int64_t)c * M0 + t];
            if (e >= 0 && claim(vis, e)) cid[atomicAdd(&sh.nnew, 1u)] = e;
        }
        for (int i0 = (int)first + 1 + (tid & ~(kWave - 1)); i0 < (int)nbeam; i0 += NT) {
            const int i = i0 + lane;
            const uint64_t ball = __ballot(i < (int)nbeam && !flag[i]);
            if (ball && lane == 0) atomicMin(&sh.second, (uint32_t)(i0 + __ffsll((long long)ball) - 1));
        }
        __syncthreads();
        const int nn = (int)sh.nnew;
        n_dist += nn;
        const uint32_t second = sh.second;
        const int32_t ida = second < nbeam ? key_id(beam[second]) : -1;
        // spare threads fetch the second entry's list while the rows load
        int32_t pfv = -1;
        const int pft = tid - (NT - M0);  // the last M0 threads
        if (ida >= 0 && pft >= 0) pfv = adj0[(int64_t)ida * M0 + pft];
        const uint64_t worst = nbeam == (uint32_t)ef ? beam[nbeam - 1] : 0ull;
        uint64_t gbest = 0ull;  // best key this group scored, and its node's list
        int32_t glist[kPfbPerLane];
        for (int j = grp; j < nn; j += kGroups) {
            const int32_t e = cid[j];
            int32_t l[kPfbPerLane];
            if (pfb_on) {
#pragma unroll
                for (int u = 0; u < kPfbPerLane; ++u) {
                    const int t = gl + u * G;
                    l[u] = t < M0 ? adj0[(int64_t)e * M0 + t] : -1;
                }
            }
            const float s = row_dot<VEC, BF16, G>(W, e, row_bytes, hs, gl);
            const uint64_t key = make_key(s, e);
            if (gl == 0 && key > worst) ckey[atomicAdd(&sh.nkeep, 1u)] = key;
            if (key > gbest) {
                gbest = key;
#pragma unroll
                for (int u = 0; u < kPfbPerLane; ++u) glist[u] = l[u];
            }
        }
        if (gl == 0 && gbest > worst) atomicMax(&sh.best, (unsigned long long)gbest);
        __syncthreads();
        if (ida >= 0 && pft >= 0) pfa[pft] = pfv;
        const uint64_t bestnew = sh.best;
        if (pfb_on && bestnew != 0ull && gbest == bestnew) {
#pragma unroll
            for (int u = 0; u < kPfbPerLane; ++u) {
                const int t = gl + u * G;
                if (t < M0) pfb[t] = glist[u];
            }
        }
        if (tid == 0) {
            sh.pfa_id = ida;
            sh.pfb_id = pfb_on && bestnew != 0ull ? key_id(bestnew) : -1;
            sh.first = 0xFFFFFFFFu;
        }
        const int nk = (int)sh.nkeep;
        // order the kept keys (rank sort; keys are distinct)
        for (int j = tid; j < nk; j += NT) {
            const uint64_t key = ckey[j];
            int rank = 0;
            for (int t = 0; t < nk; ++t) rank += ckey[t] > key;
            csort[rank] = key;
        }
        __syncthreads();
        // merge beam (nbeam) and csort (nk) into beam2, keep the best ef; the
        // new first unexpanded entry is the best kept key or the old second
        const int total = min((int)nbeam + nk, ef);
        for (int j = tid; j < nk; j += NT) {
            const uint64_t key = csort[j];
            int lo = 0, hi = (int)nbeam;  // count beam keys > key
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (beam[mid] > key) lo = mid + 1; else hi = mid;
            }
            const int pos = lo + j;
            if (pos < total) {
                beam2[pos] = key;
                flag2[pos] = 0;
                if (j == 0) atomicMin(&sh.first, (uint32_t)pos);
            }
        }
        for (int i = tid; i < (int)nbeam; i += NT) {
            const uint64_t key = beam[i];
            int lo = 0, hi = nk;  // count new keys > key
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (csort[mid] > key) lo = mid + 1; else hi = mid;
            }
            const int pos = lo + i;
            if (pos < total) {
                beam2[pos] = key;
                flag2[pos] = flag[i];
                if (i == (int)second) atomicMin(&sh.first, (uint32_t)pos);
            }
        }
        if (tid == 0) sh.nbeam = (uint32_t)total;
        __syncthreads();
        uint64_t *tb = beam;
        beam = beam2;
        beam2 = tb;
        uint8_t *tf = flag;
        flag = flag2;
        flag2 = tf;
    }

    const int nb = (int)sh.nbeam;
    for (int t = tid; t < k; t += NT) {
        ids[(int64_t)q * k + t] = t < nb ? key_id(beam[t]) : -1;
        logits[(int64_t)q * k + t] = t < nb ? key_logit(beam[t]) : -__builtin_inff();
    }
    if (stats && tid == 0) {
        stats[2 * q] = n_dist;
        stats[2 * q + 1] = n_expand;
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

template <int VEC, bool BF16, int NB>
hipError_t dense_launch(const void *W, int64_t V, int row_bytes, const char *h, int nq, int k, const DensePlan &p,
                        float *zbuf, uint64_t *maxes, int32_t *ids, float *logits, hipStream_t s)
{
    const size_t lds = dense_lds(NB, row_bytes, p.rpw);
    auto kern = dense_slab_kernel<VEC, BF16, NB>;
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    kern<<<p.nwg, kDenseThreads, lds, s>>>(static_cast<const char *>(W), V, row_bytes, h, nq, p.rpw, zbuf, maxes);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dense_merge_kernel<<<nq, kMergeThreads, 0, s>>>(zbuf, maxes, V, p.rpw, p.nwg, k, ids, logits);
    return hipGetLastError();
}

template <int VEC, bool BF16>
hipError_t dense_launch_nb(int nb, const void *W, int64_t V, int row_bytes, const char *h, int nq, int k,
                           const DensePlan &p, float *zbuf, uint64_t *maxes, int32_t *ids, float *logits,
                           hipStream_t s)
{
    switch (nb) {
    case 1: return dense_launch<VEC, BF16, 1>(W, V, row_bytes, h, nq, k, p, zbuf, maxes, ids, logits, s);
    case 2: return dense_launch<VEC, BF16, 2>(W, V, row_bytes, h, nq, k, p, zbuf, maxes, ids, logits, s);
    case 4: return dense_launch<VEC, BF16, 4>(W, V, row_bytes, h, nq, k, p, zbuf, maxes, ids, logits, s);
    default: return dense_launch<VEC, BF16, 8>(W, V, row_bytes, h, nq, k, p, zbuf, maxes, ids, logits, s);
    }
}

}  // namespace

// Workspace: the logits [min(B, 8)][V] fp32 (256-byte padded), then the slab
// maxima [min(B, 8)][slabs] u64.
size_t dense_workspace_bytes(int64_t V, int d, int B, int k)
{
    (void)d;
    (void)k;
    const int nb = B < kDenseMaxNB ? B : kDenseMaxNB;
    return (((size_t)nb * V * 4 + 255) & ~(size_t)255) + (size_t)nb * dense_grid(V) * 8;
}

vie_status launch_dense_topk(const void *W, int dtype, int64_t V, int d, const void *h, int B, int k, int32_t *ids,
                             float *logits, void *ws, hipStream_t s)
{
    const int row_bytes = d * elem_bytes(dtype);
    DensePlan p;
    if (!dense_plan(V, row_bytes, p))
        return fail(VIE_EUNSUPPORTED, "dense top-k: V = %lld rows of %d bytes exceed one pass's slab", (long long)V,
                    row_bytes);
    const int nbw = B < kDenseMaxNB ? B : kDenseMaxNB;
    float *zbuf = static_cast<float *>(ws);
    uint64_t *maxes = reinterpret_cast<uint64_t *>(static_cast<char *>(ws) +
                                                   (((size_t)nbw * V * 4 + 255) & ~(size_t)255));
    const char *hb = static_cast<const char *>(h);
    const int vec = pick_vec(row_bytes, W);
    const bool bf = dtype == VIE_BF16;
    for (int q0 = 0; q0 < B; q0 += p.nbmax) {
        const int nq = B - q0 < p.nbmax ? B - q0 : p.nbmax;
        const int nb = nq == 1 ? 1 : nq == 2 ? 2 : nq <= 4 ? 4 : 8;
        const char *hp = hb + (int64_t)q0 * row_bytes;
        int32_t *ip = ids + (int64_t)q0 * k;
        float *lp = logits + (int64_t)q0 * k;
        hipError_t e;
        if (vec == 16)
            e = bf ? dense_launch_nb<16, true>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, maxes, ip, lp, s)
                   : dense_launch_nb<16, false>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, maxes, ip, lp, s);
        else if (vec == 8)
            e = bf ? dense_launch_nb<8, true>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, maxes, ip, lp, s)
                   : dense_launch_nb<8, false>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, maxes, ip, lp, s);
        else if (vec == 4)
            e = bf ? dense_launch_nb<4, true>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, maxes, ip, lp, s)
                   : dense_launch_nb<4, false>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, maxes, ip, lp, s);
        else
            e = dense_launch_nb<2, true>(nb, W, V, row_bytes, hp, nq, k, p, zbuf, maxes, ip, lp, s);
        if (e != hipSuccess) return launched(e, "dense top-k launch");
    }
    return VIE_OK;
}

size_t hnsw_lds_bytes(int64_t V, int d, int dtype, int ef_eff, int M0, int M)
{
    const int row_bytes = d * elem_bytes(dtype);
    const size_t hbytes = (size_t)((row_bytes + 15) & ~15);
    const size_t maxdeg = (size_t)(M0 > M ? M0 : M);
    size_t n = hbytes + (size_t)ef_eff * 8 * 2 + maxdeg * (8 + 8 + 4) + (size_t)M0 * 8 + (size_t)ef_eff * 2;
    n = (n + 15) & ~(size_t)15;
    return n + (size_t)((V + 31) / 32) * 4;
}

size_t hnsw_lds_limit()
{
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 64 * 1024;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0)
        return 64 * 1024;
    return (size_t)v;
}

namespace {
template <int NT, int VEC, bool BF16, int G>
hipError_t hnsw_launch(const HnswLaunch &a, size_t lds, hipStream_t s)
{
    auto kern = hnsw_kernel<NT, VEC, BF16, G>;
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    kern<<<a.B, NT, lds, s>>>(static_cast<const char *>(a.W), a.V, a.d * elem_bytes(a.dtype), a.adj0, a.M0,
                               a.upper_off, a.upper, a.M, a.maxlevel, a.entry, static_cast<const char *>(a.h), a.k,
                               a.ef_eff, a.ids, a.logits, a.stats);
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
    const bool wide = a.B < kHnswWideBatch;
    if (nchunk <= 16 * CPL)
        return wide ? hnsw_launch<1024, VEC, BF16, 16>(a, lds, s) : hnsw_launch<256, VEC, BF16, 16>(a, lds, s);
    if (nchunk <= 32 * CPL)
        return wide ? hnsw_launch<1024, VEC, BF16, 32>(a, lds, s) : hnsw_launch<256, VEC, BF16, 32>(a, lds, s);
    return wide ? hnsw_launch<1024, VEC, BF16, 64>(a, lds, s) : hnsw_launch<256, VEC, BF16, 64>(a, lds, s);
}
}  // namespace

vie_status launch_hnsw_search(const HnswLaunch &a, hipStream_t s)
{
    const size_t lds = hnsw_lds_bytes(a.V, a.d, a.dtype, a.ef_eff, a.M0, a.M);
    const size_t lim = hnsw_lds_limit();
    if (lds > lim)
        return fail(VIE_EUNSUPPORTED, "HNSW search needs %zu bytes of LDS per workgroup; the device allows %zu", lds,
                    lim);
    if (a.M0 > 256 || a.M > 256) return fail(VIE_EUNSUPPORTED, "HNSW search: degree caps above 256");
    const int row_bytes = a.d * elem_bytes(a.dtype);
    const int vec = pick_vec(row_bytes, a.W);
    const bool bf = a.dtype == VIE_BF16;
    hipError_t e;
    if (vec == 16) e = bf ? hnsw_launch_g<16, true>(a, lds, s) : hnsw_launch_g<16, false>(a, lds, s);
    else if (vec == 8) e = bf ? hnsw_launch_g<8, true>(a, lds, s) : hnsw_launch_g<8, false>(a, lds, s);
    else if (vec == 4) e = bf ? hnsw_launch_g<4, true>(a, lds, s) : hnsw_launch_g<4, false>(a, lds, s);
    else e = hnsw_launch_g<2, true>(a, lds, s);
    return launched(e, "HNSW search launch");
}

}  // namespace vie
