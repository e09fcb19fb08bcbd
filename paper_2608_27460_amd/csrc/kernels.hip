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

// Radix selection of the `need` largest of `n` distinct 64-bit keys, produced
// by key_at(i).  On return (every thread) s_sel->prefix / s_sel->shift
// describe the threshold: key i is selected iff
// (key >> shift) >= (prefix >> shift); exactly `need` keys qualify.
struct SelState {
    uint64_t prefix;
    int shift;
    int need;
    int done;
};

template <int NT, typename KeyAt>
__device__ void radix_select(int n, int need, KeyAt key_at, uint32_t *s_hist /*256*/, uint32_t *s_wave,
                             SelState *s_sel)
{
    const int tid = threadIdx.x;
    if (tid == 0) {
        s_sel->prefix = 0;
        s_sel->shift = 0;
        s_sel->need = need;
        s_sel->done = 0;
    }
    __syncthreads();
    for (int shift = 56; shift >= 0; shift -= 8) {
        const uint64_t prefix = s_sel->prefix;
        const int want = s_sel->need;
        const uint64_t hi_mask = shift == 56 ? 0ull : (~0ull << (shift + 8));
        for (int b = tid; b < 256; b += NT) s_hist[b] = 0;
        __syncthreads();
        for (int i = tid; i < n; i += NT) {
            const uint64_t key = key_at(i);
            if ((key & hi_mask) == prefix) atomicAdd(&s_hist[(key >> shift) & 255u], 1u);
        }
        __syncthreads();
        // suffix counts: digit 255 - t is handled by thread t
        const uint32_t c = tid < 256 ? s_hist[255 - tid] : 0u;
        const uint32_t incl = block_inclusive_scan<NT>(c, s_wave);
        if (tid < 256) {
            const uint32_t above = incl - c;  // keys with a larger digit
            if (above < (uint32_t)want && (uint32_t)want <= incl) {
                const uint32_t digit = 255 - tid;
                s_sel->prefix = prefix | ((uint64_t)digit << shift);
                s_sel->need = want - (int)above;
                s_sel->shift = shift;
                s_sel->done = (c == (uint32_t)(want - (int)above));
            }
        }
        __syncthreads();
        if (s_sel->done) break;
    }
}

__device__ __forceinline__ bool selected(uint64_t key, const SelState &s)
{
    return (key >> s.shift) >= (s.prefix >> s.shift);
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
// dense head: GEMV + fused top-k
// ---------------------------------------------------------------------------
//
// Workgroup w owns rows [w * rows_per_wg, ...) of W_out and streams them once
// with 16-lane row groups (VEC-byte loads, fp32 accumulation), keeping the
// logits of its rows in LDS.  It then radix-selects its own best
// min(k, rows) keys per query into the workspace.  The last workgroup to
// finish (ticket counter) selects the global top-k from those candidates,
// orders it and writes ids/logits.  The counter is left at zero.

constexpr int kDenseThreads = 512;
constexpr int kDenseGroup = 16;
constexpr int kDenseWgs = 512;   // workgroups per launch (two per CU on MI355X)
constexpr int kDenseMaxNB = 8;   // queries per pass
constexpr int kDenseMaxRows = 2048;

struct DenseShared {
    uint32_t hist[256];
    uint32_t wave[kDenseThreads / kWave];
    SelState sel;
    uint32_t count;
    int last;
};

template <typename T>
__device__ __forceinline__ T *align_up(char *p, size_t a)
{
    return reinterpret_cast<T *>(((uintptr_t)p + a - 1) & ~(uintptr_t)(a - 1));
}

template <int VEC, bool BF16, int NB>
__global__ __launch_bounds__(kDenseThreads) void dense_topk_kernel(
    const char *__restrict__ W, int64_t V, int row_bytes, const char *__restrict__ hq, int nq, int k,
    int rows_per_wg, uint64_t *__restrict__ cand, uint32_t *__restrict__ counter, int32_t *__restrict__ ids,
    float *__restrict__ logits)
{
    extern __shared__ __align__(16) char smem[];
    __shared__ DenseShared sh;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int nwg = gridDim.x;
    const int hbytes = (row_bytes + 15) & ~15;
    char *hs = smem;                                                  // [NB][hbytes]
    float *z = reinterpret_cast<float *>(smem + (size_t)NB * hbytes);  // [NB][rows_per_wg]

    // queries into LDS (bytewise: rows need not be 4-byte aligned), zero padded
    for (int i = tid; i < NB * hbytes; i += kDenseThreads) {
        const int q = i / hbytes, c = i - q * hbytes;
        hs[i] = (q < nq && c < row_bytes) ? hq[(int64_t)q * row_bytes + c] : 0;
    }
    __syncthreads();

    const int64_t r0 = (int64_t)blockIdx.x * rows_per_wg;
    const int nrows = (int)max<int64_t>(0, min<int64_t>(rows_per_wg, V - r0));
    const int gl = lane % kDenseGroup;
    const int groups = kDenseThreads / kDenseGroup;
    const int grp = wave * (kWave / kDenseGroup) + lane / kDenseGroup;
    const int nchunk = row_bytes / VEC;
    typedef typename Vec<VEC>::T TV;
    for (int r = grp; r < nrows; r += groups) {
        const TV *w = reinterpret_cast<const TV *>(W + (r0 + r) * (int64_t)row_bytes);
        float acc[NB];
#pragma unroll
        for (int q = 0; q < NB; ++q) acc[q] = 0.0f;
#pragma unroll 4
        for (int c = gl; c < nchunk; c += kDenseGroup) {
            const TV wv = __builtin_nontemporal_load(w + c);
#pragma unroll
            for (int q = 0; q < NB; ++q)
                acc[q] = dot_vec<VEC, BF16>(wv, reinterpret_cast<const TV *>(hs + q * hbytes)[c], acc[q]);
        }
#pragma unroll
        for (int q = 0; q < NB; ++q) {
            float a = acc[q];
#pragma unroll
            for (int m = kDenseGroup / 2; m >= 1; m >>= 1) a += __shfl_xor(a, m, kDenseGroup);
            if (gl == 0) z[q * rows_per_wg + r] = a;
        }
    }
    __syncthreads();

    // per-workgroup candidates: the best min(k, nrows) of its rows
    const int kk = min(k, nrows);
    for (int q = 0; q < nq; ++q) {
        uint64_t *out = cand + ((int64_t)q * nwg + blockIdx.x) * k;
        const float *zq = z + q * rows_per_wg;
        auto key_at = [&](int i) { return make_key(zq[i], (int32_t)(r0 + i)); };
        if (kk > 0) radix_select<kDenseThreads>(nrows, kk, key_at, sh.hist, sh.wave, &sh.sel);
        if (tid == 0) sh.count = 0;
        __syncthreads();
        const SelState s = sh.sel;
        for (int i = tid; i < nrows && kk > 0; i += kDenseThreads) {
            const uint64_t key = key_at(i);
            if (selected(key, s)) {
                const uint32_t slot = atomicAdd(&sh.count, 1u);
                if (slot < (uint32_t)kk) out[slot] = key;
            }
        }
        for (int i = kk + tid; i < k; i += kDenseThreads) out[i] = 0;  // empty slots
        __syncthreads();
    }

    // ticket: the last workgroup merges
    __threadfence();
    __syncthreads();
    if (tid == 0) {
        const uint32_t prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        sh.last = prev == (uint32_t)(nwg - 1);
    }
    __syncthreads();
    if (!sh.last) return;
    __threadfence();

    uint64_t *sorted = reinterpret_cast<uint64_t *>(smem);  // reuse: [k] keys
    const int n = nwg * k;
    for (int q = 0; q < nq; ++q) {
        const uint64_t *cq = cand + (int64_t)q * n;
        auto key_at = [&](int i) { return __builtin_nontemporal_load(cq + i); };
        radix_select<kDenseThreads>(n, k, key_at, sh.hist, sh.wave, &sh.sel);
        if (tid == 0) sh.count = 0;
        __syncthreads();
        const SelState s = sh.sel;
        uint64_t *pick = sorted + k;  // [k] unordered picks
        for (int i = tid; i < n; i += kDenseThreads) {
            const uint64_t key = key_at(i);
            if (key != 0 && selected(key, s)) {
                const uint32_t slot = atomicAdd(&sh.count, 1u);
                if (slot < (uint32_t)k) pick[slot] = key;
            }
        }
        __syncthreads();
        // rank sort (keys are distinct)
        for (int t = tid; t < k; t += kDenseThreads) {
            const uint64_t key = pick[t];
            int rank = 0;
            for (int j = 0; j < k; ++j) rank += pick[j] > key;
            sorted[rank] = key;
        }
        __syncthreads();
        for (int t = tid; t < k; t += kDenseThreads) {
            const uint64_t key = sorted[t];
            ids[(int64_t)q * k + t] = key_id(key);
            logits[(int64_t)q * k + t] = key_logit(key);
        }
        __syncthreads();
    }
    if (tid == 0) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// HNSW search, one workgroup per query
// ---------------------------------------------------------------------------
//
// Exact restatement of K-NN-SEARCH over SEARCH-LAYER: greedy descent (result
// set of 1) through layers maxlevel..1, then a sorted beam of ef_eff keys on
// layer 0.  Each step expands the best unexpanded beam entry: its neighbour
// list is read by one thread per slot, unseen ids are claimed in the LDS
// visited bitmap, their rows are dotted with h by 16-lane groups, and the new
// keys are merged into the beam (which keeps the best ef_eff).  The search
// ends when every beam entry is expanded.  This visits, scores and expands
// exactly the nodes the sequential algorithm does (a node evicted from the
// result set is worse than all of it and would only be popped to stop the
// search), so the distance and expansion counts match it.

constexpr int kHnswThreads = 256;
constexpr int kHnswGroup = 16;

struct HnswShared {
    uint64_t best;
    uint32_t nnew;
    uint32_t first;  // first unexpanded beam slot
    uint32_t nbeam;
};

__device__ __forceinline__ void clear_bits(uint32_t *vis, int words)
{
    for (int i = threadIdx.x; i < words; i += kHnswThreads) vis[i] = 0u;
}

// Returns true if id was not yet marked (and marks it).
__device__ __forceinline__ bool claim(uint32_t *vis, int32_t id)
{
    const uint32_t bit = 1u << (id & 31);
    return (atomicOr(&vis[id >> 5], bit) & bit) == 0u;
}

template <int VEC, bool BF16>
__global__ __launch_bounds__(kHnswThreads) void hnsw_kernel(
    const char *__restrict__ W, int64_t V, int row_bytes, const int32_t *__restrict__ adj0, int M0,
    const int32_t *__restrict__ upper_off, const int32_t *__restrict__ upper, int M, int maxlevel, int32_t entry,
    const char *__restrict__ hq, int k, int ef, int32_t *__restrict__ ids, float *__restrict__ logits,
    uint32_t *__restrict__ stats)
{
    extern __shared__ __align__(16) char smem[];
    __shared__ HnswShared sh;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int q = blockIdx.x;
    const int hbytes = (row_bytes + 15) & ~15;
    const int vwords = (int)((V + 31) / 32);
    const int maxdeg = M0 > M ? M0 : M;
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
    uint8_t *flag = reinterpret_cast<uint8_t *>(p);
    p += (size_t)ef;
    uint8_t *flag2 = reinterpret_cast<uint8_t *>(p);
    p += (size_t)ef;
    uint32_t *vis = reinterpret_cast<uint32_t *>(((uintptr_t)p + 15) & ~(uintptr_t)15);

    const char *h = hq + (int64_t)q * row_bytes;
    for (int i = tid; i < hbytes; i += kHnswThreads) hs[i] = i < row_bytes ? h[i] : 0;
    __syncthreads();

    const int gl = lane % kHnswGroup;
    const int grp = wave * (kWave / kHnswGroup) + lane / kHnswGroup;
    const int ngroups = kHnswThreads / kHnswGroup;
    uint32_t n_dist = 0, n_expand = 0;

    // score the entry point
    if (tid == 0) sh.best = 0;
    __syncthreads();
    if (grp == 0) {
        const float s = group_row_dot<VEC, BF16, kHnswGroup>(W, entry, row_bytes, hs, gl);
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
            if (tid < M) {
                const int32_t e = lst[tid];
                if (e >= 0 && claim(vis, e)) cid[atomicAdd(&sh.nnew, 1u)] = e;
            }
            __syncthreads();
            const int nn = (int)sh.nnew;
            for (int j = grp; j < nn; j += ngroups) {
                const float s = group_row_dot<VEC, BF16, kHnswGroup>(W, cid[j], row_bytes, hs, gl);
                if (gl == 0) atomicMax(reinterpret_cast<unsigned long long *>(&sh.best),
                                       (unsigned long long)make_key(s, cid[j]));
            }
            __syncthreads();
            n_dist += nn;
            const uint64_t best = sh.best;
            __syncthreads();
            if (best <= cur) break;
            cur = best;
        }
    }

    // layer 0: beam of ef keys, sorted descending, with expanded flags
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
        __syncthreads();
        if (tid == 0) {
            flag[first] = 1;
            sh.nnew = 0;
        }
        ++n_expand;
        __syncthreads();
        const int32_t *lst = adj0 + (int64_t)c * M0;
        for (int t = tid; t < M0; t += kHnswThreads) {
            const int32_t e = lst[t];
            if (e >= 0 && claim(vis, e)) cid[atomicAdd(&sh.nnew, 1u)] = e;
        }
        __syncthreads();
        const int nn = (int)sh.nnew;
        n_dist += nn;
        for (int j = grp; j < nn; j += ngroups) {
            const float s = group_row_dot<VEC, BF16, kHnswGroup>(W, cid[j], row_bytes, hs, gl);
            if (gl == 0) ckey[j] = make_key(s, cid[j]);
        }
        __syncthreads();
        // order the new keys (rank sort; keys are distinct)
        for (int j = tid; j < nn; j += kHnswThreads) {
            const uint64_t key = ckey[j];
            int rank = 0;
            for (int t = 0; t < nn; ++t) rank += ckey[t] > key;
            csort[rank] = key;
        }
        __syncthreads();
        // merge beam (nbeam) and csort (nn) into beam2, keep the best ef
        const int total = min((int)nbeam + nn, ef);
        for (int j = tid; j < nn; j += kHnswThreads) {
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
            }
        }
        for (int i = tid; i < (int)nbeam; i += kHnswThreads) {
            const uint64_t key = beam[i];
            int lo = 0, hi = nn;  // count new keys > key
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (csort[mid] > key) lo = mid + 1; else hi = mid;
            }
            const int pos = lo + i;
            if (pos < total) {
                beam2[pos] = key;
                flag2[pos] = flag[i];
            }
        }
        if (tid == 0) sh.first = 0xFFFFFFFFu;
        __syncthreads();
        for (int i = tid; i < total; i += kHnswThreads) {
            beam[i] = beam2[i];
            flag[i] = flag2[i];
            if (!flag2[i]) atomicMin(&sh.first, (uint32_t)i);
        }
        if (tid == 0) sh.nbeam = (uint32_t)total;
        __syncthreads();
    }

    const int nb = (int)sh.nbeam;
    for (int t = tid; t < k; t += kHnswThreads) {
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

size_t dense_workspace_bytes(int64_t V, int d, int B, int k)
{
    (void)V;
    (void)d;
    const int nb = B < kDenseMaxNB ? B : kDenseMaxNB;
    return 256 + (size_t)nb * kDenseWgs * (size_t)k * 8;
}

namespace {

size_t dense_lds(int nb, int row_bytes, int rows_per_wg, int k)
{
    const size_t hbytes = (size_t)((row_bytes + 15) & ~15);
    const size_t a = (size_t)nb * hbytes + (size_t)nb * rows_per_wg * 4;
    const size_t b = (size_t)k * 16;  // final merge reuse
    return a > b ? a : b;
}

template <int VEC, bool BF16, int NB>
hipError_t dense_launch(const void *W, int64_t V, int row_bytes, const char *h, int nq, int k, int rpw, int nwg,
                        uint64_t *cand, uint32_t *counter, int32_t *ids, float *logits, hipStream_t s)
{
    const size_t lds = dense_lds(NB, row_bytes, rpw, k);
    auto kern = dense_topk_kernel<VEC, BF16, NB>;
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    kern<<<nwg, kDenseThreads, lds, s>>>(static_cast<const char *>(W), V, row_bytes, h, nq, k, rpw, cand, counter,
                                          ids, logits);
    return hipGetLastError();
}

template <int VEC, bool BF16>
hipError_t dense_launch_nb(int nb, const void *W, int64_t V, int row_bytes, const char *h, int nq, int k, int rpw,
                           int nwg, uint64_t *cand, uint32_t *counter, int32_t *ids, float *logits, hipStream_t s)
{
    switch (nb) {
    case 1: return dense_launch<VEC, BF16, 1>(W, V, row_bytes, h, nq, k, rpw, nwg, cand, counter, ids, logits, s);
    case 2: return dense_launch<VEC, BF16, 2>(W, V, row_bytes, h, nq, k, rpw, nwg, cand, counter, ids, logits, s);
    case 4: return dense_launch<VEC, BF16, 4>(W, V, row_bytes, h, nq, k, rpw, nwg, cand, counter, ids, logits, s);
    default: return dense_launch<VEC, BF16, 8>(W, V, row_bytes, h, nq, k, rpw, nwg, cand, counter, ids, logits, s);
    }
}

}  // namespace

vie_status launch_dense_topk(const void *W, int dtype, int64_t V, int d, const void *h, int B, int k, int32_t *ids,
                             float *logits, void *ws, hipStream_t s)
{
    const int row_bytes = d * elem_bytes(dtype);
    const int hbytes = (row_bytes + 15) & ~15;
    // queries per pass: at most 8, and their rows must fit in 48 KB of LDS
    int nbmax = kDenseMaxNB;
    while (nbmax > 1 && (size_t)nbmax * hbytes > 48 * 1024) nbmax >>= 1;
    int nwg = kDenseWgs;
    int rpw = (int)((V + nwg - 1) / nwg);
    if (rpw > kDenseMaxRows)
        return fail(VIE_EUNSUPPORTED, "V = %lld needs more than %d rows per workgroup", (long long)V, kDenseMaxRows);
    if (rpw < 1) rpw = 1;
    nwg = (int)((V + rpw - 1) / rpw);
    uint32_t *counter = static_cast<uint32_t *>(ws);
    uint64_t *cand = reinterpret_cast<uint64_t *>(static_cast<char *>(ws) + 256);
    const char *hb = static_cast<const char *>(h);
    const int vec = pick_vec(row_bytes, W);
    for (int q0 = 0; q0 < B; q0 += nbmax) {
        const int nq = B - q0 < nbmax ? B - q0 : nbmax;
        const int nb = nq == 1 ? 1 : nq == 2 ? 2 : nq <= 4 ? 4 : 8;
        const char *hp = hb + (int64_t)q0 * row_bytes;
        int32_t *ip = ids + (int64_t)q0 * k;
        float *lp = logits + (int64_t)q0 * k;
        hipError_t e;
        const bool bf = dtype == VIE_BF16;
        if (vec == 16)
            e = bf ? dense_launch_nb<16, true>(nb, W, V, row_bytes, hp, nq, k, rpw, nwg, cand, counter, ip, lp, s)
                   : dense_launch_nb<16, false>(nb, W, V, row_bytes, hp, nq, k, rpw, nwg, cand, counter, ip, lp, s);
        else if (vec == 8)
            e = bf ? dense_launch_nb<8, true>(nb, W, V, row_bytes, hp, nq, k, rpw, nwg, cand, counter, ip, lp, s)
                   : dense_launch_nb<8, false>(nb, W, V, row_bytes, hp, nq, k, rpw, nwg, cand, counter, ip, lp, s);
        else if (vec == 4)
            e = bf ? dense_launch_nb<4, true>(nb, W, V, row_bytes, hp, nq, k, rpw, nwg, cand, counter, ip, lp, s)
                   : dense_launch_nb<4, false>(nb, W, V, row_bytes, hp, nq, k, rpw, nwg, cand, counter, ip, lp, s);
        else
            e = dense_launch_nb<2, true>(nb, W, V, row_bytes, hp, nq, k, rpw, nwg, cand, counter, ip, lp, s);
        if (e != hipSuccess) return launched(e, "dense top-k launch");
    }
    return VIE_OK;
}

size_t hnsw_lds_bytes(int64_t V, int d, int dtype, int ef_eff, int M0, int M)
{
    const int row_bytes = d * elem_bytes(dtype);
    const size_t hbytes = (size_t)((row_bytes + 15) & ~15);
    const size_t maxdeg = (size_t)(M0 > M ? M0 : M);
    size_t n = hbytes + (size_t)ef_eff * 8 * 2 + maxdeg * (8 + 8 + 4) + (size_t)ef_eff * 2;
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
template <int VEC, bool BF16>
hipError_t hnsw_launch(const HnswLaunch &a, size_t lds, hipStream_t s)
{
    auto kern = hnsw_kernel<VEC, BF16>;
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    kern<<<a.B, kHnswThreads, lds, s>>>(static_cast<const char *>(a.W), a.V, a.d * elem_bytes(a.dtype), a.adj0,
                                         a.M0, a.upper_off, a.upper, a.M, a.maxlevel, a.entry,
                                         static_cast<const char *>(a.h), a.k, a.ef_eff, a.ids, a.logits, a.stats);
    return hipGetLastError();
}
}  // namespace

vie_status launch_hnsw_search(const HnswLaunch &a, hipStream_t s)
{
    const size_t lds = hnsw_lds_bytes(a.V, a.d, a.dtype, a.ef_eff, a.M0, a.M);
    const size_t lim = hnsw_lds_limit();
    if (lds > lim)
        return fail(VIE_EUNSUPPORTED, "HNSW search needs %zu bytes of LDS per workgroup; the device allows %zu", lds,
                    lim);
    const int row_bytes = a.d * elem_bytes(a.dtype);
    const int vec = pick_vec(row_bytes, a.W);
    const bool bf = a.dtype == VIE_BF16;
    hipError_t e;
    if (vec == 16) e = bf ? hnsw_launch<16, true>(a, lds, s) : hnsw_launch<16, false>(a, lds, s);
    else if (vec == 8) e = bf ? hnsw_launch<8, true>(a, lds, s) : hnsw_launch<8, false>(a, lds, s);
    else if (vec == 4) e = bf ? hnsw_launch<4, true>(a, lds, s) : hnsw_launch<4, false>(a, lds, s);
    else e = hnsw_launch<2, true>(a, lds, s);
    return launched(e, "HNSW search launch");
}

}  // namespace vie
