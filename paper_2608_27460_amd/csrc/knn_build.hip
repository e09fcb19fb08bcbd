// Batch construction of a single-layer graph over the rows of W_out on the
// GPU.  Section 3 builds the index offline and prioritises its quality;
// Section 5 names GPU construction as future work.  The graph is the batch
// form also written out by the CPU oracle:
//
//   1. cand(i): the K rows nearest to row i by inner product (j != i), in the
//      (score desc, id asc) order of the search;
//   2. fwd(i): the neighbour-selection heuristic of Malkov & Yashunin
//      (Algorithm 4) over cand(i) with cap M0: in candidate order, e is kept
//      iff <w_e, w_i> > <w_e, w_r> for every r kept before it (a list of at
//      most M0 candidates is kept whole);
//   3. rev(j): every i with j in fwd(i);
//   4. the list of j: fwd(j), then the nodes of rev(j) not in fwd(j) in
//      (score desc, id asc) order, cut at M0 entries;
//   5. entry point: the row of largest squared norm (ties: smaller id).
//
// Step 1 is a dense contraction: the Gram block S = W[rows] W^T of a chunk of
// rows comes from this file's matrix-core kernel (fp32 accumulation), and
// one workgroup per row selects its exact top K from S.  Scores are fp32 throughout; ties of equal scores are
// broken by id exactly as the oracle breaks them.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <type_traits>
#include <vector>

#include "index.hpp"
#include "keys.hpp"

namespace vie {

namespace {

constexpr int kWave = 64;
constexpr int kTopkThreads = 256;
constexpr int kDigitBits = 12;               // radix digit of the selection
constexpr int kDigitBuckets = 1 << kDigitBits;
constexpr int kGatherCap = 2048;             // keys a selection sorts in LDS
constexpr int kSelectThreads = 256;
constexpr int kSelectRows = 128;             // candidate rows of one Gram block (K <= 128)
constexpr int kChunkBytes = 256;             // bytes of a row per staged chunk
constexpr int kChunkPitch = kChunkBytes + 32;  // padded: the matrix-core operand reads hit every LDS bank once
constexpr int kGramPitch = kSelectRows + 1;  // floats per Gram row in LDS

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

// 16 x 16 tile += A (16 rows x 32 columns) B^T, bf16 operands, fp32 accumulation
__device__ __forceinline__ f32x4 mfma_bf16(u32x4 a, u32x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
}

struct TopkShared {
    uint32_t hist[kDigitBuckets];
    uint64_t gat[kGatherCap];
    uint32_t wsum[kTopkThreads / kWave];
    uint32_t n, bucket, above, count;
};

// Exclusive prefix sum over the block of one value per thread.
template <int NT>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t *wsum)
{
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    uint32_t incl = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t t = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += t;
    }
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    uint32_t base = 0;
    for (int w = 0; w < wave; ++w) base += wsum[w];
    __syncthreads();
    return base + incl - v;
}

// Sorts n <= kGatherCap keys in LDS, largest first (bitonic network over the
// next power of two; the padding is 0, the smallest key).
template <int NT>
__device__ void block_sort_desc(uint64_t *a, int n)
{
    int p = 1;
    while (p < n) p <<= 1;
    for (int i = n + threadIdx.x; i < p; i += NT) a[i] = 0ull;
    __syncthreads();
    for (int size = 2; size <= p; size <<= 1)
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = threadIdx.x; i < p / 2; i += NT) {
                const int lo = 2 * i - (i & (stride - 1)), hi = lo + stride;
                const bool desc = (lo & size) == 0;
                const uint64_t x = a[lo], y = a[hi];
                if (desc ? x < y : x > y) {
                    a[lo] = y;
                    a[hi] = x;
                }
            }
            __syncthreads();
        }
}

// The K largest of the keys key_at(0 .. n-1) (0 = no key), sorted, into
// sh.gat[0 .. K).  Exact: a radix select over the 64-bit keys, kDigitBits
// per round from the top, narrows the bucket of the K-th largest until every
// key at or above that bucket fits in LDS; those are gathered and sorted.
// Keys are distinct, so at most 6 rounds are needed.  Returns the number of
// keys found (< K only when fewer than K keys exist).
template <int NT, typename KeyAt>
__device__ int block_topk(int64_t n, int K, KeyAt key_at, TopkShared &sh)
{
    const int tid = threadIdx.x;
    uint64_t prefix = 0ull;
    int known = 0;
    uint32_t want = (uint32_t)K;
    uint64_t T = 0ull;
    for (;;) {
        const int width = 64 - known < kDigitBits ? 64 - known : kDigitBits;
        const int shift = 64 - known - width;
        const uint32_t nb = 1u << width;
        for (int b = tid; b < kDigitBuckets; b += NT) sh.hist[b] = 0u;
        if (tid == 0) {
            sh.bucket = 0u;
            sh.above = 0u;
            sh.count = 0u;
        }
        __syncthreads();
        for (int64_t i = tid; i < n; i += NT) {
            const uint64_t key = key_at(i);
            if (key != 0ull && (known == 0 || (key >> (64 - known)) == (prefix >> (64 - known))))
                atomicAdd(&sh.hist[(uint32_t)(key >> shift) & (nb - 1)], 1u);
        }
        __syncthreads();
        // buckets from the top: thread t holds buckets nb-1-16t .. nb-16-16t
        constexpr int per = kDigitBuckets / NT;
        uint32_t c[per], sum = 0;
#pragma unroll
        for (int j = 0; j < per; ++j) {
            const int b = (int)nb - 1 - (per * tid + j);
            c[j] = b >= 0 ? sh.hist[b] : 0u;
            sum += c[j];
        }
        uint32_t above = block_exclusive_scan<NT>(sum, sh.wsum);
        bool found = false;
#pragma unroll
        for (int j = 0; j < per; ++j) {
            if (!found && above < want && want <= above + c[j]) {
                sh.bucket = (uint32_t)((int)nb - 1 - (per * tid + j));
                sh.above = above;
                sh.count = c[j];
                found = true;
            }
            above += c[j];
        }
        __syncthreads();
        if (sh.count == 0u) {
            // fewer than want keys match the prefix: take every key >= prefix
            T = prefix == 0ull ? 1ull : prefix;
            break;
        }
        const uint64_t lo = prefix | ((uint64_t)sh.bucket << shift);
        const uint32_t total = ((uint32_t)K - want) + sh.above + sh.count;
        if (total <= (uint32_t)kGatherCap || shift == 0) {
            T = lo == 0ull ? 1ull : lo;
            break;
        }
        prefix = lo;
        known += width;
        want -= sh.above;
        __syncthreads();
    }
    if (tid == 0) sh.n = 0u;
    __syncthreads();
    for (int64_t i = tid; i < n; i += NT) {
        const uint64_t key = key_at(i);
        if (key >= T) {
            const uint32_t slot = atomicAdd(&sh.n, 1u);
            if (slot < (uint32_t)kGatherCap) sh.gat[slot] = key;
        }
    }
    __syncthreads();
    const int m = (int)min(sh.n, (uint32_t)kGatherCap);
    block_sort_desc<NT>(sh.gat, m);
    return m < K ? m : K;
}

// Step 1, per row of a chunk: the K nearest other rows from the chunk's
// scores S [rows][ld] (row r of the chunk is row r0 + r of W_out; rows start
// 16-byte aligned).  A sample of the row (every kSampleEvery-th block of
// kTopkThreads scores) gives a threshold T0 with about twice the sample's
// share of K keys above it; one vectorized pass then gathers every key >= T0.
// If at least K and at most kGatherCap keys were gathered, every key of the
// answer is among them (K keys are >= T0, so the K-th largest is too) and a
// sort finishes; otherwise the exact radix select runs.  The sample only
// decides the speed, never the result.
constexpr int kSampleEvery = 8;

// ---------------------------------------------------------------------------
// Gram blocks on the matrix cores
// ---------------------------------------------------------------------------
//
// S[c][j] = <w_{r0 + c}, w_j> for the rows c of a chunk and every row j, fp32
// accumulation, written with row pitch ld.  A workgroup of eight waves owns
// a 256 x 128 tile (256 chunk rows c by 128 rows j); wave (wm, wn) computes
// its 64 x 64 block as 4 x 4 tiles of 16 x 16 on the matrix cores
// (v_mfma_f32_16x16x32_bf16 for bf16 rows, v_mfma_f32_16x16x4_f32 for fp32
// rows).  The reduction over the row width runs in stages of kGramKC bytes
// of each row: both slices of a stage (256 and 128 rows) are staged in LDS,
// the stages two ahead loading into registers while the current one is
// multiplied.  (128 x 128 tiles of four waves, two workgroups per CU, read a
// quarter more through the CU for the same products and measured the same
// per chunk but 2-5% slower per build.)
// Lane (r, g) of a wave (r = lane % 16, g = lane / 16) feeds row r of a
// 16-row operand with its g-th quarter of the k step, and ends holding rows
// 4 g + i of column r of each 16 x 16 result.  Every score is the same
// sequence of products and sums whichever tile computes it.
//
// Staged rows are not padded: the 16-byte piece p of staged row x sits at
// piece p ^ ((x >> 1) & 7) of the row.  Measured with the LDS counters on
// gfx950, the operand reads (16 rows, four consecutive pieces or four
// consecutive floats each) then use every bank once per cycle, where rows
// padded by 16 bytes took twice the cycles (half of them bank conflicts).  Every load of a stage is issued with
// no branch around it (pieces past the row are clamped to its last piece and
// replaced by zeros when staged), in the order they are consumed, so the
// compiler waits only for the stage being staged.

#ifndef VIE_GRAM_TILE_C
#define VIE_GRAM_TILE_C 256
#endif
constexpr int kGramTileC = VIE_GRAM_TILE_C;        // chunk rows c per workgroup (128 or 256)
constexpr int kGramTile = 128;                     // rows j per workgroup
constexpr int kGramThreads = 2 * kGramTileC;       // (kGramTileC / 64) x 2 waves of 64 x 64 quarters
#ifndef VIE_GRAM_KC
#define VIE_GRAM_KC 128
#endif
constexpr int kGramKC = VIE_GRAM_KC;               // bytes of a row per stage
static_assert(kGramKC == 128, "the piece swizzle is laid out for 8 pieces a staged row");
constexpr int kGramRowPitch = kGramKC;                 // LDS bytes per staged row
constexpr int kGramStage = (kGramTileC + kGramTile) * kGramRowPitch;  // A and B slices of one stage

// byte offset of 16-byte piece p of staged row x
__device__ __forceinline__ int gram_piece(int x, int p) { return x * kGramRowPitch + ((p ^ ((x >> 1) & 7)) << 4); }
constexpr int kGramLoads = (kGramTileC + kGramTile) * (kGramKC / 16) / kGramThreads;  // 16-byte loads per thread
static_assert(kGramLoads * kGramThreads == (kGramTileC + kGramTile) * (kGramKC / 16), "staging shape");

__device__ __forceinline__ f32x4 mfma_f32(float a, float b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

template <bool BF16>
__global__ __launch_bounds__(kGramThreads) __attribute__((amdgpu_waves_per_eu(2))) void knn_gram_kernel(const char *__restrict__ W, int64_t V, int row_bytes,
                                                                int64_t r0, int64_t rows, float *__restrict__ S,
                                                                int64_t ld)
{
    extern __shared__ __align__(16) char smem[];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int r = lane & 15, g = lane >> 4;
    const int wm = wave >> 1, wn = wave & 1;
    // Launch order for the eight XCDs, each with its own L2: workgroups are
    // dealt to the XCDs in turn (workgroup L runs on XCD L % 8).  XCD x
    // takes half of the chunk's tiles c (the first half for even x) and the
    // tiles of rows j numbered x / 2, x / 2 + 4, ..., each with all of its
    // tiles c in a row: a tile of j is fetched by two XCDs, and each XCD
    // re-reads only its half of the chunk's rows.  The grid rounds the tiles
    // of c up to an even count and those of j up to a multiple of 4; the
    // workgroups past the last tile return at once.
    const int nc = (int)((rows + kGramTileC - 1) / kGramTileC);
    const int nch = (nc + 1) / 2;
    const int64_t nj = (V + kGramTile - 1) / kGramTile;
    const int64_t wg = blockIdx.x, i = wg >> 3, x = wg & 7;
    const int64_t jt = (i / nch) * 4 + (x >> 1), ct = (x & 1) * nch + i % nch;
    if (jt >= nj || ct >= nc) return;
    const int64_t c0 = ct * kGramTileC, j0 = jt * kGramTile;
    const int nstage = (row_bytes + kGramKC - 1) / kGramKC;
    const u32x4 zero = {0u, 0u, 0u, 0u};
    // staging: load t of a thread covers staged row (L / 8) of A (the first
    // kGramTileC rows) or of B, 16 bytes at byte (L % 8) * 16 of the stage,
    // L = t * kGramThreads + tid
    const char *src[kGramLoads];
    int soff[kGramLoads], scol[kGramLoads];
#pragma unroll
    for (int t = 0; t < kGramLoads; ++t) {
        const int L = t * kGramThreads + tid;
        const int srow = L / (kGramKC / 16);  // 0..255: A rows then B rows
        scol[t] = (L % (kGramKC / 16)) * 16;
        const int64_t grow = srow < kGramTileC ? r0 + min<int64_t>(c0 + srow, rows - 1)
                                               : min<int64_t>(j0 + srow - kGramTileC, V - 1);
        src[t] = W + grow * (int64_t)row_bytes;
        soff[t] = gram_piece(srow, scol[t] >> 4);
    }
    auto load_stage = [&](int st, u32x4(&buf)[kGramLoads]) {
#pragma unroll
        for (int t = 0; t < kGramLoads; ++t)
            buf[t] = *reinterpret_cast<const u32x4 *>(src[t] + min(st * kGramKC + scol[t], row_bytes - 16));
        __builtin_amdgcn_sched_barrier(0);  // keep the issue order
    };
    f32x4 acc[4][4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int n = 0; n < 4; ++n) acc[m][n] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    // stages load two ahead: stage st's loads sit in register buffer st % 2
    // (the stage pairs are written out over the buffers, so no load in
    // flight is ever copied) and in LDS buffer st % 2
    u32x4 pre[2][kGramLoads];
    load_stage(0, pre[0]);
    load_stage(min(1, nstage - 1), pre[1]);
    // one stage: into LDS buffer PB from register buffer PB, the loads of the
    // stage two ahead into that register buffer, then the products.  The
    // stage pairs run in a loop without any branch inside (so the compiler
    // keeps the loads of the next stage in flight across it) and an odd last
    // stage after it.
    auto run_stage = [&](auto pbc, int st) {
        constexpr int pb = decltype(pbc)::value;
        char *buf = smem + pb * kGramStage;
#pragma unroll
        for (int t = 0; t < kGramLoads; ++t)
            *reinterpret_cast<u32x4 *>(buf + soff[t]) = st * kGramKC + scol[t] + 16 <= row_bytes ? pre[pb][t] : zero;
        __builtin_amdgcn_sched_barrier(0);
        load_stage(min(st + 2, nstage - 1), pre[pb]);  // past the end: the last stage again (cached)
        __syncthreads();  // the stage is in LDS (and the stage before it is no longer read)
        const char *A = buf + (wm * 64) * kGramRowPitch;
        const char *B = buf + (kGramTileC + wn * 64) * kGramRowPitch;
        if constexpr (BF16) {
#pragma unroll
            for (int kk = 0; kk < kGramKC; kk += 64) {  // 32 bf16 per MFMA step
                u32x4 a[4], b[4];
#pragma unroll
                for (int m = 0; m < 4; ++m)
                    a[m] = *reinterpret_cast<const u32x4 *>(A + gram_piece(m * 16 + r, kk / 16 + g));
#pragma unroll
                for (int n = 0; n < 4; ++n)
                    b[n] = *reinterpret_cast<const u32x4 *>(B + gram_piece(n * 16 + r, kk / 16 + g));
#pragma unroll
                for (int m = 0; m < 4; ++m)
#pragma unroll
                    for (int n = 0; n < 4; ++n) acc[m][n] = mfma_bf16(a[m], b[n], acc[m][n]);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < kGramKC; kk += 16) {  // 4 floats per MFMA step
                float a[4], b[4];
#pragma unroll
                for (int m = 0; m < 4; ++m)
                    a[m] = *reinterpret_cast<const float *>(A + gram_piece(m * 16 + r, kk / 16) + 4 * g);
#pragma unroll
                for (int n = 0; n < 4; ++n)
                    b[n] = *reinterpret_cast<const float *>(B + gram_piece(n * 16 + r, kk / 16) + 4 * g);
#pragma unroll
                for (int m = 0; m < 4; ++m)
#pragma unroll
                    for (int n = 0; n < 4; ++n) acc[m][n] = mfma_f32(a[m], b[n], acc[m][n]);
            }
        }
    };
    int st = 0;
    for (; st + 1 < nstage; st += 2) {
        run_stage(std::integral_constant<int, 0>(), st);
        run_stage(std::integral_constant<int, 1>(), st + 1);
    }
    if (st < nstage) run_stage(std::integral_constant<int, 0>(), st);
    // lane (r, g) holds chunk rows 16 m + 4 g + i of the quarter, column 16 n + r
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t c = c0 + wm * 64 + m * 16 + 4 * g + i;
            if (c >= rows) continue;
            float *out = S + c * ld + j0 + wn * 64;
#pragma unroll
            for (int n = 0; n < 4; ++n)
                if (j0 + wn * 64 + n * 16 + r < V) out[n * 16 + r] = acc[m][n][i];
        }
}

__global__ __launch_bounds__(kTopkThreads) void knn_topk_kernel(const float *__restrict__ S, int64_t ld, int64_t r0,
                                                                int64_t V, int K, int32_t *__restrict__ cand,
                                                                float *__restrict__ cand_score)
{
    __shared__ TopkShared sh;
    const int tid = threadIdx.x;
    const int64_t i = r0 + blockIdx.x;
    const float *row = S + (int64_t)blockIdx.x * ld;
    auto key_at = [&](int64_t j) -> uint64_t { return j == i ? 0ull : make_key(row[j], (int32_t)j); };

    // sample: blocks 0, kSampleEvery, 2 kSampleEvery, ... of kTopkThreads scores
    for (int bkt = tid; bkt < kDigitBuckets; bkt += kTopkThreads) sh.hist[bkt] = 0u;
    if (tid == 0) {
        sh.n = 0u;
        sh.bucket = 0u;
        sh.count = 0u;
    }
    __syncthreads();
    // (kSampleBatch sampled blocks per round: their loads are all in flight
    // before the first histogram update)
    // (the next round's loads are issued before this round's updates)
    constexpr int kSampleBatch = 8;
    constexpr int64_t kRound = (int64_t)kSampleBatch * kSampleEvery * kTopkThreads;
    uint32_t ns = 0;
    auto load_round = [&](int64_t j0, float(&x)[kSampleBatch]) {
#pragma unroll
        for (int u = 0; u < kSampleBatch; ++u)
            x[u] = row[min<int64_t>(j0 + (int64_t)u * kSampleEvery * kTopkThreads + tid, V - 1)];
        __builtin_amdgcn_sched_barrier(0);  // keep the issue order
    };
    auto count_round = [&](int64_t j0, const float(&x)[kSampleBatch]) {
#pragma unroll
        for (int u = 0; u < kSampleBatch; ++u) {
            const int64_t jb = j0 + (int64_t)u * kSampleEvery * kTopkThreads, j = jb + tid;
            if (jb < V) ns += (uint32_t)min<int64_t>(kTopkThreads, V - jb);
            if (j < V && j != i) atomicAdd(&sh.hist[(uint32_t)(make_key(x[u], (int32_t)j) >> (64 - kDigitBits))], 1u);
        }
    };
    {
        float xa[kSampleBatch], xb[kSampleBatch];
        load_round(0, xa);
        for (int64_t j0 = 0; j0 < V; j0 += 2 * kRound) {
            load_round(j0 + kRound, xb);
            count_round(j0, xa);
            load_round(j0 + 2 * kRound, xa);
            count_round(j0 + kRound, xb);
        }
    }
    const uint32_t want = (uint32_t)((2 * (int64_t)K * ns + V - 1) / V) + 4;
    __syncthreads();
    {
        constexpr int per = kDigitBuckets / kTopkThreads;
        uint32_t c[per], sum = 0;
#pragma unroll
        for (int j = 0; j < per; ++j) {
            c[j] = sh.hist[kDigitBuckets - 1 - (per * tid + j)];
            sum += c[j];
        }
        uint32_t above = block_exclusive_scan<kTopkThreads>(sum, sh.wsum);
#pragma unroll
        for (int j = 0; j < per; ++j) {
            if (above < want && want <= above + c[j]) {
                sh.bucket = (uint32_t)(kDigitBuckets - 1 - (per * tid + j));
                sh.count = 1u;
            }
            above += c[j];
        }
    }
    __syncthreads();
    // (fewer sampled keys than want: T0 = 1, every key)
    const uint64_t T0 = sh.count ? ((uint64_t)sh.bucket << (64 - kDigitBits)) | 1ull : 1ull;
    // gather every key >= T0, four scores per load: batches of kGatherLoads
    // loads per thread, the next batch issued before the current one is
    // sifted so that the row keeps streaming (indices clamped, no branch
    // around a load; the keys past the row are skipped when sifted)
    constexpr int kGatherLoads = 8;
    constexpr int64_t kBatch = (int64_t)kGatherLoads * kTopkThreads;
    const int64_t n4 = (V + 3) / 4;
    const float4 *row4 = reinterpret_cast<const float4 *>(row);
    auto load_batch = [&](int64_t b0, float4(&v)[kGatherLoads]) {
#pragma unroll
        for (int u = 0; u < kGatherLoads; ++u) v[u] = row4[min(b0 + u * kTopkThreads + tid, n4 - 1)];
        __builtin_amdgcn_sched_barrier(0);  // keep the issue order
    };
    auto sift_batch = [&](int64_t b0, const float4(&v)[kGatherLoads]) {
#pragma unroll
        for (int u = 0; u < kGatherLoads; ++u) {
            const int64_t j = 4 * (b0 + u * kTopkThreads + tid);
            const float x[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (j + e < V && j + e != i) {
                    const uint64_t key = make_key(x[e], (int32_t)(j + e));
                    if (key >= T0) {
                        const uint32_t slot = atomicAdd(&sh.n, 1u);
                        if (slot < (uint32_t)kGatherCap) sh.gat[slot] = key;
                    }
                }
            }
        }
    };
    float4 va[kGatherLoads], vb[kGatherLoads];
    load_batch(0, va);
    for (int64_t b0 = 0; b0 < n4; b0 += 2 * kBatch) {
        load_batch(b0 + kBatch, vb);
        sift_batch(b0, va);
        load_batch(b0 + 2 * kBatch, va);
        sift_batch(b0 + kBatch, vb);
    }
    __syncthreads();
    const uint32_t ng = sh.n;
    int m;
    if (ng >= (uint32_t)K && ng <= (uint32_t)kGatherCap) {
        block_sort_desc<kTopkThreads>(sh.gat, (int)ng);
        m = K;
    } else {
        __syncthreads();
        m = block_topk<kTopkThreads>(V, K, key_at, sh);
    }
    for (int t = tid; t < K; t += kTopkThreads) {
        const uint64_t key = t < m ? sh.gat[t] : 0ull;
        cand[i * K + t] = t < m ? key_id(key) : -1;
        cand_score[i * K + t] = t < m ? key_logit(key) : 0.0f;
    }
}

// Two bf16 products per 32-bit word (the words are passed as plain integers:
// bit-casting a vector lane in place compiled to the first lane here).
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float acc)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), acc,
                                           false);
}

__device__ __forceinline__ float dot16(u32x4 a, u32x4 b, float acc, bool bf16)
{
    const uint32_t a0 = a.x, a1 = a.y, a2 = a.z, a3 = a.w;
    const uint32_t b0 = b.x, b1 = b.y, b2 = b.z, b3 = b.w;
    if (bf16) {
        acc = dot2_bf16(a0, b0, acc);
        acc = dot2_bf16(a1, b1, acc);
        acc = dot2_bf16(a2, b2, acc);
        return dot2_bf16(a3, b3, acc);
    }
    acc = fmaf(__uint_as_float(a0), __uint_as_float(b0), acc);
    acc = fmaf(__uint_as_float(a1), __uint_as_float(b1), acc);
    acc = fmaf(__uint_as_float(a2), __uint_as_float(b2), acc);
    return fmaf(__uint_as_float(a3), __uint_as_float(b3), acc);
}

constexpr size_t kSelectBig = (size_t)kSelectRows * kChunkPitch > (size_t)kSelectRows * kGramPitch * 4
                                   ? (size_t)kSelectRows * kChunkPitch
                                   : (size_t)kSelectRows * kGramPitch * 4;
constexpr size_t kSelectLds = kSelectBig + (size_t)kSelectRows * 8 + 256 * 4;

// Step 2, one workgroup per node: the Gram matrix of its candidates (rows
// staged through LDS in chunks of kChunkBytes, fp32 accumulation; matrix
// cores for bf16 rows, vector ALUs for fp32 rows), then the heuristic scan
// in candidate order by one wave.  A node with at most M0 candidates keeps
// them all.
template <bool BF16>
__global__ __launch_bounds__(kSelectThreads) void knn_select_kernel(const char *__restrict__ W, int row_bytes,
                                                                    int K, int M0, const int32_t *__restrict__ cand,
                                                                    const float *__restrict__ cand_score,
                                                                    int32_t *__restrict__ fwd,
                                                                    float *__restrict__ fwd_score,
                                                                    int32_t *__restrict__ nfwd)
{
    extern __shared__ __align__(16) char smem[];
    char *tile = smem;                                            // [128][kChunkPitch] staged rows
    float *G = reinterpret_cast<float *>(smem);                   // [128][kGramPitch] after the tile
    int32_t *cid = reinterpret_cast<int32_t *>(smem + kSelectBig);  // [128]
    float *cs = reinterpret_cast<float *>(cid + kSelectRows);     // [128]
    int32_t *kept = reinterpret_cast<int32_t *>(cs + kSelectRows);  // [<= 256]
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int64_t i = blockIdx.x;
    int nc = 0;
    for (int t = tid; t < kSelectRows; t += kSelectThreads) {
        const int32_t c = t < K ? cand[i * K + t] : -1;
        cid[t] = c;
        cs[t] = t < K ? cand_score[i * K + t] : 0.0f;
    }
    __syncthreads();
    for (int t = 0; t < K; ++t) nc += cid[t] >= 0;  // uniform
    if (nc <= M0) {
        for (int t = tid; t < M0; t += kSelectThreads) {
            fwd[i * M0 + t] = t < nc ? cid[t] : -1;
            fwd_score[i * M0 + t] = t < nc ? cs[t] : 0.0f;
        }
        if (tid == 0) nfwd[i] = nc;
        return;
    }
    // Gram block.  bf16 rows: on the matrix cores, wave w owns the 64 x 64
    // block (rows 64 (w / 2), columns 64 (w % 2)) as 4 x 4 tiles of
    // v_mfma_f32_16x16x32_bf16, lane (r, g) supplying columns 8 g .. 8 g + 7
    // of each 32-column step for row r of a tile.  fp32 rows: on the vector
    // ALUs, thread (ta, tb) owns pairs (ta + 16 x, tb + 16 y) (rows 16 apart
    // keep the 16-byte reads of a wave on distinct LDS banks).
    const int ta = tid / 16, tb = tid % 16;
    const int wv = tid / kWave, mr = lane & 15, mg = lane >> 4;
    const int rb = 64 * (wv >> 1), cb = 64 * (wv & 1);
    constexpr int NX = BF16 ? 1 : 8;
    float acc[NX][NX];
    f32x4 macc[4][4];
#pragma unroll
    for (int x = 0; x < NX; ++x)
#pragma unroll
        for (int y = 0; y < NX; ++y) acc[x][y] = 0.0f;
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int n = 0; n < 4; ++n) macc[m][n] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    const u32x4 zero = {0u, 0u, 0u, 0u};
    // stage 128 rows x 256 bytes per chunk (16 pieces of 16 bytes per row,
    // kPieces per thread); for bf16 rows the next chunk's pieces load into
    // registers while the current one is multiplied
    constexpr int kPieces = kSelectRows * (kChunkBytes / 16) / kSelectThreads;
    static_assert(kPieces * kSelectThreads == kSelectRows * (kChunkBytes / 16), "staging shape");
    u32x4 pre[kPieces];
    auto load_chunk = [&](int c0) {
#pragma unroll
        for (int j = 0; j < kPieces; ++j) {
            const int p = tid + j * kSelectThreads;
            const int r = p / (kChunkBytes / 16), off = c0 + 16 * (p % (kChunkBytes / 16));
            const int32_t c = cid[r];
            pre[j] = c >= 0 && off < row_bytes ? *reinterpret_cast<const u32x4 *>(W + (int64_t)c * row_bytes + off)
                                               : zero;
        }
    };
    // (bf16 rows only: fp32 rows hold an 8 x 8 block of sums per thread, and
    // the extra registers would halve their occupancy)
    if constexpr (BF16) load_chunk(0);
    for (int c0 = 0; c0 < row_bytes; c0 += kChunkBytes) {
        __syncthreads();  // every wave is done with the previous chunk
        if constexpr (!BF16) load_chunk(c0);
#pragma unroll
        for (int j = 0; j < kPieces; ++j) {
            const int p = tid + j * kSelectThreads;
            *reinterpret_cast<u32x4 *>(tile + (p / (kChunkBytes / 16)) * kChunkPitch + 16 * (p % (kChunkBytes / 16))) =
                pre[j];
        }
        if constexpr (BF16)
            if (c0 + kChunkBytes < row_bytes) load_chunk(c0 + kChunkBytes);
        __syncthreads();
        if constexpr (BF16) {
#pragma unroll
            for (int t = 0; t < kChunkBytes / 64; ++t) {  // 32 bf16 columns per step
                u32x4 a[4], b[4];
#pragma unroll
                for (int m = 0; m < 4; ++m)
                    a[m] = *reinterpret_cast<const u32x4 *>(tile + (rb + 16 * m + mr) * kChunkPitch + 64 * t + 16 * mg);
#pragma unroll
                for (int n = 0; n < 4; ++n)
                    b[n] = *reinterpret_cast<const u32x4 *>(tile + (cb + 16 * n + mr) * kChunkPitch + 64 * t + 16 * mg);
#pragma unroll
                for (int m = 0; m < 4; ++m)
#pragma unroll
                    for (int n = 0; n < 4; ++n) macc[m][n] = mfma_bf16(a[m], b[n], macc[m][n]);
            }
        } else {
#pragma unroll 2
            for (int piece = 0; piece < kChunkBytes / 16; ++piece) {
                u32x4 a[NX], b[NX];
#pragma unroll
                for (int x = 0; x < NX; ++x)
                    a[x] = *reinterpret_cast<const u32x4 *>(tile + (ta + 16 * x) * kChunkPitch + 16 * piece);
#pragma unroll
                for (int y = 0; y < NX; ++y)
                    b[y] = *reinterpret_cast<const u32x4 *>(tile + (tb + 16 * y) * kChunkPitch + 16 * piece);
#pragma unroll
                for (int x = 0; x < NX; ++x)
#pragma unroll
                    for (int y = 0; y < NX; ++y) acc[x][y] = dot16(a[x], b[y], acc[x][y], false);
            }
        }
    }
    __syncthreads();
    if constexpr (BF16) {
        // lane (r, g) holds rows 4 g + i of tile m against row r of tile n
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int n = 0; n < 4; ++n)
#pragma unroll
                for (int e = 0; e < 4; ++e) G[(rb + 16 * m + 4 * mg + e) * kGramPitch + cb + 16 * n + mr] = macc[m][n][e];
    } else {
#pragma unroll
        for (int x = 0; x < NX; ++x)
#pragma unroll
            for (int y = 0; y < NX; ++y) G[(ta + 16 * x) * kGramPitch + tb + 16 * y] = acc[x][y];
    }
    __syncthreads();
    if (tid < kWave) {
        // heuristic scan: e is kept iff s_e > <w_e, w_r> for every kept r
        int nk = 0;
        for (int e = 0; e < nc && nk < M0; ++e) {
            const float se = cs[e];
            bool bad = false;
            for (int r = lane; r < nk; r += kWave) bad |= G[e * kGramPitch + kept[r]] >= se;
            if (!__any(bad)) {
                if (lane == 0) kept[nk] = e;
                ++nk;
                __builtin_amdgcn_wave_barrier();
            }
        }
        for (int t = lane; t < M0; t += kWave) {
            fwd[i * M0 + t] = t < nk ? cid[kept[t]] : -1;
            fwd_score[i * M0 + t] = t < nk ? cs[kept[t]] : 0.0f;
        }
        if (lane == 0) nfwd[i] = nk;
    }
}

__device__ __forceinline__ bool in_list(const int32_t *lst, int n, int32_t x)
{
    bool f = false;
    for (int t = 0; t < n; ++t) f |= lst[t] == x;
    return f;
}

// Step 3: reverse edges not already forward edges of their target.  Pass 0
// counts them per target, pass 1 (after the scan) writes their keys.
__global__ void knn_reverse_kernel(int64_t V, int M0, const int32_t *__restrict__ fwd,
                                   const float *__restrict__ fwd_score, const int32_t *__restrict__ nfwd,
                                   uint32_t *__restrict__ count, const int64_t *__restrict__ roff,
                                   uint64_t *__restrict__ rev, int pass)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= V * M0) return;
    const int64_t i = e / M0;
    const int t = (int)(e - i * M0);
    if (t >= nfwd[i]) return;
    const int32_t j = fwd[e];
    if (in_list(fwd + (int64_t)j * M0, nfwd[j], (int32_t)i)) return;
    const uint32_t slot = atomicAdd(&count[j], 1u);
    if (pass == 1) rev[roff[j] + slot] = make_key(fwd_score[e], (int32_t)i);
}

// Exclusive prefix sum of count[0 .. V) into roff[0 .. V] (one workgroup).
__global__ __launch_bounds__(1024) void knn_scan_kernel(const uint32_t *__restrict__ count, int64_t V,
                                                        int64_t *__restrict__ roff)
{
    __shared__ uint32_t wsum[16];
    __shared__ int64_t s_base;
    if (threadIdx.x == 0) s_base = 0;
    __syncthreads();
    for (int64_t b0 = 0; b0 < V; b0 += 1024) {
        const int64_t j = b0 + threadIdx.x;
        const uint32_t v = j < V ? count[j] : 0u;
        const uint32_t ex = block_exclusive_scan<1024>(v, wsum);
        const int64_t base = s_base;
        if (j < V) roff[j] = base + ex;
        __syncthreads();
        if (threadIdx.x == 1023) s_base = base + ex + v;
        __syncthreads();
    }
    if (threadIdx.x == 0) roff[V] = s_base;
}

// Step 4, one workgroup per node: the forward list, then the best reverse
// edges in the free slots.
__global__ __launch_bounds__(kTopkThreads) void knn_lists_kernel(int M0, const int32_t *__restrict__ fwd,
                                                                 const int32_t *__restrict__ nfwd,
                                                                 const int64_t *__restrict__ roff,
                                                                 const uint64_t *__restrict__ rev,
                                                                 int32_t *__restrict__ adj0)
{
    __shared__ TopkShared sh;
    const int64_t j = blockIdx.x;
    const int nf = nfwd[j];
    const int free_slots = M0 - nf;
    const int64_t off = roff[j], nr = roff[j + 1] - off;
    int m = 0;
    if (free_slots > 0 && nr > 0) {
        auto key_at = [&](int64_t t) -> uint64_t { return rev[off + t]; };
        m = block_topk<kTopkThreads>(nr, free_slots, key_at, sh);
    }
    for (int t = threadIdx.x; t < M0; t += kTopkThreads)
        adj0[j * M0 + t] = t < nf ? fwd[j * M0 + t] : t < nf + m ? key_id(sh.gat[t - nf]) : -1;
}

// Step 5: the key (squared norm, id) of every row, the largest kept.  Each
// wave takes rows grid-stride and keeps its best key; the workgroup's best
// goes to *best with one atomic (one per row would serialise on the word).
constexpr int kEntryThreads = 256;
constexpr int kEntryBlocks = 2048;

template <bool BF16>
__global__ __launch_bounds__(kEntryThreads) void knn_entry_kernel(const char *__restrict__ W, int64_t V,
                                                                  int row_bytes, unsigned long long *__restrict__ best)
{
    __shared__ unsigned long long wbest[kEntryThreads / kWave];
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
    const int64_t nwaves = (int64_t)gridDim.x * (kEntryThreads / kWave);
    unsigned long long mine = 0ull;
    for (int64_t i = (int64_t)blockIdx.x * (kEntryThreads / kWave) + wv; i < V; i += nwaves) {
        const char *w = W + i * row_bytes;
        float acc = 0.0f;
        for (int c = 16 * lane; c < row_bytes; c += 16 * kWave) {
            const u32x4 v = *reinterpret_cast<const u32x4 *>(w + c);
            acc = dot16(v, v, acc, BF16);
        }
#pragma unroll
        for (int o = kWave / 2; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, kWave);
        const unsigned long long key = make_key(acc, (int32_t)i);
        mine = key > mine ? key : mine;
    }
    if (lane == 0) wbest[wv] = mine;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long m = wbest[0];
#pragma unroll
        for (int x = 1; x < kEntryThreads / kWave; ++x) m = wbest[x] > m ? wbest[x] : m;
        if (m) atomicMax(best, m);
    }
}

struct Buffers {
    float *S = nullptr;
    int32_t *cand = nullptr, *fwd = nullptr, *nfwd = nullptr, *adj0 = nullptr, *upper_off = nullptr,
            *upper = nullptr;
    float *cand_score = nullptr, *fwd_score = nullptr;
    uint32_t *count = nullptr;
    int64_t *roff = nullptr;
    uint64_t *rev = nullptr;
    unsigned long long *best = nullptr;
    char *sample = nullptr;  // the rows of W_out the fingerprint samples, gathered
    void release()
    {
        void *p[] = {S, cand, fwd, nfwd, cand_score, fwd_score, count, roff, rev, best, sample};
        for (void *q : p)
            if (q) (void)hipFree(q);
        S = nullptr;
        cand = fwd = nfwd = nullptr;
        cand_score = fwd_score = nullptr;
        count = nullptr;
        roff = nullptr;
        rev = nullptr;
        best = nullptr;
        sample = nullptr;
    }
    void release_graph()
    {
        void *p[] = {adj0, upper_off, upper};
        for (void *q : p)
            if (q) (void)hipFree(q);
        adj0 = upper_off = upper = nullptr;
    }
};

template <typename T>
bool dalloc(T *&p, size_t bytes)
{
    void *q = nullptr;
    if (hipMalloc(&q, bytes < 16 ? 16 : bytes) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    p = static_cast<T *>(q);
    return true;
}

}  // namespace

vie_status build_knn_graph_gpu(const void *W_dev, int dtype, int64_t V, int d, int K, int M0, int64_t chunk_rows,
                               hipStream_t s, Graph &g, DeviceGraph &dg)
{
    const int row_bytes = d * elem_bytes(dtype);
    const int64_t ld = (V + 3) & ~(int64_t)3;  // 16-byte aligned rows of scores
    int64_t R = chunk_rows > 0 ? chunk_rows : ((int64_t)2 << 30) / (ld * 4);
    R = std::max<int64_t>(1, std::min<int64_t>(R, V));
    if (R * ld > ((int64_t)1 << 31)) return fail(VIE_EUNSUPPORTED, "GPU build: a score chunk of %lld rows is too large", (long long)R);
    int dev = 0;
    hipError_t he = hipGetDevice(&dev);
    if (he != hipSuccess) return fail(VIE_EHIP, "hipGetDevice: %s", hipGetErrorString(he));
    const size_t lds = kSelectLds;
    auto sel = dtype == VIE_BF16 ? knn_select_kernel<true> : knn_select_kernel<false>;
    he = hipFuncSetAttribute((const void *)sel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (he != hipSuccess) return fail(VIE_EHIP, "GPU build: %s", hipGetErrorString(he));

    Buffers b;
    const int64_t edges = V * M0;
    // the rows the W_out fingerprint samples: every step-th row, then the last
    const int64_t step = V / 1024 > 1 ? V / 1024 : 1;
    const int64_t nreg = (V + step - 1) / step;
    if (!dalloc(b.S, (size_t)R * ld * 4) || !dalloc(b.cand, (size_t)V * K * 4) ||
        !dalloc(b.cand_score, (size_t)V * K * 4) || !dalloc(b.fwd, (size_t)edges * 4) ||
        !dalloc(b.fwd_score, (size_t)edges * 4) || !dalloc(b.nfwd, (size_t)V * 4) ||
        !dalloc(b.count, (size_t)V * 4) || !dalloc(b.roff, (size_t)(V + 1) * 8) ||
        !dalloc(b.rev, (size_t)edges * 8) || !dalloc(b.best, 8) || !dalloc(b.adj0, (size_t)edges * 4) ||
        !dalloc(b.upper_off, (size_t)V * 4) || !dalloc(b.upper, 4) ||
        !dalloc(b.sample, (size_t)(nreg + 1) * row_bytes)) {
        b.release();
        b.release_graph();
        return fail(VIE_ENOMEM, "GPU build: device allocation failed (V = %lld, chunk of %lld rows)", (long long)V,
                    (long long)R);
    }
    auto bail = [&](vie_status st) {
        (void)hipStreamSynchronize(s);
        b.release();
        b.release_graph();
        return st;
    };

    const int64_t gram_nj4 = ((V + kGramTile - 1) / kGramTile + 3) / 4 * 4;  // tiles of j, rounded up to 4
    if (gram_nj4 * ((R + kGramTileC - 1) / kGramTileC + 1) > 0x7FFFFFFF)
        return bail(fail(VIE_EUNSUPPORTED, "GPU build: V = %lld rows exceed the Gram grid", (long long)V));
    auto gram = dtype == VIE_BF16 ? knn_gram_kernel<true> : knn_gram_kernel<false>;
    he = hipFuncSetAttribute((const void *)gram, hipFuncAttributeMaxDynamicSharedMemorySize, 2 * kGramStage);
    if (he != hipSuccess) return bail(fail(VIE_EHIP, "GPU build: %s", hipGetErrorString(he)));
    for (int64_t r0 = 0; r0 < V; r0 += R) {
        const int64_t rows = std::min(R, V - r0);
        const dim3 grid((unsigned)((((rows + kGramTileC - 1) / kGramTileC + 1) / 2 * 2) * gram_nj4));
        gram<<<grid, kGramThreads, 2 * kGramStage, s>>>(static_cast<const char *>(W_dev), V, row_bytes, r0, rows, b.S,
                                                        ld);
        he = hipGetLastError();
        if (he != hipSuccess) break;
        knn_topk_kernel<<<(unsigned)rows, kTopkThreads, 0, s>>>(b.S, ld, r0, V, K, b.cand, b.cand_score);
        he = hipGetLastError();
        if (he != hipSuccess) break;
    }
    if (he != hipSuccess) return bail(fail(VIE_EHIP, "GPU build: Gram / top-k launch: %s", hipGetErrorString(he)));

    sel<<<(unsigned)V, kSelectThreads, lds, s>>>(static_cast<const char *>(W_dev), row_bytes, K, M0, b.cand,
                                                 b.cand_score, b.fwd, b.fwd_score, b.nfwd);
    he = hipMemsetAsync(b.count, 0, (size_t)V * 4, s);
    const unsigned eg = (unsigned)((edges + 255) / 256);
    if (he == hipSuccess) {
        knn_reverse_kernel<<<eg, 256, 0, s>>>(V, M0, b.fwd, b.fwd_score, b.nfwd, b.count, b.roff, b.rev, 0);
        knn_scan_kernel<<<1, 1024, 0, s>>>(b.count, V, b.roff);
        he = hipMemsetAsync(b.count, 0, (size_t)V * 4, s);
    }
    if (he == hipSuccess) {
        knn_reverse_kernel<<<eg, 256, 0, s>>>(V, M0, b.fwd, b.fwd_score, b.nfwd, b.count, b.roff, b.rev, 1);
        knn_lists_kernel<<<(unsigned)V, kTopkThreads, 0, s>>>(M0, b.fwd, b.nfwd, b.roff, b.rev, b.adj0);
        he = hipMemsetAsync(b.best, 0, 8, s);
    }
    if (he == hipSuccess) {
        const unsigned eb = (unsigned)std::min<int64_t>((V + 3) / 4, kEntryBlocks);
        if (dtype == VIE_BF16)
            knn_entry_kernel<true><<<eb, kEntryThreads, 0, s>>>(static_cast<const char *>(W_dev), V, row_bytes, b.best);
        else
            knn_entry_kernel<false><<<eb, kEntryThreads, 0, s>>>(static_cast<const char *>(W_dev), V, row_bytes, b.best);
        he = hipMemsetAsync(b.upper_off, 0xFF, (size_t)V * 4, s);  // every node on layer 0 only: -1
    }
    if (he == hipSuccess) he = hipGetLastError();
    if (he != hipSuccess) return bail(fail(VIE_EHIP, "GPU build: %s", hipGetErrorString(he)));

    // host form of the graph (the index file and vie_index_export read it)
    g = Graph();
    g.V = V;
    g.d = d;
    g.dtype = dtype;
    g.M0 = M0;
    g.M = std::min(M0, std::max(2, M0 / 2));
    g.efC = K;
    g.seed = 0;
    g.maxlevel = 0;
    g.levels.assign((size_t)V, 0);
    g.upper_off.assign((size_t)V, -1);
    // (the layer-0 lists stay on the device: the index copies them to the
    // host when a host-side call first needs them)
    unsigned long long best = 0;
    he = hipMemcpyAsync(&best, b.best, 8, hipMemcpyDeviceToHost, s);
    // the sampled rows of W_out gathered on the device (one strided copy
    // and the last row), then one copy to the host: a copy per row, or a
    // strided copy straight to host memory, took 7-15 ms of host time
    std::vector<char> sample((size_t)(nreg + 1) * row_bytes);
    if (he == hipSuccess)
        he = hipMemcpy2DAsync(b.sample, (size_t)row_bytes, W_dev, (size_t)step * row_bytes, (size_t)row_bytes,
                              (size_t)nreg, hipMemcpyDeviceToDevice, s);
    if (he == hipSuccess)
        he = hipMemcpyAsync(b.sample + nreg * row_bytes, static_cast<const char *>(W_dev) + (V - 1) * row_bytes,
                            row_bytes, hipMemcpyDeviceToDevice, s);
    if (he == hipSuccess) he = hipMemcpyAsync(sample.data(), b.sample, sample.size(), hipMemcpyDeviceToHost, s);
    if (he == hipSuccess) he = hipStreamSynchronize(s);
    if (he != hipSuccess) return bail(fail(VIE_EHIP, "GPU build: %s", hipGetErrorString(he)));
    g.entry = (int32_t)(~(uint32_t)best);
    g.fingerprint = w_fingerprint_rows(sample.data(), dtype, V, d, nreg + 1);
    b.release();

    dg = DeviceGraph();
    dg.device = dev;
    dg.W = W_dev;
    dg.adj0 = b.adj0;
    dg.upper_off = b.upper_off;
    dg.upper = b.upper;
    return VIE_OK;
}

}  // namespace vie
