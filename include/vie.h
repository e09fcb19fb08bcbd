/*
 * vie.h -- C ABI of libvie.so, an MI355X (gfx950) output head that treats
 * "output projection + top-k token selection" as maximum inner product search
 * over the rows of the output-embedding matrix W_out.
 *
 * Method: Loretz & Hochreiter, "Accelerating LLM Inference via Vector Index
 * Based Output Embeddings", Section 3.  The logits are z = W_out h with
 * z_i = <w_i, h>; top-k decoding only needs the k largest, which is exactly
 * MIPS with query h.  An HNSW graph (Malkov & Yashunin 2018) built offline over
 * the rows with inner product as the similarity answers it approximately; the
 * retrieved logits are scattered into a full-vocabulary tensor that is -inf
 * elsewhere.  The exact dense head (vie_dense_topk) is the baseline the paper
 * compares against (Section 4.1).
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 * - Every function returns a vie_status; none throws or aborts.  On failure
 *   vie_last_error() gives a detail string (thread-local, valid until the
 *   next call on the same thread).
 * - Device pointers are plain HIP device addresses on the current device;
 *   the caller allocates and owns every device buffer.  The library owns only
 *   a vie_index and the device copy of its graph.  W_out on the device is
 *   borrowed, never copied.
 * - Calls that take a stream (hipStream_t passed as void*, NULL = the null
 *   stream) enqueue their kernels and return without waiting.  Argument errors
 *   are reported synchronously, before anything is enqueued.  Device data
 *   (ids, queries) is not validated by the host.
 * - Layouts are row-major and densely packed.  W_out is [V][d] of the index
 *   dtype; a batch of queries h is [B][d] of the same dtype.  bf16 values are
 *   raw bit patterns (the top 16 bits of the fp32 value).
 * - Returned top-k lists are ordered by logit descending; equal logits are
 *   ordered by id ascending.  Logits are always fp32.
 * - Sizes: 1 <= d <= 8192, 1 <= V < 2^31, 1 <= k <= min(V, 1024),
 *   1 <= B <= 65535.
 */
#ifndef VIE_H
#define VIE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    VIE_OK = 0,
    VIE_EINVAL = 1,       /* bad argument (NULL, size, dtype, k > V, ...) */
    VIE_ENOMEM = 2,       /* host or device allocation failed */
    VIE_EHIP = 3,         /* a HIP runtime call or kernel launch failed */
    VIE_EIO = 4,          /* file could not be opened, read or written */
    VIE_EFORMAT = 5,      /* index file corrupt, truncated, or for another W */
    VIE_ESTATE = 6,       /* index not on the device yet, or on another one */
    VIE_EUNSUPPORTED = 7  /* valid request this build cannot serve */
} vie_status;

typedef enum { VIE_F32 = 0, VIE_BF16 = 1 } vie_dtype;

typedef struct vie_index vie_index; /* opaque, library owned */

/* HNSW construction parameters (Section 3: the index is built offline from
 * the rows of W_out with inner product as the similarity; Section 4 uses
 * M = 32, ef_construction = 5000). */
typedef struct {
    int32_t M;               /* neighbour cap on layers >= 1; 2 <= M <= 128 */
    int32_t M0;              /* neighbour cap on layer 0; 0 selects 2*M (the
                                |V|(4d + 8M) memory formula of Section 3);
                                M <= M0 <= 256 */
    int32_t ef_construction; /* candidate list size while inserting; >= 1 */
    int32_t n_threads;       /* build threads; 0 = hardware concurrency.  With
                                1 thread the graph is deterministic. */
    uint64_t seed;           /* seeds the level of every node */
    int32_t select;          /* 0 = neighbour-selection heuristic (Malkov &
                                Yashunin Algorithm 4), 1 = the m nearest */
} vie_build_params;

/* Plain description of an index. */
typedef struct {
    int64_t V;
    int32_t d;
    int32_t dtype;           /* vie_dtype */
    int32_t M, M0, ef_construction;
    int32_t maxlevel;        /* top layer */
    int32_t entry;           /* entry node (Section 2: the predefined entry node) */
    int64_t n_upper_blocks;  /* sum over nodes of their level */
    uint64_t seed;
    uint64_t w_fingerprint;  /* see the file format below */
    int32_t on_device;       /* 1 after vie_index_to_device */
    int32_t device;          /* HIP device of the device copy, -1 if none */
} vie_index_desc;

/* ------------------------------------------------------------------------
 * Index life cycle
 * ------------------------------------------------------------------------ */

/* Builds an HNSW graph over the V rows of W_host (host memory, [V][d] of
 * dtype) on the CPU.  Rows are inserted in id order; the level of node i is
 * floor(-ln(u_i) / ln M) with u_i = ((splitmix64(seed ^ i) >> 11) + 1) 2^-53,
 * capped at 16.  W_host is only read during the call.  *out receives a new
 * index that the caller releases with vie_index_free.
 * Errors: VIE_EINVAL (NULL, sizes, params), VIE_ENOMEM. */
vie_status vie_index_build(const void *W_host, vie_dtype dtype, int64_t V, int32_t d,
                           const vie_build_params *params, vie_index **out);

/* Parameters of the GPU batch construction (vie_index_build_gpu). */
typedef struct {
    int32_t K;          /* candidates per node: the K rows nearest by inner
                           product; 1 <= K <= min(V - 1, 128) */
    int32_t M0;         /* list cap; 2 <= M0 <= 256 */
    int64_t chunk_rows; /* rows of W_out per Gram block: the library holds
                           chunk_rows x V fp32 scores in device scratch; 0
                           selects about 2 GiB */
} vie_gpu_build_params;

/* Builds a single-layer graph over the V rows of W_dev (device memory,
 * [V][d] of dtype, 16-byte aligned rows) on the current HIP device, as a
 * batch: (1) the K rows nearest to each row i by inner product (j != i, fp32
 * accumulation), ordered by (score desc, id asc); (2) the forward list of i:
 * the neighbour-selection heuristic of Malkov & Yashunin (Algorithm 4) over
 * those candidates with cap M0 -- in candidate order e is kept iff
 * <w_e, w_i> > <w_e, w_r> for every r kept before it; at most M0 candidates
 * are kept whole; (3) reverse edges: i joins the list of every j in its
 * forward list, after j's forward list, in (score desc, id asc) order, up to
 * M0 entries.  The entry point is the row of largest squared norm (ties: the
 * smaller id).  Section 3 builds the index offline from the rows of W_out
 * with inner product as the similarity; construction on the GPU is the
 * future work of Section 5, and this batch form (one layer, maxlevel 0) is
 * the library's own.  The graph searches with vie_query like any index: the
 * greedy upper layers are empty.  On return the graph is complete and on the
 * device (as after vie_index_to_device with W_dev, which must stay allocated);
 * its layer-0 lists reach the host when a call first needs them there
 * (vie_index_save, vie_index_export, vie_index_to_device copy them from the
 * device, so these may also fail with VIE_EHIP for such an index; the first
 * of them should not race with another on the same index).  The index
 * reports M = max(2, M0 / 2)
 * (capped at M0), ef_construction = K, seed 0.  The call allocates device
 * scratch (chunk_rows x V x 4 bytes of scores plus about V (8K + 16 M0)
 * bytes) and releases it before returning; it enqueues on hip_stream and
 * waits for it.
 * Errors: VIE_EINVAL (NULL, sizes, params), VIE_EUNSUPPORTED (rows not
 * 16-byte aligned), VIE_ENOMEM, VIE_EHIP (a HIP call or launch failed). */
vie_status vie_index_build_gpu(const void *W_dev, vie_dtype dtype, int64_t V, int32_t d,
                               const vie_gpu_build_params *params, void *hip_stream, vie_index **out);

/* Writes the index file (format below).  Section 3: the index is built once,
 * offline, and shipped with the model checkpoint; this file is that artifact
 * (the graph plus a fingerprint of the W_out it was built on).
 * Errors: VIE_EINVAL, VIE_EIO, VIE_EHIP (a GPU-built index whose lists could
 * not be copied from the device). */
vie_status vie_index_save(const vie_index *index, const char *path);

/* Loads the shipped index (Section 3: precomputed and distributed with the
 * checkpoint, so inference never builds it).
 * Reads and validates an index file (checksum, sizes, every id in range, no
 * self loops or duplicates, degree caps, nested levels, entry on the top
 * level).  If W_host is not NULL it must be the [V][d] matrix the index was
 * built on: its fingerprint is compared with the stored one.
 * Errors: VIE_EINVAL, VIE_EIO, VIE_EFORMAT, VIE_ENOMEM. */
vie_status vie_index_load(const char *path, const void *W_host, vie_index **out);

/* Copies the graph to the current HIP device and records W_dev, the device
 * copy of W_out ([V][d] of the index dtype), which must stay allocated and
 * unchanged while the index is used.  The copy is complete when the call
 * returns.  May be called again to move the index or swap W_dev.
 * Errors: VIE_EINVAL, VIE_ENOMEM, VIE_EHIP. */
vie_status vie_index_to_device(vie_index *index, const void *W_dev, void *hip_stream);

vie_status vie_index_info(const vie_index *index, vie_index_desc *out);

/* Copies the graph into caller arrays: levels uint8[V], adj0 int32[V][M0],
 * upper_off int32[V], upper int32[n_upper_blocks][M] (layout as in the file).
 * Any pointer may be NULL to skip that array.  Errors: VIE_EINVAL, VIE_EHIP
 * (a GPU-built index whose lists could not be copied from the device). */
vie_status vie_index_export(const vie_index *index, uint8_t *levels, int32_t *adj0,
                            int32_t *upper_off, int32_t *upper);

/* Releases the index and its device graph.  NULL is ignored. */
void vie_index_free(vie_index *index);

/* ------------------------------------------------------------------------
 * Queries
 * ------------------------------------------------------------------------ */

/* HNSW k-NN search (Section 3; Malkov & Yashunin Algorithms 2 and 5) for B
 * queries h_dev [B][d] (index dtype), one workgroup per query: greedy descent
 * with a candidate list of 1 through layers maxlevel..1, then a candidate
 * list of ef_eff = max(ef, k) on layer 0.  Writes ids_dev int32[B][k] and
 * logits_dev fp32[B][k] (<w_id, h> accumulated in fp32); if fewer than k
 * nodes are reachable the tail holds id -1 and logit -inf.  stats_dev, if
 * not NULL, receives uint32[B][2] = (distance evaluations, expanded nodes)
 * over all layers.  Needs vie_index_to_device on the current device first.
 * Limits: ef_eff <= 8192, M0 <= 256, and one workgroup's LDS must hold the
 * query, the beam twice (16 bytes + 2 flag bytes per entry), the visited
 * bitmap (V/8 bytes) and per-step lists of about 20 bytes per layer-0 slot
 * (160 KiB on gfx950: ef_eff = 4096 fits next to a 262144-row bitmap).
 * Errors: VIE_EINVAL, VIE_ESTATE, VIE_EUNSUPPORTED, VIE_EHIP. */
vie_status vie_query(const vie_index *index, const void *h_dev, int32_t B, int32_t k, int32_t ef,
                     int32_t *ids_dev, float *logits_dev, uint32_t *stats_dev, void *hip_stream);

/* Options of vie_query_ex and vie_query_forced. */
typedef struct {
    int32_t expand_width; /* beam entries expanded per layer-0 step, 1..128 */
    int32_t int8_rows;    /* 1: layer-0 scores from the int8 rows attached with
                             vie_index_attach_int8, final beam re-ranked on
                             the stored rows; 0: stored rows throughout */
    int32_t *trace_dev;   /* NULL, or a device buffer int32[B][trace_cap]
                             (caller owned) that receives each query's
                             expansions in order: entry t is
                             (layer << 27) | (s << 26) | node for
                             t < min(expanded nodes, trace_cap), s = 1 for
                             the first node of a step (every node of a
                             one-expansion step); the nodes one layer-0 step
                             expands together appear best first; entries
                             past the last expansion are not written.
                             Needs V < 2^26.  A diagnostic: it lets a
                             caller replay and compare a traversal. */
    int32_t trace_cap;    /* entries per query of trace_dev (>= 1 when set) */
    int32_t team;         /* workgroups that search each query together:
                             a power of two up to 256 (0 counts as 1).  Each
                             member keeps the whole search state and takes
                             every decision itself, scores only the new
                             nodes whose id modulo team is its member
                             index, and passes the scores that can enter
                             the beam to the others through
                             workspace_dev, so the traversal, the
                             results and stats are those of team = 1 (a
                             query's distance evaluations are shared, its
                             dependent steps are not).  All B * team
                             workgroups must be resident on the device at
                             once (else VIE_EUNSUPPORTED).  Should a member
                             wait for another for seconds (the device kept
                             busy by other work), the query's row holds
                             ids -1, logits NaN and stats 0xFFFFFFFF. */
    void *workspace_dev;  /* team > 1 or share > 1: device buffer of at
                             least vie_query_workspace() bytes, 256-byte
                             aligned, caller owned, no initialisation
                             needed; calls that share it must not overlap
                             in time.  Ignored for team <= 1 and
                             share <= 1. */
    size_t workspace_bytes;
    int32_t share;        /* row sharing between the call's queries: 1, 2,
                             4, 8 or 16 (0 counts as 1) queries per group
                             (query b is in group b / share).  The workgroup
                             that fetches a row scores it for every query of
                             its group and publishes the others' scores in
                             workspace_dev; a query that later claims that
                             node takes its score from there and reads no
                             row.  Each score is computed by the same
                             instructions the query's own workgroup would
                             use, so results, stats and expansion records
                             are those of share = 1; the rows read drop
                             where the group's walks overlap.  Needs
                             team <= 1 and workspace_dev (vie_query_workspace
                             bytes, 256-byte aligned), which the library
                             clears on its first use and then keeps valid
                             across calls of any index; calls that share it
                             must not overlap in time.  Each workgroup also
                             holds its group's queries in LDS (share times
                             the query's size). */
} vie_search_params;

/* Bytes of device workspace that vie_query_ex / vie_query_forced need with
 * these arguments (0 unless params->team > 1 or params->share > 1; with
 * share, about 8 V bytes per query).
 * Errors: VIE_EINVAL (as the query would report for its arguments). */
vie_status vie_query_workspace(const vie_index *index, int32_t B, int32_t k, int32_t ef,
                               const vie_search_params *params, size_t *bytes);

/* vie_query with a layer-0 step that expands the expand_width best
 * unexpanded beam entries at once (their unvisited neighbours are scored
 * together and merged into the beam, which keeps its ef_eff best; the search
 * ends when every beam entry is expanded).  expand_width = 1 is exactly
 * vie_query.  Wider steps trade extra distance evaluations for fewer
 * dependent steps, which is what a GPU pays for (the paper names the
 * sequential traversal as the obstacle to GPU execution, Section 5).  The
 * results follow the same rule on any hardware; the test oracle implements
 * it independently.  Limits as vie_query, and LDS must also hold about
 * 16 bytes per claimed neighbour (expand_width * M0 of them; 12 in a team,
 * which keeps no list cache): a shape that does not fit is refused with
 * VIE_EUNSUPPORTED before any launch (on gfx950, 128 per step at
 * ef_eff = 2048 fits a 128256-row head with bf16 queries of 3072 values
 * only in a team).
 * Errors: as vie_query; VIE_EINVAL also for params NULL or expand_width
 * outside 1..128. */
vie_status vie_query_ex(const vie_index *index, const void *h_dev, int32_t B, int32_t k, int32_t ef,
                        const vie_search_params *params, int32_t *ids_dev, float *logits_dev,
                        uint32_t *stats_dev, void *hip_stream);

/* vie_query_ex (params NULL: expand_width 1) followed by the forced-inclusion
 * tokens of Section 3, whose logits are computed explicitly so that they are
 * never missing from the reconstructed logits.  forced_dev int32[n_forced]
 * (device; distinct ids, ids outside [0, V) are skipped) is caller owned.
 * ids_dev / logits_dev are [B][k + n_forced]: the union of the search's
 * top k and the forced ids, each id once, ordered by logit descending (ties:
 * id ascending), padded with -1 / -inf where an id occurred in both.  Forced
 * logits are computed like the search's (fp32 accumulation).
 * Limits: 0 <= n_forced <= 1024 and as vie_query_ex.
 * Errors: as vie_query_ex; VIE_EINVAL also for n_forced out of range or
 * forced_dev NULL with n_forced > 0. */
vie_status vie_query_forced(const vie_index *index, const void *h_dev, int32_t B, int32_t k, int32_t ef,
                            const vie_search_params *params, const int32_t *forced_dev, int32_t n_forced,
                            int32_t *ids_dev, float *logits_dev, uint32_t *stats_dev, void *hip_stream);

/* int8 copy of W_out for the traversal (quantized data types are the
 * paper's future work, Section 5).  Per row: scale = max_j |w_j| / 127 as an
 * fp32 division, q_j = rint(w_j / scale) (fp32 division, ties to even)
 * clamped to [-127, 127]; a row of zeros gets scale 0 and q = 0.  W_dev [V][d]
 * of dtype; q_dev int8[V][d] and scale_dev fp32[V] are caller-owned device
 * buffers.  Enqueued on the stream.  Errors: VIE_EINVAL, VIE_EHIP. */
vie_status vie_quantize_rows(const void *W_dev, vie_dtype dtype, int64_t V, int32_t d, int8_t *q_dev,
                             float *scale_dev, void *hip_stream);

/* Lets searches with int8_rows = 1 use q_dev / scale_dev (as written by
 * vie_quantize_rows for the index's W_dev; borrowed, must stay allocated and
 * unchanged while used; both NULL detaches).  With int8 rows, layer 0 is
 * walked on int8 scores: the query is quantized by the same rule, a score is
 * fp32(integer dot) times the row scale, times the query scale, each product
 * rounded to fp32; the layer-0 entry point is scored again that way.  The
 * upper layers use the stored rows, and the final beam is ranked again on
 * the stored rows (fp32 accumulation), so returned logits are exact-path
 * logits.  vie_index_to_device detaches.  Needs d divisible by 16.
 * Errors: VIE_EINVAL, VIE_ESTATE (not on a device), VIE_EUNSUPPORTED. */
vie_status vie_index_attach_int8(vie_index *index, const int8_t *q_dev, const float *scale_dev);

/* Bytes of device workspace vie_dense_topk needs for these sizes. */
vie_status vie_dense_topk_workspace(int64_t V, int32_t d, int32_t B, int32_t k, size_t *bytes);

/* Exact dense head: z = W_out h for B queries (fp32 accumulation over the
 * stored values), fused with the selection of the k largest (Section 3 and
 * the dense baseline of Section 4.1).  W_dev [V][d] and h_dev [B][d] of
 * dtype; ids_dev int32[B][k], logits_dev fp32[B][k].  workspace_dev must
 * hold at least vie_dense_topk_workspace() bytes and be 256-byte aligned; it
 * carries per-slab candidates between the call's two kernels and needs no
 * initialisation.  Calls that share a workspace must not overlap in time.
 * Errors: VIE_EINVAL, VIE_EHIP. */
vie_status vie_dense_topk(const void *W_dev, vie_dtype dtype, int64_t V, int32_t d, const void *h_dev,
                          int32_t B, int32_t k, int32_t *ids_dev, float *logits_dev, void *workspace_dev,
                          size_t workspace_bytes, void *hip_stream);

/* vie_dense_topk for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops, harnesses that forbid hipMalloc): the
 * same kernels and results, with the workspace taken from a 16 MiB array
 * that the library holds on each GPU until the process ends (set up on the
 * first call on a device).  The call allocates nothing.  Calls on one GPU
 * share that array, so calls that overlap in time on one GPU (other streams,
 * other threads) race and must be ordered by the caller.  Limit:
 * vie_dense_topk_workspace(V, d, B, k) <= 16 MiB (for example B <= 15 at
 * V = 262144, B <= 30 at V = 128256); larger requests fail with
 * VIE_EUNSUPPORTED before anything is enqueued.
 * Errors: VIE_EINVAL, VIE_EUNSUPPORTED, VIE_EHIP. */
vie_status vie_dense_topk_noalloc(const void *W_dev, vie_dtype dtype, int64_t V, int32_t d, const void *h_dev,
                                  int32_t B, int32_t k, int32_t *ids_dev, float *logits_dev, void *hip_stream);

/* Reconstructs full-vocabulary logits (Section 3): out_dev fp32[B][V] is -inf
 * everywhere except out[b][ids[b][j]] = logits[b][j].  Ids outside [0, V) are
 * skipped (so -1 padding is harmless); ids within a row must be distinct.
 * Errors: VIE_EINVAL, VIE_EHIP. */
vie_status vie_scatter(const int32_t *ids_dev, const float *logits_dev, int32_t B, int32_t k, int64_t V,
                       float *out_dev, void *hip_stream);

/* ------------------------------------------------------------------------
 * Diagnostics
 * ------------------------------------------------------------------------ */

const char *vie_status_string(vie_status status);
const char *vie_last_error(void);
int32_t vie_version(void); /* 10000 * major + 100 * minor + patch */

/* ------------------------------------------------------------------------
 * Index file format (little endian), version 1
 * ------------------------------------------------------------------------
 *   0   char[8]  "VIEHNSW1"
 *   8   u32      version = 1
 *   12  u32      dtype (0 fp32, 1 bf16)
 *   16  i64      V
 *   24  i32      d
 *   28  i32      M
 *   32  i32      M0
 *   36  i32      ef_construction
 *   40  u64      seed
 *   48  i32      maxlevel
 *   52  i32      entry
 *   56  i64      n_upper_blocks (nb)
 *   64  u64      fingerprint of W
 *   72  zero bytes up to 128
 *   128 u8   levels[V], then zero bytes up to a multiple of 8
 *       i32  adj0[V][M0]     layer-0 neighbours in stored order, -1 padded
 *       i32  upper_off[V]    first upper block of a node, -1 at level 0
 *       i32  upper[nb][M]    block upper_off[u] + l - 1 = level-l list of u
 *       u64  FNV-1a-64 checksum of every preceding byte
 * Fingerprint: FNV-1a-64 over V (8 bytes), d (4 bytes), dtype (4 bytes), then
 * the bytes of rows 0, s, 2s, ... below V with s = max(1, V / 1024), then the
 * bytes of row V - 1.
 */

#ifdef __cplusplus
}
#endif

#endif /* VIE_H */
