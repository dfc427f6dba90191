/*
 * eahr.h -- C ABI of libeahr.so: the PVS dense channel on an MI355X (gfx950),
 * the PBM sparse channel and exact adaptive weighted-RRF fusion on the host.
 *
 * Paper: "Exact Adaptive Hybrid Retrieval Without Fixed Top-L Cutoffs".
 *
 * Conventions (all entry points):
 *  - Every function returning int returns EAHR_OK (0) or a negative EAHR_E_*.
 *    On error nothing is returned through output pointers except where stated.
 *  - Item identifiers are int64 at the ABI.  Dense ids are row numbers in a
 *    pvs_index (0 .. rows-1, inserts get new, larger ids); sparse document ids
 *    must use the same numbering, so one identifier names one item in both
 *    channels.  The total identifier order used for every tie is ascending id.
 *  - Input pointers are borrowed for the duration of the call only.  Handles
 *    are owned by the library and released with their *_free / *_close call.
 *    Output buffers are caller-owned host memory unless stated otherwise.
 *  - Pointers tagged with a ptr_kind argument may be host (EAHR_PTR_HOST) or
 *    device (EAHR_PTR_DEVICE, memory of the GPU the index lives on).
 *  - Calls on one handle are not thread-safe; a pvs_state must not be used
 *    while its pvs_index is being modified.
 */
#ifndef EAHR_H
#define EAHR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status */
enum {
    EAHR_OK = 0,
    EAHR_E_INVALID = -1,    /* bad argument (null pointer, size, unknown epoch, ...) */
    EAHR_E_NONFINITE = -2,  /* NaN or Inf in a corpus row or a query (App. A.1)      */
    EAHR_E_RANGE = -3,      /* dimension too large: a_m >= 1, or 127^2 d >= 2^31      */
    EAHR_E_OOM = -4,        /* device or host allocation failed                       */
    EAHR_E_HIP = -5,        /* HIP runtime error                                      */
    EAHR_E_FAILED = -6      /* a ranked list failed (Sec. 2.1): see per-query status  */
};

/* Ranked-list states (Sec. 2.1): an Open list may extend its exact prefix, an
 * Exhausted list is complete, a Failed list invalidates the request. */
enum { EAHR_LIST_OPEN = 0, EAHR_LIST_EXHAUSTED = 1, EAHR_LIST_FAILED = 2 };

enum { EAHR_PTR_HOST = 0, EAHR_PTR_DEVICE = 1 };

typedef struct pvs_index pvs_index;
typedef struct pvs_state pvs_state;
typedef struct pbm_index pbm_index;
typedef struct pbm_state pbm_state;
typedef struct pbm_gpu_state pbm_gpu_state;

/* ------------------------------------------------------------ PVS (dense) */

/* pvs_build -- quantise a float32 corpus (Sec. 2.3.1).
 *   corpus  n x d float32, row-major, host or device (ptr_kind).
 *   stream  hipStream_t every later call on this index and its states uses
 *           (NULL: the default stream).
 * Per row v the index stores the scale s_v = fl32(||v||_inf / 127) (1 for a zero
 * row), the codes z_v = clip(round_half_away(fl32(v_j / s_v)), -127, 127), the
 * float32 norms ||v||_2 and ||v - s_v z_v||_2 rounded up, and a copy of the
 * float32 row for authoritative scoring.  Epoch 0 (all n rows visible) is
 * created.  Errors: EAHR_E_NONFINITE for NaN/Inf anywhere in the corpus,
 * EAHR_E_RANGE when d > 4096 (guard and Int32 accumulator range, App. A.1). */
int pvs_build(const float* corpus, int64_t n, int32_t d, int32_t ptr_kind,
              void* stream, pvs_index** out);

/* Quantisation modes of pvs_build_quant. */
enum { EAHR_QUANT_PER_VECTOR = 0, EAHR_QUANT_GLOBAL = 1 };

/* pvs_build_quant -- pvs_build with a choice of scale: EAHR_QUANT_PER_VECTOR
 * is pvs_build (one scale per row, Sec. 2.3.1); EAHR_QUANT_GLOBAL gives every
 * row one shared scale s = fl32(max |x| / 127) over the corpus (1 for an
 * all-zero corpus), the scalar-quantisation interval generator that Sec. 3.5
 * and Sec. 4.4 (Table 4-1) compare PVS with.  Codes, norms, intervals,
 * rescoring and the pvs_next contract are otherwise identical, so the two
 * modes rank identically and differ only in how many pairs are rescored.
 * The shared scale is fixed by the first non-empty pvs_build_quant or
 * pvs_insert; later inserts reuse it, and their codes clip at +-127 (the
 * error norm is computed from the clipped codes, so intervals stay valid).
 * Errors: those of pvs_build, and EAHR_E_INVALID for an unknown mode. */
int pvs_build_quant(const float* corpus, int64_t n, int32_t d, int32_t ptr_kind,
                    void* stream, int32_t quant, pvs_index** out);

/* pvs_insert -- append n_new rows (quantised on insert); their ids are
 * *first_id .. *first_id + n_new - 1.  They are visible in the live state and
 * in epochs taken afterwards, never in earlier epochs. */
int pvs_insert(pvs_index* idx, const float* rows, int64_t n_new, int32_t ptr_kind,
               int64_t* first_id);

/* pvs_delete -- hide ids (host array) from the live state; earlier epochs are
 * unchanged (the visible set of a request is fixed by its snapshot, Sec. 2.4). */
int pvs_delete(pvs_index* idx, const int64_t* ids, int64_t n);

/* pvs_snapshot -- freeze the live visible set as a new epoch. */
int pvs_snapshot(pvs_index* idx, int64_t* epoch);

/* pvs_info -- rows, dimension and visible-row count of an epoch. */
int pvs_info(const pvs_index* idx, int64_t epoch, int64_t* rows, int32_t* d,
             int64_t* visible);

/* pvs_open -- encode a batch of B queries (B x d float32, host or device) the
 * same way as corpus rows and create resumable state on epoch `epoch`.
 * Errors: EAHR_E_NONFINITE for NaN/Inf in a query. */
int pvs_open(const pvs_index* idx, int64_t epoch, const float* q, int32_t B,
             int32_t ptr_kind, pvs_state** out);

/* Dense rank generators of pvs_open_gen. */
enum { EAHR_GEN_INTERVALS = 0, EAHR_GEN_FULL_SCAN = 1 };

/* pvs_open_gen -- pvs_open with a choice of dense rank generator:
 * EAHR_GEN_INTERVALS is pvs_open (interval scans over the index's codes,
 * Sec. 2.3.1); EAHR_GEN_FULL_SCAN scores every visible row in float32 on the
 * first pvs_next that needs ranks, sorts them once and serves every later
 * rank from that complete ranking: the exhaustive float32 scan that Sec. 3.5
 * and Sec. 4.4 (Table 4-1) compare PVS with.  Scores are the same
 * authoritative float32 dot products, so both generators emit identical
 * ranks.  The full scan needs 16 bytes of device memory per row of the epoch
 * and query of a group (groups are sized to 4 GiB) and keeps 8 bytes per
 * visible row and query on the host.  Errors: those of pvs_open, and
 * EAHR_E_INVALID for an unknown generator. */
int pvs_open_gen(const pvs_index* idx, int64_t epoch, const float* q, int32_t B,
                 int32_t ptr_kind, int32_t generator, pvs_state** out);

/* pvs_next -- extend each active query's exact dense prefix by up to m ranks
 * (Sec. 2.3.1 resumable generation).  The complete list orders the visible
 * rows by (authoritative float32 inner product descending, id ascending);
 * the authoritative score is one float32 dot product in a fixed order.
 *   active  B flags (NULL: all active); inactive queries are left untouched.
 *   ids     B x m, scores B x m: row b receives count[b] (id, score) pairs.
 *   count   B: number written; count[b] < m only when status[b] is
 *           EAHR_LIST_EXHAUSTED.
 *   status  B: EAHR_LIST_* after the call.  Failed is sticky: it is set when a
 *           rescored score lies outside its interval (App. A.1); such a query
 *           returns count 0 from then on.
 * Returns EAHR_OK even when some queries failed (see status).
 * Test hook: with the environment variable EAHR_TEST_FAIL_QUERY=b set when a
 * state is opened, rescoring judges query b's scores against a zero-width
 * interval around c, so that query fails through this containment check. */
int pvs_next(pvs_state* st, int32_t m, const uint8_t* active, int64_t* ids,
             float* scores, int32_t* count, int32_t* status);

/* Counters of one state (summed over its queries). */
typedef struct {
    int64_t scans;           /* full interval scans over the codes             */
    int64_t sample_scans;    /* threshold-estimation passes over sampled rows  */
    int64_t rows_scanned;    /* visible-or-not rows streamed by full scans     */
    int64_t bytes_scanned;   /* code + metadata bytes streamed by full scans   */
    int64_t candidates;      /* (query, row) pairs rescored in float32         */
    int64_t certified;       /* ranks certified by scans                       */
    int64_t emitted;         /* ranks returned by pvs_next                     */
    int64_t rescans;         /* scans repeated with a lower threshold          */
    int64_t overflows;       /* query scans repeated because the candidate pool
                              * or the query's key region was too small       */
} pvs_counters;

int pvs_stats(const pvs_state* st, pvs_counters* out);

/* Process-wide kernel timing of the dense channel, measured with HIP events
 * recorded on the index's stream around each kernel group of a scan (all
 * states, all threads).  Disabled by default; enabling adds event records and
 * no synchronisation.  Times in milliseconds, bytes algorithmic:
 * rows * (d + 12) + 8 bytes per 64-row visibility word for a full scan pass. */
typedef struct {
    double scan_ms;          /* full interval scans (kernel time)            */
    int64_t scan_launches;   /* kernel launches those scans used             */
    int64_t scan_bytes;      /* algorithmic bytes those launches streamed    */
    double sample_ms;        /* threshold sampling + selection               */
    double rescore_ms;       /* float32 rescoring of candidates              */
    int64_t rescore_rows;    /* candidate pairs rescored                     */
    double sort_ms;          /* candidate sort and packing                   */
    int64_t scan_rounds;
    int64_t mfma_launches;   /* scan launches that used the Int8 MFMA kernel */
    double host_dense_ms;    /* eahr_topk: wall time of its pvs_next calls   */
    double host_sparse_ms;   /* eahr_topk: wall time of its PBM rounds       */
    double host_fuse_ms;     /* eahr_topk: wall time of certification        */
    /* Full scans per kernel variant: [0..7] dot4 GEMV with 1..8 queries per
     * launch, [8..11] Int8 MFMA with 1, 2, 4, 8 tiles of 32 queries.  A scan
     * pass of one variant is one launch. */
    double variant_ms[12];
    int64_t variant_launches[12];
    int64_t variant_bytes[12];
    int64_t rescore_certified;   /* candidates certified by rescoring (keys written) */
    int64_t rescore_row_reads;   /* row loads of rescoring: one per run of pairs of one
                                  * row inside a wavefront's share */
} pvs_profile;

int pvs_profile_enable(int32_t on);   /* also clears the accumulators */
int pvs_profile_read(pvs_profile* out);

/* Debug / test entry points (not on the retrieval path):
 * pvs_read_index -- copy rows [row0, row0+n) of the index to host: codes
 *   n x d int8 (row-major), meta n x 3 float32 (s_v, ||v||_2 up, ||e_v||_2 up).
 * pvs_read_query -- copy the encoded batch: codes B x d int8, meta B x 4
 *   float32 (s_q, ||q||_2 up, ||q_hat||_2 up, ||e_q||_2 up).
 * pvs_intervals -- score intervals [lo, hi] of query b against n host-listed
 *   rows, computed by the scan's own device code.
 * pvs_scores -- authoritative float32 scores of query b against n rows. */
int pvs_read_index(const pvs_index* idx, int64_t row0, int64_t n, int8_t* codes,
                   float* meta);
int pvs_read_query(const pvs_state* st, int8_t* codes, float* meta);
int pvs_intervals(const pvs_state* st, int32_t b, const int64_t* rows, int64_t n,
                  float* lo, float* hi);
int pvs_scores(const pvs_state* st, int32_t b, const int64_t* rows, int64_t n,
               float* scores);

/* Largest n of one pvs_scores_noalloc call. */
#define EAHR_NOALLOC_MAX_ROWS 65536

/* pvs_scores_noalloc -- pvs_scores for callers that cannot allocate memory
 * (code under HIP stream capture, tight serving loops, harnesses that forbid
 * allocation): the same arguments (host rows and scores), results and
 * errors, plus EAHR_E_RANGE when n > EAHR_NOALLOC_MAX_ROWS.  It calls no
 * allocator: the row ids and scores are staged in one fixed array of device
 * memory per GPU (EAHR_NOALLOC_MAX_ROWS * 12 bytes, held until the process
 * ends) that every call on that GPU shares, so calls that overlap on one GPU
 * race. */
int pvs_scores_noalloc(const pvs_state* st, int32_t b, const int64_t* rows, int64_t n,
                       float* scores);

/* pvs_close releases a state.  pvs_free releases an index; while states
 * opened on it are still open (also states held by a merge) the release
 * waits for the last of them to be closed, and the index accepts no new
 * pvs_open.  Both accept NULL. */
void pvs_close(pvs_state* st);
void pvs_free(pvs_index* idx);

/* ------------------------------------------- hierarchical merging (dense) */

/* Hierarchical merging of exact dense rankings (Sec. 2.4).  A Segment is a
 * pvs_index whose rows stand for global item ids; a Shard merges the
 * rankings of its Segments, and a request merges its Shards, each by (score
 * descending, global id ascending), into one resumable ranking with the
 * pvs_next contract.  An item visible in more than one Segment is emitted
 * once when its copies agree on score and version.  Copies that disagree
 * invalidate the request whatever depth it reaches, so they are compared
 * when the merge is opened (pvs_merge_open within a Shard, pvs_merge_shards
 * across Shards): a version conflict fails every query, a score conflict the
 * queries it occurs for, and such a query's merged list is Failed (sticky)
 * from its first pvs_merge_next, as it is when a Segment's list fails. */
typedef struct pvs_merge pvs_merge;

/* pvs_merge_open -- open a Shard over n_segs Segments for B queries.
 *   segs[s]      the Segment's index; epochs[s] its snapshot (NULL: all 0).
 *   gids[s]      host array, one global id in [0, 2^31 - 1) per row of the snapshot,
 *                strictly ascending (so the Segment's own id order is the
 *                global one); copied.
 *   versions[s]  host array of per-row versions, or NULL (all 0); versions
 *                may be NULL.  Copied.
 *   q            B x d float32 queries (host or device, ptr_kind).
 * Errors: EAHR_E_INVALID for null arguments or ids that are negative or
 * not ascending; those of pvs_open. */
int pvs_merge_open(const pvs_index* const* segs, const int64_t* epochs,
                   const int64_t* const* gids, const int64_t* const* versions,
                   int32_t n_segs, const float* q, int32_t B, int32_t ptr_kind,
                   pvs_merge** out);

/* pvs_merge_shards -- the request-level merge over n_shards Shards opened by
 * pvs_merge_open on the same B queries and not read yet.  The request takes
 * ownership of the Shards: close only the returned handle. */
int pvs_merge_shards(pvs_merge** shards, int32_t n_shards, pvs_merge** out);

/* pvs_merge_next -- next m merged ranks per active query; ids are global
 * ids.  Same count/status contract as pvs_next. */
int pvs_merge_next(pvs_merge* mg, int32_t m, const uint8_t* active, int64_t* ids,
                   float* scores, int32_t* count, int32_t* status);

/* pvs_merge_close -- release a merge (and, for a request, its Shards). */
void pvs_merge_close(pvs_merge* mg);

/* ------------------------------------------------------------ PBM (sparse) */

/* pbm_build -- Posting Block-Max index over term-major postings (Sec. 2.3.2).
 *   term_ptr  vocab+1 offsets into docs/impacts; docs of one term strictly
 *             ascending and < n_docs; impacts finite and >= 0 (App. A.2).
 *   range_size  documents per contiguous id range (>= 1).
 * The index stores, per term and range, the maximum impact m_t(R) and where
 * the term's postings for R start.  Copies its inputs.  Host only. */
int pbm_build(const int64_t* term_ptr, int32_t vocab, const int32_t* docs,
              const float* impacts, int64_t n_docs, int32_t range_size,
              pbm_index** out);
/* pbm_free -- release the index; while states opened on it are still open
 * the release waits for the last pbm_close (no new pbm_open meanwhile). */
void pbm_free(pbm_index* idx);

/* A sparse query: n_terms distinct term ids with weights q_t >= 0. */
typedef struct {
    const int32_t* terms;
    const float* weights;
    int32_t n_terms;
} eahr_sparse_query;

/* pbm_open / pbm_next -- resumable exact sparse ranking of one query: items
 * with S(x) > 0 in (S descending, id ascending) order, S accumulated in float32
 * in ascending term order.  Same count/status contract as pvs_next. */
int pbm_open(const pbm_index* idx, const eahr_sparse_query* q, pbm_state** out);
int pbm_next(pbm_state* st, int32_t m, int64_t* ids, float* scores, int32_t* count,
             int32_t* status);
void pbm_close(pbm_state* st);

/* Sparse rank generators of pbm_open_gen (EAHR_SPARSE_PBM_GPU only for
 * eahr_params.sparse_generator: its states are pbm_gpu_open batches). */
enum { EAHR_SPARSE_PBM = 0, EAHR_SPARSE_COMPLETE = 1, EAHR_SPARSE_PBM_GPU = 2 };

/* pbm_open_gen -- pbm_open with a choice of generator: EAHR_SPARSE_PBM is
 * pbm_open (ranges expanded in bound order, ranks published when no
 * unexpanded range can precede them, Sec. 2.3.2); EAHR_SPARSE_COMPLETE scores
 * every document of every range with a positive bound at the first pbm_next
 * and sorts them once: the complete exact sparse ranking that Sec. 3.5 and
 * Sec. 4.4 (Table 4-1) compare PBM with.  Both give identical rankings and
 * scores.  Errors: those of pbm_open, and EAHR_E_INVALID for an unknown
 * generator. */
int pbm_open_gen(const pbm_index* idx, const eahr_sparse_query* q, int32_t generator,
                 pbm_state** out);

/* pbm_debug_set_blockmax -- test hook: overwrite m_t(R) of one (term, range)
 * entry so that a later pbm_open sees metadata that no longer covers its
 * postings; pbm_next then reports EAHR_LIST_FAILED (App. A.2).  Returns
 * EAHR_E_INVALID when the term has no postings in that range. */
int pbm_debug_set_blockmax(pbm_index* idx, int32_t term, int64_t range, float value);

/* ------------------------------------------------- PBM on the GPU (sparse) */

/* Largest range_size the GPU generator handles (a range's scores live in
 * the LDS of one workgroup). */
#define EAHR_PBM_GPU_MAX_RANGE 16384

/* pbm_upload -- copy the index's postings and block-max table to the
 * current GPU (about 8 bytes per posting and 20 per block-max entry).  The
 * first pbm_gpu_open does it when no copy exists; later calls do nothing.
 * The copy lives until pbm_free; pbm_debug_set_blockmax updates it too.
 * Errors: EAHR_E_INVALID (NULL), EAHR_E_OOM / EAHR_E_HIP. */
int pbm_upload(const pbm_index* idx);

/* pbm_gpu_open -- B sparse queries ranked by Posting Block-Max with the
 * posting work on the GPU (Sec. 2.3.2, App. A.2): the bounds H(R) of every
 * (query, range) pair in one kernel, one thread per pair; later, every
 * expanded range's documents scored by one workgroup in LDS.  Each query's
 * ranking, scores and work counters equal those of pbm_open + pbm_next on the
 * same query (H and S are accumulated in the same order with the same
 * roundings; the host keeps the bound order, the expansion batches and the
 * publication rule of the host generator).  The index must stay alive and
 * unmodified while the state is open (pbm_free waits for pbm_gpu_close).
 * Errors: those of pbm_open for any query; EAHR_E_RANGE when range_size >
 * EAHR_PBM_GPU_MAX_RANGE; EAHR_E_OOM / EAHR_E_HIP. */
int pbm_gpu_open(const pbm_index* idx, const eahr_sparse_query* q, int32_t B, pbm_gpu_state** out);
/* pbm_gpu_next -- the next m[b] ranks of every query b with m[b] > 0, as
 * pbm_next(m[b]) would give them, into the host arrays ids[b] / scores[b]
 * (m[b] entries each; unused when m[b] == 0).  Queries with m[b] == 0 are
 * untouched (count 0, their current status).  The expansions of all queries
 * that need one run in the same device rounds.  A range whose scores exceed
 * its bound fails its query only (EAHR_LIST_FAILED, count 0, sticky).
 * Errors: EAHR_E_INVALID (NULL pointers, m[b] < 0), EAHR_E_OOM / EAHR_E_HIP. */
int pbm_gpu_next(pbm_gpu_state* st, const int32_t* m, int64_t* const* ids, float* const* scores,
                 int32_t* count, int32_t* status);
/* pbm_gpu_counters -- work of query b so far: out[0] postings visited,
 * out[1] documents scored, out[2] ranges expanded (Sec. 3.5 counters). */
int pbm_gpu_counters(const pbm_gpu_state* st, int32_t b, int64_t* out);
void pbm_gpu_close(pbm_gpu_state* st);

/* -------------------------------------------------------- EAHR (fusion) */

typedef struct {
    int32_t K;           /* requested result size                                */
    int32_t depth0;      /* first cumulative depth requested from each list (20)  */
    int32_t growth;      /* depth multiplier per round (2)                        */
    int32_t k_rrf;       /* rank constant k >= 1                                  */
    int32_t w_dense;     /* rank-scaled weights w_i >= 0 (Sec. 2.1), integers     */
    int32_t w_sparse;
    int32_t dense_generator;   /* EAHR_GEN_* of the dense channel (0: intervals)  */
    int32_t schedule;          /* EAHR_SCHED_*: depth doubling (0) or the frozen
                                * scheduler of Sec. 3.5 (1); the result is the same */
    int32_t sparse_generator;  /* EAHR_SPARSE_* of the sparse channel (0: PBM on the
                                * host, 2: PBM with its posting work on the GPU) */
} eahr_params;

/* Depth schedules of eahr_params.schedule.  EAHR_SCHED_DOUBLING: every Open
 * list advances to depth0 * growth^j per round.  EAHR_SCHED_FROZEN (Sec. 3.5):
 * one list per step, at most 16 ranks, the one with the larger weighted-RRF
 * contribution at its next unread rank (ties: dense) unless the other was
 * skipped 16 steps in a row; certification after every step through the
 * first 4K ranks of cumulative access, then after a further 1/8 of the
 * access (64 to 1,024 ranks), and at once when a list is read to its end.
 * eahr_fuse_lists ignores its step argument under the frozen schedule. */
enum { EAHR_SCHED_DOUBLING = 0, EAHR_SCHED_FROZEN = 1 };

typedef struct {
    int64_t dense_depth;    /* d_i: ranks read from each list        */
    int64_t sparse_depth;
    int64_t dense_len;      /* n_i, or -1 while unknown (list Open)  */
    int64_t sparse_len;
    int32_t dense_status;   /* EAHR_LIST_* at the end                */
    int32_t sparse_status;
    int32_t rounds;         /* depth rounds taken                    */
    int32_t resolved;       /* 1 when the ordered Top-K was fixed    */
    /* work counters of Sec. 3.5 (0 for a merged dense channel) */
    int64_t dense_evals;     /* (query, item) pairs scored in float32  */
    int64_t sparse_postings; /* postings read by the sparse channel    */
    int64_t sparse_scored;   /* sparse items given an exact score      */
} eahr_query_stats;

/* eahr_topk -- the ordered Top-K of complete-list weighted RRF (Sec. 2.1) for
 * B queries, without a preset per-list depth: every Open list with positive
 * weight advances to cumulative depth depth0 * growth^j, and after every round
 * positions are fixed one at a time with the unread-rank bounds (Sec. 2.2).
 * Exhausted lists contribute their complete rankings.
 *   q_dense   B x d float32 (host or device, q_ptr_kind); q_sparse: B queries.
 *   out_ids   B x K; out_count[b] = q_K = min(K, |U+|) (no zero-score padding).
 *   out_status[b] = 0 on success, EAHR_LIST_FAILED when a list failed.
 *   stats     B entries or NULL.
 * Returns EAHR_E_FAILED if any query failed (others are still valid). */
int eahr_topk(const pvs_index* dense, int64_t epoch, const pbm_index* sparse,
              const float* q_dense, int32_t q_ptr_kind,
              const eahr_sparse_query* q_sparse, int32_t B, const eahr_params* params,
              int64_t* out_ids, int32_t* out_count, int32_t* out_status,
              eahr_query_stats* stats);

/* eahr_topk_merged -- eahr_topk whose dense channel is a merged ranking
 * (pvs_merge_open / pvs_merge_shards, opened on the same B queries and not
 * read yet; it stays the caller's to close and is read on by this call).
 * Sparse document ids must be the merge's global ids.  The dense channel
 * uses interval scans (params->dense_generator must be EAHR_GEN_INTERVALS).
 * Outputs and errors as eahr_topk. */
int eahr_topk_merged(pvs_merge* dense, const pbm_index* sparse,
                     const eahr_sparse_query* q_sparse, int32_t B, const eahr_params* params,
                     int64_t* out_ids, int32_t* out_count, int32_t* out_status,
                     eahr_query_stats* stats);

/* eahr_fuse_lists -- the same fusion over two complete rankings given as host
 * arrays of distinct ids (e.g. controlled rank streams, Sec. 3.4).  Both lists
 * advance together: by `step` ranks per round (step > 0, certification after
 * every step) or to cumulative depth depth0 * growth^j (step = 0).  A list is
 * Exhausted once all of it has been read.  Host only; no GPU involved.
 *   out_ids  K entries (q_K valid, rest -1);  stats  one entry or NULL. */
int eahr_fuse_lists(const int64_t* list_d, int64_t n_d, const int64_t* list_s,
                    int64_t n_s, const eahr_params* params, int32_t step,
                    int64_t* out_ids, int32_t* out_count, eahr_query_stats* stats);

/* eahr_set_rank_observer -- register fn (process-wide; NULL clears) to see
 * every rank eahr_topk and eahr_topk_merged read from their channels, for
 * tests and tracing.  fn is called on the thread that called eahr_topk,
 * after each read and before the read ranks are certified: `list` is 0
 * (dense) or 1 (sparse), `first` the 0-based position of the first of the n
 * ranks in the query's list, ids and scores the ranks themselves (valid
 * during the call only).  Reads of a query that failed or was already
 * resolved are not reported.  The observer adds no work to the channels
 * and cannot change a result. */
typedef void (*eahr_rank_observer)(void* user, int32_t query, int32_t list, int64_t first,
                                   const int64_t* ids, const float* scores, int64_t n);
int eahr_set_rank_observer(eahr_rank_observer fn, void* user);

/* Last error message of the calling thread (static storage, never NULL). */
const char* eahr_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* EAHR_H */
