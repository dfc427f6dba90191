// Host-side structures of the PVS runtime (index in HBM, per-query state).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <vector>

#include "eahr.h"
#include "host_parallel.h"
#include "pvs_kernels.h"

// A query's certified ranks as sort keys; grown without zero-filling (the
// keys are copied in right after).
using KeyCache = std::vector<uint64_t, ::eahr::NoInit<uint64_t>>;

namespace pvs {
// Threshold estimation samples every stride-th code block, with the stride
// the largest power of two that keeps at least this many blocks sampled.
// With stride 1 tau is the target-th largest lower bound, so at least the
// target is certified.  With a larger stride tau is taken from the sampled
// interval midpoints (close to the scores, so the rows certified, s >= tau,
// number about the target scaled by the stride) with this relative margin.
constexpr int64_t kSampleBlocks = 2048;
constexpr double kSampleMargin = 1.25;
// Smallest candidate pool allocated for a scan, and the largest pool one scan
// round may use (queries beyond it wait for the next round).
constexpr int64_t kMinCap = 4096;
constexpr int64_t kPoolMax = int64_t(1) << 28;
// Candidate regions are sized from the sample: hits / sampled fraction times
// kCapSlack plus kCapPad slots.
constexpr double kCapSlack = 1.5;
constexpr int64_t kCapPad = 2048;
// Ranks a scan aims to certify per query beyond the request: about
// kTargetBudget / (queries in the scan), clamped to [kTargetMin, kTargetMax].
// A single-query scan streams the whole code array, so certifying a deep
// prefix at once is cheap; a large batch shares one scan among many queries
// and pays float32 rescoring per candidate instead.
constexpr int64_t kTargetMin = 64;
constexpr int64_t kTargetMax = 2048;
constexpr int64_t kTargetBudget = 8192;
// Callers extend prefixes geometrically, so a scan also certifies ahead:
// up to kSpecFactor times the depth reached after the request, within
// kSpecBudget ranks per scan shared by its queries.  Rescoring a row costs
// about 1/1000 of streaming the codes once, so over-certifying is cheap next
// to an extra scan.  Measured on 8.8M x 768 (queries/s at batch 256 / 1 / 64):
// factor 8 and 2^20 ranks 1,860 / 90 / 1,085; 8 and 2^22 2,355 / 106 / 1,128;
// 16 and 2^22 2,338 / 117 / 1,241; 2^23 and 2^24 are slower again.
// A scan certifies at least max(kSpecFloor, kSpecFloorBudget / queries)
// ranks per query (within the same budget): a round of a batch scan costs
// about as much as rescoring a few thousand ranks per query, and a round of
// a single-query scan (the whole code array streamed once) as much as
// rescoring about 10^5, so shallow requests are served ahead.  Measured on
// 8.8M x 768, single requests: floor budget 2^16 179 queries/s, 2^17 252,
// 2^18 247 (4096 alone: 182; batches of 64 and 256 unchanged).  Re-measured
// after the other changes (ms per batch-256 / batch-64 step): floor 4096 and
// 2^22 ranks 94.8 / 43.3; 8192 99.9 / 49.0; 2048 100.5 / 46.1; 2^23 94.4 / 44.0.
constexpr int64_t kSpecFactor = 16;
constexpr int64_t kSpecBudget = int64_t(1) << 22;
constexpr int64_t kSpecFloor = 4096;
constexpr int64_t kSpecFloorBudget = int64_t(1) << 17;
// Scans of at least this many queries use the Int8 MFMA kernel; smaller ones
// the dot4 GEMV kernel, which streams the codes at the HBM rate for up to 8
// queries in one pass.  EAHR_SCAN_PATH=gemv|mfma forces one path (testing).
constexpr int32_t kMfmaMinQueries = 9;
enum class ScanPath { Auto, Gemv, Mfma };
}  // namespace pvs

// Whether pvs_next(m) on the active queries would be served from certified
// ranks alone (no scan).
bool pvs_covered(const pvs_state* st, int32_t m, const uint8_t* active);
// pvs_next without scores: only the ids of the emitted ranks are written.
int pvs_next_ids(pvs_state* st, int32_t m, const uint8_t* active, int64_t* ids, int32_t* count,
                 int32_t* status);
// Deepen the certified caches of the active queries of a state to `depth`
// ranks each (or to exhaustion) without emitting anything; a later pvs_next
// is then served from the caches.  The host fusion calls it while the CPU
// sparse channel of a round is still running, so the GPU works ahead.
// `added` (optional) receives the number of ranks certified by the call.
int pvs_fill(pvs_state* st, int64_t depth, const uint8_t* active, int64_t* added);
// pvs_fill whose scans certify about `depth` ranks per query and nothing
// further ahead (the caller sized the depth itself).
int pvs_fill_exact(pvs_state* st, int64_t depth, const uint8_t* active, int64_t* added);
// The caller reads no further ranks of query b (its request is settled): the
// query's certified keys that are still in a scan's pinned copy are not
// moved to its cache any more, and pvs_next / pvs_fill skip the query.
void pvs_retire(pvs_state* st, int32_t b);
// Whether query b of a state has failed (a rescored score outside its
// interval), also in work-ahead that pvs_next has not reported yet.
bool pvs_query_failed(const pvs_state* st, int32_t b);
// (query, row) pairs of query b scored in float32 so far.
int64_t pvs_query_evals(const pvs_state* st, int32_t b);
// Batch size a merged ranking was opened for (pvs_merge.cpp).
int32_t eahr_merge_batch(const pvs_merge* mg);
// No rank of the merge has been returned yet (and no query failed).
bool eahr_merge_unread(const pvs_merge* mg);

// Process-wide profile hooks used by the host fusion (pvs_profile_enable).
bool pvs_profile_on();
void pvs_profile_add_host(double dense_ms, double sparse_ms, double fuse_ms);

// Scan buffers of a state (device, plus pinned host mirrors).  A closing
// state hands them to its index, and the next state opened on that index
// adopts them, so repeated requests do not re-allocate them.
struct ScanBuffers {
    int32_t buf_nq = 0;
    int64_t buf_sample = 0;
    pvs::ScanQ* scanq = nullptr;
    int32_t* counts = nullptr;
    float* sample_lo = nullptr;
    float* sample_hi = nullptr;
    void* qfrag = nullptr;
    int64_t pool_cap = 0;
    uint4* pairs = nullptr;         // candidate pair records of a scan (pool)
    uint64_t* keys = nullptr;
    uint64_t* keys_tmp = nullptr;
    uint64_t* packed = nullptr;
    pvs::ScanQ* h_scanq = nullptr;
    int32_t* h_counts = nullptr;
    uint64_t* h_packed = nullptr;
    int64_t h_packed_cap = 0;
    // certified-rank caches of the closed state (emptied, capacity kept)
    std::vector<KeyCache> caches;
};

struct pvs_index {
    struct Snapshot {
        int64_t rows = 0;      // physical rows visible to the epoch (prefix)
        int64_t visible = 0;   // set bits of vis
        uint64_t* vis = nullptr;  // device bitmap, one word per 64-row block
    };
    int device = 0;
    hipStream_t stream = nullptr;
    int32_t d = 0, dp = 0, df = 0, nchunk = 0;
    int64_t rows = 0, cap = 0;
    int8_t* codes = nullptr;   // cap x dp, chunk-major 64-row blocks
    float* scale = nullptr;    // s_v
    float* vnorm = nullptr;    // ||v||_2 rounded up
    float* enorm = nullptr;    // ||e_v||_2 rounded up
    float* frows = nullptr;    // cap x df float32 rows
    uint64_t* live = nullptr;  // live visibility bitmap
    uint32_t* flags = nullptr;
    float* staging = nullptr;  // host->device staging for quantisation
    float nv_max = 0.0f, nev_max = 0.0f;
    float gamma = 0.0f;
    int32_t quant = EAHR_QUANT_PER_VECTOR;   // per-vector scales, or one shared scale
    float global_s = 0.0f;                   // the shared scale once fixed (global mode)
    std::vector<Snapshot> snaps;
    mutable ScanBuffers spare;   // buffers of the last closed state
    mutable bool has_spare = false;
    // states opened on the index and not closed yet; pvs_free while some are
    // open only marks the index, and the last pvs_close releases it
    mutable std::mutex life_mu;
    mutable int64_t open_states = 0;
    mutable bool release_requested = false;
    ~pvs_index();
};

struct pvs_state {
    struct Query {
        float sq = 0, nq = 0, nqh = 0, neq = 0, wmax = 0;
        bool has_cert = false;          // a rank has been certified
        float s_cert = 0.0f;            // key (s_cert, id_cert) of the last certified rank
        int32_t id_cert = -1;
        // certified ranks in order, as their sort keys (~mono(s32) << 32 | id);
        // ids and scores are decoded only when emitted
        KeyCache cache;
        // the keys of its last scan that follow the cache, still in that
        // scan's pinned copy (h_packed[pend_off .. pend_off + pend_n))
        int64_t pend_off = 0, pend_n = 0;
        bool retired = false;           // no further ranks will be read (pvs_retire)
        int64_t emitted = 0;            // ranks returned by pvs_next
        bool failed = false;
        bool cert_exhausted = false;    // every visible row certified
        int retries = 0;                // consecutive scans that certified too few
        int64_t cap_hint = 0;           // candidate capacity needed by the last overflow
        int64_t evals = 0;              // (query, row) pairs rescored in float32
    };
    const pvs_index* ix = nullptr;
    int64_t epoch = 0;
    int32_t B = 0;
    int32_t generator = EAHR_GEN_INTERVALS;   // interval scans, or one exhaustive float32 scan
    int64_t n_rows = 0, n_vis = 0;
    const uint64_t* vis = nullptr;
    int8_t* qcodes = nullptr;   // B x dp row-major
    float* qrows = nullptr;     // B x df
    float *qscale = nullptr, *qnorm = nullptr, *qenorm = nullptr, *qhnorm = nullptr;
    uint32_t* qflags = nullptr;
    std::vector<Query> q;
    std::vector<KeyCache> recycled;   // caches adopted from the index
    pvs_counters stats{};
    // per-query scan buffers, sized for buf_nq queries and buf_sample rows
    int32_t buf_nq = 0;
    int64_t buf_sample = 0;
    pvs::ScanQ* scanq = nullptr;
    int32_t* counts = nullptr;
    float* sample_lo = nullptr;
    float* sample_hi = nullptr;
    void* qfrag = nullptr;             // query codes in MFMA operand order
    // candidate pool (pool_cap slots) split into per-query regions per scan
    int64_t pool_cap = 0;
    uint4* pairs = nullptr;
    uint64_t* keys = nullptr;
    uint64_t* keys_tmp = nullptr;
    uint64_t* packed = nullptr;
    pvs::ScanPath path = pvs::ScanPath::Auto;
    bool spec_off = false;             // scans certify no further ahead than asked
    // test knob: first-attempt key regions and pool divided by this, so that
    // the overflow and rescan paths run (results do not change)
    int64_t cap_shrink = 1;
    // test knob (EAHR_TEST_FAIL_QUERY): this query's rescoring judges its
    // scores against a zero-width interval, so its list fails through the
    // normal containment check (App. A.1); -1: off
    int32_t test_fail_qi = -1;
    hipEvent_t ev[7] = {};             // profiling events (created on first use)
    pvs::ScanQ* h_scanq = nullptr;     // pinned host mirrors
    int32_t* h_counts = nullptr;
    uint64_t* h_packed = nullptr;
    int64_t h_packed_cap = 0;
    void release_scan_buffers();
    ~pvs_state();
};
