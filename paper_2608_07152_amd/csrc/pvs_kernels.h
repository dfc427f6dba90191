// Internal interface between the PVS host runtime and its gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pvs {

constexpr int kBlockRows = 64;     // rows per code block (one wavefront lane per row)
constexpr int kChunk = 16;         // bytes of one code chunk (one 16-byte load per lane)
constexpr int kMaxDim = 4096;      // 127^2 * 4096 < 2^31 and a_m < 1
constexpr int kSortTile = 2048;    // keys sorted per workgroup in LDS
constexpr int kMaxGemvQueries = 8; // queries per GEMV scan pass
constexpr int kMaxMfmaQueries = 256;  // queries per MFMA scan pass (8 tiles of 32)
// The candidate pool of a scan is split into kSub sub-regions, each with its
// own append counter; the code block (or workgroup) picks the sub-region
// from its index, so concurrent appends hit kSub different counters instead
// of one.  Counters sit kCntStride ints (64 bytes) apart.
constexpr int kSub = 64;
constexpr int kCntStride = 16;

// Per scanning query, uploaded before every scan.  All fields are read
// uniformly by a wavefront (scalar loads).
struct ScanQ {
    int32_t qi;        // query index inside its state
    float tau;         // interval threshold: candidates have hi >= tau,
                       // certified ranks have s32 >= tau
    float s_cert;      // score of the last certified rank (valid if has_cert)
    int32_t id_cert;   // its row id
    int32_t has_cert;
    int32_t k;         // rank of tau among sampled lower bounds (select pass)
    float sq;          // s_q
    float nq;          // ||q||_2 rounded up
    float nqh;         // ||q_hat||_2 rounded up
    float neq;         // ||e_q||_2 rounded up
    float wmax;        // upper bound of E + G over every row of the index
    int32_t sample_hits;  // sampled eligible rows with hi >= tau (select pass)
    int64_t cand_off;  // first slot of this query's key region
    int64_t cand_cap;  // its key region holds kSub * cand_cap keys
};
static_assert(sizeof(ScanQ) == 64, "ScanQ layout");

// Row storage of an index.  Codes of 64 consecutive rows form one block laid
// out chunk-major: byte j of row r lives at
//   ((r / 64) * nchunk + j / 16) * 1024 + (r % 64) * 16 + j % 16,
// so one 16-byte load per lane streams a whole 1 KiB chunk of a block.
struct IndexView {
    const uint4* codes;
    const float* scale;
    const float* vnorm;
    const float* enorm;
    const float* rows;     // float32 rows, stride df floats
    int32_t d, dp, df, nchunk;
};

// Launchers (all asynchronous on `stream`).
void launch_quantize(const float* src, int64_t nrows, int32_t d, int64_t src_stride,
                     int64_t row0, bool tiled, int8_t* codes, int32_t dp, float* scale,
                     float* vnorm, float* enorm, float* hnorm, float* rows, int32_t df,
                     float fixed_s, uint32_t* flags, hipStream_t stream);
// Largest |x| of count floats into flags[3] (float bits), non-finite into flags[0].
void launch_maxabs(const float* src, int64_t count, uint32_t* flags, hipStream_t stream);

// Outputs of a scan pass.  Sample pass: lower and upper bounds of every
// (query, row) pair of the sampled blocks, row-major [query][sample_ld],
// -inf / -inf for ineligible rows.  Main pass: every candidate pair (hi >= tau)
// becomes one record (row, index of the query in the scan, exact integer dot
// product, 0).  A wavefront reserves all records of its block (or of its
// block and half of the query tiles, in the wide MFMA kernel) with one atomic
// on the counter of sub-region s = block or workgroup index % kSub,
// pair_cnt[s * kCntStride], and writes them at pairs[s * pair_sub + j] for
// j < pair_sub; the counter counts every record handed out, also past the
// sub-region's end (the pool overflowed).  A wavefront writes the records of
// one row next to each other, so rescoring reads the row once for all of
// them.
struct ScanOut {
    float* sample_lo = nullptr;
    float* sample_hi = nullptr;
    int64_t sample_ld = 0;
    int64_t sample_stride = 1;   // sampled blocks are multiples of this
    uint4* pairs = nullptr;
    int64_t pair_sub = 0;        // records per sub-region
    int32_t* pair_cnt = nullptr;
    // main pass: q_evals[s * q_ld + i] (zeroed by the caller), summed over
    // the kSub copies s, counts the records of the query with scan index i,
    // i.e. the float32 evaluations its rescoring will make when the pool did
    // not overflow (a block or workgroup adds to copy s = its index % kSub,
    // so the atomics of concurrent blocks spread over kSub addresses)
    int32_t* q_evals = nullptr;
    int32_t q_ld = 0;
    int32_t qbase = 0;           // scan index of the pass's first query
};

void launch_scan(const IndexView& ix, const uint64_t* vis, int64_t nblocks, const int8_t* qcodes,
                 const ScanQ* sq, int32_t nq, float gamma, bool sample, const ScanOut& o,
                 hipStream_t stream);

// Int8 MFMA variant (same outputs as launch_scan).  `frag` is device scratch
// of (dp / 32) * 8 KiB for the query codes in MFMA operand order.
void launch_scan_mfma(const IndexView& ix, const uint64_t* vis, int64_t nblocks,
                      const int8_t* qcodes, const ScanQ* sq, int32_t nq, float gamma, bool sample,
                      const ScanOut& o, void* frag, hipStream_t stream);
int mfma_tiles_for(int32_t nq);

// tau = k-th largest finite sampled lower bound (or, with midpoint, sampled
// interval midpoint); sample_hits = sampled pairs with hi >= tau (both
// written into sq).
void launch_select(const float* sample_lo, const float* sample_hi, int64_t n, int64_t ld,
                   bool midpoint, ScanQ* sq, int32_t nq, hipStream_t stream);

// Rescoring reads the kept records of every sub-region of the pool (at most
// pair_sub each, in chunks of kRescoreChunk; chunks = rescore_chunks of the
// host copy of the counters), computes each pair's float32 score and checks
// it against its interval, and appends the keys of the certified pairs of
// query b at keys[cand_off + j], j < min(cert_cnt[b], kSub * cand_cap)
// (cert_cnt zeroed by the caller counts them all; order of appends
// unspecified).  cbase is device scratch of kSub + 1 ints; the kSub counters
// row_reads[s * kCntStride] (zeroed by the caller) sum to the number of row
// loads, one per run of records of one row inside a wavefront's share.
// fail_qi (tests only, -1 otherwise): the state query whose rescored scores
// are judged against a zero-width interval, so that its list fails.  nq: the
// scan's queries (records refer to sq[0, nq)); when their float32 query rows
// fit in LDS, workgroups copy them there once instead of reloading them.
constexpr int kRescoreChunk = 256;
int64_t rescore_chunks(const int32_t* pair_cnt, int64_t pair_sub);
void launch_rescore(const IndexView& ix, const float* qrows, const ScanQ* sq, int32_t nq,
                    const int32_t* pair_cnt, const uint4* pairs, int64_t pair_sub,
                    int32_t* cbase, int64_t chunks, float gamma, uint64_t* keys,
                    int32_t* cert_cnt, int32_t* fail, int32_t* row_reads, int32_t fail_qi,
                    hipStream_t stream);

// Sorts every query's candidate keys (cnt[b] keys from cand_off) ascending;
// returns the buffer holding the result (keys or tmp).
// Exhaustive float32 keys of every row of [0, n_rows) for ng queries (state
// query indices qidx, device), query g's keys at keys + g * ld; invisible rows
// get ~0.
void launch_full_keys(const IndexView& ix, const uint64_t* vis, int64_t n_rows, const float* qrows,
                      const int32_t* qidx, int32_t ng, uint64_t* keys, int64_t ld,
                      hipStream_t stream);
uint64_t* launch_segmented_sort(uint64_t* keys, uint64_t* tmp, const int32_t* cnt,
                                const ScanQ* sq, int32_t nq, int64_t max_cnt, hipStream_t stream);

void launch_pack(const uint64_t* keys, const int32_t* cert_cnt, const ScanQ* sq, int32_t nq,
                 int64_t max_cnt, int32_t* offs, uint64_t* packed, hipStream_t stream);

void launch_intervals(const IndexView& ix, const int8_t* qcodes, const ScanQ* sq, float gamma,
                      const int64_t* rows, int64_t n, float* lo, float* hi, hipStream_t stream);

void launch_scores(const IndexView& ix, const float* qrows, int32_t qi, const int64_t* rows,
                   int64_t n, float* out, hipStream_t stream);

void launch_set_bits(uint64_t* vis, int64_t first, int64_t n, hipStream_t stream);
void launch_clear_ids(uint64_t* vis, const int64_t* ids, int64_t n, hipStream_t stream);
void launch_popcount(const uint64_t* vis, int64_t nwords, unsigned long long* out,
                     hipStream_t stream);

}  // namespace pvs
