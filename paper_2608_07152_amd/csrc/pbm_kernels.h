// Internal interface between the PBM host runtime and its gfx950 kernels
// (the sparse channel ranked on the GPU, Sec. 2.3.2, App. A.2).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pbmg {

// Largest range the expansion kernel accumulates in LDS (64 KiB of float32).
constexpr int32_t kMaxRangeSize = 16384;

// Device copy of a pbm_index: postings and the block-max table.
struct IndexView {
    const int32_t* docs;       // postings, ascending per term
    const float* imp;          // impact of each posting
    const int64_t* term_ptr;   // vocab + 1
    const int64_t* bm_ptr;     // vocab + 1: block-max entries of each term
    const int32_t* bm_range;   // range of each entry, ascending per term
    const float* bm_max;       // m_t(R)
    const int64_t* bm_off;     // first posting of the term inside the range
    int32_t range_size;
    int64_t n_docs;
    int64_t n_ranges;
};

// The terms of a batch of queries: query b owns [qptr[b], qptr[b + 1]) of
// qterm / qw, ascending term ids, every weight > 0.
struct QueryView {
    const int32_t* qptr;
    const int32_t* qterm;
    const float* qw;
    int32_t B;
};

// One range of one query to expand.
struct Task {
    int32_t b;      // query
    int32_t r;      // range
    float H;        // its bound H(R)
    int32_t pad;
};

// H[b * n_ranges + r] = H(R) of query b, accumulated in float32 over the
// query's terms in ascending order (one rounding per multiply and add), and
// post[b * n_ranges + r] = the number of the query's postings inside R.
// With ent (may be null): ent[i * n_ranges + r] = the block-max entry of term
// slot i (index into qterm) for range r, or -1.
void launch_bounds(const IndexView& ix, const QueryView& q, float* H, int32_t* post, int64_t* ent,
                   hipStream_t s);

// Scores every document of every task's range that carries a term of the
// task's query (S(x) accumulated like H, in LDS), then for each such
// document: scored[b] += 1; fail[b] = 1 when S(x) > H(R); and when S(x) > 0
// its key (~ord(S) << 32 | id) at keys[key_off[b] + atomicAdd(key_cnt[b])].
// key_off regions must hold the postings of the query's tasks.  ent: the
// table of launch_bounds for these queries, or null (entries found by
// binary search).  Returns 0, or -1 when the kernel cannot get its LDS.
int launch_expand(const IndexView& ix, const QueryView& q, const Task* tasks, int32_t ntasks,
                  const int64_t* ent, const int64_t* key_off, int32_t* key_cnt, int32_t* scored,
                  int32_t* fail, uint64_t* keys, hipStream_t s);

}  // namespace pbmg
