// Host structures of the Posting Block-Max sparse channel.
#pragma once
#include <cstdint>
#include <mutex>
#include <vector>

#include <hip/hip_runtime.h>

#include "eahr.h"

// Device copy of an index for the GPU generator (pbm_upload): postings and
// the block-max table on one GPU.
struct pbm_device {
    int device = -1;
    int32_t* docs = nullptr;
    float* imp = nullptr;
    int64_t* term_ptr = nullptr;
    int64_t* bm_ptr = nullptr;
    int32_t* bm_range = nullptr;
    float* bm_max = nullptr;
    int64_t* bm_off = nullptr;
};

struct pbm_index {
    int32_t vocab = 0;
    int64_t n_docs = 0;
    int32_t range_size = 1;
    int64_t n_ranges = 0;
    std::vector<int64_t> term_ptr;   // vocab + 1
    std::vector<int32_t> docs;       // postings, ascending per term
    std::vector<float> imp;
    // block-max entries of term t: [bm_ptr[t], bm_ptr[t+1]), ascending range
    std::vector<int64_t> bm_ptr;
    std::vector<int64_t> bm_range;   // range number
    std::vector<float> bm_max;       // m_t(R)
    std::vector<int64_t> bm_off;     // first posting of the term inside the range
    // closed states kept for reuse by later pbm_open calls (their vectors
    // keep their memory)
    mutable std::mutex free_mu;
    mutable std::vector<struct pbm_state*> free_states;
    // states opened on the index and not closed yet; pbm_free while some are
    // open only marks the index, and the last pbm_close releases it
    mutable int64_t open_states = 0;
    mutable bool release_requested = false;
    // device copy (made by pbm_upload or the first GPU open), under dev_mu
    mutable std::mutex dev_mu;
    mutable pbm_device* dev = nullptr;
    // closed GPU states kept for reuse (under free_mu)
    mutable std::vector<struct pbm_gpu_state*> free_gpu_states;
    ~pbm_index();
};

// Checks a query against the index (term ids in range, weights finite and
// non-negative, no term twice) as pbm_open does; EAHR_OK or the error code
// with the message set.
int pbm_check_query(const pbm_index* ix, const eahr_sparse_query* q);

struct pbm_state {
    struct Range {
        float H;
        int32_t post = 0;   // postings of the query inside R (GPU generator)
        int64_t r;
    };
    const pbm_index* ix = nullptr;
    std::vector<int32_t> terms;   // ascending term ids with nonzero weight
    std::vector<float> w;
    // Ranges with H(R) > 0 in expansion order (H desc, first id asc); H(R)
    // is fixed at open, so the order is sorted once.  order[next..] are the
    // unexpanded ranges.
    std::vector<Range> order;
    size_t next = 0;
    std::vector<Range> batch;     // ranges of the current expansion batch
    // ent[i * n_ranges + r]: block-max entry of terms[i] for range r, or -1
    std::vector<int64_t> ent;
    // Scored items as keys (~ord(S) << 32 | id): ascending keys are
    // (S desc, id asc), and an item precedes range R's bound exactly when its
    // key is below (~ord(H(R)) << 32 | first id of R).
    std::vector<uint64_t> pool;   // scored, not yet publishable
    std::vector<uint64_t> ready;  // publishable, sorted; ready[ready_pos..] pending
    size_t ready_pos = 0;
    std::vector<float> acc;       // per-range scratch
    std::vector<uint8_t> seen;
    std::vector<int32_t> touched;
    int64_t emitted = 0;
    int64_t ranges_expanded = 0;
    int64_t postings_visited = 0;
    int64_t items_scored = 0;     // documents given an exact score S(x)
    bool failed = false;
    bool complete = false;        // complete generator: rank everything at the first call
    bool complete_done = false;

    // empty state for another query, keeping the memory
    void reset() {
        terms.clear();
        w.clear();
        order.clear();
        next = 0;
        pool.clear();
        ready.clear();
        ready_pos = 0;
        touched.clear();   // acc and seen are all zero after every expansion
        emitted = 0;
        ranges_expanded = 0;
        postings_visited = 0;
        items_scored = 0;
        failed = false;
        complete = false;
        complete_done = false;
    }
};

// Growable device and pinned host buffers of a GPU state (kept across the
// calls that reuse the state).
struct pbm_buf {
    void* p = nullptr;
    size_t cap = 0;   // bytes
};

// A batch of queries ranked by the GPU generator: per query the host part of
// PBM (bound order, pool, published run, counters) in a pbm_state, and the
// device buffers the bound and expansion kernels use.  Closed states return
// to their index (buffers, stream and vectors keep their memory).
struct pbm_gpu_state {
    struct Call {                 // progress of one query inside pbm_gpu_next
        int32_t m = 0, n = 0;
        bool done = true;
        bool in_refill = false;
        size_t want = 0, checked = 0, batch = 0;
        std::vector<pbm_state::Range> run;   // ranges waiting for the device
        bool run_pending = false;
    };
    const pbm_index* ix = nullptr;
    int32_t B = 0;
    int device = 0;
    hipStream_t stream = nullptr;
    std::vector<pbm_state> q;
    std::vector<Call> call;
    // device: query terms (qptr, qterm, qw), bounds (H, post), per round
    // tasks, key offsets, counters (key counts, scored counts, fail flags)
    // and keys
    pbm_buf d_qptr, d_qterm, d_qw, d_H, d_post, d_tasks, d_keyoff, d_cnt, d_keys;
    // block-max entry of every (query term, range), when it fits kEntTableMax
    pbm_buf d_ent;
    bool ent_ok = false;
    // pinned host mirrors
    pbm_buf h_H, h_post, h_tasks, h_keyoff, h_cnt, h_keys;
    ~pbm_gpu_state();
};