// Posting Block-Max (PBM): resumable exact sparse ranking on the host
// (Sec. 2.3.2, App. A.2).
//
// The identifier space is cut into contiguous ranges of `range_size` ids.
// For every term and range the index keeps m_t(R), the largest impact of the
// term inside R (absent: no entry, i.e. 0).  A query's range bound
// H(R) = sum_t q_t m_t(R) and every document score S(x) = sum_t q_t p_t(x) are
// accumulated in float32 in ascending term order, one rounding per multiply
// and add, so H(R) >= S(x) for every x in R (App. A.2).  Ranges are expanded
// in (H descending, first id ascending) order; a scored item is published
// once no unexpanded range can hold an item that precedes it.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <memory>
#include <new>
#include <vector>

#include "common.h"
#include "eahr.h"
#include "host_parallel.h"
#include "pbm_internal.h"
#include "pbm_kernels.h"

extern "C" int pbm_build(const int64_t* term_ptr, int32_t vocab, const int32_t* docs,
                         const float* impacts, int64_t n_docs, int32_t range_size,
                         pbm_index** out) {
    if (!out) EAHR_FAIL(EAHR_E_INVALID, "pbm_build: out is NULL");
    *out = nullptr;
    if (!term_ptr || vocab < 0 || n_docs < 0 || range_size < 1)
        EAHR_FAIL(EAHR_E_INVALID, "pbm_build: bad arguments");
    if (term_ptr[0] != 0) EAHR_FAIL(EAHR_E_INVALID, "pbm_build: term_ptr[0] != 0");
    for (int32_t t = 0; t < vocab; ++t)
        if (term_ptr[t + 1] < term_ptr[t]) EAHR_FAIL(EAHR_E_INVALID, "pbm_build: term_ptr not monotone");
    const int64_t P = term_ptr[vocab];
    if (P > 0 && (!docs || !impacts)) EAHR_FAIL(EAHR_E_INVALID, "pbm_build: NULL postings");
    std::unique_ptr<pbm_index> ix(new (std::nothrow) pbm_index());
    if (!ix) EAHR_FAIL(EAHR_E_OOM, "pbm_build: host allocation");
    ix->vocab = vocab;
    ix->n_docs = n_docs;
    ix->range_size = range_size;
    ix->n_ranges = (n_docs + range_size - 1) / range_size;
    try {
        ix->term_ptr.assign(term_ptr, term_ptr + vocab + 1);
        ix->docs.assign(docs, docs + P);
        ix->imp.assign(impacts, impacts + P);
        ix->bm_ptr.assign(static_cast<size_t>(vocab) + 1, 0);
    } catch (const std::bad_alloc&) {
        EAHR_FAIL(EAHR_E_OOM, "pbm_build: host allocation");
    }
    for (int32_t t = 0; t < vocab; ++t) {
        int64_t cur_range = -1;
        for (int64_t p = term_ptr[t]; p < term_ptr[t + 1]; ++p) {
            const int32_t x = docs[p];
            const float v = impacts[p];
            if (x < 0 || x >= n_docs) EAHR_FAIL(EAHR_E_INVALID, "pbm_build: doc id out of range");
            if (p > term_ptr[t] && docs[p - 1] >= x)
                EAHR_FAIL(EAHR_E_INVALID, "pbm_build: docs of term %d not strictly ascending", t);
            if (!std::isfinite(v) || v < 0.0f)
                EAHR_FAIL(EAHR_E_INVALID, "pbm_build: impact must be finite and >= 0");
            const int64_t r = x / range_size;
            if (r != cur_range) {
                ix->bm_range.push_back(r);
                ix->bm_max.push_back(v);
                ix->bm_off.push_back(p);
                cur_range = r;
            } else {
                ix->bm_max.back() = std::max(ix->bm_max.back(), v);
            }
        }
        ix->bm_ptr[t + 1] = static_cast<int64_t>(ix->bm_range.size());
    }
    *out = ix.release();
    return EAHR_OK;
}

static void free_device(pbm_device* d);

pbm_index::~pbm_index() {
    for (pbm_state* st : free_states) delete st;
    for (pbm_gpu_state* st : free_gpu_states) delete st;
    free_device(dev);
}

extern "C" void pbm_free(pbm_index* ix) {
    if (!ix) return;
    {
        std::lock_guard<std::mutex> lk(ix->free_mu);
        if (ix->open_states > 0) {   // released by the last pbm_close
            ix->release_requested = true;
            return;
        }
    }
    delete ix;
}

extern "C" int pbm_debug_set_blockmax(pbm_index* ix, int32_t term, int64_t range, float value) {
    if (!ix || term < 0 || term >= ix->vocab) EAHR_FAIL(EAHR_E_INVALID, "pbm_debug_set_blockmax: bad term");
    for (int64_t e = ix->bm_ptr[term]; e < ix->bm_ptr[term + 1]; ++e) {
        if (ix->bm_range[e] == range) {
            ix->bm_max[e] = value;
            std::lock_guard<std::mutex> lk(ix->dev_mu);
            if (ix->dev) {
                int cur = 0;
                HIP_TRY(hipGetDevice(&cur));
                HIP_TRY(hipSetDevice(ix->dev->device));
                const hipError_t err = hipMemcpy(ix->dev->bm_max + e, &value, sizeof(float), hipMemcpyHostToDevice);
                (void)hipSetDevice(cur);
                HIP_TRY(err);
            }
            return EAHR_OK;
        }
    }
    EAHR_FAIL(EAHR_E_INVALID, "pbm_debug_set_blockmax: term has no postings in range");
}

int pbm_check_query(const pbm_index* ix, const eahr_sparse_query* q) {
    if (!ix || !q || q->n_terms < 0 || (q->n_terms > 0 && (!q->terms || !q->weights)))
        EAHR_FAIL(EAHR_E_INVALID, "pbm_open: bad arguments");
    for (int32_t i = 0; i < q->n_terms; ++i) {
        const int32_t t = q->terms[i];
        const float w = q->weights[i];
        if (t < 0 || t >= ix->vocab) EAHR_FAIL(EAHR_E_INVALID, "pbm_open: term id out of range");
        if (!std::isfinite(w) || w < 0.0f) EAHR_FAIL(EAHR_E_INVALID, "pbm_open: weight must be finite and >= 0");
    }
    std::vector<int32_t> t(q->terms, q->terms + q->n_terms);
    std::sort(t.begin(), t.end());
    if (std::adjacent_find(t.begin(), t.end()) != t.end()) EAHR_FAIL(EAHR_E_INVALID, "pbm_open: duplicate term");
    return EAHR_OK;
}

extern "C" int pbm_open(const pbm_index* ix, const eahr_sparse_query* q, pbm_state** out) {
    return pbm_open_gen(ix, q, EAHR_SPARSE_PBM, out);
}

extern "C" int pbm_open_gen(const pbm_index* ix, const eahr_sparse_query* q, int32_t generator,
                            pbm_state** out) {
    if (!out) EAHR_FAIL(EAHR_E_INVALID, "pbm_open: out is NULL");
    *out = nullptr;
    if (generator != EAHR_SPARSE_PBM && generator != EAHR_SPARSE_COMPLETE)
        EAHR_FAIL(EAHR_E_INVALID, "pbm_open: unknown sparse generator %d", generator);
    EAHR_TRY(pbm_check_query(ix, q));
    std::unique_ptr<pbm_state> st;
    {
        std::lock_guard<std::mutex> lk(ix->free_mu);
        if (ix->release_requested) EAHR_FAIL(EAHR_E_INVALID, "pbm_open: the index has been freed");
        if (!ix->free_states.empty()) {
            st.reset(ix->free_states.back());
            ix->free_states.pop_back();
        }
    }
    if (!st) st.reset(new (std::nothrow) pbm_state());
    if (!st) EAHR_FAIL(EAHR_E_OOM, "pbm_open: host allocation");
    st->reset();
    st->ix = ix;
    st->complete = (generator == EAHR_SPARSE_COMPLETE);
    std::vector<std::pair<int32_t, float>> tw;
    for (int32_t i = 0; i < q->n_terms; ++i) tw.emplace_back(q->terms[i], q->weights[i]);
    std::sort(tw.begin(), tw.end());
    for (auto& p : tw) {
        if (p.second == 0.0f) continue;   // a zero weight contributes exactly 0
        st->terms.push_back(p.first);
        st->w.push_back(p.second);
    }
    // H(R) in ascending term order over the ranges any query term touches;
    // each term's block-max entry per range is tabulated for expansion
    const int64_t nr = ix->n_ranges;
    std::vector<float> H(static_cast<size_t>(nr), 0.0f);
    std::vector<uint8_t> touched(static_cast<size_t>(nr), 0);
    std::vector<int64_t> list;
    try {
        st->ent.assign(st->terms.size() * static_cast<size_t>(nr), -1);
    } catch (const std::bad_alloc&) {
        EAHR_FAIL(EAHR_E_OOM, "pbm_open: host allocation");
    }
    for (size_t i = 0; i < st->terms.size(); ++i) {
        const int32_t t = st->terms[i];
        const float w = st->w[i];
        int64_t* ent = st->ent.data() + i * static_cast<size_t>(nr);
        for (int64_t e = ix->bm_ptr[t]; e < ix->bm_ptr[t + 1]; ++e) {
            const int64_t r = ix->bm_range[e];
            ent[r] = e;
            const float c = w * ix->bm_max[e];
            H[r] = H[r] + c;
            if (!touched[r]) {
                touched[r] = 1;
                list.push_back(r);
            }
        }
    }
    for (int64_t r : list)
        if (H[r] > 0.0f) st->order.push_back(pbm_state::Range{H[r], 0, r});
    std::sort(st->order.begin(), st->order.end(), [](const pbm_state::Range& a, const pbm_state::Range& b) {
        return a.H > b.H || (a.H == b.H && a.r < b.r);
    });
    {
        std::lock_guard<std::mutex> lk(ix->free_mu);
        ix->open_states += 1;
    }
    *out = st.release();
    return EAHR_OK;
}

// Score every document of range r that carries a query term and queue the
// positive ones; fails when a score exceeds the range bound (metadata that
// does not cover its postings, App. A.2).
static inline uint32_t ord32(float f) {
    uint32_t b;
    std::memcpy(&b, &f, 4);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
static inline float unord32(uint32_t k) {
    const uint32_t b = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    float f;
    std::memcpy(&f, &b, 4);
    return f;
}
static inline uint64_t item_key(float s, int64_t id) {
    return (static_cast<uint64_t>(~ord32(s + 0.0f)) << 32) | static_cast<uint64_t>(id);
}
static inline bool ranges_left(const pbm_state* st) { return st->next < st->order.size(); }
static inline uint64_t bound_key(const pbm_state* st) {
    if (!ranges_left(st)) return ~0ull;
    const auto& R = st->order[st->next];
    return (static_cast<uint64_t>(~ord32(R.H)) << 32) | static_cast<uint64_t>(R.r * st->ix->range_size);
}

// Score every document of range R that carries a query term and add the
// positive ones to the pool; fails when a score exceeds the range bound
// (metadata that does not cover its postings, App. A.2).
static bool expand(pbm_state* st, const pbm_state::Range& R) {
    const pbm_index* ix = st->ix;
    const int64_t start = R.r * ix->range_size;
    const int64_t len = std::min<int64_t>(ix->range_size, ix->n_docs - start);
    if (st->acc.size() < static_cast<size_t>(len)) {
        st->acc.assign(static_cast<size_t>(len), 0.0f);
        st->seen.assign(static_cast<size_t>(len), 0);
    }
    st->touched.clear();
    for (size_t i = 0; i < st->terms.size(); ++i) {
        const int32_t t = st->terms[i];
        const int64_t e = st->ent[i * static_cast<size_t>(ix->n_ranges) + R.r];
        if (e < 0) continue;
        const int64_t p_end = (e + 1 < ix->bm_ptr[t + 1]) ? ix->bm_off[e + 1] : ix->term_ptr[t + 1];
        const float w = st->w[i];
        st->postings_visited += p_end - ix->bm_off[e];
        for (int64_t p = ix->bm_off[e]; p < p_end; ++p) {
            const int64_t off = ix->docs[p] - start;
            const float c = w * ix->imp[p];
            st->acc[off] = st->acc[off] + c;
            if (!st->seen[off]) {
                st->seen[off] = 1;
                st->touched.push_back(static_cast<int32_t>(off));
            }
        }
    }
    bool ok = true;
    st->items_scored += static_cast<int64_t>(st->touched.size());
    for (int32_t off : st->touched) {
        const float s = st->acc[off];
        if (s > R.H) ok = false;
        if (s > 0.0f) st->pool.push_back(item_key(s, start + off));
        st->acc[off] = 0.0f;
        st->seen[off] = 0;
    }
    return ok;
}

// Ascending sort of 64-bit keys: least-significant-digit radix sort with
// 8-bit digits (256 scatter targets stay in cache), skipping digits that are
// equal in every key (the high bits of the identifiers); short runs use a
// comparison sort.
static void sort_keys(std::vector<uint64_t>& a) {
    const size_t n = a.size();
    if (n < 1024) {
        std::sort(a.begin(), a.end());
        return;
    }
    // scratch reused by every state sorted on this thread
    thread_local std::vector<uint64_t> tmp;
    thread_local std::vector<uint32_t> cnt;
    if (tmp.size() < n) tmp.resize(n);
    cnt.assign(8 * 256, 0u);
    for (size_t i = 0; i < n; ++i) {
        const uint64_t k = a[i];
        for (int d = 0; d < 8; ++d) ++cnt[d * 256 + ((k >> (8 * d)) & 0xff)];
    }
    for (int d = 0; d < 8; ++d) {
        uint32_t* c = cnt.data() + d * 256;
        if (c[(a[0] >> (8 * d)) & 0xff] == n) continue;   // one digit value
        uint32_t sum = 0;
        for (int v = 0; v < 256; ++v) {
            const uint32_t t = c[v];
            c[v] = sum;
            sum += t;
        }
        uint64_t* out = tmp.data();
        for (size_t i = 0; i < n; ++i) out[c[(a[i] >> (8 * d)) & 0xff]++] = a[i];
        std::copy(out, out + n, a.begin());
    }
}

// Ranges are expanded in batches: the next `batch` ranges of the bound order,
// visited in id order so that each term's postings are read front to back.
// Expanding a range beyond the ones the stopping rule needs only adds work;
// publication still waits for the bound of the first unexpanded range.  The
// batch doubles (kBatchMin .. kBatchMax) while a refill goes on.
constexpr size_t kBatchMin = 8;
constexpr size_t kBatchMax = 1024;

// Move the publishable pool items (keys below the bound key bk) to the
// ready run, sorted.  When far more are publishable than wanted, only the
// smallest keys go (at least kPublishMin and 4 * want, cut at a boundary of
// the top 16 key bits found from one histogram pass): they are still the
// smallest keys of everything unpublished, and the rest stay pooled for a
// later refill, so a query whose every range had to be expanded does not
// sort its whole scored set up front.
constexpr size_t kPublishMin = 65536;

static void publish(pbm_state* st, uint64_t bk, size_t want) {
    auto& pool = st->pool;
    const auto mid = std::partition(pool.begin(), pool.end(), [bk](uint64_t k) { return k < bk; });
    const size_t np = static_cast<size_t>(mid - pool.begin());
    const size_t take = std::max(kPublishMin, 4 * want);
    auto cut_end = mid;
    if (np > take + take / 2) {
        thread_local std::vector<uint32_t> hist;
        hist.assign(65536, 0u);
        for (auto it = pool.begin(); it != mid; ++it) ++hist[*it >> 48];
        size_t cum = 0;
        uint32_t cut = 0;
        for (; cut < 65535; ++cut) {
            cum += hist[cut];
            if (cum >= take) break;
        }
        if (cut < 65535) {
            const uint64_t lim = static_cast<uint64_t>(cut + 1) << 48;
            cut_end = std::partition(pool.begin(), mid, [lim](uint64_t k) { return k < lim; });
        }
    }
    st->ready.assign(pool.begin(), cut_end);
    pool.erase(pool.begin(), cut_end);
    sort_keys(st->ready);
}

// Refill the ready run with at least `want` publishable items when the
// remaining ranges allow: expand ranges in bound order until enough pooled
// items precede the next range's bound (counted whenever the pool has grown
// by half since the last count), then move those items out of the pool and
// sort them.  Returns false on a failed expansion.
static bool refill(pbm_state* st, size_t want) {
    st->ready.clear();
    st->ready_pos = 0;
    size_t checked = 0;
    size_t batch = kBatchMin;
    std::vector<pbm_state::Range>& run = st->batch;
    for (;;) {
        if (!ranges_left(st)) break;
        if (st->pool.size() >= want && st->pool.size() >= checked + checked / 2) {
            const uint64_t bk = bound_key(st);
            size_t n = 0;
            for (uint64_t k : st->pool) n += (k < bk);
            if (n >= want) break;
            checked = st->pool.size();
        }
        const size_t take = std::min(batch, st->order.size() - st->next);
        run.assign(st->order.begin() + st->next, st->order.begin() + st->next + take);
        st->next += take;
        std::sort(run.begin(), run.end(),
                  [](const pbm_state::Range& a, const pbm_state::Range& b) { return a.r < b.r; });
        for (const auto& R : run) {
            st->ranges_expanded += 1;
            if (!expand(st, R)) return false;
        }
        batch = std::min(batch * 2, kBatchMax);
    }
    publish(st, bound_key(st), want);
    return true;
}

extern "C" int pbm_next(pbm_state* st, int32_t m, int64_t* ids, float* scores, int32_t* count,
                        int32_t* status) {
    if (!st || m < 0 || (m > 0 && (!ids || !scores)) || !count || !status)
        EAHR_FAIL(EAHR_E_INVALID, "pbm_next: bad arguments");
    int32_t n = 0;
    if (!st->failed && st->complete && !st->complete_done) {
        // complete generator: score every document of every range with a
        // positive bound (ascending ranges), then one sort of all of them
        st->complete_done = true;
        std::vector<pbm_state::Range> all(st->order.begin(), st->order.end());
        std::sort(all.begin(), all.end(),
                  [](const pbm_state::Range& a, const pbm_state::Range& b) { return a.r < b.r; });
        for (const auto& R : all) {
            st->ranges_expanded += 1;
            if (!expand(st, R)) st->failed = true;
        }
        st->next = st->order.size();
        if (!st->failed) {
            sort_keys(st->pool);
            st->ready.swap(st->pool);
            st->ready_pos = 0;
        }
        st->pool.clear();
    }
    if (!st->failed) {
        while (n < m) {
            if (st->ready_pos < st->ready.size()) {
                const uint64_t k = st->ready[st->ready_pos++];
                ids[n] = static_cast<int64_t>(k & 0xffffffffu);
                scores[n] = unord32(~static_cast<uint32_t>(k >> 32));
                ++n;
                continue;
            }
            if (!ranges_left(st) && st->pool.empty()) break;   // list complete
            if (!refill(st, static_cast<size_t>(m - n))) {
                st->failed = true;
                n = 0;
                break;
            }
        }
    }
    st->emitted += n;
    *count = n;
    if (st->failed) *status = EAHR_LIST_FAILED;
    else if (!ranges_left(st) && st->pool.empty() && st->ready_pos >= st->ready.size())
        *status = EAHR_LIST_EXHAUSTED;
    else *status = EAHR_LIST_OPEN;
    return EAHR_OK;
}

// Closed states go back to their index for reuse (up to this many).
constexpr size_t kFreeStates = 1024;

extern "C" void pbm_close(pbm_state* st) {
    if (!st) return;
    const pbm_index* ix = st->ix;
    bool release = false;
    if (ix) {
        std::lock_guard<std::mutex> lk(ix->free_mu);
        ix->open_states -= 1;
        release = ix->release_requested && ix->open_states == 0;
        if (!release && ix->free_states.size() < kFreeStates) {
            ix->free_states.push_back(st);
            return;
        }
    }
    delete st;
    if (release) delete ix;   // pbm_free came first
}

// ---------------------------------------------------------------- GPU PBM
//
// The host keeps, per query, exactly the state machine of pbm_next/refill
// above (bound order, expansion batches doubling from kBatchMin, the pool
// count before each batch, publication); only the expansions of a batch run
// on the device, and they run for every query of the call that needs one in
// the same device round.  Pool order never matters (publication partitions
// and sorts by key), so a query's ranks, scores and counters are those of
// the host generator.

namespace {

template <class T>
int dev_alloc_n(T** p, size_t n) {
    *p = nullptr;
    if (n == 0) n = 1;
    HIP_TRY(hipMalloc(reinterpret_cast<void**>(p), n * sizeof(T)));
    return EAHR_OK;
}

template <class T>
int dev_upload(T** p, const T* src, size_t n) {
    EAHR_TRY(dev_alloc_n(p, n));
    if (n > 0) HIP_TRY(hipMemcpy(*p, src, n * sizeof(T), hipMemcpyHostToDevice));
    return EAHR_OK;
}

}  // namespace

static void free_device(pbm_device* d) {
    if (!d) return;
    int cur = 0;
    const bool switch_dev = hipGetDevice(&cur) == hipSuccess && cur != d->device;
    if (switch_dev) (void)hipSetDevice(d->device);
    void* ptrs[] = {d->docs, d->imp, d->term_ptr, d->bm_ptr, d->bm_range, d->bm_max, d->bm_off};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
    if (switch_dev) (void)hipSetDevice(cur);
    delete d;
}

namespace {

// Runs with ix->dev_mu held.
int upload_locked(const pbm_index* ix) {
    if (ix->dev) return EAHR_OK;
    std::unique_ptr<pbm_device, void (*)(pbm_device*)> d(new (std::nothrow) pbm_device(), free_device);
    if (!d) EAHR_FAIL(EAHR_E_OOM, "pbm_upload: host allocation");
    HIP_TRY(hipGetDevice(&d->device));
    std::vector<int32_t> range32(ix->bm_range.size());
    for (size_t i = 0; i < range32.size(); ++i) range32[i] = static_cast<int32_t>(ix->bm_range[i]);
    EAHR_TRY(dev_upload(&d->docs, ix->docs.data(), ix->docs.size()));
    EAHR_TRY(dev_upload(&d->imp, ix->imp.data(), ix->imp.size()));
    EAHR_TRY(dev_upload(&d->term_ptr, ix->term_ptr.data(), ix->term_ptr.size()));
    EAHR_TRY(dev_upload(&d->bm_ptr, ix->bm_ptr.data(), ix->bm_ptr.size()));
    EAHR_TRY(dev_upload(&d->bm_range, range32.data(), range32.size()));
    EAHR_TRY(dev_upload(&d->bm_max, ix->bm_max.data(), ix->bm_max.size()));
    EAHR_TRY(dev_upload(&d->bm_off, ix->bm_off.data(), ix->bm_off.size()));
    ix->dev = d.release();
    return EAHR_OK;
}

pbmg::IndexView view_of(const pbm_index* ix) {
    const pbm_device* d = ix->dev;
    pbmg::IndexView v;
    v.docs = d->docs;
    v.imp = d->imp;
    v.term_ptr = d->term_ptr;
    v.bm_ptr = d->bm_ptr;
    v.bm_range = d->bm_range;
    v.bm_max = d->bm_max;
    v.bm_off = d->bm_off;
    v.range_size = ix->range_size;
    v.n_docs = ix->n_docs;
    v.n_ranges = ix->n_ranges;
    return v;
}

// Keys of one device round at most (a query whose batch needs more still
// runs, alone in its round).
constexpr size_t kRoundKeys = size_t(1) << 25;
// (query, range) bound pairs computed per bound launch
constexpr int64_t kBoundPairs = int64_t(1) << 26;

// Restores the caller's device on every return path.
struct DeviceGuard {
    int prev = -1;
    bool switched = false;
    int enter(int dev) {
        HIP_TRY(hipGetDevice(&prev));
        if (prev != dev) {
            HIP_TRY(hipSetDevice(dev));
            switched = true;
        }
        return EAHR_OK;
    }
    ~DeviceGuard() {
        if (switched) (void)hipSetDevice(prev);
    }
};

}  // namespace

extern "C" int pbm_upload(const pbm_index* ix) {
    if (!ix) EAHR_FAIL(EAHR_E_INVALID, "pbm_upload: index is NULL");
    std::lock_guard<std::mutex> lk(ix->dev_mu);
    return upload_locked(ix);
}

pbm_gpu_state::~pbm_gpu_state() {
    int cur = 0;
    const bool sw = hipGetDevice(&cur) == hipSuccess && cur != device;
    if (sw) (void)hipSetDevice(device);
    if (stream) (void)hipStreamSynchronize(stream);
    for (pbm_buf* b : {&d_qptr, &d_qterm, &d_qw, &d_H, &d_post, &d_tasks, &d_keyoff, &d_cnt, &d_keys, &d_ent})
        if (b->p) (void)hipFree(b->p);
    for (pbm_buf* b : {&h_H, &h_post, &h_tasks, &h_keyoff, &h_cnt, &h_keys})
        if (b->p) (void)hipHostFree(b->p);
    if (stream) (void)hipStreamDestroy(stream);
    if (sw) (void)hipSetDevice(cur);
}

namespace {

// At least `bytes` in b (contents not kept when it grows).
int grow_dev(pbm_buf& b, size_t bytes) {
    if (bytes <= b.cap) return EAHR_OK;
    const size_t cap = std::max<size_t>({bytes, b.cap + b.cap / 2, 256});
    if (b.p) HIP_TRY(hipFree(b.p));
    b.p = nullptr;
    b.cap = 0;
    HIP_TRY(hipMalloc(&b.p, cap));
    b.cap = cap;
    return EAHR_OK;
}

int grow_pinned(pbm_buf& b, size_t bytes) {
    if (bytes <= b.cap) return EAHR_OK;
    const size_t cap = std::max<size_t>({bytes, b.cap + b.cap / 2, 256});
    if (b.p) HIP_TRY(hipHostFree(b.p));
    b.p = nullptr;
    b.cap = 0;
    HIP_TRY(hipHostMalloc(&b.p, cap, hipHostMallocDefault));
    b.cap = cap;
    return EAHR_OK;
}

template <class T>
T* as(const pbm_buf& b) {
    return static_cast<T*>(b.p);
}

// Closed GPU states kept per index for reuse.
constexpr size_t kFreeGpuStates = 4;
// Largest table of block-max entries per (query term, range) a state keeps
// on the device; beyond it the expansions find entries by binary search.
constexpr size_t kEntTableMax = size_t(1) << 30;

}  // namespace

extern "C" int pbm_gpu_open(const pbm_index* ix, const eahr_sparse_query* q, int32_t B, pbm_gpu_state** out) {
    if (!out) EAHR_FAIL(EAHR_E_INVALID, "pbm_gpu_open: out is NULL");
    *out = nullptr;
    if (!ix || B < 0 || (B > 0 && !q)) EAHR_FAIL(EAHR_E_INVALID, "pbm_gpu_open: bad arguments");
    if (ix->range_size > pbmg::kMaxRangeSize)
        EAHR_FAIL(EAHR_E_RANGE, "pbm_gpu_open: range_size %d exceeds %d", ix->range_size,
                  static_cast<int>(pbmg::kMaxRangeSize));
    for (int32_t b = 0; b < B; ++b) EAHR_TRY(pbm_check_query(ix, &q[b]));
    const auto t_open = std::chrono::steady_clock::now();
    {
        std::lock_guard<std::mutex> lk(ix->dev_mu);
        EAHR_TRY(upload_locked(ix));
    }
    std::unique_ptr<pbm_gpu_state> st;
    {
        std::lock_guard<std::mutex> lk(ix->free_mu);
        if (ix->release_requested) EAHR_FAIL(EAHR_E_INVALID, "pbm_gpu_open: the index has been freed");
        if (!ix->free_gpu_states.empty()) {
            st.reset(ix->free_gpu_states.back());
            ix->free_gpu_states.pop_back();
        }
    }
    if (!st) st.reset(new (std::nothrow) pbm_gpu_state());
    if (!st) EAHR_FAIL(EAHR_E_OOM, "pbm_gpu_open: host allocation");
    st->ix = ix;
    st->B = B;
    st->device = ix->dev->device;
    DeviceGuard guard;
    EAHR_TRY(guard.enter(st->device));
    if (!st->stream) HIP_TRY(hipStreamCreateWithFlags(&st->stream, hipStreamNonBlocking));
    hipStream_t s = st->stream;
    try {
        st->q.resize(static_cast<size_t>(B));
        st->call.resize(static_cast<size_t>(B));
    } catch (const std::bad_alloc&) {
        EAHR_FAIL(EAHR_E_OOM, "pbm_gpu_open: host allocation");
    }
    // the query terms, ascending, zero weights dropped (they add exactly 0)
    std::vector<int32_t> qptr(static_cast<size_t>(B) + 1, 0), qterm;
    std::vector<float> qw;
    for (int32_t b = 0; b < B; ++b) {
        std::vector<std::pair<int32_t, float>> tw;
        for (int32_t i = 0; i < q[b].n_terms; ++i) tw.emplace_back(q[b].terms[i], q[b].weights[i]);
        std::sort(tw.begin(), tw.end());
        pbm_state& S = st->q[b];
        S.reset();
        S.ix = ix;
        for (auto& p : tw) {
            if (p.second == 0.0f) continue;
            S.terms.push_back(p.first);
            S.w.push_back(p.second);
            qterm.push_back(p.first);
            qw.push_back(p.second);
        }
        qptr[b + 1] = static_cast<int32_t>(qterm.size());
    }
    EAHR_TRY(grow_dev(st->d_qptr, qptr.size() * sizeof(int32_t)));
    EAHR_TRY(grow_dev(st->d_qterm, std::max<size_t>(1, qterm.size()) * sizeof(int32_t)));
    EAHR_TRY(grow_dev(st->d_qw, std::max<size_t>(1, qw.size()) * sizeof(float)));
    HIP_TRY(hipMemcpyAsync(st->d_qptr.p, qptr.data(), qptr.size() * sizeof(int32_t), hipMemcpyHostToDevice, s));
    if (!qterm.empty()) {
        HIP_TRY(hipMemcpyAsync(st->d_qterm.p, qterm.data(), qterm.size() * sizeof(int32_t),
                               hipMemcpyHostToDevice, s));
        HIP_TRY(hipMemcpyAsync(st->d_qw.p, qw.data(), qw.size() * sizeof(float), hipMemcpyHostToDevice, s));
    }
    EAHR_TRY(grow_dev(st->d_keyoff, std::max<size_t>(1, B) * sizeof(int64_t)));
    EAHR_TRY(grow_dev(st->d_cnt, 3 * std::max<size_t>(1, B) * sizeof(int32_t)));
    EAHR_TRY(grow_pinned(st->h_keyoff, std::max<size_t>(1, B) * sizeof(int64_t)));
    EAHR_TRY(grow_pinned(st->h_cnt, 3 * std::max<size_t>(1, B) * sizeof(int32_t)));
    // H(R) and the postings count of every (query, range), a chunk of
    // queries per launch; each query's ranges with H > 0 in bound order
    const int64_t nr = ix->n_ranges;
    const size_t ent_bytes = qterm.size() * static_cast<size_t>(std::max<int64_t>(nr, 0)) * sizeof(int64_t);
    st->ent_ok = nr > 0 && !qterm.empty() && ent_bytes <= kEntTableMax;
    if (st->ent_ok) EAHR_TRY(grow_dev(st->d_ent, ent_bytes));
    if (nr > 0 && B > 0) {
        const int32_t chunk = static_cast<int32_t>(std::max<int64_t>(1, std::min<int64_t>(B, kBoundPairs / nr)));
        const size_t pairs = static_cast<size_t>(chunk) * static_cast<size_t>(nr);
        EAHR_TRY(grow_dev(st->d_H, pairs * sizeof(float)));
        EAHR_TRY(grow_dev(st->d_post, pairs * sizeof(int32_t)));
        EAHR_TRY(grow_pinned(st->h_H, pairs * sizeof(float)));
        EAHR_TRY(grow_pinned(st->h_post, pairs * sizeof(int32_t)));
        const pbmg::IndexView v = view_of(ix);
        for (int32_t b0 = 0; b0 < B; b0 += chunk) {
            const int32_t nb = std::min(chunk, B - b0);
            const pbmg::QueryView qv{as<int32_t>(st->d_qptr) + b0, as<int32_t>(st->d_qterm), as<float>(st->d_qw), nb};
            pbmg::launch_bounds(v, qv, as<float>(st->d_H), as<int32_t>(st->d_post),
                                st->ent_ok ? as<int64_t>(st->d_ent) : nullptr, s);
            HIP_TRY(hipGetLastError());
            const size_t n = static_cast<size_t>(nb) * static_cast<size_t>(nr);
            HIP_TRY(hipMemcpyAsync(st->h_H.p, st->d_H.p, n * sizeof(float), hipMemcpyDeviceToHost, s));
            HIP_TRY(hipMemcpyAsync(st->h_post.p, st->d_post.p, n * sizeof(int32_t), hipMemcpyDeviceToHost, s));
            HIP_TRY(hipStreamSynchronize(s));
            const float* H = as<float>(st->h_H);
            const int32_t* post = as<int32_t>(st->h_post);
            ::eahr::parallel_for(nb, ::eahr::host_threads(), [&](int64_t i) {
                pbm_state& S = st->q[b0 + i];
                const float* h = H + i * nr;
                const int32_t* p = post + i * nr;
                for (int64_t r = 0; r < nr; ++r)
                    if (h[r] > 0.0f) S.order.push_back(pbm_state::Range{h[r], p[r], r});
                std::sort(S.order.begin(), S.order.end(), [](const pbm_state::Range& a, const pbm_state::Range& c) {
                    return a.H > c.H || (a.H == c.H && a.r < c.r);
                });
            });
        }
    }
    {
        std::lock_guard<std::mutex> lk(ix->free_mu);
        ix->open_states += 1;
    }
    if (::eahr::trace_on())
        std::fprintf(stderr, "pbm_gpu open queries=%d ranges=%lld ms=%.2f\n", B, static_cast<long long>(nr),
                     std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_open).count());
    *out = st.release();
    return EAHR_OK;
}

extern "C" int pbm_gpu_next(pbm_gpu_state* st, const int32_t* m, int64_t* const* ids, float* const* scores,
                            int32_t* count, int32_t* status) {
    if (!st || !m || !count || !status || (st->B > 0 && (!ids || !scores)))
        EAHR_FAIL(EAHR_E_INVALID, "pbm_gpu_next: bad arguments");
    const int32_t B = st->B;
    for (int32_t b = 0; b < B; ++b) {
        if (m[b] < 0) EAHR_FAIL(EAHR_E_INVALID, "pbm_gpu_next: m[%d] < 0", b);
        if (m[b] > 0 && (!ids[b] || !scores[b])) EAHR_FAIL(EAHR_E_INVALID, "pbm_gpu_next: NULL output");
    }
    const pbm_index* ix = st->ix;
    DeviceGuard guard;
    EAHR_TRY(guard.enter(st->device));
    hipStream_t s = st->stream;
    for (int32_t b = 0; b < B; ++b) {
        auto& c = st->call[b];
        c.m = m[b];
        c.n = 0;
        c.done = m[b] == 0;
        c.in_refill = false;
        c.run_pending = false;
    }
    // The host generator's pbm_next and refill as a resumable step: serve
    // published ranks, start a refill, count the pool against the bound,
    // publish; returns true with c.run set when a batch must be expanded.
    auto advance = [&](int32_t b) -> bool {
        pbm_state& S = st->q[b];
        auto& c = st->call[b];
        int64_t* oid = ids[b];
        float* osc = scores[b];
        for (;;) {
            if (S.failed) {
                c.done = true;
                return false;
            }
            if (!c.in_refill) {
                while (c.n < c.m && S.ready_pos < S.ready.size()) {
                    const uint64_t k = S.ready[S.ready_pos++];
                    oid[c.n] = static_cast<int64_t>(k & 0xffffffffu);
                    osc[c.n] = unord32(~static_cast<uint32_t>(k >> 32));
                    ++c.n;
                }
                if (c.n >= c.m || (!ranges_left(&S) && S.pool.empty())) {
                    c.done = true;
                    return false;
                }
                c.want = static_cast<size_t>(c.m - c.n);
                S.ready.clear();
                S.ready_pos = 0;
                c.checked = 0;
                c.batch = kBatchMin;
                c.in_refill = true;
            }
            if (ranges_left(&S)) {
                bool enough = false;
                if (S.pool.size() >= c.want && S.pool.size() >= c.checked + c.checked / 2) {
                    const uint64_t bk = bound_key(&S);
                    size_t n = 0;
                    for (uint64_t k : S.pool) n += (k < bk);
                    if (n >= c.want) enough = true;
                    else c.checked = S.pool.size();
                }
                if (!enough) {
                    const size_t take = std::min(c.batch, S.order.size() - S.next);
                    c.run.assign(S.order.begin() + S.next, S.order.begin() + S.next + take);
                    S.next += take;
                    std::sort(c.run.begin(), c.run.end(),
                              [](const pbm_state::Range& a, const pbm_state::Range& x) { return a.r < x.r; });
                    c.batch = std::min(c.batch * 2, kBatchMax);
                    return true;
                }
            }
            publish(&S, bound_key(&S), c.want);
            c.in_refill = false;
        }
    };
    const pbmg::IndexView v = view_of(ix);
    const pbmg::QueryView qv{as<int32_t>(st->d_qptr), as<int32_t>(st->d_qterm), as<float>(st->d_qw), B};
    const auto t0 = std::chrono::steady_clock::now();
    int64_t rounds = 0;
    size_t all_tasks = 0, all_keys = 0;
    double t_host = 0, t_dev = 0, t_pool = 0;   // trace: host steps, device rounds, pool appends
    auto since = [](std::chrono::steady_clock::time_point t) {
        return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t).count();
    };
    std::vector<int32_t> round;
    std::vector<size_t> need(static_cast<size_t>(B), 0);
    for (;;) {
        auto tr = std::chrono::steady_clock::now();
        ::eahr::parallel_for(B, ::eahr::host_threads(), [&](int64_t b) {
            auto& c = st->call[b];
            if (!c.done && !c.run_pending) c.run_pending = advance(static_cast<int32_t>(b));
        });
        t_host += since(tr);
        // the runs of this round: queries in order while the keys fit (the
        // first one always runs)
        round.clear();
        size_t keys = 0, tasks = 0;
        for (int32_t b = 0; b < B; ++b) {
            const auto& c = st->call[b];
            if (!c.run_pending) continue;
            size_t n = 0;
            for (const auto& R : c.run) n += static_cast<size_t>(R.post);
            if (!round.empty() && keys + n > kRoundKeys) continue;
            need[b] = n;
            round.push_back(b);
            keys += n;
            tasks += c.run.size();
        }
        if (round.empty()) break;
        tr = std::chrono::steady_clock::now();
        EAHR_TRY(grow_dev(st->d_tasks, tasks * sizeof(pbmg::Task)));
        EAHR_TRY(grow_pinned(st->h_tasks, tasks * sizeof(pbmg::Task)));
        EAHR_TRY(grow_dev(st->d_keys, std::max<size_t>(1, keys) * sizeof(uint64_t)));
        EAHR_TRY(grow_pinned(st->h_keys, std::max<size_t>(1, keys) * sizeof(uint64_t)));
        pbmg::Task* ht = as<pbmg::Task>(st->h_tasks);
        int64_t* hoff = as<int64_t>(st->h_keyoff);
        size_t t = 0, off = 0;
        for (int32_t b : round) {
            hoff[b] = static_cast<int64_t>(off);
            off += need[b];
            for (const auto& R : st->call[b].run) ht[t++] = pbmg::Task{b, static_cast<int32_t>(R.r), R.H, 0};
        }
        int32_t* dcnt = as<int32_t>(st->d_cnt);
        HIP_TRY(hipMemcpyAsync(st->d_tasks.p, ht, tasks * sizeof(pbmg::Task), hipMemcpyHostToDevice, s));
        HIP_TRY(hipMemcpyAsync(st->d_keyoff.p, hoff, static_cast<size_t>(B) * sizeof(int64_t),
                               hipMemcpyHostToDevice, s));
        HIP_TRY(hipMemsetAsync(dcnt, 0, 3 * static_cast<size_t>(B) * sizeof(int32_t), s));
        if (pbmg::launch_expand(v, qv, as<pbmg::Task>(st->d_tasks), static_cast<int32_t>(tasks),
                                st->ent_ok ? as<int64_t>(st->d_ent) : nullptr, as<int64_t>(st->d_keyoff), dcnt,
                                dcnt + B, dcnt + 2 * B, as<uint64_t>(st->d_keys), s) != 0)
            EAHR_FAIL(EAHR_E_HIP, "pbm_gpu_next: the expansion kernel cannot get %d ids of LDS", ix->range_size);
        HIP_TRY(hipGetLastError());
        HIP_TRY(hipMemcpyAsync(st->h_cnt.p, dcnt, 3 * static_cast<size_t>(B) * sizeof(int32_t),
                               hipMemcpyDeviceToHost, s));
        if (keys > 0)
            HIP_TRY(hipMemcpyAsync(st->h_keys.p, st->d_keys.p, keys * sizeof(uint64_t), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
        ++rounds;
        all_tasks += tasks;
        all_keys += keys;
        t_dev += since(tr);
        tr = std::chrono::steady_clock::now();
        const int32_t* kc = as<int32_t>(st->h_cnt);
        const int32_t* sc = kc + B;
        const int32_t* fl = kc + 2 * B;
        ::eahr::parallel_for(static_cast<int64_t>(round.size()), ::eahr::host_threads(), [&](int64_t i) {
            const int32_t b = round[i];
            pbm_state& S = st->q[b];
            auto& c = st->call[b];
            S.ranges_expanded += static_cast<int64_t>(c.run.size());
            S.postings_visited += static_cast<int64_t>(need[b]);
            S.items_scored += sc[b];
            if (fl[b]) {   // a score above its range's bound (App. A.2)
                S.failed = true;
                c.n = 0;
                c.done = true;
            } else {
                const uint64_t* k = as<uint64_t>(st->h_keys) + hoff[b];
                S.pool.insert(S.pool.end(), k, k + kc[b]);
            }
            c.run_pending = false;
        });
        t_pool += since(tr);
    }
    for (int32_t b = 0; b < B; ++b) {
        pbm_state& S = st->q[b];
        const auto& c = st->call[b];
        const int32_t n = (m[b] > 0) ? c.n : 0;
        S.emitted += n;
        count[b] = n;
        if (S.failed) status[b] = EAHR_LIST_FAILED;
        else if (!ranges_left(&S) && S.pool.empty() && S.ready_pos >= S.ready.size())
            status[b] = EAHR_LIST_EXHAUSTED;
        else status[b] = EAHR_LIST_OPEN;
    }
    if (::eahr::trace_on())
        std::fprintf(stderr,
                     "pbm_gpu next queries=%d device_rounds=%lld tasks=%zu keys=%zu ms=%.2f host_ms=%.2f "
                     "device_ms=%.2f pool_ms=%.2f\n",
                     B, static_cast<long long>(rounds), all_tasks, all_keys, since(t0), t_host, t_dev, t_pool);
    return EAHR_OK;
}

extern "C" int pbm_gpu_counters(const pbm_gpu_state* st, int32_t b, int64_t* out) {
    if (!st || !out || b < 0 || b >= st->B) EAHR_FAIL(EAHR_E_INVALID, "pbm_gpu_counters: bad arguments");
    const pbm_state& S = st->q[b];
    out[0] = S.postings_visited;
    out[1] = S.items_scored;
    out[2] = S.ranges_expanded;
    return EAHR_OK;
}

extern "C" void pbm_gpu_close(pbm_gpu_state* st) {
    if (!st) return;
    const pbm_index* ix = st->ix;
    if (st->stream) (void)hipStreamSynchronize(st->stream);
    bool release = false;
    if (ix) {
        std::lock_guard<std::mutex> lk(ix->free_mu);
        ix->open_states -= 1;
        release = ix->release_requested && ix->open_states == 0;
        if (!release && ix->free_gpu_states.size() < kFreeGpuStates) {
            ix->free_gpu_states.push_back(st);
            return;
        }
    }
    delete st;
    if (release) delete ix;   // pbm_free came first
}
