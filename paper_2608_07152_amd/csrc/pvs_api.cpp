// Host runtime of the PVS dense channel: index storage in HBM, snapshots,
// per-query resumable state and the scan -> rescore -> sort -> certify driver.
//
// Certification rule (Sec. 2.3.1 exact prefixes): a scan with threshold tau
// collects every eligible visible row with hi >= tau, rescores them in float32
// and certifies those with s32 >= tau.  Any row left out has
// s32 <= hi < tau, so the certified rows, in (s32 desc, id asc) order, are
// exactly the next ranks after the last certified key.  tau only changes the
// work done, never the result; it is estimated from a sampled subset of
// blocks and lowered when a scan certifies too few ranks.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <atomic>
#include <memory>
#include <mutex>
#include <new>
#include <vector>

#include "common.h"
#include "eahr.h"
#include "host_parallel.h"
#include "pvs_internal.h"
#include "pvs_kernels.h"

using pvs::ScanQ;

namespace {

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Smallest float32 >= a / (1 - a), a = (8m + 64) * 2^-23 (App. A.1): num/den
// with num = 8m + 64 and den = 2^23 - num, compared exactly in integers.
float gamma_of(int32_t m) {
    const int64_t num = 8LL * m + 64;
    const int64_t den = (1LL << 23) - num;
    float f = static_cast<float>(static_cast<double>(num) / static_cast<double>(den));
    auto ge = [&](float x) {  // x >= num / den  <=>  M * den >= num * 2^-e
        int e;
        const double mant = std::frexp(static_cast<double>(x), &e);   // x = mant * 2^e
        const __int128 M = static_cast<__int128>(std::ldexp(mant, 53));  // x = M * 2^(e-53)
        const int sh = 53 - e;                                          // > 0 here
        return M * den >= static_cast<__int128>(num) << sh;
    };
    while (!ge(f)) f = std::nextafter(f, std::numeric_limits<float>::infinity());
    while (ge(std::nextafter(f, 0.0f))) f = std::nextafter(f, 0.0f);
    return f;
}

template <typename T>
int dev_alloc(T** p, size_t count) {
    *p = nullptr;
    if (count == 0) count = 1;
    HIP_TRY(hipMalloc(reinterpret_cast<void**>(p), count * sizeof(T)));
    return EAHR_OK;
}

template <typename T>
void dev_free(T*& p) {
    if (p) (void)hipFree(p);
    p = nullptr;
}

std::atomic<int> g_prof_on{0};
std::mutex g_prof_mu;
pvs_profile g_prof{};

bool is_device_ptr(const void* p) {
    hipPointerAttribute_t a;
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    return a.type == hipMemoryTypeDevice;
}

}  // namespace

static void free_buffers(ScanBuffers& b);

// ======================================================================= index
pvs_index::~pvs_index() {
    dev_free(codes);
    dev_free(scale);
    dev_free(vnorm);
    dev_free(enorm);
    dev_free(frows);
    dev_free(live);
    dev_free(flags);
    dev_free(staging);
    for (auto& s : snaps) dev_free(s.vis);
    free_buffers(spare);
}

static int index_grow(pvs_index* ix, int64_t need_rows) {
    if (need_rows <= ix->cap) return EAHR_OK;
    int64_t cap = std::max<int64_t>(need_rows, ix->cap + ix->cap / 2);
    cap = round_up(std::max<int64_t>(cap, 64), 64);
    int8_t* codes;
    float *scale, *vnorm, *enorm, *frows;
    uint64_t* live;
    EAHR_TRY(dev_alloc(&codes, static_cast<size_t>(cap) * ix->dp));
    EAHR_TRY(dev_alloc(&scale, cap));
    EAHR_TRY(dev_alloc(&vnorm, cap));
    EAHR_TRY(dev_alloc(&enorm, cap));
    EAHR_TRY(dev_alloc(&frows, static_cast<size_t>(cap) * ix->df));
    EAHR_TRY(dev_alloc(&live, cap / 64));
    hipStream_t s = ix->stream;
    HIP_TRY(hipMemsetAsync(codes, 0, static_cast<size_t>(cap) * ix->dp, s));
    HIP_TRY(hipMemsetAsync(scale, 0, cap * sizeof(float), s));
    HIP_TRY(hipMemsetAsync(vnorm, 0, cap * sizeof(float), s));
    HIP_TRY(hipMemsetAsync(enorm, 0, cap * sizeof(float), s));
    HIP_TRY(hipMemsetAsync(live, 0, cap / 64 * sizeof(uint64_t), s));
    if (ix->cap > 0) {
        HIP_TRY(hipMemcpyAsync(codes, ix->codes, static_cast<size_t>(ix->cap) * ix->dp,
                               hipMemcpyDeviceToDevice, s));
        HIP_TRY(hipMemcpyAsync(scale, ix->scale, ix->cap * sizeof(float), hipMemcpyDeviceToDevice, s));
        HIP_TRY(hipMemcpyAsync(vnorm, ix->vnorm, ix->cap * sizeof(float), hipMemcpyDeviceToDevice, s));
        HIP_TRY(hipMemcpyAsync(enorm, ix->enorm, ix->cap * sizeof(float), hipMemcpyDeviceToDevice, s));
        HIP_TRY(hipMemcpyAsync(frows, ix->frows, static_cast<size_t>(ix->cap) * ix->df * sizeof(float),
                               hipMemcpyDeviceToDevice, s));
        HIP_TRY(hipMemcpyAsync(live, ix->live, ix->cap / 64 * sizeof(uint64_t), hipMemcpyDeviceToDevice, s));
        HIP_TRY(hipStreamSynchronize(s));
    }
    dev_free(ix->codes);
    dev_free(ix->scale);
    dev_free(ix->vnorm);
    dev_free(ix->enorm);
    dev_free(ix->frows);
    dev_free(ix->live);
    ix->codes = codes;
    ix->scale = scale;
    ix->vnorm = vnorm;
    ix->enorm = enorm;
    ix->frows = frows;
    ix->live = live;
    ix->cap = cap;
    return EAHR_OK;
}

// The shared scale of a global-scale index: fl32(max |x| / 127) over the n
// rows given (its first non-empty build or insert), 1 if they are all zero,
// the smallest positive float32 if the quotient underflows (the per-row rule
// applied to the whole matrix).
static int global_scale_of(pvs_index* ix, const float* src, int64_t n, bool dev, float* out) {
    hipStream_t s = ix->stream;
    HIP_TRY(hipMemsetAsync(ix->flags, 0, 4 * sizeof(uint32_t), s));
    const int64_t chunk = 65536;
    for (int64_t r = 0; r < n; r += chunk) {
        const int64_t k = std::min(chunk, n - r);
        const float* p = src + r * ix->d;
        if (!dev) {
            if (!ix->staging) EAHR_TRY(dev_alloc(&ix->staging, static_cast<size_t>(chunk) * ix->d));
            HIP_TRY(hipMemcpyAsync(ix->staging, p, static_cast<size_t>(k) * ix->d * sizeof(float),
                                   hipMemcpyHostToDevice, s));
            p = ix->staging;
        }
        pvs::launch_maxabs(p, k * ix->d, ix->flags, s);
        HIP_TRY(hipGetLastError());
        if (!dev) HIP_TRY(hipStreamSynchronize(s));   // staging buffer is reused
    }
    uint32_t fl[4];
    HIP_TRY(hipMemcpyAsync(fl, ix->flags, sizeof(fl), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (fl[0]) EAHR_FAIL(EAHR_E_NONFINITE, "non-finite value in corpus rows");
    float mu;
    std::memcpy(&mu, &fl[3], 4);
    float sc = mu / 127.0f;
    if (mu > 0.0f && sc == 0.0f) sc = std::numeric_limits<float>::denorm_min();
    if (mu == 0.0f) sc = 1.0f;
    *out = sc;
    return EAHR_OK;
}

// Quantise n rows (host or device) into rows [row0, row0 + n) of the index.
static int index_quantize(pvs_index* ix, const float* src, int64_t n, int32_t ptr_kind, int64_t row0) {
    hipStream_t s = ix->stream;
    const bool dev = (ptr_kind == EAHR_PTR_DEVICE);
    if (ix->quant == EAHR_QUANT_GLOBAL && ix->global_s == 0.0f && n > 0)
        EAHR_TRY(global_scale_of(ix, src, n, dev, &ix->global_s));
    const float fixed_s = (ix->quant == EAHR_QUANT_GLOBAL) ? ix->global_s : 0.0f;
    HIP_TRY(hipMemsetAsync(ix->flags, 0, 4 * sizeof(uint32_t), s));
    const int64_t chunk = 65536;
    for (int64_t r = 0; r < n; r += chunk) {
        const int64_t k = std::min(chunk, n - r);
        const float* p = src + r * ix->d;
        if (!dev) {
            if (!ix->staging) EAHR_TRY(dev_alloc(&ix->staging, static_cast<size_t>(chunk) * ix->d));
            HIP_TRY(hipMemcpyAsync(ix->staging, p, static_cast<size_t>(k) * ix->d * sizeof(float),
                                   hipMemcpyHostToDevice, s));
            p = ix->staging;
        }
        pvs::launch_quantize(p, k, ix->d, ix->d, row0 + r, true, ix->codes, ix->dp, ix->scale,
                             ix->vnorm, ix->enorm, nullptr, ix->frows, ix->df, fixed_s, ix->flags, s);
        HIP_TRY(hipGetLastError());
        if (!dev) HIP_TRY(hipStreamSynchronize(s));   // staging buffer is reused
    }
    uint32_t fl[4];
    HIP_TRY(hipMemcpyAsync(fl, ix->flags, sizeof(fl), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (fl[0]) EAHR_FAIL(EAHR_E_NONFINITE, "non-finite value in corpus rows");
    float nv, nev;
    std::memcpy(&nv, &fl[1], 4);
    std::memcpy(&nev, &fl[2], 4);
    ix->nv_max = std::max(ix->nv_max, nv);
    ix->nev_max = std::max(ix->nev_max, nev);
    return EAHR_OK;
}

static int take_snapshot(pvs_index* ix, int64_t* epoch) {
    pvs_index::Snapshot sn;
    sn.rows = ix->rows;
    const int64_t words = std::max<int64_t>(1, (ix->rows + 63) / 64);
    EAHR_TRY(dev_alloc(&sn.vis, words));
    HIP_TRY(hipMemcpyAsync(sn.vis, ix->live, words * sizeof(uint64_t), hipMemcpyDeviceToDevice,
                           ix->stream));
    unsigned long long* cnt;
    EAHR_TRY(dev_alloc(&cnt, 1));
    HIP_TRY(hipMemsetAsync(cnt, 0, sizeof(unsigned long long), ix->stream));
    pvs::launch_popcount(sn.vis, words, cnt, ix->stream);
    unsigned long long h = 0;
    HIP_TRY(hipMemcpyAsync(&h, cnt, sizeof(h), hipMemcpyDeviceToHost, ix->stream));
    HIP_TRY(hipStreamSynchronize(ix->stream));
    dev_free(cnt);
    sn.visible = static_cast<int64_t>(h);
    ix->snaps.push_back(sn);
    if (epoch) *epoch = static_cast<int64_t>(ix->snaps.size()) - 1;
    return EAHR_OK;
}

extern "C" int pvs_build(const float* corpus, int64_t n, int32_t d, int32_t ptr_kind, void* stream,
                         pvs_index** out) {
    return pvs_build_quant(corpus, n, d, ptr_kind, stream, EAHR_QUANT_PER_VECTOR, out);
}

extern "C" int pvs_build_quant(const float* corpus, int64_t n, int32_t d, int32_t ptr_kind,
                               void* stream, int32_t quant, pvs_index** out) {
    if (!out) EAHR_FAIL(EAHR_E_INVALID, "pvs_build: out is NULL");
    *out = nullptr;
    if (quant != EAHR_QUANT_PER_VECTOR && quant != EAHR_QUANT_GLOBAL)
        EAHR_FAIL(EAHR_E_INVALID, "pvs_build: unknown quantisation mode %d", quant);
    if (n < 0 || d <= 0 || (n > 0 && !corpus)) EAHR_FAIL(EAHR_E_INVALID, "pvs_build: bad arguments");
    if (d > pvs::kMaxDim) EAHR_FAIL(EAHR_E_RANGE, "pvs_build: d=%d exceeds %d", d, pvs::kMaxDim);
    if (n >= (1LL << 31) - 64) EAHR_FAIL(EAHR_E_RANGE, "pvs_build: too many rows");
    if (ptr_kind != EAHR_PTR_HOST && ptr_kind != EAHR_PTR_DEVICE)
        EAHR_FAIL(EAHR_E_INVALID, "pvs_build: bad ptr_kind");
    std::unique_ptr<pvs_index> ix(new (std::nothrow) pvs_index());
    if (!ix) EAHR_FAIL(EAHR_E_OOM, "pvs_build: host allocation");
    HIP_TRY(hipGetDevice(&ix->device));
    ix->stream = static_cast<hipStream_t>(stream);
    ix->d = d;
    ix->dp = static_cast<int32_t>(round_up(d, 64));
    ix->df = static_cast<int32_t>(round_up(d, 4));
    ix->nchunk = ix->dp / 16;
    ix->gamma = gamma_of(d);
    ix->quant = quant;
    EAHR_TRY(dev_alloc(&ix->flags, 4));
    EAHR_TRY(index_grow(ix.get(), std::max<int64_t>(n, 64)));
    if (n > 0) {
        EAHR_TRY(index_quantize(ix.get(), corpus, n, ptr_kind, 0));
        pvs::launch_set_bits(ix->live, 0, n, ix->stream);
        HIP_TRY(hipGetLastError());
    }
    ix->rows = n;
    EAHR_TRY(take_snapshot(ix.get(), nullptr));
    *out = ix.release();
    return EAHR_OK;
}

extern "C" int pvs_insert(pvs_index* ix, const float* rows, int64_t n_new, int32_t ptr_kind,
                          int64_t* first_id) {
    if (!ix || n_new < 0 || (n_new > 0 && !rows)) EAHR_FAIL(EAHR_E_INVALID, "pvs_insert: bad arguments");
    if (ix->rows + n_new >= (1LL << 31) - 64) EAHR_FAIL(EAHR_E_RANGE, "pvs_insert: too many rows");
    if (first_id) *first_id = ix->rows;
    if (n_new == 0) return EAHR_OK;
    EAHR_TRY(index_grow(ix, ix->rows + n_new));
    EAHR_TRY(index_quantize(ix, rows, n_new, ptr_kind, ix->rows));
    pvs::launch_set_bits(ix->live, ix->rows, n_new, ix->stream);
    HIP_TRY(hipGetLastError());
    ix->rows += n_new;
    return EAHR_OK;
}

extern "C" int pvs_delete(pvs_index* ix, const int64_t* ids, int64_t n) {
    if (!ix || n < 0 || (n > 0 && !ids)) EAHR_FAIL(EAHR_E_INVALID, "pvs_delete: bad arguments");
    for (int64_t i = 0; i < n; ++i)
        if (ids[i] < 0 || ids[i] >= ix->rows) EAHR_FAIL(EAHR_E_INVALID, "pvs_delete: id out of range");
    if (n == 0) return EAHR_OK;
    int64_t* d_ids;
    EAHR_TRY(dev_alloc(&d_ids, n));
    HIP_TRY(hipMemcpyAsync(d_ids, ids, n * sizeof(int64_t), hipMemcpyHostToDevice, ix->stream));
    pvs::launch_clear_ids(ix->live, d_ids, n, ix->stream);
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipStreamSynchronize(ix->stream));
    dev_free(d_ids);
    return EAHR_OK;
}

extern "C" int pvs_snapshot(pvs_index* ix, int64_t* epoch) {
    if (!ix) EAHR_FAIL(EAHR_E_INVALID, "pvs_snapshot: NULL index");
    return take_snapshot(ix, epoch);
}

extern "C" int pvs_info(const pvs_index* ix, int64_t epoch, int64_t* rows, int32_t* d,
                        int64_t* visible) {
    if (!ix || epoch < 0 || epoch >= static_cast<int64_t>(ix->snaps.size()))
        EAHR_FAIL(EAHR_E_INVALID, "pvs_info: bad index or epoch");
    if (rows) *rows = ix->snaps[epoch].rows;
    if (d) *d = ix->d;
    if (visible) *visible = ix->snaps[epoch].visible;
    return EAHR_OK;
}

extern "C" void pvs_free(pvs_index* ix) {
    if (!ix) return;
    {
        std::lock_guard<std::mutex> lk(ix->life_mu);
        if (ix->open_states > 0) {   // released by the last pvs_close
            ix->release_requested = true;
            return;
        }
    }
    delete ix;
}

extern "C" int pvs_read_index(const pvs_index* ix, int64_t row0, int64_t n, int8_t* codes,
                              float* meta) {
    if (!ix || row0 < 0 || n < 0 || row0 + n > ix->rows) EAHR_FAIL(EAHR_E_INVALID, "pvs_read_index: bad range");
    if (n == 0) return EAHR_OK;
    const int64_t b0 = row0 / 64, b1 = (row0 + n - 1) / 64 + 1;
    std::vector<int8_t> blk(static_cast<size_t>(b1 - b0) * 64 * ix->dp);
    HIP_TRY(hipMemcpy(blk.data(), ix->codes + b0 * 64 * ix->dp, blk.size(), hipMemcpyDeviceToHost));
    if (codes) {
        for (int64_t i = 0; i < n; ++i) {
            const int64_t r = row0 + i;
            const int64_t rb = r / 64 - b0, rr = r % 64;
            for (int32_t j = 0; j < ix->d; ++j) {
                const int64_t off = ((rb * ix->nchunk + j / 16) * 64 + rr) * 16 + j % 16;
                codes[i * ix->d + j] = blk[off];
            }
        }
    }
    if (meta) {
        std::vector<float> s(n), a(n), e(n);
        HIP_TRY(hipMemcpy(s.data(), ix->scale + row0, n * sizeof(float), hipMemcpyDeviceToHost));
        HIP_TRY(hipMemcpy(a.data(), ix->vnorm + row0, n * sizeof(float), hipMemcpyDeviceToHost));
        HIP_TRY(hipMemcpy(e.data(), ix->enorm + row0, n * sizeof(float), hipMemcpyDeviceToHost));
        for (int64_t i = 0; i < n; ++i) {
            meta[3 * i] = s[i];
            meta[3 * i + 1] = a[i];
            meta[3 * i + 2] = e[i];
        }
    }
    return EAHR_OK;
}

// ======================================================================= state
pvs_state::~pvs_state() {
    dev_free(qcodes);
    dev_free(qrows);
    dev_free(qscale);
    dev_free(qnorm);
    dev_free(qenorm);
    dev_free(qhnorm);
    dev_free(qflags);
    release_scan_buffers();
    for (auto& e : ev)
        if (e) (void)hipEventDestroy(e);
}

void pvs_state::release_scan_buffers() {
    dev_free(scanq);
    dev_free(counts);
    dev_free(sample_lo);
    dev_free(sample_hi);
    dev_free(qfrag);
    dev_free(pairs);
    dev_free(keys);
    dev_free(keys_tmp);
    dev_free(packed);
    if (h_scanq) (void)hipHostFree(h_scanq);
    if (h_counts) (void)hipHostFree(h_counts);
    if (h_packed) (void)hipHostFree(h_packed);
    h_scanq = nullptr;
    h_counts = nullptr;
    h_packed = nullptr;
    buf_nq = 0;
    buf_sample = 0;
    pool_cap = 0;
    h_packed_cap = 0;
}

// Move the scan buffers between a state and an index's spare slot.
#define PVS_BUFFER_FIELDS(X)                                                                 \
    X(buf_nq) X(buf_sample) X(scanq) X(counts) X(sample_lo) X(sample_hi) X(qfrag) X(pool_cap) \
    X(pairs) X(keys) X(keys_tmp) X(packed) X(h_scanq) X(h_counts)    \
    X(h_packed) X(h_packed_cap)

static void adopt_buffers(pvs_state* st, ScanBuffers& b) {
#define PVS_MOVE_IN(f) st->f = b.f;
    PVS_BUFFER_FIELDS(PVS_MOVE_IN)
#undef PVS_MOVE_IN
    st->recycled.swap(b.caches);
    b = ScanBuffers{};
}

// Caches kept for the next state, at most this many bytes in all: reusing
// their memory spares the page faults of fresh allocations.
constexpr size_t kRecycleBytes = size_t(2) << 30;

static void donate_buffers(pvs_state* st, ScanBuffers& b) {
#define PVS_MOVE_OUT(f) b.f = st->f;
    PVS_BUFFER_FIELDS(PVS_MOVE_OUT)
#undef PVS_MOVE_OUT
    b.caches.clear();
    size_t kept = 0;
    for (auto& Q : st->q) {
        const size_t bytes = Q.cache.capacity() * sizeof(uint64_t);
        if (kept + bytes > kRecycleBytes) break;
        kept += bytes;
        Q.cache.clear();
        Q.pend_n = 0;
        b.caches.push_back(std::move(Q.cache));
    }
    st->buf_nq = 0;
    st->buf_sample = 0;
    st->pool_cap = 0;
    st->h_packed_cap = 0;
    st->scanq = nullptr;
    st->counts = nullptr;
    st->sample_lo = nullptr;
    st->sample_hi = nullptr;
    st->qfrag = nullptr;
    st->pairs = nullptr;
    st->keys = nullptr;
    st->keys_tmp = nullptr;
    st->packed = nullptr;
    st->h_scanq = nullptr;
    st->h_counts = nullptr;
    st->h_packed = nullptr;
}

static void free_buffers(ScanBuffers& b) {
    dev_free(b.scanq);
    dev_free(b.counts);
    dev_free(b.sample_lo);
    dev_free(b.sample_hi);
    dev_free(b.qfrag);
    dev_free(b.pairs);
    dev_free(b.keys);
    dev_free(b.keys_tmp);
    dev_free(b.packed);
    if (b.h_scanq) (void)hipHostFree(b.h_scanq);
    if (b.h_counts) (void)hipHostFree(b.h_counts);
    if (b.h_packed) (void)hipHostFree(b.h_packed);
    b = ScanBuffers{};
}

// Per-query scan buffers for nq queries and samples of sample_ld rows.
// counts layout: [cert nq][fail nq][offs nq + 1][unused 1]
// [rescore chunk base kSub + 1], then from pair_counts_at(nq) the kSub append
// counters of the pair pool, from reads_counts_at(nq) the kSub row-load
// counters of rescoring, kCntStride ints apart, and from evals_counts_at(nq)
// the records of each query.  h_counts mirrors it.
static size_t pair_counts_at(int32_t nq) {
    return (3 * static_cast<size_t>(nq) + 2 + pvs::kSub + 1 + 63) / 64 * 64;
}
static size_t reads_counts_at(int32_t nq) {
    return pair_counts_at(nq) + static_cast<size_t>(pvs::kSub) * pvs::kCntStride;
}
static size_t evals_counts_at(int32_t nq) {
    return reads_counts_at(nq) + static_cast<size_t>(pvs::kSub) * pvs::kCntStride;
}
static size_t all_counts(int32_t nq) {
    return evals_counts_at(nq) + static_cast<size_t>(pvs::kSub) * nq;
}

static int ensure_query_buffers(pvs_state* st, int32_t nq, int64_t sample_ld) {
    if (nq <= st->buf_nq && sample_ld <= st->buf_sample) return EAHR_OK;
    nq = std::max(nq, st->buf_nq);
    sample_ld = std::max(sample_ld, st->buf_sample);
    HIP_TRY(hipStreamSynchronize(st->ix->stream));
    dev_free(st->scanq);
    dev_free(st->counts);
    dev_free(st->sample_lo);
    dev_free(st->sample_hi);
    dev_free(st->qfrag);
    if (st->h_scanq) (void)hipHostFree(st->h_scanq);
    if (st->h_counts) (void)hipHostFree(st->h_counts);
    st->h_scanq = nullptr;
    st->h_counts = nullptr;
    EAHR_TRY(dev_alloc(&st->scanq, nq));
    EAHR_TRY(dev_alloc(&st->counts, all_counts(nq)));
    EAHR_TRY(dev_alloc(&st->sample_lo, static_cast<size_t>(nq) * sample_ld));
    EAHR_TRY(dev_alloc(&st->sample_hi, static_cast<size_t>(nq) * sample_ld));
    int8_t* f;
    EAHR_TRY(dev_alloc(&f, static_cast<size_t>(st->ix->dp / 32) * 8 * 64 * 16));
    st->qfrag = f;
    HIP_TRY(hipHostMalloc(reinterpret_cast<void**>(&st->h_scanq), nq * sizeof(ScanQ)));
    HIP_TRY(hipHostMalloc(reinterpret_cast<void**>(&st->h_counts), all_counts(nq) * sizeof(int32_t)));
    st->buf_nq = nq;
    st->buf_sample = sample_ld;
    return EAHR_OK;
}

// Pair pool and key regions of `slots` entries for one scan.
static int ensure_pool(pvs_state* st, int64_t slots) {
    if (slots <= st->pool_cap) return EAHR_OK;
    slots = std::max<int64_t>(slots + slots / 4, pvs::kMinCap);
    HIP_TRY(hipStreamSynchronize(st->ix->stream));
    dev_free(st->pairs);
    dev_free(st->keys);
    dev_free(st->keys_tmp);
    dev_free(st->packed);
    st->pool_cap = 0;
    const size_t n = static_cast<size_t>(slots);
    EAHR_TRY(dev_alloc(&st->pairs, n));
    EAHR_TRY(dev_alloc(&st->keys, n));
    EAHR_TRY(dev_alloc(&st->keys_tmp, n));
    EAHR_TRY(dev_alloc(&st->packed, n));
    st->pool_cap = slots;
    return EAHR_OK;
}

static int ensure_host_packed(pvs_state* st, int64_t n) {
    if (n <= st->h_packed_cap) return EAHR_OK;
    n = std::max<int64_t>(n + n / 4, 4096);
    if (st->h_packed) (void)hipHostFree(st->h_packed);
    st->h_packed = nullptr;
    st->h_packed_cap = 0;
    HIP_TRY(hipHostMalloc(reinterpret_cast<void**>(&st->h_packed), n * sizeof(uint64_t)));
    st->h_packed_cap = n;
    return EAHR_OK;
}

extern "C" int pvs_open(const pvs_index* ix, int64_t epoch, const float* q, int32_t B,
                        int32_t ptr_kind, pvs_state** out) {
    return pvs_open_gen(ix, epoch, q, B, ptr_kind, EAHR_GEN_INTERVALS, out);
}

extern "C" int pvs_open_gen(const pvs_index* ix, int64_t epoch, const float* q, int32_t B,
                            int32_t ptr_kind, int32_t generator, pvs_state** out) {
    if (!out) EAHR_FAIL(EAHR_E_INVALID, "pvs_open: out is NULL");
    *out = nullptr;
    if (generator != EAHR_GEN_INTERVALS && generator != EAHR_GEN_FULL_SCAN)
        EAHR_FAIL(EAHR_E_INVALID, "pvs_open: unknown generator %d", generator);
    if (!ix || B <= 0 || !q) EAHR_FAIL(EAHR_E_INVALID, "pvs_open: bad arguments");
    if (epoch < 0 || epoch >= static_cast<int64_t>(ix->snaps.size()))
        EAHR_FAIL(EAHR_E_INVALID, "pvs_open: unknown epoch %lld", static_cast<long long>(epoch));
    if (ptr_kind != EAHR_PTR_HOST && ptr_kind != EAHR_PTR_DEVICE)
        EAHR_FAIL(EAHR_E_INVALID, "pvs_open: bad ptr_kind");
    {
        std::lock_guard<std::mutex> lk(ix->life_mu);
        if (ix->release_requested) EAHR_FAIL(EAHR_E_INVALID, "pvs_open: the index has been freed");
    }
    std::unique_ptr<pvs_state> st(new (std::nothrow) pvs_state());
    if (!st) EAHR_FAIL(EAHR_E_OOM, "pvs_open: host allocation");
    st->ix = ix;
    st->epoch = epoch;
    st->B = B;
    st->generator = generator;
    if (const char* p = std::getenv("EAHR_SCAN_PATH")) {
        if (std::strcmp(p, "gemv") == 0) st->path = pvs::ScanPath::Gemv;
        else if (std::strcmp(p, "mfma") == 0) st->path = pvs::ScanPath::Mfma;
    }
    if (const char* p = std::getenv("EAHR_CAP_SHRINK")) st->cap_shrink = std::max(1L, std::atol(p));
    if (const char* p = std::getenv("EAHR_TEST_FAIL_QUERY")) st->test_fail_qi = static_cast<int32_t>(std::atol(p));
    st->n_rows = ix->snaps[epoch].rows;
    st->n_vis = ix->snaps[epoch].visible;
    st->vis = ix->snaps[epoch].vis;
    if (ix->has_spare) {
        adopt_buffers(st.get(), ix->spare);
        ix->has_spare = false;
    }
    hipStream_t s = ix->stream;
    EAHR_TRY(dev_alloc(&st->qcodes, static_cast<size_t>(B) * ix->dp));
    EAHR_TRY(dev_alloc(&st->qrows, static_cast<size_t>(B) * ix->df));
    EAHR_TRY(dev_alloc(&st->qscale, B));
    EAHR_TRY(dev_alloc(&st->qnorm, B));
    EAHR_TRY(dev_alloc(&st->qenorm, B));
    EAHR_TRY(dev_alloc(&st->qhnorm, B));
    EAHR_TRY(dev_alloc(&st->qflags, 4));
    HIP_TRY(hipMemsetAsync(st->qflags, 0, 4 * sizeof(uint32_t), s));
    const float* src = q;
    float* tmp = nullptr;
    if (ptr_kind == EAHR_PTR_HOST) {
        EAHR_TRY(dev_alloc(&tmp, static_cast<size_t>(B) * ix->d));
        HIP_TRY(hipMemcpyAsync(tmp, q, static_cast<size_t>(B) * ix->d * sizeof(float),
                               hipMemcpyHostToDevice, s));
        src = tmp;
    }
    pvs::launch_quantize(src, B, ix->d, ix->d, 0, false, st->qcodes, ix->dp, st->qscale, st->qnorm,
                         st->qenorm, st->qhnorm, st->qrows, ix->df, 0.0f, st->qflags, s);
    HIP_TRY(hipGetLastError());
    std::vector<float> sc(B), nq(B), ne(B), nh(B);
    uint32_t fl[4];
    HIP_TRY(hipMemcpyAsync(sc.data(), st->qscale, B * sizeof(float), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(nq.data(), st->qnorm, B * sizeof(float), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(ne.data(), st->qenorm, B * sizeof(float), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(nh.data(), st->qhnorm, B * sizeof(float), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(fl, st->qflags, sizeof(fl), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    dev_free(tmp);
    if (fl[0]) EAHR_FAIL(EAHR_E_NONFINITE, "pvs_open: non-finite value in a query");
    st->q.resize(B);
    for (size_t b = 0; b < st->recycled.size() && b < static_cast<size_t>(B); ++b)
        st->q[b].cache.swap(st->recycled[b]);
    st->recycled.clear();
    const double NV = ix->nv_max, NEV = ix->nev_max, g = ix->gamma;
    for (int32_t b = 0; b < B; ++b) {
        auto& Q = st->q[b];
        Q.sq = sc[b];
        Q.nq = nq[b];
        Q.neq = ne[b];
        Q.nqh = nh[b];
        // bound of E + G over every row: |c| <= ||q_hat|| (||v|| + ||e_v||)
        const double E = ne[b] * NV + nh[b] * NEV;
        const double c = nh[b] * (NV + NEV);
        const double G = (c + E + nq[b] * NV) * g;
        Q.wmax = static_cast<float>((E + G) * 1.01 + 1e-30);
    }
    {
        std::lock_guard<std::mutex> lk(ix->life_mu);
        ix->open_states += 1;
    }
    *out = st.release();
    return EAHR_OK;
}

extern "C" void pvs_close(pvs_state* st) {
    if (!st) return;
    const pvs_index* ix = st->ix;
    if (ix) {
        (void)hipStreamSynchronize(ix->stream);
        if (!ix->has_spare) {
            donate_buffers(st, ix->spare);
            ix->has_spare = true;
        }
    }
    delete st;
    if (!ix) return;
    bool release = false;
    {
        std::lock_guard<std::mutex> lk(ix->life_mu);
        ix->open_states -= 1;
        release = ix->release_requested && ix->open_states == 0;
    }
    if (release) delete ix;   // pvs_free came first
}

extern "C" int pvs_read_query(const pvs_state* st, int8_t* codes, float* meta) {
    if (!st) EAHR_FAIL(EAHR_E_INVALID, "pvs_read_query: NULL state");
    const pvs_index* ix = st->ix;
    if (codes) {
        std::vector<int8_t> all(static_cast<size_t>(st->B) * ix->dp);
        HIP_TRY(hipMemcpy(all.data(), st->qcodes, all.size(), hipMemcpyDeviceToHost));
        for (int32_t b = 0; b < st->B; ++b)
            std::memcpy(codes + static_cast<size_t>(b) * ix->d, all.data() + static_cast<size_t>(b) * ix->dp, ix->d);
    }
    if (meta) {
        for (int32_t b = 0; b < st->B; ++b) {
            meta[4 * b] = st->q[b].sq;
            meta[4 * b + 1] = st->q[b].nq;
            meta[4 * b + 2] = st->q[b].nqh;
            meta[4 * b + 3] = st->q[b].neq;
        }
    }
    return EAHR_OK;
}

static ScanQ make_scanq(const pvs_state* st, int32_t b) {
    const auto& Q = st->q[b];
    ScanQ s{};
    s.qi = b;
    s.tau = -std::numeric_limits<float>::infinity();
    s.has_cert = Q.has_cert ? 1 : 0;
    s.s_cert = Q.s_cert;
    s.id_cert = Q.id_cert;
    s.k = 0;
    s.sq = Q.sq;
    s.nq = Q.nq;
    s.nqh = Q.nqh;
    s.neq = Q.neq;
    s.wmax = Q.wmax;
    return s;
}

static pvs::IndexView view_of(const pvs_index* ix) {
    pvs::IndexView v;
    v.codes = reinterpret_cast<const uint4*>(ix->codes);
    v.scale = ix->scale;
    v.vnorm = ix->vnorm;
    v.enorm = ix->enorm;
    v.rows = ix->frows;
    v.d = ix->d;
    v.dp = ix->dp;
    v.df = ix->df;
    v.nchunk = ix->nchunk;
    return v;
}

extern "C" int pvs_intervals(const pvs_state* st, int32_t b, const int64_t* rows, int64_t n,
                             float* lo, float* hi) {
    if (!st || b < 0 || b >= st->B || n < 0 || (n > 0 && (!rows || !lo || !hi)))
        EAHR_FAIL(EAHR_E_INVALID, "pvs_intervals: bad arguments");
    for (int64_t i = 0; i < n; ++i)
        if (rows[i] < 0 || rows[i] >= st->n_rows) EAHR_FAIL(EAHR_E_INVALID, "pvs_intervals: row out of range");
    if (n == 0) return EAHR_OK;
    const pvs_index* ix = st->ix;
    hipStream_t s = ix->stream;
    ScanQ q = make_scanq(st, b);
    ScanQ* dq;
    int64_t* dr;
    float *dlo, *dhi;
    EAHR_TRY(dev_alloc(&dq, 1));
    EAHR_TRY(dev_alloc(&dr, n));
    EAHR_TRY(dev_alloc(&dlo, n));
    EAHR_TRY(dev_alloc(&dhi, n));
    HIP_TRY(hipMemcpyAsync(dq, &q, sizeof(q), hipMemcpyHostToDevice, s));
    HIP_TRY(hipMemcpyAsync(dr, rows, n * sizeof(int64_t), hipMemcpyHostToDevice, s));
    pvs::launch_intervals(view_of(ix), st->qcodes, dq, ix->gamma, dr, n, dlo, dhi, s);
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipMemcpyAsync(lo, dlo, n * sizeof(float), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(hi, dhi, n * sizeof(float), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    dev_free(dq);
    dev_free(dr);
    dev_free(dlo);
    dev_free(dhi);
    return EAHR_OK;
}

extern "C" int pvs_scores(const pvs_state* st, int32_t b, const int64_t* rows, int64_t n,
                          float* scores) {
    if (!st || b < 0 || b >= st->B || n < 0 || (n > 0 && (!rows || !scores)))
        EAHR_FAIL(EAHR_E_INVALID, "pvs_scores: bad arguments");
    for (int64_t i = 0; i < n; ++i)
        if (rows[i] < 0 || rows[i] >= st->n_rows) EAHR_FAIL(EAHR_E_INVALID, "pvs_scores: row out of range");
    if (n == 0) return EAHR_OK;
    const pvs_index* ix = st->ix;
    hipStream_t s = ix->stream;
    int64_t* dr;
    float* dout;
    EAHR_TRY(dev_alloc(&dr, n));
    EAHR_TRY(dev_alloc(&dout, n));
    HIP_TRY(hipMemcpyAsync(dr, rows, n * sizeof(int64_t), hipMemcpyHostToDevice, s));
    pvs::launch_scores(view_of(ix), st->qrows, b, dr, n, dout, s);
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipMemcpyAsync(scores, dout, n * sizeof(float), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    dev_free(dr);
    dev_free(dout);
    return EAHR_OK;
}

// ============================================================== scan driver
static inline int32_t key_id(uint64_t key) { return static_cast<int32_t>(key & 0xffffffffu); }
static inline float key_score(uint64_t key) {
    const uint32_t k = ~static_cast<uint32_t>(key >> 32);
    const uint32_t bits = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    float f;
    std::memcpy(&f, &bits, 4);
    return f;
}

// Certified ranks of a query: its cache, then the keys of its last scan
// still in the pinned copy.
static int64_t certified_count(const pvs_state::Query& Q) {
    return static_cast<int64_t>(Q.cache.size()) + Q.pend_n;
}

// Appends every query's keys still in the pinned copy to its cache (before
// a scan overwrites the copy), in pieces over the host threads.
static void flush_pending(pvs_state* st) {
    const int32_t B = st->B;
    std::vector<int64_t> n(B, 0), at(B, 0);
    bool any = false;
    for (int32_t b = 0; b < B; ++b) {
        auto& Q = st->q[b];
        if (Q.pend_n <= 0) continue;
        at[b] = static_cast<int64_t>(Q.cache.size());
        n[b] = Q.pend_n;
        Q.cache.resize(Q.cache.size() + static_cast<size_t>(Q.pend_n));
        any = true;
    }
    if (!any) return;
    eahr::parallel_pieces(n, int64_t(1) << 18, eahr::host_threads(), [&](int64_t b, int64_t lo, int64_t hi) {
        const auto& Q = st->q[b];
        std::memcpy(st->q[b].cache.data() + at[b] + lo, st->h_packed + Q.pend_off + lo,
                    static_cast<size_t>(hi - lo) * sizeof(uint64_t));
    });
    for (int32_t b = 0; b < B; ++b) {
        st->q[b].pend_off = 0;
        st->q[b].pend_n = 0;
    }
}

// Certified ranks of query b that may still have lo <= s_cert: they score at
// most s_cert + 2 * wmax, because lo >= s32 - 2 * wmax.
static int64_t lower_overlap(const pvs_state* st, int32_t b) {
    const auto& Q = st->q[b];
    if (!Q.has_cert) return 0;
    const double lim = static_cast<double>(Q.s_cert) + 2.0 * Q.wmax;
    int64_t a = 0;
    for (int64_t i = static_cast<int64_t>(Q.cache.size()) - 1; i >= 0; --i) {
        if (key_score(Q.cache[i]) > lim) break;
        ++a;
    }
    return a;
}

// Exhaustive float32 generator: every visible row of the epoch is scored in
// float32 (the same authoritative order as rescoring), each query's keys are
// sorted once and the whole ranking becomes its certified cache, so the
// query is finished after one round.  Queries go in groups whose keys and
// sort buffer fit in 4 GiB.
static int full_scan_round(pvs_state* st, std::vector<int32_t>& todo) {
    const pvs_index* ix = st->ix;
    hipStream_t s = ix->stream;
    const int64_t n = st->n_rows;
    const bool prof = g_prof_on.load(std::memory_order_relaxed) != 0;
    if (prof && !st->ev[0])
        for (auto& e : st->ev) HIP_TRY(hipEventCreate(&e));
    const int64_t per = std::min<int64_t>(65535, std::max<int64_t>(1, (int64_t(4) << 30) / std::max<int64_t>(1, 16 * n)));
    const pvs::IndexView v = view_of(ix);
    for (size_t g0 = 0; g0 < todo.size() && n > 0; g0 += static_cast<size_t>(per)) {
        const int32_t ng = static_cast<int32_t>(std::min<int64_t>(per, static_cast<int64_t>(todo.size() - g0)));
        uint64_t *keys = nullptr, *tmp = nullptr;
        int32_t *d_qidx = nullptr, *d_cnt = nullptr;
        ScanQ* d_sq = nullptr;
        std::vector<int32_t> qidx(ng), cnt(ng, static_cast<int32_t>(n));
        std::vector<ScanQ> sq(ng);
        for (int32_t i = 0; i < ng; ++i) {
            qidx[i] = todo[g0 + i];
            sq[i] = ScanQ{};
            sq[i].qi = qidx[i];
            sq[i].cand_off = static_cast<int64_t>(i) * n;
        }
        int rc = EAHR_OK;
        auto body = [&]() -> int {
            EAHR_TRY(dev_alloc(&keys, static_cast<size_t>(ng) * n));
            EAHR_TRY(dev_alloc(&tmp, static_cast<size_t>(ng) * n));
            EAHR_TRY(dev_alloc(&d_qidx, ng));
            EAHR_TRY(dev_alloc(&d_cnt, ng));
            EAHR_TRY(dev_alloc(&d_sq, ng));
            HIP_TRY(hipMemcpyAsync(d_qidx, qidx.data(), ng * sizeof(int32_t), hipMemcpyHostToDevice, s));
            HIP_TRY(hipMemcpyAsync(d_cnt, cnt.data(), ng * sizeof(int32_t), hipMemcpyHostToDevice, s));
            HIP_TRY(hipMemcpyAsync(d_sq, sq.data(), ng * sizeof(ScanQ), hipMemcpyHostToDevice, s));
            if (prof) HIP_TRY(hipEventRecord(st->ev[0], s));
            pvs::launch_full_keys(v, st->vis, n, st->qrows, d_qidx, ng, keys, n, s);
            HIP_TRY(hipGetLastError());
            if (prof) HIP_TRY(hipEventRecord(st->ev[1], s));
            const uint64_t* sorted = pvs::launch_segmented_sort(keys, tmp, d_cnt, d_sq, ng, n, s);
            HIP_TRY(hipGetLastError());
            if (prof) HIP_TRY(hipEventRecord(st->ev[2], s));
            for (int32_t i = 0; i < ng; ++i) {
                auto& Q = st->q[qidx[i]];
                Q.cache.resize(static_cast<size_t>(st->n_vis));
                if (st->n_vis > 0)
                    HIP_TRY(hipMemcpyAsync(Q.cache.data(), sorted + static_cast<int64_t>(i) * n,
                                           st->n_vis * sizeof(uint64_t), hipMemcpyDeviceToHost, s));
            }
            HIP_TRY(hipStreamSynchronize(s));
            return EAHR_OK;
        };
        rc = body();
        dev_free(keys);
        dev_free(tmp);
        dev_free(d_qidx);
        dev_free(d_cnt);
        dev_free(d_sq);
        if (rc != EAHR_OK) return rc;
        if (prof) {
            float t0 = 0.0f, t1 = 0.0f;
            HIP_TRY(hipEventElapsedTime(&t0, st->ev[0], st->ev[1]));
            HIP_TRY(hipEventElapsedTime(&t1, st->ev[1], st->ev[2]));
            std::lock_guard<std::mutex> lk(g_prof_mu);
            g_prof.rescore_ms += t0;
            g_prof.rescore_rows += static_cast<int64_t>(ng) * st->n_vis;
            g_prof.rescore_row_reads += static_cast<int64_t>(ng) * st->n_vis;
            g_prof.rescore_certified += static_cast<int64_t>(ng) * st->n_vis;
            g_prof.sort_ms += t1;
            g_prof.scan_rounds += 1;
        }
        for (int32_t i = 0; i < ng; ++i) {
            auto& Q = st->q[qidx[i]];
            Q.evals += st->n_vis;
            st->stats.scans += 1;
            st->stats.candidates += st->n_vis;
            st->stats.certified += st->n_vis;
            if (st->n_vis > 0) {
                Q.has_cert = true;
                Q.s_cert = key_score(Q.cache.back());
                Q.id_cert = key_id(Q.cache.back());
            }
        }
    }
    for (int32_t b : todo) st->q[b].cert_exhausted = true;
    todo.clear();
    return EAHR_OK;
}

// One scan round over the queries in `todo`; removes the queries it finished.
//  1. sample pass + select: tau and the sampled hit count of every query;
//  2. candidate regions sized from the hits (host), main scan;
//  3. rescore, sort, pack; certified ranks appended to each query's cache.
// Queries whose region overflowed are scanned again with room for all of
// their candidates; queries that certified too few ranks again with a lower
// threshold.
static int scan_round(pvs_state* st, std::vector<int32_t>& todo, int32_t m) {
    // the pinned copy is about to be reused, and the targets below read
    // complete caches
    flush_pending(st);
    if (st->generator == EAHR_GEN_FULL_SCAN) return full_scan_round(st, todo);
    const pvs_index* ix = st->ix;
    hipStream_t s = ix->stream;
    int32_t nq = static_cast<int32_t>(todo.size());
    const int64_t nblocks = (st->n_rows + 63) / 64;
    if (nblocks == 0) {
        for (int32_t b : todo) st->q[b].cert_exhausted = true;
        todo.clear();
        return EAHR_OK;
    }
    int64_t stride = 1;
    while (nblocks / (stride * 2) >= pvs::kSampleBlocks) stride *= 2;
    const int64_t nsb = (nblocks + stride - 1) / stride;
    const int64_t sample_ld = nsb * 64;
    const double frac = static_cast<double>(nsb) / static_cast<double>(nblocks);
    EAHR_TRY(ensure_query_buffers(st, nq, sample_ld));

    const int64_t mmin = std::max<int64_t>(pvs::kTargetMin, std::min<int64_t>(pvs::kTargetMax, pvs::kTargetBudget / nq));
    for (int32_t i = 0; i < nq; ++i) {
        const int32_t b = todo[i];
        auto& Q = st->q[b];
        ScanQ sq = make_scanq(st, b);
        const int64_t have = static_cast<int64_t>(Q.cache.size());
        const int64_t avail = have - Q.emitted;
        const int64_t need = std::max<int64_t>(1, m - avail);
        const int64_t spec_floor = std::max(pvs::kSpecFloor, pvs::kSpecFloorBudget / nq);
        const int64_t spec = st->spec_off ? 0
                           : std::min(std::max(pvs::kSpecFactor * (Q.emitted + m), spec_floor) - have,
                                      pvs::kSpecBudget / nq);
        const int64_t target = std::max({need, mmin, spec}) + lower_overlap(st, b);
        double k = (stride == 1) ? static_cast<double>(target)
                                 : std::max(4.0, std::ceil(pvs::kSampleMargin * target * frac));
        for (int r = 0; r < Q.retries; ++r) k *= 4.0;
        sq.k = static_cast<int32_t>(std::min(k, 2.0e9));
        st->h_scanq[i] = sq;
    }
    const bool mfma = st->path == pvs::ScanPath::Mfma ||
                      (st->path == pvs::ScanPath::Auto && nq >= pvs::kMfmaMinQueries);
    const bool prof = g_prof_on.load(std::memory_order_relaxed) != 0;
    if (prof && !st->ev[0])
        for (auto& e : st->ev) HIP_TRY(hipEventCreate(&e));
    auto mark = [&](int i) -> int {
        if (prof) HIP_TRY(hipEventRecord(st->ev[i], s));
        return EAHR_OK;
    };
    const pvs::IndexView v = view_of(ix);
    auto scan = [&](bool sample, const pvs::ScanOut& o, int32_t n) {
        if (mfma) pvs::launch_scan_mfma(v, st->vis, nblocks, st->qcodes, st->scanq, n, ix->gamma, sample, o, st->qfrag, s);
        else pvs::launch_scan(v, st->vis, nblocks, st->qcodes, st->scanq, n, ix->gamma, sample, o, s);
    };

    const bool trace = ::eahr::trace_on();
    using clk = std::chrono::steady_clock;
    clk::time_point tp[5];
    tp[0] = clk::now();
    // 1. threshold and candidate estimate from the sampled blocks
    HIP_TRY(hipMemcpyAsync(st->scanq, st->h_scanq, nq * sizeof(ScanQ), hipMemcpyHostToDevice, s));
    pvs::ScanOut so;
    so.sample_lo = st->sample_lo;
    so.sample_hi = st->sample_hi;
    so.sample_ld = sample_ld;
    so.sample_stride = stride;
    EAHR_TRY(mark(0));
    scan(true, so, nq);
    pvs::launch_select(st->sample_lo, st->sample_hi, sample_ld, sample_ld, stride > 1, st->scanq, nq, s);
    EAHR_TRY(mark(1));
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipMemcpyAsync(st->h_scanq, st->scanq, nq * sizeof(ScanQ), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    tp[1] = clk::now();

    // 2. candidate regions: the sample saw every block when stride == 1.
    //    Queries past the pool limit wait for the next round (kept in todo).
    int64_t total = 0;
    int32_t run = 0;
    const int64_t max_sub = round_up(st->n_rows, 64);
    for (; run < nq; ++run) {
        ScanQ& sq = st->h_scanq[run];
        const auto& Q = st->q[todo[run]];
        // exact count when the sample saw every block, plus room for the
        // unused tails of per-workgroup slices (at most cap / 16)
        const int64_t cap = (stride == 1)
                          ? static_cast<int64_t>(sq.sample_hits) + sq.sample_hits / 8 + 64
                          : static_cast<int64_t>(std::ceil(sq.sample_hits / frac * pvs::kCapSlack)) + pvs::kCapPad;
        // per sub-region, with room for an uneven split
        int64_t sub = (cap + pvs::kSub - 1) / pvs::kSub;
        sub += sub / 4 + 16;
        if (Q.cap_hint == 0 && st->cap_shrink > 1) sub = std::max<int64_t>(1, sub / st->cap_shrink);
        sub = std::max(sub, Q.cap_hint);
        sub = std::min(sub, max_sub);
        if (run > 0 && total + sub * pvs::kSub > pvs::kPoolMax) break;
        // a pool counter must not wrap: at most (blocks / kSub + 32) * 64 rows
        // of one sub-region times the queries
        if (run > 0 && (nblocks + 2048) * (run + 1) >= (int64_t(1) << 31)) break;
        sq.cand_off = total;
        sq.cand_cap = sub;
        total += sub * pvs::kSub;
    }
    std::vector<int32_t> later(todo.begin() + run, todo.end());
    todo.resize(run);
    nq = run;
    EAHR_TRY(ensure_pool(st, total));
    HIP_TRY(hipMemcpyAsync(st->scanq, st->h_scanq, nq * sizeof(ScanQ), hipMemcpyHostToDevice, s));
    int32_t* d_cert = st->counts;
    int32_t* d_fail = st->counts + nq;
    int32_t* d_offs = st->counts + 2 * nq;
    int32_t* d_reads = st->counts + reads_counts_at(nq);
    int32_t* d_cbase = st->counts + 3 * nq + 2;
    int32_t* d_pcnt = st->counts + pair_counts_at(nq);
    const int32_t* h_pcnt = st->h_counts + pair_counts_at(nq);
    const int64_t pair_sub = total / pvs::kSub;
    HIP_TRY(hipMemsetAsync(st->counts, 0, all_counts(nq) * sizeof(int32_t), s));
    pvs::ScanOut mo;
    mo.pairs = st->pairs;
    mo.pair_sub = pair_sub;
    mo.pair_cnt = d_pcnt;
    mo.q_evals = st->counts + evals_counts_at(nq);
    mo.q_ld = nq;
    EAHR_TRY(mark(2));
    scan(false, mo, nq);
    EAHR_TRY(mark(3));
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipMemcpyAsync(st->h_counts + pair_counts_at(nq), d_pcnt,
                           static_cast<size_t>(pvs::kSub) * pvs::kCntStride * sizeof(int32_t),
                           hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(st->h_counts + evals_counts_at(nq), mo.q_evals,
                           static_cast<size_t>(pvs::kSub) * nq * sizeof(int32_t), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    tp[2] = clk::now();
    int64_t kept = 0, fullest = 0;   // records kept; the fullest sub-region's count
    for (int i = 0; i < pvs::kSub; ++i) {
        const int64_t c = h_pcnt[i * pvs::kCntStride];
        kept += std::min(c, pair_sub);
        fullest = std::max(fullest, c);
    }
    const bool pool_over = fullest > pair_sub;   // records were dropped
    st->stats.scans += 1;
    st->stats.sample_scans += 1;
    st->stats.rows_scanned += nblocks * 64;
    st->stats.bytes_scanned += st->n_rows * (static_cast<int64_t>(ix->d) + 12) + nblocks * 8;
    if (pool_over) {
        // records were dropped: nothing of this scan is used, so nothing is
        // rescored, and every query scans again with room for all of its
        // candidates
        const double grow = static_cast<double>(fullest) / static_cast<double>(pair_sub);
        std::vector<int32_t> again;
        for (int32_t i = 0; i < nq; ++i) {
            auto& Q = st->q[todo[i]];
            const int64_t cap = st->h_scanq[i].cand_cap;
            Q.cap_hint = std::max(Q.cap_hint, static_cast<int64_t>(std::ceil(cap * grow * 1.25)) + 16);
            st->stats.overflows += 1;
            again.push_back(todo[i]);
        }
        if (prof) {
            float t[2];
            HIP_TRY(hipEventElapsedTime(&t[0], st->ev[0], st->ev[1]));
            HIP_TRY(hipEventElapsedTime(&t[1], st->ev[2], st->ev[3]));
            std::lock_guard<std::mutex> lk(g_prof_mu);
            g_prof.sample_ms += t[0];
            g_prof.scan_ms += t[1];
        }
        again.insert(again.end(), later.begin(), later.end());
        todo.swap(again);
        return EAHR_OK;
    }
    {
        const int32_t* ev = st->h_counts + evals_counts_at(nq);
        for (int c = 0; c < pvs::kSub; ++c)
            for (int32_t i = 0; i < nq; ++i) st->q[todo[i]].evals += ev[c * nq + i];
    }

    // 3. rescore, order and pack the certified ranks
    const int64_t chunks = pvs::rescore_chunks(h_pcnt, pair_sub);
    pvs::launch_rescore(v, st->qrows, st->scanq, nq, d_pcnt, st->pairs, pair_sub, d_cbase, chunks,
                        ix->gamma, st->keys, d_cert, d_fail, d_reads, st->test_fail_qi, s);
    EAHR_TRY(mark(4));
    // only the certified keys are ordered; a query whose key region overflowed
    // (it is scanned again) keeps the region's worth
    HIP_TRY(hipMemcpyAsync(st->h_counts, d_cert, 2 * static_cast<size_t>(nq) * sizeof(int32_t),
                           hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    tp[3] = clk::now();
    const std::vector<int32_t> cert_all(st->h_counts, st->h_counts + nq);
    int64_t max_cert = 0;
    bool clamped = false;
    for (int32_t i = 0; i < nq; ++i) {
        const int64_t region = pvs::kSub * st->h_scanq[i].cand_cap;
        if (st->h_counts[i] > region) {
            st->h_counts[i] = static_cast<int32_t>(region);
            clamped = true;
        }
        max_cert = std::max<int64_t>(max_cert, st->h_counts[i]);
    }
    if (clamped)
        HIP_TRY(hipMemcpyAsync(d_cert, st->h_counts, nq * sizeof(int32_t), hipMemcpyHostToDevice, s));
    // the packed layout: query i's keys at h_offs[i] (the pack kernel's
    // exclusive prefix of the same counts)
    const int32_t* h_cert = st->h_counts;
    const int32_t* h_fail = st->h_counts + nq;
    std::vector<int64_t> h_offs(static_cast<size_t>(nq) + 1, 0);
    for (int32_t i = 0; i < nq; ++i) h_offs[i + 1] = h_offs[i] + h_cert[i];
    const int64_t n_packed = h_offs[nq];
    EAHR_TRY(ensure_host_packed(st, n_packed));
    EAHR_TRY(mark(6));
    uint64_t* sorted = pvs::launch_segmented_sort(st->keys, st->keys_tmp, d_cert, st->scanq, nq, max_cert, s);
    pvs::launch_pack(sorted, d_cert, st->scanq, nq, max_cert, d_offs, st->packed, s);
    EAHR_TRY(mark(5));
    HIP_TRY(hipGetLastError());
    if (prof)
        HIP_TRY(hipMemcpyAsync(st->h_counts + reads_counts_at(nq), d_reads,
                               static_cast<size_t>(pvs::kSub) * pvs::kCntStride * sizeof(int32_t),
                               hipMemcpyDeviceToHost, s));
    // The keys come back into the pinned copy; they stay there (pending)
    // until the next scan round, which appends them to the caches, while the
    // ranks they hold are emitted straight from the copy.
    if (n_packed > 0)
        HIP_TRY(hipMemcpyAsync(st->h_packed, st->packed, static_cast<size_t>(n_packed) * sizeof(uint64_t),
                               hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    tp[4] = clk::now();
    int64_t row_reads = 0;
    if (prof)
        for (int i = 0; i < pvs::kSub; ++i) row_reads += st->h_counts[reads_counts_at(nq) + i * pvs::kCntStride];
    std::vector<uint8_t> usable(nq, 0);
    for (int32_t i = 0; i < nq; ++i) {
        usable[i] = !h_fail[i] && cert_all[i] == h_cert[i];
        if (!usable[i] || h_cert[i] == 0) continue;
        auto& Q = st->q[todo[i]];
        Q.pend_off = h_offs[i];
        Q.pend_n = h_cert[i];
    }
    if (prof) {
        float t[4];
        HIP_TRY(hipEventElapsedTime(&t[0], st->ev[0], st->ev[1]));
        HIP_TRY(hipEventElapsedTime(&t[1], st->ev[2], st->ev[3]));
        HIP_TRY(hipEventElapsedTime(&t[2], st->ev[3], st->ev[4]));
        HIP_TRY(hipEventElapsedTime(&t[3], st->ev[6], st->ev[5]));
        std::lock_guard<std::mutex> lk(g_prof_mu);
        g_prof.sample_ms += t[0];
        g_prof.scan_ms += t[1];
        const int64_t per = mfma ? pvs::kMaxMfmaQueries : pvs::kMaxGemvQueries;
        const int64_t launches = (nq + per - 1) / per;
        g_prof.scan_launches += launches;
        if (mfma) g_prof.mfma_launches += launches;
        const int64_t pass_bytes = st->n_rows * (static_cast<int64_t>(ix->d) + 12) + nblocks * 8;
        g_prof.scan_bytes += launches * pass_bytes;
        // kernel variant of the first launch (the only one when nq fits one pass)
        const int first_q = static_cast<int>(std::min<int64_t>(nq, per));
        int v = mfma ? 8 + (pvs::mfma_tiles_for(first_q) == 1 ? 0 : pvs::mfma_tiles_for(first_q) == 2 ? 1
                            : pvs::mfma_tiles_for(first_q) == 4 ? 2 : 3)
                     : first_q - 1;
        g_prof.variant_ms[v] += t[1];
        g_prof.variant_launches[v] += launches;
        g_prof.variant_bytes[v] += launches * pass_bytes;
        g_prof.rescore_ms += t[2];
        g_prof.rescore_rows += kept;
        g_prof.rescore_row_reads += row_reads;
        for (int32_t i = 0; i < nq; ++i) g_prof.rescore_certified += h_cert[i];
        g_prof.sort_ms += t[3];
        g_prof.scan_rounds += 1;
    }
    if (trace) {
        auto ms = [&](int a, int b) { return std::chrono::duration<double, std::milli>(tp[b] - tp[a]).count(); };
        int64_t certified = 0;
        for (int32_t i = 0; i < nq; ++i) certified += h_cert[i];
        std::fprintf(stderr,
                     "pvs scan_round queries=%d path=%s stride=%lld pool=%lld kept=%lld certified=%lld "
                     "sample_ms=%.2f scan_ms=%.2f rescore_ms=%.2f order_copy_ms=%.2f\n",
                     nq, mfma ? "mfma" : "gemv", static_cast<long long>(stride),
                     static_cast<long long>(total), static_cast<long long>(kept),
                     static_cast<long long>(certified), ms(0, 1), ms(1, 2), ms(2, 3), ms(3, 4));
    }
    st->stats.candidates += kept;
    std::vector<int32_t> keep;
    for (int32_t i = 0; i < nq; ++i) {
        const int32_t b = todo[i];
        auto& Q = st->q[b];
        if (h_fail[i]) {
            Q.failed = true;
            continue;
        }
        if (cert_all[i] != h_cert[i]) {   // its key region overflowed: again with room for all
            const int64_t per = (cert_all[i] + pvs::kSub - 1) / pvs::kSub;
            Q.cap_hint = per + per / 4 + 16;
            st->stats.overflows += 1;
            keep.push_back(b);
            continue;
        }
        Q.cap_hint = 0;
        const int64_t c = h_cert[i];
        st->stats.certified += c;
        if (c > 0) {
            const uint64_t last = st->h_packed[h_offs[i] + c - 1];
            Q.has_cert = true;
            Q.s_cert = key_score(last);
            Q.id_cert = key_id(last);
        }
        const int64_t avail = certified_count(Q) - Q.emitted;
        if (certified_count(Q) >= st->n_vis) {
            Q.cert_exhausted = true;
            Q.retries = 0;
        } else if (avail >= m) {
            Q.retries = 0;
        } else {
            Q.retries += 1;
            st->stats.rescans += 1;
            keep.push_back(b);
        }
    }
    keep.insert(keep.end(), later.begin(), later.end());
    todo.swap(keep);
    return EAHR_OK;
}

// pvs_next; scores may be null (then only ids are written).
static int next_ranks(pvs_state* st, int32_t m, const uint8_t* active, int64_t* ids, float* scores,
                      int32_t* count, int32_t* status) {
    const int32_t B = st->B;
    std::vector<int32_t> todo;
    for (int32_t b = 0; b < B; ++b) {
        if (active && !active[b]) continue;
        auto& Q = st->q[b];
        if (Q.retired) EAHR_FAIL(EAHR_E_INVALID, "pvs_next: query %d was retired", b);
        if (Q.failed || Q.cert_exhausted) continue;
        const int64_t avail = certified_count(Q) - Q.emitted;
        if (avail < m) todo.push_back(b);
    }
    for (int guard = 0; !todo.empty(); ++guard) {
        if (guard > 200) EAHR_FAIL(EAHR_E_HIP, "pvs_next: scan loop did not converge");
        EAHR_TRY(scan_round(st, todo, m));
    }
    // decode the emitted ranks of every query, in pieces over the host threads
    std::vector<int64_t> took(B, 0);
    for (int32_t b = 0; b < B; ++b) {
        if (active && !active[b]) continue;
        const auto& Q = st->q[b];
        if (Q.failed) {
            count[b] = 0;
            status[b] = EAHR_LIST_FAILED;
            continue;
        }
        took[b] = std::min<int64_t>(m, certified_count(Q) - Q.emitted);
    }
    eahr::parallel_pieces(took, int64_t(1) << 17, eahr::host_threads(), [&](int64_t b, int64_t lo, int64_t hi) {
        // ranks emitted + j: from the cache, then from the pinned copy
        const auto& Q = st->q[b];
        const int64_t in_cache = static_cast<int64_t>(Q.cache.size()) - Q.emitted;
        int64_t* oi = ids + b * static_cast<int64_t>(m);
        float* os = scores ? scores + b * static_cast<int64_t>(m) : nullptr;
        auto decode = [&](const uint64_t* kp, int64_t j0, int64_t j1) {   // kp[0] is rank emitted + j0
            if (scores)
                for (int64_t j = j0; j < j1; ++j) {
                    oi[j] = key_id(kp[j - j0]);
                    os[j] = key_score(kp[j - j0]);
                }
            else
                for (int64_t j = j0; j < j1; ++j) oi[j] = key_id(kp[j - j0]);
        };
        const int64_t mid = std::min(std::max(in_cache, lo), hi);
        if (mid > lo) decode(Q.cache.data() + Q.emitted + lo, lo, mid);
        if (hi > mid) decode(st->h_packed + Q.pend_off + (mid - in_cache), mid, hi);
    });
    for (int32_t b = 0; b < B; ++b) {
        if ((active && !active[b]) || st->q[b].failed) continue;
        auto& Q = st->q[b];
        Q.emitted += took[b];
        count[b] = static_cast<int32_t>(took[b]);
        status[b] = (Q.emitted >= st->n_vis) ? EAHR_LIST_EXHAUSTED : EAHR_LIST_OPEN;
        st->stats.emitted += took[b];
    }
    return EAHR_OK;
}


extern "C" int pvs_next(pvs_state* st, int32_t m, const uint8_t* active, int64_t* ids,
                        float* scores, int32_t* count, int32_t* status) {
    if (!st || m < 0 || (m > 0 && (!ids || !scores)) || !count || !status)
        EAHR_FAIL(EAHR_E_INVALID, "pvs_next: bad arguments");
    return next_ranks(st, m, active, ids, scores, count, status);
}

int pvs_next_ids(pvs_state* st, int32_t m, const uint8_t* active, int64_t* ids, int32_t* count,
                 int32_t* status) {
    if (!st || m < 0 || (m > 0 && !ids) || !count || !status)
        EAHR_FAIL(EAHR_E_INVALID, "pvs_next: bad arguments");
    return next_ranks(st, m, active, ids, nullptr, count, status);
}
int pvs_fill(pvs_state* st, int64_t depth, const uint8_t* active, int64_t* added) {
    if (!st || depth < 0) EAHR_FAIL(EAHR_E_INVALID, "pvs_fill: bad arguments");
    std::vector<int32_t> todo;
    int64_t m = 0, before = 0;
    for (int32_t b = 0; b < st->B; ++b) {
        if (active && !active[b]) continue;
        const auto& Q = st->q[b];
        before += certified_count(Q);
        if (Q.failed || Q.cert_exhausted || Q.retired) continue;
        if (certified_count(Q) >= depth) continue;
        todo.push_back(b);
        m = std::max<int64_t>(m, depth - Q.emitted);
    }
    m = std::min<int64_t>(m, int64_t(1) << 30);
    for (int guard = 0; !todo.empty(); ++guard) {
        if (guard > 200) EAHR_FAIL(EAHR_E_HIP, "pvs_fill: scan loop did not converge");
        EAHR_TRY(scan_round(st, todo, static_cast<int32_t>(m)));
    }
    if (added) {
        int64_t after = 0;
        for (int32_t b = 0; b < st->B; ++b)
            if (!active || active[b]) after += certified_count(st->q[b]);
        *added = after - before;
    }
    return EAHR_OK;
}

int pvs_fill_exact(pvs_state* st, int64_t depth, const uint8_t* active, int64_t* added) {
    if (!st) EAHR_FAIL(EAHR_E_INVALID, "pvs_fill: bad arguments");
    st->spec_off = true;
    const int rc = pvs_fill(st, depth, active, added);
    st->spec_off = false;
    return rc;
}

bool pvs_covered(const pvs_state* st, int32_t m, const uint8_t* active) {
    if (!st) return false;
    for (int32_t b = 0; b < st->B; ++b) {
        if (active && !active[b]) continue;
        const auto& Q = st->q[b];
        if (Q.failed || Q.cert_exhausted || Q.retired) continue;
        if (certified_count(Q) - Q.emitted < m) return false;
    }
    return true;
}

void pvs_retire(pvs_state* st, int32_t b) {
    if (!st || b < 0 || b >= st->B) return;
    auto& Q = st->q[b];
    Q.retired = true;
    Q.pend_n = 0;
}

bool pvs_query_failed(const pvs_state* st, int32_t b) {
    return st && b >= 0 && b < st->B && st->q[b].failed;
}

int64_t pvs_query_evals(const pvs_state* st, int32_t b) {
    return (st && b >= 0 && b < st->B) ? st->q[b].evals : 0;
}

extern "C" int pvs_stats(const pvs_state* st, pvs_counters* out) {
    if (!st || !out) EAHR_FAIL(EAHR_E_INVALID, "pvs_stats: bad arguments");
    *out = st->stats;
    return EAHR_OK;
}

extern "C" int pvs_profile_enable(int32_t on) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof = pvs_profile{};
    g_prof_on.store(on ? 1 : 0);
    return EAHR_OK;
}

extern "C" int pvs_profile_read(pvs_profile* out) {
    if (!out) EAHR_FAIL(EAHR_E_INVALID, "pvs_profile_read: NULL");
    std::lock_guard<std::mutex> lk(g_prof_mu);
    *out = g_prof;
    return EAHR_OK;
}

bool pvs_profile_on() { return g_prof_on.load(std::memory_order_relaxed) != 0; }

void pvs_profile_add_host(double dense_ms, double sparse_ms, double fuse_ms) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof.host_dense_ms += dense_ms;
    g_prof.host_sparse_ms += sparse_ms;
    g_prof.host_fuse_ms += fuse_ms;
}
