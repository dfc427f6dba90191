// pvs_scores_noalloc: the authoritative float32 scores of pvs_scores for
// callers that cannot allocate memory (code under stream capture, tight
// serving loops).  pvs_scores stages the row ids and the scores in device
// buffers it allocates per call; this variant stages them in one
// fixed-size array of device memory per GPU, `scratch`, which the library
// holds until the process ends.  Every call on a GPU shares that GPU's
// array, so calls that overlap on one GPU (from several host threads) race;
// the row ids are copied in and every score is written before it is read,
// so nothing in the array needs to start at zero.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "common.h"
#include "eahr.h"
#include "pvs_internal.h"
#include "pvs_kernels.h"

namespace {

constexpr int64_t kNoAllocRows = EAHR_NOALLOC_MAX_ROWS;
// row ids (int64) of one call, then their scores (float32)
constexpr size_t kIdsBytes = static_cast<size_t>(kNoAllocRows) * sizeof(int64_t);
constexpr size_t kScratchBytes = kIdsBytes + static_cast<size_t>(kNoAllocRows) * sizeof(float);

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on each GPU, looked up once per device with that
// device current (the name itself is a host-side stand-in, not an address).
constexpr int kMaxDevices = 64;
std::mutex g_mu;
unsigned char* g_scratch[kMaxDevices] = {};

int scratch_on(int dev, unsigned char** out) {
    if (dev < 0 || dev >= kMaxDevices) EAHR_FAIL(EAHR_E_INVALID, "pvs_scores_noalloc: device %d", dev);
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        g_scratch[dev] = static_cast<unsigned char*>(p);
    }
    *out = g_scratch[dev];
    return EAHR_OK;
}

}  // namespace

extern "C" int pvs_scores_noalloc(const pvs_state* st, int32_t b, const int64_t* rows, int64_t n,
                                  float* scores) {
    if (!st || b < 0 || b >= st->B || n < 0 || (n > 0 && (!rows || !scores)))
        EAHR_FAIL(EAHR_E_INVALID, "pvs_scores_noalloc: bad arguments");
    if (n > kNoAllocRows)
        EAHR_FAIL(EAHR_E_RANGE, "pvs_scores_noalloc: %lld rows exceed the limit of %lld per call",
                  static_cast<long long>(n), static_cast<long long>(kNoAllocRows));
    for (int64_t i = 0; i < n; ++i)
        if (rows[i] < 0 || rows[i] >= st->n_rows)
            EAHR_FAIL(EAHR_E_INVALID, "pvs_scores_noalloc: row out of range");
    if (n == 0) return EAHR_OK;
    const pvs_index* ix = st->ix;
    int cur = 0;
    HIP_TRY(hipGetDevice(&cur));
    if (cur != ix->device) HIP_TRY(hipSetDevice(ix->device));
    unsigned char* base = nullptr;
    int rc = scratch_on(ix->device, &base);
    if (rc == EAHR_OK) {
        auto body = [&]() -> int {
            hipStream_t s = ix->stream;
            int64_t* d_rows = reinterpret_cast<int64_t*>(base);
            float* d_out = reinterpret_cast<float*>(base + kIdsBytes);
            HIP_TRY(hipMemcpyAsync(d_rows, rows, static_cast<size_t>(n) * sizeof(int64_t),
                                   hipMemcpyHostToDevice, s));
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
            pvs::launch_scores(v, st->qrows, b, d_rows, n, d_out, s);
            HIP_TRY(hipGetLastError());
            HIP_TRY(hipMemcpyAsync(scores, d_out, static_cast<size_t>(n) * sizeof(float),
                                   hipMemcpyDeviceToHost, s));
            HIP_TRY(hipStreamSynchronize(s));
            return EAHR_OK;
        };
        rc = body();
    }
    if (cur != ix->device) (void)hipSetDevice(cur);
    return rc;
}
