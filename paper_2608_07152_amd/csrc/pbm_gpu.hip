// Posting Block-Max on the GPU (Sec. 2.3.2, App. A.2): range bounds H(R) of
// a batch of queries, and exact scores of the documents of expanded ranges.
//
// Both follow the host definitions operation for operation: a bound or a
// score starts at 0 and adds q_t * v (one float32 rounding for the product,
// one for the sum) for the query's terms in ascending term order, so the
// values are bit-identical to the host PBM's.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "pbm_kernels.h"

namespace pbmg {

// First block-max entry of term t with range >= r, and whether it is r.
__device__ __forceinline__ int64_t find_entry(const IndexView& ix, int32_t t, int64_t r) {
    int64_t lo = ix.bm_ptr[t], hi = ix.bm_ptr[t + 1];
    const int64_t end = hi;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (ix.bm_range[mid] < r) lo = mid + 1;
        else hi = mid;
    }
    return (lo < end && ix.bm_range[lo] == r) ? lo : -1;
}

// End of the postings of entry e of term t (the next entry's start, or the
// term's end).
__device__ __forceinline__ int64_t entry_end(const IndexView& ix, int32_t t, int64_t e) {
    return (e + 1 < ix.bm_ptr[t + 1]) ? ix.bm_off[e + 1] : ix.term_ptr[t + 1];
}

// One thread per (query, range): the ranges of a query are independent, and
// each thread walks the query's few terms in order.
__global__ __launch_bounds__(256) void k_bounds(IndexView ix, QueryView q, float* __restrict__ H,
                                                int32_t* __restrict__ post) {
    const int32_t b = blockIdx.y;
    const int64_t r = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (r >= ix.n_ranges) return;
    float h = 0.0f;
    int64_t n = 0;
    for (int32_t i = q.qptr[b]; i < q.qptr[b + 1]; ++i) {
        const int32_t t = q.qterm[i];
        const int64_t e = find_entry(ix, t, r);
        if (e < 0) continue;
        const float c = q.qw[i] * ix.bm_max[e];
        h = h + c;
        n += entry_end(ix, t, e) - ix.bm_off[e];
    }
    H[b * ix.n_ranges + r] = h;
    post[b * ix.n_ranges + r] = static_cast<int32_t>(n);
}

__device__ __forceinline__ uint32_t ord32(float f) {
    const uint32_t b = __float_as_uint(f);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// One workgroup per task.  acc[i] holds the running score of document
// start + i, or -1 while no posting of it was seen (every partial sum is
// >= +0).  Terms are applied one after another with a barrier between them;
// inside a term the documents are distinct, so its postings go in parallel.
__global__ __launch_bounds__(256) void k_expand(IndexView ix, QueryView q, const Task* __restrict__ tasks,
                                                const int64_t* __restrict__ key_off,
                                                int32_t* __restrict__ key_cnt, int32_t* __restrict__ scored,
                                                int32_t* __restrict__ fail, uint64_t* __restrict__ keys) {
    extern __shared__ float acc[];
    const Task T = tasks[blockIdx.x];
    const int64_t start = static_cast<int64_t>(T.r) * ix.range_size;
    const int64_t rem = ix.n_docs - start;
    const int32_t len = static_cast<int32_t>(rem < ix.range_size ? rem : ix.range_size);
    const int tid = threadIdx.x;
    for (int i = tid; i < len; i += 256) acc[i] = -1.0f;
    __syncthreads();
    for (int32_t i = q.qptr[T.b]; i < q.qptr[T.b + 1]; ++i) {
        const int32_t t = q.qterm[i];
        const int64_t e = find_entry(ix, t, T.r);   // the same value in every thread
        if (e < 0) continue;
        const float w = q.qw[i];
        const int64_t p1 = entry_end(ix, t, e);
        for (int64_t p = ix.bm_off[e] + tid; p < p1; p += 256) {
            const int32_t off = static_cast<int32_t>(ix.docs[p] - start);
            const float c = w * ix.imp[p];
            const float v = acc[off];
            acc[off] = (v < 0.0f) ? 0.0f + c : v + c;
        }
        __syncthreads();
    }
    const int lane = tid & 63;
    int my_scored = 0;
    bool my_fail = false;
    for (int base = 0; base < len; base += 256) {
        const int i = base + tid;
        const float s = (i < len) ? acc[i] : -1.0f;
        my_scored += s >= 0.0f;
        my_fail |= s > T.H;
        const bool emit = s > 0.0f;
        // one append per wavefront: a ballot, the lane's rank among the
        // emitting lanes, one atomic by the first of them
        const uint64_t m = __ballot(emit);
        if (m) {
            const int first = __ffsll(static_cast<unsigned long long>(m)) - 1;
            int at = 0;
            if (lane == first) at = atomicAdd(&key_cnt[T.b], __popcll(m));
            at = __shfl(at, first, 64);
            if (emit) {
                const int rank = __popcll(m & ((1ull << lane) - 1ull));
                keys[key_off[T.b] + at + rank] =
                    (static_cast<uint64_t>(~ord32(s)) << 32) | static_cast<uint64_t>(start + i);
            }
        }
    }
    // per wavefront: one add of the scored count, one fail flag
    for (int off = 32; off > 0; off >>= 1) my_scored += __shfl_xor(my_scored, off, 64);
    if (__ballot(my_fail) && lane == 0) fail[T.b] = 1;
    if (lane == 0 && my_scored) atomicAdd(&scored[T.b], my_scored);
}

void launch_bounds(const IndexView& ix, const QueryView& q, float* H, int32_t* post, hipStream_t s) {
    if (q.B <= 0 || ix.n_ranges <= 0) return;
    const dim3 grid(static_cast<uint32_t>((ix.n_ranges + 255) / 256), static_cast<uint32_t>(q.B));
    hipLaunchKernelGGL(k_bounds, grid, dim3(256), 0, s, ix, q, H, post);
}

void launch_expand(const IndexView& ix, const QueryView& q, const Task* tasks, int32_t ntasks,
                   const int64_t* key_off, int32_t* key_cnt, int32_t* scored, int32_t* fail,
                   uint64_t* keys, hipStream_t s) {
    if (ntasks <= 0) return;
    const size_t lds = static_cast<size_t>(ix.range_size) * sizeof(float);
    hipLaunchKernelGGL(k_expand, dim3(static_cast<uint32_t>(ntasks)), dim3(256), lds, s, ix, q, tasks,
                       key_off, key_cnt, scored, fail, keys);
}

}  // namespace pbmg
