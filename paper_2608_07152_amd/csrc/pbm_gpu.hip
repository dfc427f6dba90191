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
// each thread walks the query's few terms in order.  With ent, the entry of
// term slot i (global index into qterm) for range r is kept at
// ent[i * n_ranges + r] (-1: none) for the expansions.
__global__ __launch_bounds__(256) void k_bounds(IndexView ix, QueryView q, float* __restrict__ H,
                                                int32_t* __restrict__ post, int64_t* __restrict__ ent) {
    const int32_t b = blockIdx.y;
    const int64_t r = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (r >= ix.n_ranges) return;
    float h = 0.0f;
    int64_t n = 0;
    for (int32_t i = q.qptr[b]; i < q.qptr[b + 1]; ++i) {
        const int32_t t = q.qterm[i];
        const int64_t e = find_entry(ix, t, r);
        if (ent) ent[static_cast<int64_t>(i) * ix.n_ranges + r] = e;
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

// One workgroup per task.  A bitmap in LDS marks the documents of the range
// that a posting of the query reached (bit i: document start + i); acc[i]
// holds the running score of a marked document.  Terms are applied one after
// another with a barrier between them; inside a term the documents are
// distinct, so its postings go in parallel (the bitmap words are set with
// LDS atomics, and a document's first posting starts its sum at 0 + c).
// Only the bitmap is cleared, so a task costs O(its postings + range / 32).
// Afterwards each marked document is counted as scored, checked against the
// bound, and appended as a key when its score is positive: one atomic per
// wavefront, positions from a wavefront prefix sum of the per-lane counts.
__device__ __forceinline__ int wave_excl_scan(int v, int lane, int& total) {
    int x = v;
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    total = __shfl(x, 63, 64);
    return x - v;
}

__global__ __launch_bounds__(256) void k_expand(IndexView ix, QueryView q, const Task* __restrict__ tasks,
                                                const int64_t* __restrict__ ent, const int64_t* __restrict__ key_off,
                                                int32_t* __restrict__ key_cnt, int32_t* __restrict__ scored,
                                                int32_t* __restrict__ fail, uint64_t* __restrict__ keys) {
    extern __shared__ uint32_t smem[];
    const Task T = tasks[blockIdx.x];
    const int64_t start = static_cast<int64_t>(T.r) * ix.range_size;
    const int64_t rem = ix.n_docs - start;
    const int32_t len = static_cast<int32_t>(rem < ix.range_size ? rem : ix.range_size);
    const int32_t nwords = (len + 31) >> 5;
    uint32_t* seen = smem;
    float* acc = reinterpret_cast<float*>(smem + ((ix.range_size + 31) >> 5));
    const int tid = threadIdx.x;
    for (int i = tid; i < nwords; i += 256) seen[i] = 0u;
    __syncthreads();
    for (int32_t i = q.qptr[T.b]; i < q.qptr[T.b + 1]; ++i) {
        const int32_t t = q.qterm[i];
        const int64_t e = ent ? ent[static_cast<int64_t>(i) * ix.n_ranges + T.r] : find_entry(ix, t, T.r);
        if (e < 0) continue;   // the same value in every thread
        const float w = q.qw[i];
        const int64_t p1 = entry_end(ix, t, e);
        for (int64_t p = ix.bm_off[e] + tid; p < p1; p += 256) {
            const int32_t off = static_cast<int32_t>(ix.docs[p] - start);
            const float c = w * ix.imp[p];
            const uint32_t bit = 1u << (off & 31);
            const uint32_t old = atomicOr(&seen[off >> 5], bit);
            acc[off] = (old & bit) ? acc[off] + c : 0.0f + c;
        }
        __syncthreads();
    }
    const int lane = tid & 63;
    for (int w0 = 0; w0 < nwords; w0 += 256) {   // the same trip count in every thread
        const int wi = w0 + tid;
        const uint32_t bits = wi < nwords ? seen[wi] : 0u;
        int npos = 0, nscored = 0;
        bool bad = false;
        for (uint32_t m = bits; m; m &= m - 1) {
            const float sc = acc[(wi << 5) + (__ffs(m) - 1)];
            ++nscored;
            bad |= sc > T.H;
            npos += sc > 0.0f;
        }
        int tot = 0;
        const int at = wave_excl_scan(npos, lane, tot);
        int base = 0;
        if (tot) {
            if (lane == 0) base = atomicAdd(&key_cnt[T.b], tot);
            base = __shfl(base, 0, 64);
            int k = base + at;
            for (uint32_t m = bits; m; m &= m - 1) {
                const int i = (wi << 5) + (__ffs(m) - 1);
                const float sc = acc[i];
                if (sc > 0.0f)
                    keys[key_off[T.b] + k++] = (static_cast<uint64_t>(~ord32(sc)) << 32) | static_cast<uint64_t>(start + i);
            }
        }
        for (int off = 32; off > 0; off >>= 1) nscored += __shfl_xor(nscored, off, 64);
        if (__ballot(bad) && lane == 0) fail[T.b] = 1;
        if (lane == 0 && nscored) atomicAdd(&scored[T.b], nscored);
    }
}

void launch_bounds(const IndexView& ix, const QueryView& q, float* H, int32_t* post, int64_t* ent,
                   hipStream_t s) {
    if (q.B <= 0 || ix.n_ranges <= 0) return;
    const dim3 grid(static_cast<uint32_t>((ix.n_ranges + 255) / 256), static_cast<uint32_t>(q.B));
    hipLaunchKernelGGL(k_bounds, grid, dim3(256), 0, s, ix, q, H, post, ent);
}

int launch_expand(const IndexView& ix, const QueryView& q, const Task* tasks, int32_t ntasks,
                  const int64_t* ent, const int64_t* key_off, int32_t* key_cnt, int32_t* scored,
                  int32_t* fail, uint64_t* keys, hipStream_t s) {
    if (ntasks <= 0) return 0;
    const size_t lds = static_cast<size_t>((ix.range_size + 31) / 32) * sizeof(uint32_t) +
                       static_cast<size_t>(ix.range_size) * sizeof(float);
    if (lds > 65536) {   // ranges of more than 16,256 ids need the larger LDS allowance
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_expand),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (e != hipSuccess) return -1;
    }
    hipLaunchKernelGGL(k_expand, dim3(static_cast<uint32_t>(ntasks)), dim3(256), lds, s, ix, q, tasks, ent,
                       key_off, key_cnt, scored, fail, keys);
    return 0;
}

}  // namespace pbmg
