// Candidate rescoring, ordering and packing of the PVS dense channel.
//
// Every candidate pair gets its authoritative float32 score (the fixed
// order of group_dot) and is checked against its interval (App. A.1: a score
// outside it fails the request), recomputed from the integer dot product the
// scan recorded with the scan's own arithmetic, so identical to it.  A scan
// with threshold tau certifies exactly the candidates with s32 >= tau whose
// key follows the last certified key; their keys (~mono(s32) << 32 | row) are
// appended to the query's key region, so ascending keys are (score
// descending, id ascending).  Keys are unique inside a query; the segmented
// sort orders each query's certified keys.
#include <algorithm>
#include <atomic>

#include "pvs_device.h"

namespace pvs {

// Records of a scan round are cut into chunks of kRescoreChunk per pool
// sub-region; cbase[s] is the first chunk of sub-region s (exclusive prefix).
__global__ __launch_bounds__(64) void k_chunk_base(const int32_t* __restrict__ pair_cnt,
                                                   int64_t pair_sub, int32_t* __restrict__ cbase) {
    if (threadIdx.x == 0) {
        int32_t acc = 0;
        for (int s = 0; s < kSub; ++s) {
            cbase[s] = acc;
            const int64_t n = pair_cnt[s * kCntStride] < pair_sub ? pair_cnt[s * kCntStride] : pair_sub;
            acc += static_cast<int32_t>((n + kRescoreChunk - 1) / kRescoreChunk);
        }
        cbase[kSub] = acc;
    }
}

// The records of quarter `wave` of chunk x (one wavefront, 64 records).
// Lane j first prepares record j (its interval from the recorded dot with
// the scan's arithmetic, its query's tau and last certified key); each
// 16-lane group g then scores records 16 g .. 16 g + 15 one after another
// (the group's lanes hold the record's row and query row in the fixed order
// of the authoritative score, so four records are scored at once), and the
// record's own lane judges its score.  Records of one row are adjacent, so a
// group loads the row once for them; likewise the query row, which comes
// from LDS (slot = the record's query in the scan) when LDSQ.  At the end
// the keys of each query are appended to its region with one atomic.
// J: chunks per lane (0: rows scored in segments); FULL: df / 4 == 16 J.
template <int J, bool FULL, bool LDSQ>
__device__ __forceinline__ void rescore_quarter(
    int x, int wave, const float4* __restrict__ rows, int32_t df4, const float4* __restrict__ qsrc,
    const ScanQ* __restrict__ sq, const int32_t* __restrict__ cbase,
    const int32_t* __restrict__ pair_cnt, const uint4* __restrict__ pairs, int64_t pair_sub,
    const float* __restrict__ scale, const float* __restrict__ vnorm,
    const float* __restrict__ enorm, float gamma, uint64_t* __restrict__ keys,
    int32_t* __restrict__ cert_cnt, int32_t* __restrict__ fail, int32_t* __restrict__ row_reads,
    int32_t fail_qi) {
    constexpr int PER_WAVE = kRescoreChunk / 4;
    static_assert(PER_WAVE == 64, "one record per lane");
    const int lane = threadIdx.x & 63;
    // the sub-region of this chunk: the last s with cbase[s] <= chunk
    int slo = 0, shi = kSub;
    while (shi - slo > 1) {
        const int mid = (slo + shi) >> 1;
        if (cbase[mid] <= x) slo = mid;
        else shi = mid;
    }
    const int s = slo;
    const int64_t cnt = pair_cnt[s * kCntStride];
    const int64_t n_s = cnt < pair_sub ? cnt : pair_sub;
    const int64_t i0 = static_cast<int64_t>(x - cbase[s]) * kRescoreChunk + wave * PER_WAVE;
    const int n = static_cast<int>(n_s - i0 < PER_WAVE ? n_s - i0 : PER_WAVE);
    if (n <= 0) return;
    // this lane's record
    const bool mine = lane < n;
    const uint4 rec = mine ? pairs[s * pair_sub + i0 + lane] : make_uint4(0u, 0u, 0u, 0u);
    const int32_t my_row = static_cast<int32_t>(rec.x);
    const int32_t my_b = static_cast<int32_t>(rec.y);
    const ScanQ& MQ = sq[my_b];
    const int32_t my_qi = MQ.qi;
    float my_lo, my_hi;
    pair_interval(MQ, scale[my_row], vnorm[my_row], enorm[my_row], static_cast<int32_t>(rec.z), gamma,
                  my_lo, my_hi);
    if (my_qi == fail_qi) {
        // failure injection (tests only): the judged interval of this query
        // shrinks to the ulps around c, so its scores fall outside it
        const float c = (MQ.sq * scale[my_row]) * static_cast<float>(static_cast<int32_t>(rec.z));
        my_lo = next_down(c);
        my_hi = next_up(c);
    }
    const float my_tau = MQ.tau, my_scert = MQ.s_cert;
    const int32_t my_idcert = MQ.id_cert;
    const bool my_hascert = MQ.has_cert != 0;
    uint64_t mykey = 0;
    bool cert = false, bad = false;
    const int g = lane >> 4, j = lane & 15;
    float4 v[J > 0 ? J : 1], q[J > 0 ? J : 1];
    int32_t prow = -1, pqi = -1;
    int reads = 0;   // row loads of this lane's group
    static_for(
        [&](auto I_) {
            constexpr int i = decltype(I_)::value;
            // the group's record i, held by lane 16 g + i
            const int32_t row = bcast16<i>(my_row);
            const int32_t qi = bcast16<i>(LDSQ ? my_b : my_qi);   // LDSQ: the LDS slot
            if (16 * g + i < n) {   // the same in every lane of the group
                float sc;
                if constexpr (J > 0) {
                    if (row != prow) {
                        load_chunks<J, FULL>(rows + static_cast<int64_t>(row) * df4, j, df4, v);
                        prow = row;
                        ++reads;
                    }
                    if (qi != pqi) {   // from LDS when LDSQ
                        load_chunks<J, FULL>(qsrc + static_cast<int64_t>(qi) * df4, j, df4, q);
                        pqi = qi;
                    }
                    sc = group_dot<J, FULL>(v, q, j, df4);
                } else {
                    sc = group_score_seg(rows + static_cast<int64_t>(row) * df4,
                                         qsrc + static_cast<int64_t>(qi) * df4, j, df4);
                    ++reads;
                }
                if (j == i) {
                    bad = !(my_lo <= sc && sc <= my_hi);
                    const bool dropped = my_hascert && (sc > my_scert || (sc == my_scert && row <= my_idcert));
                    if (!dropped && sc >= my_tau) {
                        mykey = (static_cast<uint64_t>(~mono32(sc)) << 32) | static_cast<uint32_t>(row);
                        cert = true;
                    }
                }
            }
        },
        std::make_integer_sequence<int, 16>{});
    reads = __builtin_amdgcn_readlane(reads, 0) + __builtin_amdgcn_readlane(reads, 16) +
            __builtin_amdgcn_readlane(reads, 32) + __builtin_amdgcn_readlane(reads, 48);
    // one of kSub counters (one address for every wavefront would serialise)
    if (lane == 0) atomicAdd(&row_reads[(blockIdx.x & (kSub - 1)) * kCntStride], reads);
    if (bad) fail[my_b] = 1;
    // group the certified lanes by query (one pass per distinct query, ALU
    // only), then the first lane of each group appends the group with one
    // atomic, all groups in the same instruction
    const int myb = cert ? my_b : -1;
    uint64_t todo = __ballot(cert);
    if (!todo) return;
    int leader = 0, rank = 0, size = 0;
    while (todo) {
        const int l0 = __ffsll(static_cast<unsigned long long>(todo)) - 1;
        const int b0 = __builtin_amdgcn_readlane(myb, l0);
        const uint64_t grp = __ballot(myb == b0);
        if (myb == b0) {
            leader = l0;
            rank = __popcll(grp & ((1ull << lane) - 1ull));
            size = __popcll(grp);
        }
        todo &= ~grp;
    }
    int base = 0;
    if (cert && lane == leader) base = atomicAdd(&cert_cnt[myb], size);
    base = __shfl(base, leader, 64);
    if (!cert) return;
    const int64_t pos = static_cast<int64_t>(base) + rank;
    if (pos < kSub * MQ.cand_cap) keys[MQ.cand_off + pos] = mykey;
}

// One wavefront per quarter of a chunk of kRescoreChunk records.  LDSQ: a
// workgroup of sixteen wavefronts takes four chunks and first copies the
// scan's nq float32 query rows to LDS, and the groups read their query rows
// from there instead of reloading them from L2 per record (the loads that
// bound the kernel when records of one row belong to different queries).
// Workgroups that each loop over many chunks after one copy measured slower
// (on a three-query scan, 9.3 against 3.8 ms).
template <int J, bool FULL, bool LDSQ>
__global__ __launch_bounds__(LDSQ ? 1024 : 256) void k_rescore(
    const float4* __restrict__ rows, int32_t df4, const float4* __restrict__ qrows,
    const ScanQ* __restrict__ sq, int32_t nq, const int32_t* __restrict__ cbase,
    const int32_t* __restrict__ pair_cnt, const uint4* __restrict__ pairs, int64_t pair_sub,
    const float* __restrict__ scale, const float* __restrict__ vnorm,
    const float* __restrict__ enorm, float gamma, uint64_t* __restrict__ keys,
    int32_t* __restrict__ cert_cnt, int32_t* __restrict__ fail, int32_t* __restrict__ row_reads,
    int32_t fail_qi) {
    if constexpr (LDSQ) {
        extern __shared__ float4 s_q[];   // query row b at s_q[b * df4]
        for (int k = threadIdx.x; k < nq * df4; k += blockDim.x) {
            const int b = k / df4;
            s_q[k] = qrows[static_cast<int64_t>(sq[b].qi) * df4 + (k - b * df4)];
        }
        __syncthreads();
        const int x = static_cast<int>(blockIdx.x) * 4 + static_cast<int>(threadIdx.x >> 8);
        if (x < cbase[kSub])
            rescore_quarter<J, FULL, true>(x, (threadIdx.x >> 6) & 3, rows, df4, s_q, sq, cbase, pair_cnt, pairs,
                                           pair_sub, scale, vnorm, enorm, gamma, keys, cert_cnt, fail, row_reads,
                                           fail_qi);
    } else {
        rescore_quarter<J, FULL, false>(blockIdx.x, threadIdx.x >> 6, rows, df4, qrows, sq, cbase, pair_cnt, pairs,
                                        pair_sub, scale, vnorm, enorm, gamma, keys, cert_cnt, fail, row_reads,
                                        fail_qi);
    }
}

// LDS of the query-row variant: at most a gfx950 CU's 160 KiB.
constexpr size_t kRescoreLdsMax = 160 * 1024;

template <int J, bool FULL>
static void rescore_j(const IndexView& ix, const float* qrows, const ScanQ* sq, int32_t nq,
                      const int32_t* cbase, int64_t chunks, const int32_t* pair_cnt,
                      const uint4* pairs, int64_t pair_sub, float gamma, uint64_t* keys,
                      int32_t* cert_cnt, int32_t* fail, int32_t* row_reads, int32_t fail_qi,
                      hipStream_t stream) {
    const int32_t df4 = ix.df / 4;
    const size_t lds = static_cast<size_t>(nq) * df4 * sizeof(float4);
    // one query: its row stays in the groups' registers anyway
    if constexpr (J > 0) {
        static std::atomic<int> ready{0};   // 1: LDS attribute set, -1: refused
        if (nq > 1 && lds <= kRescoreLdsMax && ready.load() == 0) {
            const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_rescore<J, FULL, true>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     static_cast<int>(kRescoreLdsMax));
            ready.store(e == hipSuccess ? 1 : -1);
            if (e != hipSuccess) (void)hipGetLastError();
        }
        if (nq > 1 && lds <= kRescoreLdsMax && ready.load() > 0) {
            const uint32_t groups = static_cast<uint32_t>((chunks + 3) / 4);
            hipLaunchKernelGGL((k_rescore<J, FULL, true>), dim3(groups), dim3(1024), lds, stream,
                               reinterpret_cast<const float4*>(ix.rows), df4,
                               reinterpret_cast<const float4*>(qrows), sq, nq, cbase, pair_cnt, pairs, pair_sub,
                               ix.scale, ix.vnorm, ix.enorm, gamma, keys, cert_cnt, fail, row_reads, fail_qi);
            return;
        }
    }
    hipLaunchKernelGGL((k_rescore<J, FULL, false>), dim3(static_cast<uint32_t>(chunks)), dim3(256), 0, stream,
                       reinterpret_cast<const float4*>(ix.rows), df4, reinterpret_cast<const float4*>(qrows), sq,
                       nq, cbase, pair_cnt, pairs, pair_sub, ix.scale, ix.vnorm, ix.enorm, gamma, keys, cert_cnt,
                       fail, row_reads, fail_qi);
}

int64_t rescore_chunks(const int32_t* pair_cnt, int64_t pair_sub) {
    int64_t c = 0;
    for (int s = 0; s < kSub; ++s) {
        const int64_t n = std::min<int64_t>(pair_cnt[s * kCntStride], pair_sub);
        c += (n + kRescoreChunk - 1) / kRescoreChunk;
    }
    return c;
}

void launch_rescore(const IndexView& ix, const float* qrows, const ScanQ* sq, int32_t nq,
                    const int32_t* pair_cnt, const uint4* pairs, int64_t pair_sub,
                    int32_t* cbase, int64_t chunks, float gamma, uint64_t* keys,
                    int32_t* cert_cnt, int32_t* fail, int32_t* row_reads, int32_t fail_qi,
                    hipStream_t stream) {
    hipLaunchKernelGGL(k_chunk_base, dim3(1), dim3(64), 0, stream, pair_cnt, pair_sub, cbase);
    if (chunks <= 0) return;
    const int J = group_chunks(ix.df);
    const bool full = J > 0 && ix.df / 4 == 16 * J;
#define PVS_RS(N)                                                                                      \
    case N:                                                                                            \
        if (full)                                                                                      \
            rescore_j<N, true>(ix, qrows, sq, nq, cbase, chunks, pair_cnt, pairs, pair_sub, gamma, keys, \
                               cert_cnt, fail, row_reads, fail_qi, stream);                            \
        else                                                                                           \
            rescore_j<N, false>(ix, qrows, sq, nq, cbase, chunks, pair_cnt, pairs, pair_sub, gamma,     \
                                keys, cert_cnt, fail, row_reads, fail_qi, stream);                     \
        break;
    switch (J) {
        PVS_RS(1)
        PVS_RS(2)
        PVS_RS(3)
        PVS_RS(4)
        PVS_RS(6)
        PVS_RS(8)
        PVS_RS(12)
        PVS_RS(16)
        default:
            rescore_j<0, false>(ix, qrows, sq, nq, cbase, chunks, pair_cnt, pairs, pair_sub, gamma, keys,
                                cert_cnt, fail, row_reads, fail_qi, stream);
            break;
    }
#undef PVS_RS
}

// ------------------------------------------------------------------ sorting
// Ascending sort of every tile of kSortTile keys of every query's region
// (bitonic network in LDS; keys past the region's count are padded with ~0
// and not written back).
__global__ __launch_bounds__(256) void k_sort_tiles(uint64_t* __restrict__ keys,
                                                    const int32_t* __restrict__ cnt,
                                                    const ScanQ* __restrict__ sq) {
    __shared__ uint64_t s[kSortTile];
    const int b = blockIdx.y;
    const int64_t n = cnt[b];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kSortTile;
    if (base >= n) return;
    uint64_t* k = keys + sq[b].cand_off + base;
    const int64_t m = min(static_cast<int64_t>(kSortTile), n - base);
    for (int i = threadIdx.x; i < kSortTile; i += 256) s[i] = (i < m) ? k[i] : ~0ull;
    __syncthreads();
    for (int size = 2; size <= kSortTile; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = threadIdx.x; i < kSortTile; i += 256) {
                const int j = i ^ stride;
                if (j > i) {
                    const bool asc = (i & size) == 0;
                    const uint64_t a = s[i], c = s[j];
                    if ((a > c) == asc) {
                        s[i] = c;
                        s[j] = a;
                    }
                }
            }
            __syncthreads();
        }
    }
    for (int i = threadIdx.x; i < m; i += 256) k[i] = s[i];
}

// One merge level: runs of length `run` (a multiple of kSortTile) are merged
// pairwise, by merge path.  Workgroup (x, b) writes outputs
// [x kSortTile, (x + 1) kSortTile) of query b, which lie in one pair of runs:
// searches on the pair's cross diagonals give the parts of the left and
// right runs that fill them (the left run first among equal keys; keys are
// unique inside a query), those are staged in LDS, and each thread merges
// eight consecutive outputs after a search of its own diagonal there.
__global__ __launch_bounds__(256) void k_merge(const uint64_t* __restrict__ src,
                                               uint64_t* __restrict__ dst,
                                               const int32_t* __restrict__ cnt,
                                               const ScanQ* __restrict__ sq, int64_t run) {
    constexpr int T = kSortTile;
    constexpr int PER = T / 256;
    static_assert(T % 256 == 0, "eight outputs per thread");
    __shared__ uint64_t seg[T];   // the left part, then the right part
    __shared__ uint64_t out[T];
    __shared__ int64_t s_split[2];
    const int b = blockIdx.y;
    const int64_t n = cnt[b];
    const int64_t o0 = static_cast<int64_t>(blockIdx.x) * T;
    if (o0 >= n) return;
    const int64_t o1 = min(o0 + T, n);
    const uint64_t* s = src + sq[b].cand_off;
    uint64_t* d = dst + sq[b].cand_off;
    const int64_t start = (o0 / (2 * run)) * (2 * run);
    const int64_t mid = min(start + run, n);
    const int64_t end = min(start + 2 * run, n);
    const int64_t la = mid - start, lb = end - mid;
    const uint64_t* A = s + start;
    const uint64_t* B = s + mid;
    // Left-run elements among the first `diag` outputs of the pair: the
    // first m with A[m] > B[diag - 1 - m], searched by a wavefront 64 ways at
    // a time (four dependent loads for runs of millions, not twenty).
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    if (wave < 2) {
        const int64_t diag = (wave == 0 ? o0 : o1) - start;
        int64_t lo = diag > lb ? diag - lb : 0, hi = diag < la ? diag : la;
        while (lo < hi) {   // the same in every lane
            const int64_t m = lo + ((hi - lo) * lane) / 64;   // in [lo, hi), ascending with the lane
            const bool p = A[m] <= B[diag - 1 - m];           // true exactly below the answer
            const int c = __popcll(__ballot(p));              // lanes below the answer
            const int64_t m_below = __shfl(m, c > 0 ? c - 1 : 0, 64);
            const int64_t m_at = __shfl(m, c < 64 ? c : 63, 64);
            const int64_t nlo = c > 0 ? m_below + 1 : lo;
            hi = c < 64 ? m_at : hi;
            lo = nlo;
        }
        if (lane == 0) s_split[wave] = lo;
    }
    __syncthreads();
    const int64_t a0 = s_split[0], a1 = s_split[1];
    const int64_t b0 = (o0 - start) - a0, b1 = (o1 - start) - a1;
    const int na = static_cast<int>(a1 - a0), nb = static_cast<int>(b1 - b0);
    for (int i = threadIdx.x; i < na + nb; i += 256) seg[i] = i < na ? A[a0 + i] : B[b0 + i - na];
    __syncthreads();
    // this thread's outputs [t0, t0 + PER) of the tile
    const int t0 = threadIdx.x * PER;
    if (t0 < na + nb) {
        const uint64_t* sa = seg;
        const uint64_t* sb = seg + na;
        int lo = t0 > nb ? t0 - nb : 0, hi = t0 < na ? t0 : na;
        while (lo < hi) {
            const int m = (lo + hi) >> 1;
            if (sa[m] <= sb[t0 - 1 - m]) lo = m + 1;
            else hi = m;
        }
        int ia = lo, ib = t0 - lo;
        const int t1 = min(t0 + PER, na + nb);
        for (int t = t0; t < t1; ++t) {
            const bool takea = ib >= nb || (ia < na && sa[ia] <= sb[ib]);
            out[t] = takea ? sa[ia++] : sb[ib++];
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < na + nb; i += 256) d[o0 + i] = out[i];
}

uint64_t* launch_segmented_sort(uint64_t* keys, uint64_t* tmp, const int32_t* cnt,
                                const ScanQ* sq, int32_t nq, int64_t max_cnt, hipStream_t stream) {
    if (nq <= 0 || max_cnt <= 0) return keys;
    const int64_t tiles = (max_cnt + kSortTile - 1) / kSortTile;
    hipLaunchKernelGGL(k_sort_tiles, dim3(static_cast<uint32_t>(tiles), nq), dim3(256), 0, stream,
                       keys, cnt, sq);
    uint64_t* a = keys;
    uint64_t* b = tmp;
    for (int64_t run = kSortTile; run < max_cnt; run *= 2) {
        const int64_t g = (max_cnt + kSortTile - 1) / kSortTile;
        hipLaunchKernelGGL(k_merge, dim3(static_cast<uint32_t>(g), nq), dim3(256), 0, stream, a, b,
                           cnt, sq, run);
        uint64_t* t = a;
        a = b;
        b = t;
    }
    return a;
}

// ----------------------------------------------------------------- packing
__global__ __launch_bounds__(64) void k_offsets(const int32_t* __restrict__ cert, int32_t nq,
                                                int32_t* __restrict__ offs) {
    if (threadIdx.x == 0) {
        int32_t acc = 0;
        for (int b = 0; b < nq; ++b) {
            offs[b] = acc;
            acc += cert[b];
        }
        offs[nq] = acc;
    }
}

__global__ __launch_bounds__(256) void k_pack(const uint64_t* __restrict__ keys,
                                              const int32_t* __restrict__ cert,
                                              const int32_t* __restrict__ offs,
                                              const ScanQ* __restrict__ sq,
                                              uint64_t* __restrict__ packed) {
    const int b = blockIdx.y;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i < cert[b]) packed[offs[b] + i] = keys[sq[b].cand_off + i];
}

void launch_pack(const uint64_t* keys, const int32_t* cert_cnt, const ScanQ* sq, int32_t nq,
                 int64_t max_cnt, int32_t* offs, uint64_t* packed, hipStream_t stream) {
    if (nq <= 0) return;
    hipLaunchKernelGGL(k_offsets, dim3(1), dim3(64), 0, stream, cert_cnt, nq, offs);
    if (max_cnt <= 0) return;
    const int64_t g = (max_cnt + 255) / 256;
    hipLaunchKernelGGL(k_pack, dim3(static_cast<uint32_t>(g), nq), dim3(256), 0, stream, keys,
                       cert_cnt, offs, sq, packed);
}

}  // namespace pvs
