// Candidate rescoring, ordering and packing of the PVS dense channel.
//
// Every candidate gets its authoritative float32 score (row_score, one fixed
// order) and is checked against its interval (App. A.1: a score outside it
// fails the request), recomputed here from the integer dot product the scan
// recorded with the same arithmetic as the scan's, so identical to it.  A scan with threshold tau certifies exactly the
// candidates with s32 >= tau whose key follows the last certified key; their
// keys (~mono(s32) << 32 | row) are appended to the query's key region, so
// ascending keys are (score descending, id ascending).  Keys are unique
// inside a query; the segmented sort orders each query's certified keys.
#include "pvs_device.h"

namespace pvs {

// Candidates of a scan round are cut into chunks of kRescoreChunk per query;
// cbase[b] is the first chunk of query b (exclusive prefix over the queries).
constexpr int kRescoreChunk = 256;

__global__ __launch_bounds__(64) void k_chunk_base(const int32_t* __restrict__ total, int32_t nq,
                                                   int32_t* __restrict__ cbase) {
    if (threadIdx.x == 0) {
        int32_t acc = 0;
        for (int b = 0; b < nq; ++b) {
            cbase[b] = acc;
            acc += (total[b] + kRescoreChunk - 1) / kRescoreChunk;
        }
        cbase[nq] = acc;
    }
}

// One workgroup per chunk, one wavefront per quarter of it, R candidates in
// flight per wavefront (one candidate per wavefront pass: lane l holds
// elements 256 t + 4 l + i of the row, the fixed order of row_score).
// Candidate i of a query (sub-region order) lives in sub-region s with
// first[s] <= i < last[s]: lane s holds first[s] and last[s] (a prefix sum of
// the kept counts), and a ballot finds s.  Only certified candidates produce
// a key: s32 >= tau and the key (~mono(s32) << 32 | row) after the last
// certified key; a wavefront collects its keys in lanes 0.. and appends them
// to the query's key region with one atomic.
template <int J>
__global__ __launch_bounds__(256) void k_rescore(
    const float4* __restrict__ rows, int32_t df4, const float4* __restrict__ qrows,
    const ScanQ* __restrict__ sq, int32_t nq, const int32_t* __restrict__ cbase,
    const uint2* __restrict__ cand, const float* __restrict__ scale,
    const float* __restrict__ vnorm, const float* __restrict__ enorm, float gamma,
    const int32_t* __restrict__ sub_cnt, uint64_t* __restrict__ keys,
    int32_t* __restrict__ cert_cnt, int32_t* __restrict__ fail) {
    static_assert(kSub == 64, "one lane per sub-region");
    constexpr int PER_WAVE = kRescoreChunk / 4;
    static_assert(PER_WAVE <= 64, "one key per lane");
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    // the query of this chunk: the last b with cbase[b] <= chunk (that query
    // has chunks, as cbase[b + 1] > chunk)
    const int x = blockIdx.x;
    int blo = 0, bhi = nq;
    while (bhi - blo > 1) {
        const int mid = (blo + bhi) >> 1;
        if (cbase[mid] <= x) blo = mid;
        else bhi = mid;
    }
    const int b = blo;
    const ScanQ Q = sq[b];
    const int c = sub_cnt[(b * kSub + lane) * kCntStride];
    const int kept = static_cast<int>(c < Q.cand_cap ? c : Q.cand_cap);
    int last = kept;
    for (int off = 1; off < 64; off <<= 1) {
        const int t = __shfl_up(last, off, 64);
        if (lane >= off) last += t;
    }
    const int first = last - kept;
    const int64_t n = __builtin_amdgcn_readlane(last, 63);
    const int64_t i_begin = static_cast<int64_t>(x - cbase[b]) * kRescoreChunk + wave * PER_WAVE;
    const int64_t i_end = (i_begin + PER_WAVE < n) ? i_begin + PER_WAVE : n;
    if (i_begin >= i_end) return;
    float4 qv[J];
    load_query_row<J>(qrows, Q.qi, df4, lane, qv);
    // slot of candidate i (uniform across the wavefront)
    auto slot_of = [&](int64_t i) -> int64_t {
        const uint64_t m = __ballot(first <= i && i < last);
        const int s = __ffsll(static_cast<unsigned long long>(m)) - 1;
        const int f = __builtin_amdgcn_readlane(first, s);
        return Q.cand_off + static_cast<int64_t>(s) * Q.cand_cap + (i - f);
    };
    constexpr int R = (J <= 4) ? 4 : 1;
    uint64_t mykey = 0;
    int nk = 0;          // certified keys collected (lanes 0 .. nk - 1)
    bool bad = false;
    for (int64_t i0 = i_begin; i0 < i_end; i0 += R) {
        int32_t row[R];
        int32_t dot[R];
        float sv[R], nv[R], nev[R];
        float4 v[R][J];
#pragma unroll
        for (int k = 0; k < R; ++k) {
            const int64_t i = i0 + k;
            const uint2 rec = (i < i_end) ? cand[slot_of(i)] : make_uint2(0xffffffffu, 0u);
            row[k] = static_cast<int32_t>(rec.x);   // -1 past the chunk or for a sentinel
            dot[k] = static_cast<int32_t>(rec.y);
            const int64_t r = row[k] < 0 ? 0 : row[k];
            sv[k] = scale[r];
            nv[k] = vnorm[r];
            nev[k] = enorm[r];
            const float4* rp = rows + r * df4;
#pragma unroll
            for (int t = 0; t < J; ++t) {
                const int idx = 64 * t + lane;
                v[k][t] = (row[k] >= 0 && idx < df4) ? rp[idx] : make_float4(0, 0, 0, 0);
            }
        }
#pragma unroll
        for (int k = 0; k < R; ++k) {
            if (row[k] < 0) continue;   // past the chunk, or a sentinel slot
            // same accumulation order as row_score: (t, x, y, z, w), then the butterfly
            float acc = 0.0f;
#pragma unroll
            for (int t = 0; t < J; ++t) {
                if (64 * t + lane < df4) {
                    acc = fmaf(qv[t].x, v[k][t].x, acc);
                    acc = fmaf(qv[t].y, v[k][t].y, acc);
                    acc = fmaf(qv[t].z, v[k][t].z, acc);
                    acc = fmaf(qv[t].w, v[k][t].w, acc);
                }
            }
            for (int off = 32; off > 0; off >>= 1) acc = acc + __shfl_xor(acc, off, 64);
            const float s = acc;   // identical in every lane
            float lo, hi;
            pair_interval(Q, sv[k], nv[k], nev[k], dot[k], gamma, lo, hi);
            bad |= !(lo <= s && s <= hi);
            const bool dropped =
                Q.has_cert && (s > Q.s_cert || (s == Q.s_cert && row[k] <= Q.id_cert));
            if (!dropped && s >= Q.tau) {
                if (lane == nk)
                    mykey = (static_cast<uint64_t>(~mono32(s)) << 32) | static_cast<uint32_t>(row[k]);
                ++nk;
            }
        }
    }
    if (bad && lane == 0) fail[b] = 1;
    if (nk == 0) return;
    int base = 0;
    if (lane == 0) base = atomicAdd(&cert_cnt[b], nk);
    base = __shfl(base, 0, 64);
    if (lane < nk) keys[Q.cand_off + base + lane] = mykey;
}

template <int J>
static void rescore_j(const IndexView& ix, const float* qrows, const ScanQ* sq, int32_t nq,
                      const int32_t* cbase, int64_t chunks, const uint2* cand, float gamma,
                      const int32_t* sub_cnt, uint64_t* keys, int32_t* cert_cnt, int32_t* fail,
                      hipStream_t stream) {
    hipLaunchKernelGGL((k_rescore<J>), dim3(static_cast<uint32_t>(chunks)), dim3(256), 0, stream,
                       reinterpret_cast<const float4*>(ix.rows), ix.df / 4,
                       reinterpret_cast<const float4*>(qrows), sq, nq, cbase, cand, ix.scale,
                       ix.vnorm, ix.enorm, gamma, sub_cnt, keys, cert_cnt, fail);
}

int64_t rescore_chunks(const int32_t* total, int32_t nq) {
    int64_t c = 0;
    for (int32_t b = 0; b < nq; ++b) c += (total[b] + kRescoreChunk - 1) / kRescoreChunk;
    return c;
}

void launch_rescore(const IndexView& ix, const float* qrows, const ScanQ* sq, int32_t nq,
                    const int32_t* total, int32_t* cbase, int64_t chunks,
                    const uint2* cand, float gamma, const int32_t* sub_cnt, uint64_t* keys,
                    int32_t* cert_cnt, int32_t* fail, hipStream_t stream) {
    if (nq <= 0) return;
    hipLaunchKernelGGL(k_chunk_base, dim3(1), dim3(64), 0, stream, total, nq, cbase);
    if (chunks <= 0) return;
#define PVS_RS(N)                                                                              \
    case N:                                                                                    \
        rescore_j<N>(ix, qrows, sq, nq, cbase, chunks, cand, gamma, sub_cnt, keys, cert_cnt,  \
                     fail, stream);                                                            \
        break;
    switch (row_chunks(ix.df)) {
        PVS_RS(1)
        PVS_RS(2)
        PVS_RS(3)
        PVS_RS(4)
        PVS_RS(8)
        PVS_RS(16)
        default:
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

// One merge level: runs of length `run` are merged pairwise.  An element's
// output slot is its offset in its own run plus the number of keys of the
// partner run that precede it (binary search; smaller keys, and for the right
// run also equal ones, so the merge is stable).
__global__ __launch_bounds__(256) void k_merge(const uint64_t* __restrict__ src,
                                               uint64_t* __restrict__ dst,
                                               const int32_t* __restrict__ cnt,
                                               const ScanQ* __restrict__ sq, int64_t run) {
    const int b = blockIdx.y;
    const int64_t n = cnt[b];
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= n) return;
    const uint64_t* s = src + sq[b].cand_off;
    uint64_t* d = dst + sq[b].cand_off;
    const uint64_t key = s[i];
    const int64_t start = (i / (2 * run)) * (2 * run);
    const int64_t mid = min(start + run, n);
    const int64_t end = min(start + 2 * run, n);
    int64_t lo, hi, own;
    if (i < mid) {
        lo = mid;
        hi = end;
        own = i - start;
    } else {
        lo = start;
        hi = mid;
        own = i - mid;
    }
    const int64_t first = lo;
    const bool left = i < mid;   // ties (none expected) go to the left run first
    while (lo < hi) {
        const int64_t m = (lo + hi) >> 1;
        if (s[m] < key || (!left && s[m] == key)) lo = m + 1;
        else hi = m;
    }
    d[start + own + (lo - first)] = key;
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
        const int64_t g = (max_cnt + 255) / 256;
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
