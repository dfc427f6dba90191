// Interval scans of the PVS dense channel (Sec. 2.3.1): every visible row's
// Int8 codes are streamed once per scan; each (query, row) pair gets its exact
// integer dot product and its score interval (pvs_device.h), and rows whose
// interval can reach the query's threshold tau are appended to the query's
// candidate region.  A sample pass over every sample_stride-th block records
// the bounds from which tau is selected.
//
// Two kernels compute the same integers: a dot4 GEMV for a few queries and an
// Int8 MFMA contraction for batches.
#include <algorithm>
#include <atomic>
#include <cstdlib>
#include <cstring>

#include "pvs_device.h"

namespace pvs {

// ------------------------------------------------------------------- GEMV
// One wavefront per 64-row block (lane = row); QB queries per pass, their
// codes read through scalar loads.  The block's records (lane order, then
// query order) take one atomic per wavefront on the counter of sub-region
// blk % kSub.
template <int QB, bool SAMPLE>
__global__ __launch_bounds__(256) void k_scan_gemv(
    const uint4* __restrict__ codes, const float* __restrict__ scale,
    const float* __restrict__ vnorm, const float* __restrict__ enorm,
    const uint64_t* __restrict__ vis, int64_t nblocks, int32_t nchunk,
    const int8_t* __restrict__ qcodes, int32_t dp, const ScanQ* __restrict__ sq, float gamma,
    ScanOut o) {
    const int lane = threadIdx.x & 63;
    const int64_t w = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    const int64_t blk = SAMPLE ? w * o.sample_stride : w;
    if (blk >= nblocks) return;
    const int64_t row = blk * 64 + lane;
    const uint64_t vbits = vis[blk];
    const bool visible = (vbits >> lane) & 1ull;
    const float sv = scale[row];
    const float nv = vnorm[row];
    const float nev = enorm[row];

    const int4* qp[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b)
        qp[b] = reinterpret_cast<const int4*>(qcodes + static_cast<int64_t>(sq[b].qi) * dp);
    int acc[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) acc[b] = 0;
    const uint4* cp = codes + blk * nchunk * 64 + lane;
#pragma unroll 4
    for (int c = 0; c < nchunk; ++c) {
        const u32x4 x = load_nt(cp + c * 64);
#pragma unroll
        for (int b = 0; b < QB; ++b) {
            const int4 qc = qp[b][c];
            int a = acc[b];
            a = __builtin_amdgcn_sdot4(static_cast<int>(x.x), qc.x, a, false);
            a = __builtin_amdgcn_sdot4(static_cast<int>(x.y), qc.y, a, false);
            a = __builtin_amdgcn_sdot4(static_cast<int>(x.z), qc.z, a, false);
            a = __builtin_amdgcn_sdot4(static_cast<int>(x.w), qc.w, a, false);
            acc[b] = a;
        }
    }
    uint32_t take = 0;   // bit b: the pair (query b, this row) is a candidate
#pragma unroll
    for (int b = 0; b < QB; ++b) {
        const ScanQ Q = sq[b];
        float lo, hi;
        pair_interval(Q, sv, nv, nev, acc[b], gamma, lo, hi);
        const bool elig = visible && (!Q.has_cert || lo <= Q.s_cert);
        if (SAMPLE) {
            const int64_t i = b * o.sample_ld + w * 64 + lane;
            o.sample_lo[i] = elig ? lo : -INFINITY;
            o.sample_hi[i] = elig ? hi : -INFINITY;
        } else if (elig && hi >= Q.tau) {
            take |= 1u << b;
        }
    }
    if (SAMPLE) return;
    // records in (row, query) order: exclusive prefix of the per-lane counts
    const int mine = __popc(take);
    int incl = mine;
    for (int off = 1; off < 64; off <<= 1) {
        const int t = __shfl_up(incl, off, 64);
        if (lane >= off) incl += t;
    }
    const int total = __shfl(incl, 63, 64);
    if (total == 0) return;
#pragma unroll
    for (int b = 0; b < QB; ++b) {
        const int c = __popcll(__ballot((take >> b) & 1u));
        if (lane == 0 && c) atomicAdd(&o.q_evals[(blk & (kSub - 1)) * o.q_ld + o.qbase + b], c);
    }
    const int sub = static_cast<int>(blk & (kSub - 1));
    int base = 0;
    if (lane == 0) base = atomicAdd(&o.pair_cnt[sub * kCntStride], total);
    base = __shfl(base, 0, 64);
    uint4* dst = o.pairs + sub * o.pair_sub;
    int64_t p = static_cast<int64_t>(base) + (incl - mine);
#pragma unroll
    for (int b = 0; b < QB; ++b) {
        if ((take >> b) & 1u) {
            if (p < o.pair_sub)
                dst[p] = make_uint4(static_cast<uint32_t>(row), static_cast<uint32_t>(o.qbase + b),
                                    static_cast<uint32_t>(acc[b]), 0u);
            ++p;
        }
    }
}

template <int QB>
static void gemv_pass(const IndexView& ix, const uint64_t* vis, int64_t nblocks,
                      const int8_t* qcodes, const ScanQ* sq, float gamma, bool sample,
                      const ScanOut& o, hipStream_t stream) {
    const int64_t waves = sample ? (nblocks + o.sample_stride - 1) / o.sample_stride : nblocks;
    const uint32_t grid = static_cast<uint32_t>((waves + 3) / 4);
    if (sample) {
        hipLaunchKernelGGL((k_scan_gemv<QB, true>), dim3(grid), dim3(256), 0, stream, ix.codes,
                           ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qcodes, ix.dp,
                           sq, gamma, o);
    } else {
        hipLaunchKernelGGL((k_scan_gemv<QB, false>), dim3(grid), dim3(256), 0, stream, ix.codes,
                           ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qcodes, ix.dp,
                           sq, gamma, o);
    }
}

static ScanOut shift_out(const ScanOut& o, int32_t q0) {
    ScanOut s = o;
    if (s.sample_lo) s.sample_lo += q0 * o.sample_ld;
    if (s.sample_hi) s.sample_hi += q0 * o.sample_ld;
    s.qbase = o.qbase + q0;
    return s;
}

void launch_scan(const IndexView& ix, const uint64_t* vis, int64_t nblocks, const int8_t* qcodes,
                 const ScanQ* sq, int32_t nq, float gamma, bool sample, const ScanOut& o,
                 hipStream_t stream) {
    for (int32_t q0 = 0; q0 < nq; q0 += kMaxGemvQueries) {
        const int qb = (nq - q0 < kMaxGemvQueries) ? (nq - q0) : kMaxGemvQueries;
        const ScanOut so = shift_out(o, q0);
        const ScanQ* s = sq + q0;
#define PVS_GEMV_CASE(N)                                                    \
    case N:                                                                 \
        gemv_pass<N>(ix, vis, nblocks, qcodes, s, gamma, sample, so, stream); \
        break;
        switch (qb) {
            PVS_GEMV_CASE(1)
            PVS_GEMV_CASE(2)
            PVS_GEMV_CASE(3)
            PVS_GEMV_CASE(4)
            PVS_GEMV_CASE(5)
            PVS_GEMV_CASE(6)
            PVS_GEMV_CASE(7)
            PVS_GEMV_CASE(8)
            default:
                break;
        }
#undef PVS_GEMV_CASE
    }
}

// -------------------------------------------------------------- MFMA scan
// For query batches the code x query product is a dense Int8 contraction:
// V_MFMA_I32_32X32X32_I8 with the corpus block as A (32 rows x 32 bytes per
// instruction) and the query codes as B.  Operand layout (lane l, byte j):
// A[l % 32][16 (l / 32) + j], B[16 (l / 32) + j][l % 32]; accumulator r of lane
// l holds C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].  A 16-byte A fragment is
// therefore 32 consecutive rows of one code chunk: two contiguous 512-byte
// runs of the chunk-major block layout.

// Records of the candidate pairs of one block and NQS query tiles (q0 is the
// scan index of the first tile's first query): bit 16 t + r of mask[uu] in
// lane l marks the pair of query q0 + 32 uu + l % 32 and the row of
// accumulator element r of acc[t][uu].  One atomic reserves the wavefront's
// records; they are written row by row (rows in (t, r, l / 32) order, each
// row's queries ascending), so the records of one row are adjacent.
template <int NQS>
__device__ __forceinline__ void emit_pairs(const uint32_t (&mask)[NQS], const v16i (&acc)[2][NQS],
                                           int64_t blk, int lane, int32_t q0, int sub,
                                           const ScanOut& o) {
    int mine = 0;
#pragma unroll
    for (int uu = 0; uu < NQS; ++uu) mine += __popc(mask[uu]);
    for (int off = 32; off > 0; off >>= 1) mine += __shfl_xor(mine, off, 64);
    if (mine == 0) return;
    int base = 0;
    if (lane == 0) base = atomicAdd(&o.pair_cnt[sub * kCntStride], mine);
    // 32-bit positions and rows: the host keeps every counter and row id
    // below 2^31
    int run = __builtin_amdgcn_readfirstlane(base);
    const int cap = static_cast<int>(o.pair_sub);
    uint4* dst = o.pairs + sub * o.pair_sub;
    const uint32_t below = (1u << (lane & 31)) - 1u;
    const bool upper = lane >= 32;
    uint32_t row0 = static_cast<uint32_t>(blk * 64) + 4 * (lane >> 5);
    uint32_t qid = static_cast<uint32_t>(q0 + (lane & 31));
    // opaque here, so the 32 row numbers derived from row0 are formed at
    // their stores instead of being hoisted out of the caller's loops (where
    // they would stay live across the K loop)
    asm volatile("" : "+v"(row0), "+v"(qid));
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int bit = 16 * t + r;
            int ca = 0, cb = 0;
#pragma unroll
            for (int uu = 0; uu < NQS; ++uu) {
                const uint64_t bal = __ballot((mask[uu] >> bit) & 1u);
                ca += __popc(static_cast<uint32_t>(bal));
                cb += __popc(static_cast<uint32_t>(bal >> 32));
            }
            if (ca + cb == 0) continue;
            int at = run + (upper ? ca : 0);
#pragma unroll
            for (int uu = 0; uu < NQS; ++uu) {
                const uint64_t bal = __ballot((mask[uu] >> bit) & 1u);
                const uint32_t m = upper ? static_cast<uint32_t>(bal >> 32) : static_cast<uint32_t>(bal);
                if ((mask[uu] >> bit) & 1u) {
                    const int p = at + __popc(m & below);
                    if (p < cap)
                        dst[p] = make_uint4(row0 + 32 * t + 8 * (r >> 2) + (r & 3), qid + 32 * uu,
                                            static_cast<uint32_t>(acc[t][uu][r]), 0u);
                }
                at += __popc(m);
            }
            run += ca + cb;
        }
    }
}

// Records of a block for 8 query tiles computed in two halves: the first
// half's candidate bits m0 (tiles 0-3) with their dot products saved in
// LDS (sd, this lane's from sd[j], in (t, r, tile) order), the second half's
// bits m1 (tiles 4-7) with acc.  One atomic; each row's records (all 8 tiles)
// are adjacent, as in emit_pairs.
__device__ __forceinline__ void emit_pairs_joined(const uint32_t (&m0)[4], const int32_t* sd, int j,
                                                  const uint32_t (&m1)[4], const v16i (&acc)[2][4],
                                                  int64_t blk, int lane, int32_t q0, int sub,
                                                  const ScanOut& o) {
    int mine = 0;
#pragma unroll
    for (int uu = 0; uu < 4; ++uu) mine += __popc(m0[uu]) + __popc(m1[uu]);
    for (int off = 32; off > 0; off >>= 1) mine += __shfl_xor(mine, off, 64);
    if (mine == 0) return;
    int base = 0;
    if (lane == 0) base = atomicAdd(&o.pair_cnt[sub * kCntStride], mine);
    int run = __builtin_amdgcn_readfirstlane(base);
    const int cap = static_cast<int>(o.pair_sub);
    uint4* dst = o.pairs + sub * o.pair_sub;
    const uint32_t below = (1u << (lane & 31)) - 1u;
    const bool upper = lane >= 32;
    uint32_t row0 = static_cast<uint32_t>(blk * 64) + 4 * (lane >> 5);
    uint32_t qid = static_cast<uint32_t>(q0 + (lane & 31));
    asm volatile("" : "+v"(row0), "+v"(qid));   // as in emit_pairs
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int bit = 16 * t + r;
            int ca = 0, cb = 0;
#pragma unroll
            for (int uu = 0; uu < 4; ++uu) {
                const uint64_t b0 = __ballot((m0[uu] >> bit) & 1u);
                const uint64_t b1 = __ballot((m1[uu] >> bit) & 1u);
                ca += __popc(static_cast<uint32_t>(b0)) + __popc(static_cast<uint32_t>(b1));
                cb += __popc(static_cast<uint32_t>(b0 >> 32)) + __popc(static_cast<uint32_t>(b1 >> 32));
            }
            if (ca + cb == 0) continue;
            int at = run + (upper ? ca : 0);
            const uint32_t row = row0 + 32 * t + 8 * (r >> 2) + (r & 3);
#pragma unroll
            for (int uu = 0; uu < 4; ++uu) {
                const uint64_t bal = __ballot((m0[uu] >> bit) & 1u);
                const uint32_t m = upper ? static_cast<uint32_t>(bal >> 32) : static_cast<uint32_t>(bal);
                if ((m0[uu] >> bit) & 1u) {
                    const int p = at + __popc(m & below);
                    const int32_t dot = sd[j++];
                    if (p < cap) dst[p] = make_uint4(row, qid + 32 * uu, static_cast<uint32_t>(dot), 0u);
                }
                at += __popc(m);
            }
#pragma unroll
            for (int uu = 0; uu < 4; ++uu) {
                const uint64_t bal = __ballot((m1[uu] >> bit) & 1u);
                const uint32_t m = upper ? static_cast<uint32_t>(bal >> 32) : static_cast<uint32_t>(bal);
                if ((m1[uu] >> bit) & 1u) {
                    const int p = at + __popc(m & below);
                    if (p < cap)
                        dst[p] = make_uint4(row, qid + 32 * (4 + uu), static_cast<uint32_t>(acc[t][uu][r]), 0u);
                }
                at += __popc(m);
            }
            run += ca + cb;
        }
    }
}

// Query codes of one pass in MFMA B-fragment order:
// frag[(s * nqt + u) * 64 + lane] = 16 code bytes of query 32 u + lane % 32,
// bytes 32 s + 16 (lane / 32) .. +15; queries past nq are zero.
__global__ __launch_bounds__(64) void k_qfrag(const int8_t* __restrict__ qcodes, int32_t dp,
                                              const ScanQ* __restrict__ sq, int32_t nq, int32_t nqt,
                                              uint4* __restrict__ frag) {
    const int lane = threadIdx.x;
    const int s = blockIdx.x / nqt, u = blockIdx.x % nqt;
    const int b = 32 * u + (lane & 31);
    uint4 v = make_uint4(0, 0, 0, 0);
    if (b < nq) {
        const int64_t off = static_cast<int64_t>(sq[b].qi) * dp + 32 * s + 16 * (lane >> 5);
        v = *reinterpret_cast<const uint4*>(qcodes + off);
    }
    frag[(static_cast<int64_t>(s) * nqt + u) * 64 + lane] = v;
}

// One wavefront per 64-row block and NQT tiles of 32 queries, processed NQS
// tiles at a time (2 x NQS accumulators of 32 x 32; a second half re-reads
// the block's codes from L2).  Epilogue per query tile: lane l owns query
// 32 u + l % 32 and 32 of the block's rows; the centre-score pre-test skips
// the exact interval for rows that cannot reach tau; survivors of lanes l and
// l ^ 32 (same query) become records through emit_pairs.
template <int NQT, bool SAMPLE>
__global__ __launch_bounds__(256) void k_scan_mfma(
    const uint4* __restrict__ codes, const float* __restrict__ scale,
    const float* __restrict__ vnorm, const float* __restrict__ enorm,
    const uint64_t* __restrict__ vis, int64_t nblocks, int32_t nchunk,
    const v4i* __restrict__ qfrag, const ScanQ* __restrict__ sq, int32_t nq, float gamma,
    ScanOut o) {
    constexpr int NQS = NQT < 4 ? NQT : 4;
    const int lane = threadIdx.x & 63;
    const int64_t w = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    const int64_t blk = SAMPLE ? w * o.sample_stride : w;
    if (blk >= nblocks) return;
    const uint64_t vbits = vis[blk];
    // scale and norms of this lane's 32 rows, loaded before the K loop so the
    // epilogue's interval tests never wait on memory
    float svr[2][16], vnr[2][16], enr[2][16];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int64_t row = blk * 64 + 32 * t + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            svr[t][r] = scale[row];
            vnr[t][r] = vnorm[row];
            enr[t][r] = enorm[row];
        }
    const uint4* A = codes + blk * nchunk * 64 + (lane >> 5) * 64 + (lane & 31);
    const int nsteps = nchunk >> 1;
#pragma unroll 1
    for (int u0 = 0; u0 < NQT; u0 += NQS) {
    v16i acc[2][NQS];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < NQS; ++u) acc[t][u] = v16i{};
#pragma unroll 2
    for (int s = 0; s < nsteps; ++s) {
        const u32x4 a0 = load_nt(A + 2 * s * 64);
        const u32x4 a1 = load_nt(A + 2 * s * 64 + 32);
        v4i va0, va1;
        __builtin_memcpy(&va0, &a0, 16);
        __builtin_memcpy(&va1, &a1, 16);
#pragma unroll
        for (int u = 0; u < NQS; ++u) {
            const v4i vb = qfrag[(s * NQT + u0 + u) * 64 + lane];
            acc[0][u] = __builtin_amdgcn_mfma_i32_32x32x32_i8(va0, vb, acc[0][u], 0, 0, 0);
            acc[1][u] = __builtin_amdgcn_mfma_i32_32x32x32_i8(va1, vb, acc[1][u], 0, 0, 0);
        }
    }
    uint32_t mask[NQS];   // candidate bits (16 t + r) of each tile
#pragma unroll
    for (int uu = 0; uu < NQS; ++uu) {
        const int u = u0 + uu;
        const int b = 32 * u + (lane & 31);
        const bool valid = b < nq;
        const ScanQ Q = sq[valid ? b : 0];
        mask[uu] = 0;
        if (SAMPLE) {
            if (!valid) continue;
#pragma unroll
            for (int t = 0; t < 2; ++t) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int rib = 32 * t + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                    float lo, hi;
                    pair_interval(Q, svr[t][r], vnr[t][r], enr[t][r], acc[t][uu][r], gamma, lo, hi);
                    const bool elig = ((vbits >> rib) & 1ull) && (!Q.has_cert || lo <= Q.s_cert);
                    const int64_t i = b * o.sample_ld + w * 64 + rib;
                    o.sample_lo[i] = elig ? lo : -INFINITY;
                    o.sample_hi[i] = elig ? hi : -INFINITY;
                }
            }
            continue;
        }
        const float thr = center_threshold(Q);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rib = 32 * t + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                const float sv = svr[t][r];
                const float c = (Q.sq * sv) * static_cast<float>(acc[t][uu][r]);
                if (valid && c >= thr && ((vbits >> rib) & 1ull)) {
                    float lo, hi;
                    pair_interval(Q, sv, vnr[t][r], enr[t][r], acc[t][uu][r], gamma, lo, hi);
                    if (hi >= Q.tau && (!Q.has_cert || lo <= Q.s_cert)) mask[uu] |= 1u << (16 * t + r);
                }
            }
        }
    }
    if (!SAMPLE) {
#pragma unroll
        for (int uu = 0; uu < NQS; ++uu) {   // records per query (lanes l and l ^ 32 share one)
            int c = __popc(mask[uu]);
            c += __shfl_xor(c, 32, 64);
            if (lane < 32 && c)
                atomicAdd(&o.q_evals[(blk & (kSub - 1)) * o.q_ld + o.qbase + 32 * (u0 + uu) + lane], c);
        }
        emit_pairs<NQS>(mask, acc, blk, lane, o.qbase + 32 * u0, static_cast<int>(blk & (kSub - 1)), o);
    }
    }
}

// Wide batches (NQT = 4 or 8 tiles of 32 queries).  Persistent workgroups
// of 4 wavefronts, two per CU, take 4 consecutive blocks at a time, one per
// wavefront, and runs the K loop once per half of 4 query tiles (2 x 4
// accumulators of 32 x 32).  The K loop has no branches: it advances PA steps
// per stage (PA divides the step count), the A fragments of the next stage
// stream into a register ring while the current stage multiplies, and the B
// fragments of one stage (PA x 4 KiB) are loaded once per workgroup one stage
// ahead and shared by the 4 wavefronts through double-buffered LDS, with one
// barrier per stage.  A second half re-reads the block's codes from cache.
//
// Epilogue: lane l owns query 32 u + l % 32 and 32 of the block's rows.  A
// per-block bound of E + G (from the block's largest norms) gives a centre
// threshold below which no row of the block can reach tau; invisible rows
// carry a NaN scale so they fail it.  Each wavefront writes the records of
// its block and half through emit_pairs into sub-region blk % kSub (blocks,
// not workgroups, spread the records evenly over the sub-regions).
template <int NQT, int PA>
__global__ __launch_bounds__(256, 2) void k_scan_mfma_wide(
    const uint4* __restrict__ codes, const float* __restrict__ scale,
    const float* __restrict__ vnorm, const float* __restrict__ enorm,
    const uint64_t* __restrict__ vis, int64_t nblocks, int32_t nchunk,
    const v4i* __restrict__ qfrag, const ScanQ* __restrict__ sq, int32_t nq, float gamma,
    ScanOut o) {
    constexpr int NQS = 4;                     // tiles per half
    __shared__ v4i bsm[2][PA][NQS * 64];       // B fragments of two stages
    __shared__ float s_meta[4][3][64];         // scale (NaN if invisible), norm, error norm
    __shared__ ScanQ s_q[NQT * 32];            // the scanning queries
    // 8 tiles: dot products of the first half's candidates, written with the
    // second half's (at most kSavedDots per wavefront, else written at once)
    constexpr int kSavedDots = 512;
    __shared__ int32_t s_dots[4][NQT == 8 ? kSavedDots : 1];
    __shared__ int32_t s_evals[NQT * 32];      // records per query of this workgroup
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    for (int b = tid; b < nq && b < NQT * 32; b += 256) s_q[b] = sq[b];
    for (int b = tid; b < NQT * 32; b += 256) s_evals[b] = 0;
    __syncthreads();
    const int nsteps = nchunk >> 1;            // a multiple of PA
    const int64_t ngroups = (nblocks + 3) / 4;
    for (int64_t grp = blockIdx.x; grp < ngroups; grp += gridDim.x) {
        const int64_t blk = grp * 4 + wave;
        const bool have = blk < nblocks;
        const uint4* A = codes + (have ? blk : 0) * nchunk * 64 + (lane >> 5) * 64 + (lane & 31);
        float nvb = 0.0f, nevb = 0.0f;         // largest norms of the block's visible rows
        {
            const int64_t row = (have ? blk : 0) * 64 + lane;
            const bool v = have && ((vis[have ? blk : 0] >> lane) & 1ull);
            const float nv = vnorm[row], nev = enorm[row];
            s_meta[wave][0][lane] = v ? scale[row] : __builtin_nanf("");
            s_meta[wave][1][lane] = nv;
            s_meta[wave][2][lane] = nev;
            nvb = wave_max(v ? nv : 0.0f);
            nevb = wave_max(v ? nev : 0.0f);
        }
        uint32_t mask0[NQS] = {};   // first half's candidates kept for the joined write
        int j0 = 0;                 // this lane's first saved dot product
#pragma unroll 1
        for (int u0 = 0; u0 < NQT; u0 += NQS) {
            v16i acc[2][NQS];
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int u = 0; u < NQS; ++u) acc[t][u] = v16i{};
            // stage 0: B into LDS, A into the register ring
            v4i bst[PA];
            v4i a[PA][2];
#pragma unroll
            for (int p = 0; p < PA; ++p) bst[p] = qfrag[(p * NQT + u0) * 64 + tid];
#pragma unroll
            for (int p = 0; p < PA; ++p) bsm[0][p][tid] = bst[p];
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int p = 0; p < PA; ++p) {
                const u32x4 x0 = load_nt(A + 2 * p * 64);
                const u32x4 x1 = load_nt(A + 2 * p * 64 + 32);
                __builtin_memcpy(&a[p][0], &x0, 16);
                __builtin_memcpy(&a[p][1], &x1, 16);
            }
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
            // Scheduling barriers pin the order: the B loads of the next stage
            // are issued first and stored to LDS at the end of the stage, the
            // A load of step + PA right after step's MFMAs, and the LDS reads
            // of step + 1 before step's MFMAs, so each load has about a stage
            // of MFMA work to arrive.
            for (int s0 = 0; s0 < nsteps; s0 += PA) {
                const int cur = (s0 / PA) & 1;
#pragma unroll
                for (int p = 0; p < PA; ++p) {
                    const int sn = min(s0 + PA + p, nsteps - 1);
                    bst[p] = qfrag[(sn * NQT + u0) * 64 + tid];
                }
                v4i vb[2][NQS];
#pragma unroll
                for (int u = 0; u < NQS; ++u) vb[0][u] = bsm[cur][0][u * 64 + lane];
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int p = 0; p < PA; ++p) {
                    if (p + 1 < PA) {
#pragma unroll
                        for (int u = 0; u < NQS; ++u) vb[(p + 1) & 1][u] = bsm[cur][p + 1][u * 64 + lane];
                    }
#pragma unroll
                    for (int u = 0; u < NQS; ++u) {
                        acc[0][u] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[p][0], vb[p & 1][u], acc[0][u], 0, 0, 0);
                        acc[1][u] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[p][1], vb[p & 1][u], acc[1][u], 0, 0, 0);
                    }
                    const int sn = min(s0 + PA + p, nsteps - 1);
                    const u32x4 y0 = load_nt(A + 2 * sn * 64);
                    const u32x4 y1 = load_nt(A + 2 * sn * 64 + 32);
                    __builtin_memcpy(&a[p][0], &y0, 16);
                    __builtin_memcpy(&a[p][1], &y1, 16);
                    __builtin_amdgcn_sched_barrier(0);
                }
#pragma unroll
                for (int p = 0; p < PA; ++p) bsm[cur ^ 1][p][tid] = bst[p];
                __syncthreads();
            }
            // Candidate masks of this half; lanes l and l ^ 32 hold one query.
            // Tiles run outermost so a query's fields are read from LDS once
            // per tile (rows outermost re-read them for every pair that
            // passes: 7 % slower); the per-pair pre-test is one convert, one
            // multiply and one compare against the block threshold divided
            // by s_q (with a margin that covers the rounding of both
            // products), and only pairs that pass it evaluate the exact
            // interval.
            uint32_t mask[NQS];
#pragma unroll
            for (int uu = 0; uu < NQS; ++uu) {
                mask[uu] = 0;
                const int b = 32 * (u0 + uu) + (lane & 31);
                const bool valid = have && b < nq;
                const ScanQ Q = s_q[valid ? b : 0];   // this tile's query, in registers
                const float thq = valid ? scaled_threshold(block_threshold(Q, nvb, nevb, gamma), Q.sq) : INFINITY;
#pragma unroll
                for (int t = 0; t < 2; ++t) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int rib = 32 * t + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                        const float sv = s_meta[wave][0][rib];   // NaN for invisible rows
                        if (sv * static_cast<float>(acc[t][uu][r]) >= thq) {
                            float lo, hi;
                            pair_interval(Q, sv, s_meta[wave][1][rib], s_meta[wave][2][rib],
                                          acc[t][uu][r], gamma, lo, hi);
                            if (hi >= Q.tau && (!Q.has_cert || lo <= Q.s_cert))
                                mask[uu] |= 1u << (16 * t + r);
                        }
                    }
                }
            }
            // no code motion across the epilogue (the next half's loads would
            // raise the register pressure past 256)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int uu = 0; uu < NQS; ++uu) {   // records per query (lanes l and l ^ 32 share one)
                int c = __popc(mask[uu]);
                c += __shfl_xor(c, 32, 64);
                if (lane < 32 && c) atomicAdd(&s_evals[32 * (u0 + uu) + lane], c);
            }
            const int sub = static_cast<int>(blk & (kSub - 1));
            if (have && NQT == 8 && u0 == 0) {
                // first of two halves: save the dot products of its candidates
                // (lane order, then (t, r, tile)) to write them with the second
                int cnt = 0;
#pragma unroll
                for (int uu = 0; uu < NQS; ++uu) cnt += __popc(mask[uu]);
                int incl = cnt;
                for (int off = 1; off < 64; off <<= 1) {
                    const int v = __shfl_up(incl, off, 64);
                    if (lane >= off) incl += v;
                }
                if (__shfl(incl, 63, 64) > kSavedDots) {
                    emit_pairs<NQS>(mask, acc, blk, lane, o.qbase, sub, o);
                } else {
                    int j = incl - cnt;
                    j0 = j;
#pragma unroll
                    for (int t = 0; t < 2; ++t)
#pragma unroll
                        for (int r = 0; r < 16; ++r)
#pragma unroll
                            for (int uu = 0; uu < NQS; ++uu)
                                if ((mask[uu] >> (16 * t + r)) & 1u) s_dots[wave][j++] = acc[t][uu][r];
#pragma unroll
                    for (int uu = 0; uu < NQS; ++uu) mask0[uu] = mask[uu];
                }
            } else if (have && NQT == 8) {
                emit_pairs_joined(mask0, s_dots[wave], j0, mask, acc, blk, lane, o.qbase, sub, o);
            } else if (have) {
                emit_pairs<NQS>(mask, acc, blk, lane, o.qbase + 32 * u0, sub, o);
            }
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();   // bsm and the metadata are reused next
        }
    }
    for (int b = tid; b < nq && b < NQT * 32; b += 256)
        if (s_evals[b]) atomicAdd(&o.q_evals[(blockIdx.x & (kSub - 1)) * o.q_ld + o.qbase + b], s_evals[b]);
}

// ------------------------------------------------ single-pass MFMA scan, LDS queries
// Query batches of up to 32 NQT queries in one pass over the codes.  A
// workgroup of W wavefronts per CU (three per SIMD with four tiles, two
// with eight) holds the query fragments of the first NQT - NG tiles for
// every K step in LDS for the whole kernel; the last NG tiles are read from
// global memory (L2-resident, shared by every workgroup) two steps ahead.
// Each wavefront takes one 32-row half of a 64-row code block at a time and
// computes all NQT tiles for it (NQT accumulators of 32 x 32): the LDS
// fragments of the next K step are read while the current one multiplies,
// and its code fragments stream into a register ring P steps deep that runs
// on into the next half-block, so the epilogue of one half-block overlaps
// the loads of the next and the other wavefronts' MFMAs.  Vector memory
// loads complete in issue order for the wait counters, so every load is
// issued at least two steps before the step that waits for it.
//
// Epilogue: one compare per accumulator pre-tests s_v * dot against the
// half-block's threshold thq (scaled_threshold of block_threshold over the
// half-block's largest norms); the compare's lane mask places the passing
// pairs in a per-wavefront list in LDS, and each list is given the exact
// interval test densely, one pair per lane, with one atomic per 64 pairs
// for the records.
struct QFields {          // the fields of a scanning query the epilogue reads
    float tau, s_cert, sq, nq, nqh, neq, wmax;
    int32_t has_cert;
};

// Largest value of lanes 0..31 (lanes 32..63 hold copies of them), in every
// lane: four DPP steps inside each row of 16 lanes (partners j ^ 1, j ^ 2,
// the mirrored lane within 8 and within 16), then the two rows.
__device__ __forceinline__ float max32(float v) {
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false)));
    return fmaxf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0)),
                 __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16)));
}

template <int NQT, int NG, int NS, int P, int W>
__global__ __launch_bounds__(64 * W, 1) void k_scan_mfma_r1(
    const uint4* __restrict__ codes, const float* __restrict__ scale,
    const float* __restrict__ vnorm, const float* __restrict__ enorm,
    const uint64_t* __restrict__ vis, int64_t nblocks, int32_t nchunk,
    const v4i* __restrict__ qfrag, const ScanQ* __restrict__ sq, int32_t nq, float gamma,
    ScanOut o) {
    constexpr int NL = NQT - NG;            // tiles whose fragments stay in LDS
    // the refills of the last P steps load the next half-block's first P
    // steps into the slots step s % P names for them, which needs NS % P == 0
    static_assert(P >= 2 && P <= NS && NS % P == 0, "ring depth must divide the step count");
    extern __shared__ __align__(16) unsigned char lds[];
    v4i* bsm = reinterpret_cast<v4i*>(lds);                                    // [NS][NL][64]
    QFields* s_qf = reinterpret_cast<QFields*>(lds + static_cast<size_t>(NS) * NL * 1024);
    float* s_meta = reinterpret_cast<float*>(s_qf + NQT * 32);                 // [W][3][32]
    int32_t* s_evals = reinterpret_cast<int32_t*>(s_meta + W * 3 * 32);        // [NQT * 32]
    // pass list per wavefront: room for a row of every tile when NQT <= 4
    // (one overflow check per accumulator row), else 64 entries (a check
    // per tile and row)
    constexpr bool kRowCheck = NQT <= 4;
    constexpr int CAP = kRowCheck ? 64 * (NQT + 1) : 64;
    int32_t* s_ent = s_evals + NQT * 32;                                        // [W][2][CAP]
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar block indices
    int32_t* ent = s_ent + wave * 2 * CAP;   // this wavefront's list: dot products, then packed indices
    for (int i = tid; i < NS * NL * 64; i += 64 * W) {
        const int s = i / (NL * 64), rest = i % (NL * 64);
        bsm[i] = qfrag[s * NQT * 64 + rest];        // tiles 0 .. NL - 1 of step s
    }
    for (int b = tid; b < NQT * 32; b += 64 * W) {
        QFields f{};
        f.tau = INFINITY;
        if (b < nq) {
            const ScanQ& Q = sq[b];
            f = QFields{Q.tau, Q.s_cert, Q.sq, Q.nq, Q.nqh, Q.neq, Q.wmax, Q.has_cert};
        }
        s_qf[b] = f;
        s_evals[b] = 0;
    }
    __syncthreads();
    float* meta = s_meta + wave * 96;
    const int64_t nhalves = 2 * nblocks;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * W;
    int64_t hb = static_cast<int64_t>(blockIdx.x) * W + wave;
    const __amdgpu_buffer_rsrc_t qrs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<v4i*>(qfrag), 0, 0x7fffffff, 0x00020000);
    const int32_t qf_off = lane * 16;
    const int32_t code_off = ((lane >> 5) * 64 + (lane & 31)) * 16;
    auto half_rsrc = [&](int64_t x) {   // codes of half-block x (32 rows of block x / 2)
        return __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint4*>(codes + (x >> 1) * nchunk * 64 + 32 * (x & 1)), 0, 0x7fffffff, 0x00020000);
    };
    v4i a[P];                     // ring: slot s % P holds step s
    v4i g[2][NG > 0 ? NG : 1];    // global tiles, two steps ahead
    auto load_a = [&](__amdgpu_buffer_rsrc_t rs, int s, v4i& dst) {
        dst = __builtin_amdgcn_raw_buffer_load_b128(rs, code_off, s * 2048, 0);
    };
    auto load_g = [&](int s, v4i (&dst)[NG > 0 ? NG : 1]) {
#pragma unroll
        for (int j = 0; j < NG; ++j)
            dst[j] = __builtin_amdgcn_raw_buffer_load_b128(qrs, qf_off, (s * NQT + NL + j) * 1024, 0);
    };
    float sv0 = 0.0f, nv0 = 0.0f, nev0 = 0.0f;
    uint32_t vbits = 0;
    auto load_meta = [&](int64_t x) {
        const int64_t row = (x >> 1) * 64 + 32 * (x & 1) + (lane & 31);
        sv0 = scale[row];
        nv0 = vnorm[row];
        nev0 = enorm[row];
        vbits = static_cast<uint32_t>(vis[x >> 1] >> (32 * (x & 1)));
    };
    if (hb < nhalves) {
        load_meta(hb);
        const __amdgpu_buffer_rsrc_t rs = half_rsrc(hb);
#pragma unroll
        for (int p = 0; p < P; ++p) load_a(rs, p, a[p]);
        if (NG > 0) {
            load_g(0, g[0]);
            load_g(1, g[1]);
        }
    }
    for (; hb < nhalves; hb += stride) {
        const int64_t nxt = hb + stride;
        const bool more = nxt < nhalves;
        const __amdgpu_buffer_rsrc_t rs_cur = half_rsrc(hb);
        const __amdgpu_buffer_rsrc_t rs_nxt = half_rsrc(more ? nxt : hb);
        // this half-block's metadata (invisible rows carry a NaN scale)
        const bool visible = (vbits >> (lane & 31)) & 1u;
        if (lane < 32) {
            meta[lane] = visible ? sv0 : __builtin_nanf("");
            meta[32 + lane] = nv0;
            meta[64 + lane] = nev0;
        }
        const float nvb = max32(visible ? nv0 : 0.0f);
        const float nevb = max32(visible ? nev0 : 0.0f);
        const float s_hi = max32(visible ? sv0 : 0.0f);
        v16i acc[NQT];
#pragma unroll
        for (int u = 0; u < NQT; ++u) acc[u] = v16i{};
        // LDS tiles: the fragments of step s + 1 are read while step s
        // multiplies (two register sets, used alternately)
        v4i vb[2][NL > 0 ? NL : 1];
#pragma unroll
        for (int u = 0; u < NL; ++u) vb[0][u] = bsm[u * 64 + lane];
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int p = s % P;
            if (s + 1 < NS) {
#pragma unroll
                for (int u = 0; u < NL; ++u) vb[(s + 1) & 1][u] = bsm[((s + 1) * NL + u) * 64 + lane];
            }
#pragma unroll
            for (int u = 0; u < NL; ++u)
                acc[u] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[p], vb[s & 1][u], acc[u], 0, 0, 0);
#pragma unroll
            for (int j = 0; j < NG; ++j)
                acc[NL + j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[p], g[s & 1][j], acc[NL + j], 0, 0, 0);
            // refills: global tiles of step s + 2 (or of the next
            // half-block's first steps), then the ring slot
            if (NG > 0) {
                if (s + 2 < NS) load_g(s + 2, g[s & 1]);
                else if (more) load_g(s + 2 - NS, g[s & 1]);
            }
            if (s + P < NS) load_a(rs_cur, s + P, a[p]);
            else if (more) load_a(rs_nxt, s + P - NS, a[p]);
            __builtin_amdgcn_sched_barrier(0);   // keep each step's loads in its step
        }
        if (more) load_meta(nxt);
        // Epilogue.  Pre-test of every pair, one compare per accumulator:
        // s_v * dot >= thq, thq from the half-block's largest norms with a
        // margin for the rounding of both products (invisible rows carry a
        // NaN scale and never pass).  The compare's lane mask places the
        // passing pairs in a list of 64 in LDS (accumulator rows, then
        // tiles, then lanes), and each full list takes the exact interval
        // test densely, one pair per lane, so the divergent per-row exact
        // test of a sparse pass pattern is never run.
        float svr[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) svr[r] = meta[8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)];
        float thq[NQT];
#pragma unroll
        for (int uu = 0; uu < NQT; ++uu) {
            const int b = 32 * uu + (lane & 31);
            const QFields f = s_qf[b];
            ScanQ Q{};
            Q.tau = f.tau;
            Q.sq = f.sq;
            Q.nq = f.nq;
            Q.nqh = f.nqh;
            Q.neq = f.neq;
            Q.wmax = f.wmax;
            const bool valid = b < nq && s_hi > 0.0f;
            thq[uu] = valid ? scaled_threshold(block_threshold(Q, nvb, nevb, gamma), Q.sq) : INFINITY;
        }
        const int sub = static_cast<int>((hb >> 1) & (kSub - 1));
        const uint32_t row_base = static_cast<uint32_t>((hb >> 1) * 64 + 32 * (hb & 1));
        // the exact test of list entries [0, n), 64 at a time
        auto flush = [&](int n) {
            __builtin_amdgcn_wave_barrier();
            for (int c0 = 0; c0 < n; c0 += 64) {
                bool ok = false;
                int32_t dot = 0;
                int rih = 0, qb = 0, half = 0;
                if (c0 + lane < n) {
                    dot = ent[c0 + lane];
                    const int x = ent[CAP + c0 + lane];
                    const int r = x & 15, sl = (x >> 4) & 63;
                    half = sl >> 5;
                    rih = 8 * (r >> 2) + 4 * half + (r & 3);
                    qb = 32 * (x >> 10) + (sl & 31);
                    const QFields f = s_qf[qb];
                    ScanQ Q{};
                    Q.sq = f.sq;
                    Q.nq = f.nq;
                    Q.nqh = f.nqh;
                    Q.neq = f.neq;
                    float lo, hi;
                    pair_interval(Q, meta[rih], meta[32 + rih], meta[64 + rih], dot, gamma, lo, hi);
                    ok = hi >= f.tau && (!f.has_cert || lo <= f.s_cert);
                }
                // records of the upper rows after those of the lower ones,
                // so that the records of one row stay adjacent
                const uint64_t b0 = __ballot(ok && half == 0), b1 = __ballot(ok && half == 1);
                const int n0 = __popcll(b0), tot = n0 + __popcll(b1);
                if (tot) {
                    int base = 0;
                    if (lane == 0) base = atomicAdd(&o.pair_cnt[sub * kCntStride], tot);
                    base = __builtin_amdgcn_readfirstlane(base);
                    if (ok) {
                        const uint64_t bm = half ? b1 : b0;
                        const int pos = base + (half ? n0 : 0) +
                                        static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                                            static_cast<uint32_t>(bm >> 32),
                                            __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(bm), 0u)));
                        if (pos < o.pair_sub)
                            o.pairs[sub * o.pair_sub + pos] = make_uint4(
                                row_base + rih, static_cast<uint32_t>(o.qbase + qb), static_cast<uint32_t>(dot), 0u);
                        atomicAdd(&s_evals[qb], 1);
                    }
                }
            }
            __builtin_amdgcn_wave_barrier();
        };
        int fill = 0;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            if constexpr (kRowCheck) {   // room for the passes of every tile of this row
                if (fill > CAP - 64 * NQT) {
                    flush(fill);
                    fill = 0;
                }
            }
#pragma unroll
            for (int uu = 0; uu < NQT; ++uu) {
                const bool pass = svr[r] * static_cast<float>(acc[uu][r]) >= thq[uu];
                const uint64_t bal = __ballot(pass);
                if (!bal) continue;
                const int n = __popcll(bal);
                if (!kRowCheck && fill + n > CAP) {
                    flush(fill);
                    fill = 0;
                }
                if (pass) {
                    const int pos = fill + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                                               static_cast<uint32_t>(bal >> 32),
                                               __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(bal), 0u)));
                    ent[pos] = acc[uu][r];
                    ent[CAP + pos] = r | (lane << 4) | (uu << 10);
                }
                fill += n;
            }
        }
        if (fill) flush(fill);
    }
    __syncthreads();
    for (int b = tid; b < nq && b < NQT * 32; b += 64 * W)
        if (s_evals[b]) atomicAdd(&o.q_evals[(blockIdx.x & (kSub - 1)) * o.q_ld + o.qbase + b], s_evals[b]);
}

static int cu_count() {
    static int n = 0;
    if (n == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
    }
    return n;
}

// The single-pass kernel for an index of NS K steps (its loop is unrolled
// for them); false when the index has another step count or the kernel
// cannot get its LDS.  EAHR_MFMA_KERNEL=wide (testing) keeps the older
// kernel.
template <int NQT, int NG, int NS, int P, int W>
static bool r1_launch(const IndexView& ix, const uint64_t* vis, int64_t nblocks, const v4i* qfrag,
                      const ScanQ* sq, int32_t nq, float gamma, const ScanOut& o, hipStream_t stream) {
    if (ix.nchunk / 2 != NS) return false;
    if (const char* e = std::getenv("EAHR_MFMA_KERNEL"))
        if (std::strcmp(e, "wide") == 0) return false;
    constexpr size_t lds = static_cast<size_t>(NS) * (NQT - NG) * 1024 + NQT * 32 * sizeof(QFields) +
                           W * 96 * sizeof(float) + NQT * 32 * sizeof(int32_t) +
                           W * 2 * (NQT <= 4 ? 64 * (NQT + 1) : 64) * sizeof(int32_t);
    static std::atomic<int> ready{0};   // 1: LDS attribute set, -1: refused
    if (ready.load() == 0) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_scan_mfma_r1<NQT, NG, NS, P, W>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        ready.store(e == hipSuccess ? 1 : -1);
        if (e != hipSuccess) (void)hipGetLastError();
    }
    if (ready.load() < 0) return false;
    const int64_t groups = (2 * nblocks + W - 1) / W;
    const uint32_t g = static_cast<uint32_t>(std::min<int64_t>(groups, cu_count()));
    hipLaunchKernelGGL((k_scan_mfma_r1<NQT, NG, NS, P, W>), dim3(g), dim3(64 * W), lds, stream, ix.codes, ix.scale,
                       ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qfrag, sq, nq, gamma, o);
    return true;
}

template <int NQT>
static void mfma_pass(const IndexView& ix, const uint64_t* vis, int64_t nblocks, const v4i* qfrag,
                      const ScanQ* sq, int32_t nq, float gamma, bool sample, const ScanOut& o,
                      hipStream_t stream) {
    const int64_t waves = sample ? (nblocks + o.sample_stride - 1) / o.sample_stride : nblocks;
    const uint32_t grid = static_cast<uint32_t>((waves + 3) / 4);
    if constexpr (NQT == 8) {
        // 256 queries, d = 768: six tiles in LDS, two from L2; d = 384: all in LDS
        if (!sample && (r1_launch<8, 2, 24, 6, 8>(ix, vis, nblocks, qfrag, sq, nq, gamma, o, stream) ||
                        r1_launch<8, 0, 12, 6, 8>(ix, vis, nblocks, qfrag, sq, nq, gamma, o, stream)))
            return;
    }
    if constexpr (NQT == 4) {
        if (!sample && (r1_launch<4, 0, 24, 8, 12>(ix, vis, nblocks, qfrag, sq, nq, gamma, o, stream) ||
                        r1_launch<4, 0, 12, 6, 12>(ix, vis, nblocks, qfrag, sq, nq, gamma, o, stream)))
            return;
    }
    if (sample) {
        hipLaunchKernelGGL((k_scan_mfma<NQT, true>), dim3(grid), dim3(256), 0, stream, ix.codes,
                           ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qfrag, sq, nq,
                           gamma, o);
    } else if (NQT >= 4) {
        constexpr int W = NQT >= 4 ? NQT : 4;
        // two workgroups per CU (256 registers per lane each): one's epilogue
        // and barriers overlap the other's MFMA work
        const int64_t groups = (nblocks + 3) / 4;
        const uint32_t g = static_cast<uint32_t>(std::min<int64_t>(groups, 2 * cu_count()));
        const int nsteps = ix.nchunk / 2;
        // four tiles: a four-step stage (243 registers, no spills) keeps twice
        // the code fragments in flight per wavefront and halves the barriers;
        // eight tiles would spill at that depth
        constexpr int PA_DEEP = (W == 4) ? 4 : 2;
        if (PA_DEEP == 4 && nsteps % 4 == 0)
            hipLaunchKernelGGL((k_scan_mfma_wide<W, PA_DEEP>), dim3(g), dim3(256), 0, stream, ix.codes,
                               ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qfrag, sq, nq,
                               gamma, o);
        else if (nsteps % 2 == 0)
            hipLaunchKernelGGL((k_scan_mfma_wide<W, 2>), dim3(g), dim3(256), 0, stream, ix.codes,
                               ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qfrag, sq, nq,
                               gamma, o);
        else
            hipLaunchKernelGGL((k_scan_mfma_wide<W, 1>), dim3(g), dim3(256), 0, stream, ix.codes,
                               ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qfrag, sq, nq,
                               gamma, o);
    } else {
        hipLaunchKernelGGL((k_scan_mfma<NQT, false>), dim3(grid), dim3(256), 0, stream, ix.codes,
                           ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qfrag, sq, nq,
                           gamma, o);
    }
}

// Query tiles of an MFMA pass: one tile up to 32 queries, else the wide
// kernel with 4 or 8 tiles (33-64 queries also take 4 tiles: the wide
// kernel streams the codes faster than the two-tile kernel computes).
int mfma_tiles_for(int32_t nq) {
    const int t = (nq + 31) / 32;
    return t <= 1 ? 1 : t <= 4 ? 4 : 8;
}

void launch_scan_mfma(const IndexView& ix, const uint64_t* vis, int64_t nblocks,
                      const int8_t* qcodes, const ScanQ* sq, int32_t nq, float gamma, bool sample,
                      const ScanOut& o, void* frag, hipStream_t stream) {
    for (int32_t q0 = 0; q0 < nq; q0 += kMaxMfmaQueries) {
        const int32_t n = (nq - q0 < kMaxMfmaQueries) ? (nq - q0) : kMaxMfmaQueries;
        const int nqt = mfma_tiles_for(n);
        const ScanQ* s = sq + q0;
        hipLaunchKernelGGL(k_qfrag, dim3((ix.dp / 32) * nqt), dim3(64), 0, stream, qcodes, ix.dp, s,
                           n, nqt, static_cast<uint4*>(frag));
        const v4i* qf = static_cast<const v4i*>(frag);
        const ScanOut so = shift_out(o, q0);
#define PVS_MFMA_CASE(N)                                                          \
    case N:                                                                       \
        mfma_pass<N>(ix, vis, nblocks, qf, s, n, gamma, sample, so, stream);      \
        break;
        switch (nqt) {
            PVS_MFMA_CASE(1)
            PVS_MFMA_CASE(2)
            PVS_MFMA_CASE(4)
            PVS_MFMA_CASE(8)
            default:
                break;
        }
#undef PVS_MFMA_CASE
    }
}

// ------------------------------------------------------------ threshold
// One workgroup per query: tau = the k-th largest finite value among the
// sampled lower bounds (midpoint == 0) or the sampled interval midpoints
// (lo + hi) / 2 (midpoint == 1), by radix select over order-preserving keys,
// 8 bits per pass below the leading bits that every key shares; -inf when
// fewer than k are finite.  Then sample_hits = sampled pairs with hi >= tau.
__device__ __forceinline__ float select_value(const float* x, const float* y, int64_t i, int midpoint) {
    const float lo = x[i];
    return (midpoint && lo != -INFINITY) ? 0.5f * lo + 0.5f * y[i] : lo;
}

// Calls f(value) for every value of a query's sample (-inf: not finite),
// reading 16 bytes per lane and four of them at a time: one workgroup per
// query cannot hide the latency of 4-byte loads (a single request's select
// ran at about 30 GB/s).  Rows of the sample start 16-byte aligned (they hold
// whole 64-row blocks); a tail of n % 4 values, or a sample that is not
// aligned, is read one value at a time.
template <typename F>
__device__ __forceinline__ void for_values(const float* x, const float* y, int64_t n, int midpoint, F&& f) {
    constexpr int U = 4;
    const float4* x4 = reinterpret_cast<const float4*>(x);
    const float4* y4 = reinterpret_cast<const float4*>(y);
    const bool aligned = ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(y)) & 15u) == 0;
    const int64_t n4 = aligned ? n >> 2 : 0;
    for (int64_t i0 = threadIdx.x; i0 < n4; i0 += static_cast<int64_t>(blockDim.x) * U) {
        float4 a[U], c[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = i0 + static_cast<int64_t>(u) * blockDim.x;
            a[u] = i < n4 ? x4[i] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
            c[u] = (midpoint && i < n4) ? y4[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float lo[4] = {a[u].x, a[u].y, a[u].z, a[u].w};
            const float hi[4] = {c[u].x, c[u].y, c[u].z, c[u].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) f((midpoint && lo[e] != -INFINITY) ? 0.5f * lo[e] + 0.5f * hi[e] : lo[e]);
        }
    }
    for (int64_t i = 4 * n4 + threadIdx.x; i < n; i += blockDim.x) f(select_value(x, y, i, midpoint));
}

__global__ __launch_bounds__(1024) void k_select(const float* __restrict__ sample_lo,
                                                 const float* __restrict__ sample_hi, int64_t n,
                                                 int64_t ld, int midpoint, ScanQ* __restrict__ sq) {
    // 32 copies of the digit histogram, lane l counting into copy l % 32: the
    // keys of one query cluster in a few digits, and updates of one address
    // from many lanes would be applied one at a time (stride 257 puts a
    // digit's copies in different banks)
    constexpr int kCopies = 32, kStride = 257;
    __shared__ uint32_t hist[kCopies * kStride];
    __shared__ uint32_t s_digit;
    __shared__ uint32_t s_rest;
    __shared__ uint32_t s_total;
    __shared__ uint32_t s_hits;
    __shared__ uint32_t s_kmin;
    __shared__ uint32_t s_kmax;
    __shared__ float s_tau;
    const int b = blockIdx.x;
    const float* x = sample_lo + b * ld;
    const float* y = sample_hi + b * ld;
    uint32_t k = static_cast<uint32_t>(sq[b].k);
    if (threadIdx.x == 0) {
        s_total = 0;
        s_hits = 0;
        s_kmin = 0xffffffffu;
        s_kmax = 0u;
    }
    __syncthreads();
    // count, and the smallest and largest key: the bits they share are
    // shared by every key, so the digit passes start below them
    uint32_t local = 0, kmin = 0xffffffffu, kmax = 0u;
    for_values(x, y, n, midpoint, [&](float v) {
        if (v == -INFINITY) return;
        const uint32_t key = mono32(v);
        ++local;
        kmin = key < kmin ? key : kmin;
        kmax = key > kmax ? key : kmax;
    });
    for (int off = 32; off > 0; off >>= 1) {
        local += __shfl_xor(local, off, 64);
        const uint32_t a = __shfl_xor(kmin, off, 64), c = __shfl_xor(kmax, off, 64);
        kmin = a < kmin ? a : kmin;
        kmax = c > kmax ? c : kmax;
    }
    if ((threadIdx.x & 63) == 0) {
        atomicAdd(&s_total, local);
        atomicMin(&s_kmin, kmin);
        atomicMax(&s_kmax, kmax);
    }
    __syncthreads();
    const uint32_t total = s_total;
    if (k == 0 || k > total) {
        if (threadIdx.x == 0) s_tau = -INFINITY;
    } else {
        const uint32_t lo = s_kmin, hi = s_kmax;
        const int common = (lo == hi) ? 32 : __clz(lo ^ hi);
        uint32_t pmask = (common == 32) ? 0xffffffffu : ~(0xffffffffu >> common);
        uint32_t prefix = lo & pmask;
        // the k-th largest key, digit by digit (8 bits, the last one fewer)
        for (int bits = 32 - common; bits > 0;) {
            const int w = bits < 8 ? bits : 8;
            const int shift = bits - w;
            const uint32_t dmask = (1u << w) - 1u;
            for (int i = threadIdx.x; i < kCopies * kStride; i += blockDim.x) hist[i] = 0;
            __syncthreads();
            uint32_t* mine = hist + (threadIdx.x & (kCopies - 1)) * kStride;
            for_values(x, y, n, midpoint, [&](float v) {
                if (v == -INFINITY) return;
                const uint32_t key = mono32(v);
                if ((key & pmask) == prefix) atomicAdd(&mine[(key >> shift) & dmask], 1u);
            });
            __syncthreads();
            for (int d = threadIdx.x; d <= static_cast<int>(dmask); d += blockDim.x) {
                uint32_t c = 0;
                for (int r = 0; r < kCopies; ++r) c += hist[r * kStride + d];
                hist[d] = c;   // copy 0 holds the sums (each d read and written by one thread)
            }
            __syncthreads();
            if (threadIdx.x == 0) {
                uint32_t cum = 0;
                int dgt = static_cast<int>(dmask);
                for (; dgt > 0; --dgt) {
                    if (cum + hist[dgt] >= k) break;
                    cum += hist[dgt];
                }
                s_digit = static_cast<uint32_t>(dgt);
                s_rest = k - cum;
            }
            __syncthreads();
            prefix |= s_digit << shift;
            pmask |= dmask << shift;
            k = s_rest;
            bits -= w;
            __syncthreads();
        }
        if (threadIdx.x == 0) s_tau = unmono32(prefix);
    }
    __syncthreads();
    const float tau = s_tau;
    uint32_t hits = 0;
    for_values(y, y, n, 0, [&](float v) { hits += (v != -INFINITY && v >= tau); });
    atomicAdd(&s_hits, hits);
    __syncthreads();
    if (threadIdx.x == 0) {
        sq[b].tau = tau;
        sq[b].sample_hits = static_cast<int32_t>(s_hits);
    }
}

void launch_select(const float* sample_lo, const float* sample_hi, int64_t n, int64_t ld,
                   bool midpoint, ScanQ* sq, int32_t nq, hipStream_t stream) {
    if (nq <= 0) return;
    hipLaunchKernelGGL(k_select, dim3(nq), dim3(1024), 0, stream, sample_lo, sample_hi, n, ld,
                       midpoint ? 1 : 0, sq);
}

}  // namespace pvs
