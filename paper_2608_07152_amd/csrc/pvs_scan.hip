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

#include "pvs_device.h"

namespace pvs {

// ------------------------------------------------------------------- GEMV
// One wavefront per 64-row block (lane = row); QB queries per pass, their
// codes read through scalar loads.  Appends use one atomic per wavefront and
// query (ballot + prefix count) on the counter of sub-region blk % kSub.
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
        } else {
            const bool take = elig && hi >= Q.tau;
            const uint64_t mask = __ballot(take);
            if (mask) {
                const int sub = static_cast<int>(blk & (kSub - 1));
                const int leader = __ffsll(static_cast<unsigned long long>(mask)) - 1;
                int base = 0;
                if (lane == leader)
                    base = atomicAdd(&o.cand_cnt[(b * kSub + sub) * kCntStride], __popcll(mask));
                base = __shfl(base, leader, 64);
                if (take) {
                    const int64_t pos = base + __popcll(mask & ((1ull << lane) - 1ull));
                    if (pos < Q.cand_cap) {
                        const int64_t at = Q.cand_off + sub * Q.cand_cap + pos;
                        o.cand[at] = make_uint2(static_cast<uint32_t>(row), static_cast<uint32_t>(acc[b]));
                    }
                }
            }
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
    if (s.cand_cnt) s.cand_cnt += static_cast<int64_t>(q0) * kSub * kCntStride;
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
// l ^ 32 (same query) reserve their slots with one atomic.
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
#pragma unroll
    for (int uu = 0; uu < NQS; ++uu) {
        const int u = u0 + uu;
        const int b = 32 * u + (lane & 31);
        const bool valid = b < nq;
        const ScanQ Q = sq[valid ? b : 0];
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
        uint32_t mask = 0;
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
                    if (hi >= Q.tau && (!Q.has_cert || lo <= Q.s_cert)) mask |= 1u << (16 * t + r);
                }
            }
        }
        const int mine = __popc(mask);
        const int other = __shfl_xor(mine, 32, 64);
        const int sub = static_cast<int>(blk & (kSub - 1));
        int base = 0;
        if (lane < 32 && mine + other > 0)
            base = atomicAdd(&o.cand_cnt[(b * kSub + sub) * kCntStride], mine + other);
        base = __shfl(base, lane & 31, 64);
        if (!mask) continue;
        int64_t pos = base + ((lane >= 32) ? other : 0);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                if (!((mask >> (16 * t + r)) & 1u)) continue;
                const int rib = 32 * t + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                const int64_t row = blk * 64 + rib;
                if (pos < Q.cand_cap) {
                    const int64_t at = Q.cand_off + sub * Q.cand_cap + pos;
                    o.cand[at] = make_uint2(static_cast<uint32_t>(row), static_cast<uint32_t>(acc[t][uu][r]));
                }
                ++pos;
            }
        }
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
// carry a NaN scale so they fail it.  Candidates are appended through chunks
// of sub-region blockIdx.x % kSub of each query's region that the workgroup
// reserves with one global atomic per chunk; slots of a chunk left unused at
// the end hold the sentinel row -1, which the sub-region's count includes and
// rescoring skips.
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
    __shared__ int32_t s_wcnt[4][NQS * 32];    // per wave counts, then offsets
    __shared__ int32_t s_pos[NQT * 32];        // next free slot of each query's chunk
    __shared__ int32_t s_end[NQT * 32];        // end of that chunk
    __shared__ int32_t s_old[NQS * 32], s_room[NQS * 32], s_new[NQS * 32];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int sub = static_cast<int>(blockIdx.x & (kSub - 1));
    // workgroups sharing one sub-region
    const int64_t wg_per_sub = (static_cast<int64_t>(gridDim.x) + kSub - 1) / kSub;
    for (int b = tid; b < NQT * 32; b += 256) {
        s_pos[b] = s_end[b] = 0;
        if (b < nq) s_q[b] = sq[b];
    }
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
            // Rows run outermost so a row's scale is read once for the 4
            // tiles; the per-pair pre-test is one convert, one multiply and
            // one compare against the block threshold divided by s_q (with a
            // margin that covers the rounding of both products), and only
            // pairs that pass it evaluate the exact interval.
            uint32_t mask[NQS];
            int other[NQS];
            float thq[NQS];
#pragma unroll
            for (int uu = 0; uu < NQS; ++uu) {
                mask[uu] = 0;
                const int b = 32 * (u0 + uu) + (lane & 31);
                thq[uu] = INFINITY;
                if (have && b < nq) {
                    const ScanQ& Q = s_q[b];
                    thq[uu] = scaled_threshold(block_threshold(Q, nvb, nevb, gamma), Q.sq);
                }
            }
#pragma unroll
            for (int t = 0; t < 2; ++t) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int rib = 32 * t + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                    const float sv = s_meta[wave][0][rib];   // NaN for invisible rows
#pragma unroll
                    for (int uu = 0; uu < NQS; ++uu) {
                        if (sv * static_cast<float>(acc[t][uu][r]) >= thq[uu]) {
                            const ScanQ& Q = s_q[32 * (u0 + uu) + (lane & 31)];
                            float lo, hi;
                            pair_interval(Q, sv, s_meta[wave][1][rib], s_meta[wave][2][rib],
                                          acc[t][uu][r], gamma, lo, hi);
                            if (hi >= Q.tau && (!Q.has_cert || lo <= Q.s_cert))
                                mask[uu] |= 1u << (16 * t + r);
                        }
                    }
                }
            }
#pragma unroll
            for (int uu = 0; uu < NQS; ++uu) {
                const int mine = __popc(mask[uu]);
                other[uu] = __shfl_xor(mine, 32, 64);
                if (lane < 32) s_wcnt[wave][32 * uu + lane] = mine + other[uu];
            }
            __syncthreads();
            // one thread per query: wave offsets, and a new chunk of the
            // query's region when the current one is too small
            if (tid < NQS * 32) {
                const int b = 32 * u0 + tid;
                int tot = 0;
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const int c = s_wcnt[w][tid];
                    s_wcnt[w][tid] = tot;
                    tot += c;
                }
                const int old = s_pos[b];
                const int room = s_end[b] - old;
                int nb = 0;
                if (tot > room) {
                    const int need = tot - room;
                    const int64_t cap = s_q[b].cand_cap;
                    const int64_t per = cap / (16 * wg_per_sub);
                    const int chunk = static_cast<int>(per < 1 ? 1 : per > kMaxChunk ? kMaxChunk : per);
                    const int take = need > chunk ? need : chunk;
                    nb = atomicAdd(&o.cand_cnt[(b * kSub + sub) * kCntStride], take);
                    s_pos[b] = nb + need;
                    s_end[b] = nb + take;
                } else {
                    s_pos[b] = old + tot;
                }
                s_old[tid] = old;
                s_room[tid] = room;
                s_new[tid] = nb;
            }
            __syncthreads();
            if (have) {
#pragma unroll
                for (int uu = 0; uu < NQS; ++uu) {
                    if (!mask[uu]) continue;
                    const int ql = 32 * uu + (lane & 31);
                    const ScanQ& Q = s_q[32 * u0 + ql];
                    const int old = s_old[ql], room = s_room[ql], nb = s_new[ql];
                    int j = s_wcnt[wave][ql] + ((lane >= 32) ? other[uu] : 0);
#pragma unroll
                    for (int t = 0; t < 2; ++t) {
#pragma unroll
                        for (int r = 0; r < 16; ++r) {
                            if (!((mask[uu] >> (16 * t + r)) & 1u)) continue;
                            const int rib = 32 * t + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                            const int64_t row = blk * 64 + rib;
                            const int64_t pos = (j < room) ? old + j : nb + (j - room);
                            if (pos < Q.cand_cap) {
                                const int64_t at = Q.cand_off + sub * Q.cand_cap + pos;
                                o.cand[at] = make_uint2(static_cast<uint32_t>(row),
                                                        static_cast<uint32_t>(acc[t][uu][r]));
                            }
                            ++j;
                        }
                    }
                }
            }
            __syncthreads();   // bsm, the metadata and the chunk tables are reused next
        }
    }
    // unused tails of this workgroup's chunks become sentinel rows (-1)
    for (int b = tid; b < NQT * 32 && b < nq; b += 256) {
        const ScanQ Q = sq[b];
        const int64_t e = s_end[b] < Q.cand_cap ? s_end[b] : Q.cand_cap;
        for (int64_t p = s_pos[b]; p < e; ++p) o.cand[Q.cand_off + sub * Q.cand_cap + p] = make_uint2(0xffffffffu, 0u);
    }
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

template <int NQT>
static void mfma_pass(const IndexView& ix, const uint64_t* vis, int64_t nblocks, const v4i* qfrag,
                      const ScanQ* sq, int32_t nq, float gamma, bool sample, const ScanOut& o,
                      hipStream_t stream) {
    const int64_t waves = sample ? (nblocks + o.sample_stride - 1) / o.sample_stride : nblocks;
    const uint32_t grid = static_cast<uint32_t>((waves + 3) / 4);
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
        if (nsteps % 2 == 0)
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

// ------------------------------------------------------ candidate totals
// One wavefront per query, lane s reads the counter of sub-region s.
__global__ __launch_bounds__(64) void k_cand_totals(const int32_t* __restrict__ sub_cnt,
                                                    const ScanQ* __restrict__ sq,
                                                    int32_t* __restrict__ total,
                                                    int32_t* __restrict__ need) {
    static_assert(kSub == 64, "one lane per sub-region");
    const int b = blockIdx.x;
    const int lane = threadIdx.x;
    const int c = sub_cnt[(b * kSub + lane) * kCntStride];
    const int64_t cap = sq[b].cand_cap;
    int kept = static_cast<int>(c < cap ? c : cap);
    int mx = c;
    for (int off = 32; off > 0; off >>= 1) {
        kept += __shfl_xor(kept, off, 64);
        mx = max(mx, __shfl_xor(mx, off, 64));
    }
    if (lane == 0) {
        total[b] = kept;
        need[b] = mx;
    }
}

void launch_cand_totals(const int32_t* sub_cnt, const ScanQ* sq, int32_t nq, int32_t* total,
                        int32_t* need, hipStream_t stream) {
    if (nq <= 0) return;
    hipLaunchKernelGGL(k_cand_totals, dim3(nq), dim3(64), 0, stream, sub_cnt, sq, total, need);
}

// ------------------------------------------------------------ threshold
// One workgroup per query: tau = the k-th largest finite value among the
// sampled lower bounds (midpoint == 0) or the sampled interval midpoints
// (lo + hi) / 2 (midpoint == 1), by radix select over order-preserving keys,
// 8 bits per pass; -inf when fewer than k are finite.  Then sample_hits =
// sampled pairs with hi >= tau.
__device__ __forceinline__ float select_value(const float* x, const float* y, int64_t i, int midpoint) {
    const float lo = x[i];
    return (midpoint && lo != -INFINITY) ? 0.5f * lo + 0.5f * y[i] : lo;
}

__global__ __launch_bounds__(1024) void k_select(const float* __restrict__ sample_lo,
                                                 const float* __restrict__ sample_hi, int64_t n,
                                                 int64_t ld, int midpoint, ScanQ* __restrict__ sq) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t s_digit;
    __shared__ uint32_t s_rest;
    __shared__ uint32_t s_total;
    __shared__ uint32_t s_hits;
    __shared__ float s_tau;
    const int b = blockIdx.x;
    const float* x = sample_lo + b * ld;
    const float* y = sample_hi + b * ld;
    uint32_t k = static_cast<uint32_t>(sq[b].k);
    if (threadIdx.x == 0) {
        s_total = 0;
        s_hits = 0;
    }
    __syncthreads();
    uint32_t local = 0;
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) local += (x[i] != -INFINITY);
    atomicAdd(&s_total, local);
    __syncthreads();
    const uint32_t total = s_total;
    if (k == 0 || k > total) {
        if (threadIdx.x == 0) s_tau = -INFINITY;
    } else {
        uint32_t prefix = 0, pmask = 0;
        for (int pass = 0; pass < 4; ++pass) {
            const int shift = 24 - 8 * pass;
            for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[i] = 0;
            __syncthreads();
            for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
                const float v = select_value(x, y, i, midpoint);
                if (v == -INFINITY) continue;
                const uint32_t key = mono32(v);
                if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
            }
            __syncthreads();
            if (threadIdx.x == 0) {
                uint32_t cum = 0;
                int dgt = 255;
                for (; dgt > 0; --dgt) {
                    if (cum + hist[dgt] >= k) break;
                    cum += hist[dgt];
                }
                s_digit = static_cast<uint32_t>(dgt);
                s_rest = k - cum;
            }
            __syncthreads();
            prefix |= s_digit << shift;
            pmask |= 255u << shift;
            k = s_rest;
            __syncthreads();
        }
        if (threadIdx.x == 0) s_tau = unmono32(prefix);
    }
    __syncthreads();
    const float tau = s_tau;
    uint32_t hits = 0;
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) hits += (y[i] != -INFINITY && y[i] >= tau);
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
