// gfx950 kernels of the PVS dense channel.
//
// Numerical contract (Sec. 2.3.1, App. A.1), shared by every kernel here:
//  * quantisation: s = fl32(||v||_inf / 127) (IEEE division), smallest
//    positive float32 if that underflows, 1 for a zero vector;
//    z_j = clamp(roundf(fl32(v_j / s)), -127, 127) (roundf: halves away from 0).
//  * norms are float64 sums, inflated by (1 + 2^-40), stored as the smallest
//    float32 not below that.
//  * interval of (q, v), one float32 rounding per operation (this file is
//    compiled with -ffp-contract=off, so no operation is fused):
//      c = (s_q * s_v) * float(<z_q, z_v>)
//      E = ||e_q|| * ||v|| + ||q_hat|| * ||e_v||
//      G = ((|c| + E) + ||q|| * ||v||) * gamma_m
//      lo = down(c - (E + G)),  hi = up(c + (E + G))   (one ulp outward)
//  * authoritative float32 score: lane l of a wavefront accumulates
//    q_j * v_j with fmaf over j = 256 t + 4 l + i in (t, i) order, then the
//    64 lane sums are combined by an xor butterfly (offsets 32, 16, .., 1).
//    Every path that reports a score uses this one kernel.
#include "pvs_kernels.h"

#include <math.h>

namespace pvs {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte streaming load (codes are read once per scan)
__device__ __forceinline__ u32x4 load_nt(const uint4* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ uint32_t mono32(float f) {
    uint32_t b = __float_as_uint(f + 0.0f);   // -0 -> +0
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float unmono32(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// one ulp towards +inf / -inf (finite input)
__device__ __forceinline__ float next_up(float f) {
    uint32_t b = __float_as_uint(f);
    if (b == 0x80000000u) b = 0u;
    return (static_cast<int32_t>(b) >= 0) ? __uint_as_float(b + 1u) : __uint_as_float(b - 1u);
}
__device__ __forceinline__ float next_down(float f) { return -next_up(-f); }

__device__ __forceinline__ float up32(double x) {
    x = x * (1.0 + 0x1p-40);
    float f = static_cast<float>(x);
    if (static_cast<double>(f) < x) f = next_up(f);
    return f;
}

__device__ __forceinline__ float wave_max(float v) {
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}
__device__ __forceinline__ double wave_sum(double v) {
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ __forceinline__ int8_t code_of(float x, float s) {
    float t = roundf(x / s);
    t = fminf(fmaxf(t, -127.0f), 127.0f);
    return static_cast<int8_t>(static_cast<int>(t));
}

}  // namespace

// ---------------------------------------------------------------- quantise
// One wavefront per row.  Writes codes (chunk-major blocks when `tiled`,
// row-major otherwise), scale, ||v|| up, ||e_v|| up, ||s z|| up and the float32
// row; flags[0] |= 1 on a non-finite value, flags[1..2] = max of the norms.
__global__ __launch_bounds__(256) void k_quantize(
    const float* __restrict__ src, int64_t nrows, int32_t d, int64_t src_stride, int64_t row0,
    int tiled, int8_t* __restrict__ codes, int32_t dp, float* __restrict__ scale,
    float* __restrict__ vnorm, float* __restrict__ enorm, float* __restrict__ hnorm,
    float* __restrict__ rows, int32_t df, uint32_t* __restrict__ flags) {
    const int lane = threadIdx.x & 63;
    const int64_t r = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (r >= nrows) return;
    const float* v = src + r * src_stride;
    float mu = 0.0f;
    bool bad = false;
    for (int j = lane; j < d; j += 64) {
        const float x = v[j];
        bad |= !isfinite(x);
        mu = fmaxf(mu, fabsf(x));
    }
    mu = wave_max(mu);
    const bool any_bad = __any(bad);
    float s = mu / 127.0f;
    if (mu > 0.0f && s == 0.0f) s = __uint_as_float(1u);
    if (mu == 0.0f) s = 1.0f;
    const int64_t R = row0 + r;
    const int nchunk = dp / 16;
    double n2 = 0.0, e2 = 0.0, h2 = 0.0;
    for (int c = lane; c < nchunk; c += 64) {
        uint32_t w[4];
        for (int q = 0; q < 4; ++q) {
            uint32_t packed = 0;
            for (int i = 0; i < 4; ++i) {
                const int j = c * 16 + q * 4 + i;
                const float x = (j < d) ? v[j] : 0.0f;
                const int8_t z = code_of(x, s);
                const double vh = static_cast<double>(s) * static_cast<double>(z);
                const double e = static_cast<double>(x) - vh;
                n2 += static_cast<double>(x) * static_cast<double>(x);
                e2 += e * e;
                h2 += vh * vh;
                packed |= static_cast<uint32_t>(static_cast<uint8_t>(z)) << (8 * i);
            }
            w[q] = packed;
        }
        uint4 out = make_uint4(w[0], w[1], w[2], w[3]);
        uint4* dst;
        if (tiled) {
            dst = reinterpret_cast<uint4*>(codes) + ((R >> 6) * nchunk + c) * 64 + (R & 63);
        } else {
            dst = reinterpret_cast<uint4*>(codes + R * dp) + c;
        }
        *dst = out;
    }
    for (int j = lane; j < df; j += 64) rows[R * df + j] = (j < d) ? v[j] : 0.0f;
    n2 = wave_sum(n2);
    e2 = wave_sum(e2);
    h2 = wave_sum(h2);
    if (lane == 0) {
        const float vn = up32(sqrt(n2));
        const float en = up32(sqrt(e2));
        scale[R] = s;
        vnorm[R] = vn;
        enorm[R] = en;
        if (hnorm) hnorm[R] = up32(sqrt(h2));
        if (any_bad) atomicOr(&flags[0], 1u);
        atomicMax(&flags[1], __float_as_uint(vn));
        atomicMax(&flags[2], __float_as_uint(en));
    }
}

void launch_quantize(const float* src, int64_t nrows, int32_t d, int64_t src_stride, int64_t row0,
                     bool tiled, int8_t* codes, int32_t dp, float* scale, float* vnorm,
                     float* enorm, float* hnorm, float* rows, int32_t df, uint32_t* flags,
                     hipStream_t stream) {
    if (nrows <= 0) return;
    const int64_t grid = (nrows + 3) / 4;
    hipLaunchKernelGGL(k_quantize, dim3(static_cast<uint32_t>(grid)), dim3(256), 0, stream, src,
                       nrows, d, src_stride, row0, tiled ? 1 : 0, codes, dp, scale, vnorm, enorm,
                       hnorm, rows, df, flags);
}

// ------------------------------------------------------------------- scan
// Interval of one (query, row) pair from the exact integer dot product.
__device__ __forceinline__ void pair_interval(const ScanQ& Q, float sv, float nv, float nev,
                                              int dot, float gamma, float& lo, float& hi) {
    const float sqv = Q.sq * sv;
    const float c = sqv * static_cast<float>(dot);
    const float E = Q.neq * nv + Q.nqh * nev;
    const float G = ((fabsf(c) + E) + Q.nq * nv) * gamma;
    const float w = E + G;
    lo = next_down(c - w);
    hi = next_up(c + w);
}

// One wavefront per 64-row block (lane = row); QB queries per pass, their
// codes read through scalar loads.  SAMPLE: every pair of the sampled blocks
// writes its lower bound (or -inf when the row is invisible or already
// certified).  Otherwise rows with hi >= tau that are eligible are appended
// to the query's candidate list with one atomic per wavefront.
template <int QB, bool SAMPLE>
__global__ __launch_bounds__(256) void k_scan_gemv(
    const uint4* __restrict__ codes, const float* __restrict__ scale,
    const float* __restrict__ vnorm, const float* __restrict__ enorm,
    const uint64_t* __restrict__ vis, int64_t nblocks, int32_t nchunk,
    const int8_t* __restrict__ qcodes, int32_t dp, const ScanQ* __restrict__ sq, float gamma,
    int64_t sample_stride, float* __restrict__ sample_lo, int64_t sample_ld,
    int32_t* __restrict__ cand_row, float* __restrict__ cand_lo, float* __restrict__ cand_hi,
    int32_t* __restrict__ cand_cnt, int64_t cap) {
    const int lane = threadIdx.x & 63;
    const int64_t w = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    const int64_t blk = SAMPLE ? w * sample_stride : w;
    if (blk >= nblocks) return;
    const int64_t row = blk * 64 + lane;
    const uint64_t vbits = vis[blk];
    const bool visible = (vbits >> lane) & 1ull;
    const float sv = scale[row];
    const float nv = vnorm[row];
    const float nev = enorm[row];

    const int4* qp[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) qp[b] = reinterpret_cast<const int4*>(qcodes + static_cast<int64_t>(sq[b].qi) * dp);

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
            sample_lo[b * sample_ld + w * 64 + lane] = elig ? lo : -INFINITY;
        } else {
            const bool take = elig && hi >= Q.tau;
            const uint64_t mask = __ballot(take);
            if (mask) {
                const int leader = __ffsll(static_cast<unsigned long long>(mask)) - 1;
                int base = 0;
                if (lane == leader) base = atomicAdd(&cand_cnt[b], __popcll(mask));
                base = __shfl(base, leader, 64);
                if (take) {
                    const int64_t pos = base + __popcll(mask & ((1ull << lane) - 1ull));
                    if (pos < cap) {
                        const int64_t o = static_cast<int64_t>(b) * cap + pos;
                        cand_row[o] = static_cast<int32_t>(row);
                        cand_lo[o] = lo;
                        cand_hi[o] = hi;
                    }
                }
            }
        }
    }
}

template <int QB>
static void scan_pass(const IndexView& ix, const uint64_t* vis, int64_t nblocks,
                      const int8_t* qcodes, const ScanQ* sq, float gamma, bool sample,
                      int64_t sample_stride, float* sample_lo, int64_t sample_ld,
                      int32_t* cand_row, float* cand_lo, float* cand_hi, int32_t* cand_cnt,
                      int64_t cap, hipStream_t stream) {
    const int64_t waves = sample ? (nblocks + sample_stride - 1) / sample_stride : nblocks;
    const uint32_t grid = static_cast<uint32_t>((waves + 3) / 4);
    if (sample) {
        hipLaunchKernelGGL((k_scan_gemv<QB, true>), dim3(grid), dim3(256), 0, stream, ix.codes,
                           ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qcodes, ix.dp,
                           sq, gamma, sample_stride, sample_lo, sample_ld, cand_row, cand_lo,
                           cand_hi, cand_cnt, cap);
    } else {
        hipLaunchKernelGGL((k_scan_gemv<QB, false>), dim3(grid), dim3(256), 0, stream, ix.codes,
                           ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qcodes, ix.dp,
                           sq, gamma, sample_stride, sample_lo, sample_ld, cand_row, cand_lo,
                           cand_hi, cand_cnt, cap);
    }
}

void launch_scan(const IndexView& ix, const uint64_t* vis, int64_t nblocks, const int8_t* qcodes,
                 const ScanQ* sq, int32_t nq, float gamma, bool sample, int64_t sample_stride,
                 float* sample_lo, int64_t sample_ld, int32_t* cand_row, float* cand_lo,
                 float* cand_hi, int32_t* cand_cnt, int64_t cap, hipStream_t stream) {
    for (int32_t q0 = 0; q0 < nq; q0 += kMaxGemvQueries) {
        const int qb = (nq - q0 < kMaxGemvQueries) ? (nq - q0) : kMaxGemvQueries;
        const ScanQ* s = sq + q0;
        float* sl = sample_lo ? sample_lo + q0 * sample_ld : nullptr;
        int32_t* cr = cand_row ? cand_row + q0 * cap : nullptr;
        float* cl = cand_lo ? cand_lo + q0 * cap : nullptr;
        float* ch = cand_hi ? cand_hi + q0 * cap : nullptr;
        int32_t* cc = cand_cnt ? cand_cnt + q0 : nullptr;
#define PVS_SCAN_CASE(N)                                                                     \
    case N:                                                                                  \
        scan_pass<N>(ix, vis, nblocks, qcodes, s, gamma, sample, sample_stride, sl, sample_ld, \
                     cr, cl, ch, cc, cap, stream);                                           \
        break;
        switch (qb) {
            PVS_SCAN_CASE(1)
            PVS_SCAN_CASE(2)
            PVS_SCAN_CASE(3)
            PVS_SCAN_CASE(4)
            PVS_SCAN_CASE(5)
            PVS_SCAN_CASE(6)
            PVS_SCAN_CASE(7)
            PVS_SCAN_CASE(8)
            default:
                break;
        }
#undef PVS_SCAN_CASE
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
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

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

// One wavefront per 64-row block and NQT tiles of 32 queries: 2 x NQT
// accumulators of 32 x 32.  Epilogue per (row, query): the centre score is
// compared with tau - wmax first (wmax bounds E + G over every row, with a
// relative margin), and only rows that may reach tau get the exact interval.
template <int NQT, bool SAMPLE>
__global__ __launch_bounds__(256) void k_scan_mfma(
    const uint4* __restrict__ codes, const float* __restrict__ scale,
    const float* __restrict__ vnorm, const float* __restrict__ enorm,
    const uint64_t* __restrict__ vis, int64_t nblocks, int32_t nchunk,
    const v4i* __restrict__ qfrag, const ScanQ* __restrict__ sq, int32_t nq, float gamma,
    int64_t sample_stride, float* __restrict__ sample_lo, int64_t sample_ld,
    int32_t* __restrict__ cand_row, float* __restrict__ cand_lo, float* __restrict__ cand_hi,
    int32_t* __restrict__ cand_cnt, int64_t cap) {
    const int lane = threadIdx.x & 63;
    const int64_t w = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    const int64_t blk = SAMPLE ? w * sample_stride : w;
    if (blk >= nblocks) return;
    v16i acc[2][NQT];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < NQT; ++u) acc[t][u] = v16i{};
    const uint4* A = codes + blk * nchunk * 64 + (lane >> 5) * 64 + (lane & 31);
    const int nsteps = nchunk >> 1;
#pragma unroll 2
    for (int s = 0; s < nsteps; ++s) {
        const u32x4 a0 = load_nt(A + 2 * s * 64);
        const u32x4 a1 = load_nt(A + 2 * s * 64 + 32);
        v4i va0, va1;
        __builtin_memcpy(&va0, &a0, 16);
        __builtin_memcpy(&va1, &a1, 16);
#pragma unroll
        for (int u = 0; u < NQT; ++u) {
            const v4i vb = qfrag[(s * NQT + u) * 64 + lane];
            acc[0][u] = __builtin_amdgcn_mfma_i32_32x32x32_i8(va0, vb, acc[0][u], 0, 0, 0);
            acc[1][u] = __builtin_amdgcn_mfma_i32_32x32x32_i8(va1, vb, acc[1][u], 0, 0, 0);
        }
    }
    const uint64_t vbits = vis[blk];
#pragma unroll
    for (int u = 0; u < NQT; ++u) {
        const int b = 32 * u + (lane & 31);
        if (b >= nq) continue;
        const ScanQ Q = sq[b];
        // conservative pre-test: hi >= tau implies c >= thr
        const float thr = Q.tau - Q.wmax * 1.001f - 0x1p-20f * (fabsf(Q.tau) + Q.wmax);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rib = 32 * t + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                const int64_t row = blk * 64 + rib;
                const int dot = acc[t][u][r];
                const float sv = scale[row];
                if (SAMPLE) {
                    float lo, hi;
                    pair_interval(Q, sv, vnorm[row], enorm[row], dot, gamma, lo, hi);
                    const bool elig = ((vbits >> rib) & 1ull) && (!Q.has_cert || lo <= Q.s_cert);
                    sample_lo[b * sample_ld + w * 64 + rib] = elig ? lo : -INFINITY;
                } else {
                    const float c = (Q.sq * sv) * static_cast<float>(dot);
                    if (c >= thr && ((vbits >> rib) & 1ull)) {
                        float lo, hi;
                        pair_interval(Q, sv, vnorm[row], enorm[row], dot, gamma, lo, hi);
                        if (hi >= Q.tau && (!Q.has_cert || lo <= Q.s_cert)) {
                            const int pos = atomicAdd(&cand_cnt[b], 1);
                            if (pos < cap) {
                                const int64_t o = static_cast<int64_t>(b) * cap + pos;
                                cand_row[o] = static_cast<int32_t>(row);
                                cand_lo[o] = lo;
                                cand_hi[o] = hi;
                            }
                        }
                    }
                }
            }
        }
    }
}

template <int NQT>
static void mfma_pass(const IndexView& ix, const uint64_t* vis, int64_t nblocks, const v4i* qfrag,
                      const ScanQ* sq, int32_t nq, float gamma, bool sample, int64_t sample_stride,
                      float* sample_lo, int64_t sample_ld, int32_t* cand_row, float* cand_lo,
                      float* cand_hi, int32_t* cand_cnt, int64_t cap, hipStream_t stream) {
    const int64_t waves = sample ? (nblocks + sample_stride - 1) / sample_stride : nblocks;
    const uint32_t grid = static_cast<uint32_t>((waves + 3) / 4);
    if (sample) {
        hipLaunchKernelGGL((k_scan_mfma<NQT, true>), dim3(grid), dim3(256), 0, stream, ix.codes,
                           ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qfrag, sq, nq,
                           gamma, sample_stride, sample_lo, sample_ld, cand_row, cand_lo, cand_hi,
                           cand_cnt, cap);
    } else {
        hipLaunchKernelGGL((k_scan_mfma<NQT, false>), dim3(grid), dim3(256), 0, stream, ix.codes,
                           ix.scale, ix.vnorm, ix.enorm, vis, nblocks, ix.nchunk, qfrag, sq, nq,
                           gamma, sample_stride, sample_lo, sample_ld, cand_row, cand_lo, cand_hi,
                           cand_cnt, cap);
    }
}

int mfma_tiles_for(int32_t nq) {
    const int t = (nq + 31) / 32;
    return t <= 1 ? 1 : t <= 2 ? 2 : t <= 4 ? 4 : 8;
}

void launch_scan_mfma(const IndexView& ix, const uint64_t* vis, int64_t nblocks,
                      const int8_t* qcodes, const ScanQ* sq, int32_t nq, float gamma, bool sample,
                      int64_t sample_stride, float* sample_lo, int64_t sample_ld, int32_t* cand_row,
                      float* cand_lo, float* cand_hi, int32_t* cand_cnt, int64_t cap, void* frag,
                      hipStream_t stream) {
    for (int32_t q0 = 0; q0 < nq; q0 += kMaxMfmaQueries) {
        const int32_t n = (nq - q0 < kMaxMfmaQueries) ? (nq - q0) : kMaxMfmaQueries;
        const int nqt = mfma_tiles_for(n);
        const ScanQ* s = sq + q0;
        hipLaunchKernelGGL(k_qfrag, dim3((ix.dp / 32) * nqt), dim3(64), 0, stream, qcodes, ix.dp, s,
                           n, nqt, static_cast<uint4*>(frag));
        const v4i* qf = static_cast<const v4i*>(frag);
        float* sl = sample_lo ? sample_lo + q0 * sample_ld : nullptr;
        int32_t* cr = cand_row ? cand_row + q0 * cap : nullptr;
        float* cl = cand_lo ? cand_lo + q0 * cap : nullptr;
        float* ch = cand_hi ? cand_hi + q0 * cap : nullptr;
        int32_t* cc = cand_cnt ? cand_cnt + q0 : nullptr;
#define PVS_MFMA_CASE(N)                                                                        \
    case N:                                                                                     \
        mfma_pass<N>(ix, vis, nblocks, qf, s, n, gamma, sample, sample_stride, sl, sample_ld, cr, \
                     cl, ch, cc, cap, stream);                                                  \
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
// One workgroup per query: tau = the k-th largest finite sampled lower bound
// (radix select over order-preserving keys, 8 bits per pass); -inf when
// fewer than k are finite.
__global__ __launch_bounds__(1024) void k_select(const float* __restrict__ sample_lo, int64_t n,
                                                 int64_t ld, ScanQ* __restrict__ sq) {
    __shared__ uint32_t hist[256];
    __shared__ uint32_t s_digit;
    __shared__ uint32_t s_rest;
    __shared__ uint32_t s_total;
    const int b = blockIdx.x;
    const float* x = sample_lo + b * ld;
    uint32_t k = static_cast<uint32_t>(sq[b].k);
    if (threadIdx.x == 0) s_total = 0;
    __syncthreads();
    uint32_t local = 0;
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) local += (x[i] != -INFINITY);
    atomicAdd(&s_total, local);
    __syncthreads();
    const uint32_t total = s_total;
    if (k == 0 || k > total) {
        if (threadIdx.x == 0) sq[b].tau = -INFINITY;
        return;
    }
    uint32_t prefix = 0, pmask = 0;
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[i] = 0;
        __syncthreads();
        for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
            const float v = x[i];
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
    if (threadIdx.x == 0) sq[b].tau = unmono32(prefix);
}

void launch_select(const float* sample_lo, int64_t n, int64_t ld, ScanQ* sq, int32_t nq,
                   hipStream_t stream) {
    if (nq <= 0) return;
    hipLaunchKernelGGL(k_select, dim3(nq), dim3(1024), 0, stream, sample_lo, n, ld, sq);
}

// --------------------------------------------------------------- rescoring
// Authoritative float32 score of one row (see the file header for the order).
template <int J>
__device__ __forceinline__ float row_score(const float4* __restrict__ rp, const float4 (&qv)[J],
                                           int lane, int df4) {
    float acc = 0.0f;
#pragma unroll
    for (int t = 0; t < J; ++t) {
        const int idx = 64 * t + lane;
        if (idx < df4) {
            const float4 v = rp[idx];
            acc = fmaf(qv[t].x, v.x, acc);
            acc = fmaf(qv[t].y, v.y, acc);
            acc = fmaf(qv[t].z, v.z, acc);
            acc = fmaf(qv[t].w, v.w, acc);
        }
    }
    for (int off = 32; off > 0; off >>= 1) acc = acc + __shfl_xor(acc, off, 64);
    return acc;
}

// One wavefront per candidate; grid.y = query.  Checks lo <= s32 <= hi,
// drops rows whose key does not follow the last certified key, and writes a
// sort key: certified rows -> (~mono(s32) << 32 | row), others -> (~0 << 32 | row).
template <int J>
__global__ __launch_bounds__(256) void k_rescore(
    const float4* __restrict__ rows, int32_t df4, const float4* __restrict__ qrows,
    const ScanQ* __restrict__ sq, const int32_t* __restrict__ cand_row,
    const float* __restrict__ cand_lo, const float* __restrict__ cand_hi,
    const int32_t* __restrict__ cand_cnt, int64_t cap, uint64_t* __restrict__ keys,
    int32_t* __restrict__ cert_cnt, int32_t* __restrict__ fail) {
    const int lane = threadIdx.x & 63;
    const int b = blockIdx.y;
    const ScanQ Q = sq[b];
    float4 qv[J];
#pragma unroll
    for (int t = 0; t < J; ++t) {
        const int idx = 64 * t + lane;
        qv[t] = (idx < df4) ? qrows[static_cast<int64_t>(Q.qi) * df4 + idx] : make_float4(0, 0, 0, 0);
    }
    const int64_t n = min(static_cast<int64_t>(cand_cnt[b]), cap);
    const int64_t base = static_cast<int64_t>(b) * cap;
    int local_cert = 0;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6); i < n;
         i += static_cast<int64_t>(gridDim.x) * 4) {
        const int32_t row = cand_row[base + i];
        const float s = row_score<J>(rows + static_cast<int64_t>(row) * df4, qv, lane, df4);
        if (lane == 0) {
            const float lo = cand_lo[base + i];
            const float hi = cand_hi[base + i];
            if (!(lo <= s && s <= hi)) fail[b] = 1;
            const bool dropped = Q.has_cert && (s > Q.s_cert || (s == Q.s_cert && row <= Q.id_cert));
            const bool cert = !dropped && s >= Q.tau;
            const uint64_t hiw = cert ? static_cast<uint64_t>(~mono32(s)) : 0xffffffffull;
            keys[base + i] = (hiw << 32) | static_cast<uint32_t>(row);
            local_cert += cert;
        }
    }
    if (lane == 0 && local_cert) atomicAdd(&cert_cnt[b], local_cert);
}

template <int J>
static void rescore_j(const IndexView& ix, const float* qrows, const ScanQ* sq, int32_t nq,
                      const int32_t* cand_row, const float* cand_lo, const float* cand_hi,
                      const int32_t* cand_cnt, int64_t cap, int64_t max_cnt, uint64_t* keys,
                      int32_t* cert_cnt, int32_t* fail, hipStream_t stream) {
    int64_t gx = (max_cnt + 3) / 4;
    if (gx > 4096) gx = 4096;
    if (gx < 1) gx = 1;
    hipLaunchKernelGGL((k_rescore<J>), dim3(static_cast<uint32_t>(gx), nq), dim3(256), 0, stream,
                       reinterpret_cast<const float4*>(ix.rows), ix.df / 4,
                       reinterpret_cast<const float4*>(qrows), sq, cand_row, cand_lo, cand_hi,
                       cand_cnt, cap, keys, cert_cnt, fail);
}

void launch_rescore(const IndexView& ix, const float* qrows, const ScanQ* sq, int32_t nq,
                    const int32_t* cand_row, const float* cand_lo, const float* cand_hi,
                    const int32_t* cand_cnt, int64_t cap, int64_t max_cnt, uint64_t* keys,
                    int32_t* cert_cnt, int32_t* fail, hipStream_t stream) {
    if (nq <= 0 || max_cnt <= 0) return;
    const int j = (ix.df / 4 + 63) / 64;
#define PVS_RS(N) rescore_j<N>(ix, qrows, sq, nq, cand_row, cand_lo, cand_hi, cand_cnt, cap, max_cnt, keys, cert_cnt, fail, stream)
    if (j <= 1) PVS_RS(1);
    else if (j <= 2) PVS_RS(2);
    else if (j <= 3) PVS_RS(3);
    else if (j <= 4) PVS_RS(4);
    else if (j <= 8) PVS_RS(8);
    else PVS_RS(16);
#undef PVS_RS
}

// ------------------------------------------------------------------ sorting
// Ascending sort of every tile of kSortTile keys of every segment (bitonic
// network in LDS; keys past the segment end are padded with ~0 and dropped).
__global__ __launch_bounds__(256) void k_sort_tiles(uint64_t* __restrict__ keys,
                                                    const int32_t* __restrict__ cnt, int64_t cap) {
    __shared__ uint64_t s[kSortTile];
    const int b = blockIdx.y;
    const int64_t n = min(static_cast<int64_t>(cnt[b]), cap);
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kSortTile;
    if (base >= n) return;
    uint64_t* k = keys + static_cast<int64_t>(b) * cap + base;
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

// One merge level: runs of length `run` are merged pairwise.  Keys are unique
// inside a segment, so an element's output slot is its offset in its own run
// plus the number of smaller keys in the partner run (binary search).
__global__ __launch_bounds__(256) void k_merge(const uint64_t* __restrict__ src,
                                               uint64_t* __restrict__ dst,
                                               const int32_t* __restrict__ cnt, int64_t cap,
                                               int64_t run) {
    const int b = blockIdx.y;
    const int64_t n = min(static_cast<int64_t>(cnt[b]), cap);
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= n) return;
    const uint64_t* s = src + static_cast<int64_t>(b) * cap;
    uint64_t* d = dst + static_cast<int64_t>(b) * cap;
    const uint64_t key = s[i];
    const int64_t start = (i / (2 * run)) * (2 * run);
    const int64_t mid = min(start + run, n);
    const int64_t end = min(start + 2 * run, n);
    int64_t lo, hi;
    int64_t own;
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
    while (lo < hi) {
        const int64_t m = (lo + hi) >> 1;
        if (s[m] < key) lo = m + 1;
        else hi = m;
    }
    d[start + own + (lo - first)] = key;
}

uint64_t* launch_segmented_sort(uint64_t* keys, uint64_t* tmp, const int32_t* cnt, int32_t nq,
                                int64_t cap, int64_t max_cnt, hipStream_t stream) {
    if (nq <= 0 || max_cnt <= 0) return keys;
    const int64_t tiles = (max_cnt + kSortTile - 1) / kSortTile;
    hipLaunchKernelGGL(k_sort_tiles, dim3(static_cast<uint32_t>(tiles), nq), dim3(256), 0, stream,
                       keys, cnt, cap);
    uint64_t* a = keys;
    uint64_t* b = tmp;
    for (int64_t run = kSortTile; run < max_cnt; run *= 2) {
        const int64_t g = (max_cnt + 255) / 256;
        hipLaunchKernelGGL(k_merge, dim3(static_cast<uint32_t>(g), nq), dim3(256), 0, stream, a, b,
                           cnt, cap, run);
        uint64_t* t = a;
        a = b;
        b = t;
    }
    return a;
}

// ----------------------------------------------------------------- packing
__global__ __launch_bounds__(256) void k_offsets(const int32_t* __restrict__ cert, int32_t nq,
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
                                              const int32_t* __restrict__ offs, int64_t cap,
                                              uint64_t* __restrict__ packed) {
    const int b = blockIdx.y;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i < cert[b]) packed[offs[b] + i] = keys[static_cast<int64_t>(b) * cap + i];
}

void launch_pack(const uint64_t* keys, const int32_t* cert_cnt, int32_t nq, int64_t cap,
                 int64_t max_cnt, int32_t* offs, uint64_t* packed, hipStream_t stream) {
    if (nq <= 0) return;
    hipLaunchKernelGGL(k_offsets, dim3(1), dim3(256), 0, stream, cert_cnt, nq, offs);
    if (max_cnt <= 0) return;
    const int64_t g = (max_cnt + 255) / 256;
    hipLaunchKernelGGL(k_pack, dim3(static_cast<uint32_t>(g), nq), dim3(256), 0, stream, keys,
                       cert_cnt, offs, cap, packed);
}

// ----------------------------------------------------------- debug paths
// Intervals of one query against listed rows, by the scan's own arithmetic
// (one wavefront per row, lanes split the code bytes, integer sum exact).
__global__ __launch_bounds__(256) void k_intervals(const uint4* __restrict__ codes,
                                                   const float* __restrict__ scale,
                                                   const float* __restrict__ vnorm,
                                                   const float* __restrict__ enorm, int32_t nchunk,
                                                   const int8_t* __restrict__ qcodes, int32_t dp,
                                                   const ScanQ* __restrict__ sq, float gamma,
                                                   const int64_t* __restrict__ rows, int64_t n,
                                                   float* __restrict__ lo, float* __restrict__ hi) {
    const int lane = threadIdx.x & 63;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (i >= n) return;
    const int64_t r = rows[i];
    const ScanQ Q = sq[0];
    const int4* qp = reinterpret_cast<const int4*>(qcodes + static_cast<int64_t>(Q.qi) * dp);
    int acc = 0;
    for (int c = lane; c < nchunk; c += 64) {
        const uint4 x = codes[((r >> 6) * nchunk + c) * 64 + (r & 63)];
        const int4 qc = qp[c];
        acc = __builtin_amdgcn_sdot4(static_cast<int>(x.x), qc.x, acc, false);
        acc = __builtin_amdgcn_sdot4(static_cast<int>(x.y), qc.y, acc, false);
        acc = __builtin_amdgcn_sdot4(static_cast<int>(x.z), qc.z, acc, false);
        acc = __builtin_amdgcn_sdot4(static_cast<int>(x.w), qc.w, acc, false);
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (lane == 0) {
        float l, h;
        pair_interval(Q, scale[r], vnorm[r], enorm[r], acc, gamma, l, h);
        lo[i] = l;
        hi[i] = h;
    }
}

void launch_intervals(const IndexView& ix, const int8_t* qcodes, const ScanQ* sq, float gamma,
                      const int64_t* rows, int64_t n, float* lo, float* hi, hipStream_t stream) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_intervals, dim3(static_cast<uint32_t>((n + 3) / 4)), dim3(256), 0, stream,
                       ix.codes, ix.scale, ix.vnorm, ix.enorm, ix.nchunk, qcodes, ix.dp, sq, gamma,
                       rows, n, lo, hi);
}

template <int J>
__global__ __launch_bounds__(256) void k_scores(const float4* __restrict__ rows, int32_t df4,
                                                const float4* __restrict__ qrows, int32_t qi,
                                                const int64_t* __restrict__ ids, int64_t n,
                                                float* __restrict__ out) {
    const int lane = threadIdx.x & 63;
    float4 qv[J];
#pragma unroll
    for (int t = 0; t < J; ++t) {
        const int idx = 64 * t + lane;
        qv[t] = (idx < df4) ? qrows[static_cast<int64_t>(qi) * df4 + idx] : make_float4(0, 0, 0, 0);
    }
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6); i < n;
         i += static_cast<int64_t>(gridDim.x) * 4) {
        const float s = row_score<J>(rows + ids[i] * df4, qv, lane, df4);
        if (lane == 0) out[i] = s;
    }
}

void launch_scores(const IndexView& ix, const float* qrows, int32_t qi, const int64_t* rows,
                   int64_t n, float* out, hipStream_t stream) {
    if (n <= 0) return;
    int64_t g = (n + 3) / 4;
    if (g > 65536) g = 65536;
    const int j = (ix.df / 4 + 63) / 64;
    const float4* r4 = reinterpret_cast<const float4*>(ix.rows);
    const float4* q4 = reinterpret_cast<const float4*>(qrows);
    const dim3 grid(static_cast<uint32_t>(g));
    if (j <= 1) hipLaunchKernelGGL(k_scores<1>, grid, dim3(256), 0, stream, r4, ix.df / 4, q4, qi, rows, n, out);
    else if (j <= 2) hipLaunchKernelGGL(k_scores<2>, grid, dim3(256), 0, stream, r4, ix.df / 4, q4, qi, rows, n, out);
    else if (j <= 3) hipLaunchKernelGGL(k_scores<3>, grid, dim3(256), 0, stream, r4, ix.df / 4, q4, qi, rows, n, out);
    else if (j <= 4) hipLaunchKernelGGL(k_scores<4>, grid, dim3(256), 0, stream, r4, ix.df / 4, q4, qi, rows, n, out);
    else if (j <= 8) hipLaunchKernelGGL(k_scores<8>, grid, dim3(256), 0, stream, r4, ix.df / 4, q4, qi, rows, n, out);
    else hipLaunchKernelGGL(k_scores<16>, grid, dim3(256), 0, stream, r4, ix.df / 4, q4, qi, rows, n, out);
}

// ------------------------------------------------------------- visibility
__global__ __launch_bounds__(256) void k_set_bits(uint64_t* __restrict__ vis, int64_t first,
                                                  int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= n) return;
    const int64_t r = first + i;
    atomicOr(reinterpret_cast<unsigned long long*>(&vis[r >> 6]), 1ull << (r & 63));
}

__global__ __launch_bounds__(256) void k_clear_ids(uint64_t* __restrict__ vis,
                                                   const int64_t* __restrict__ ids, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= n) return;
    const int64_t r = ids[i];
    atomicAnd(reinterpret_cast<unsigned long long*>(&vis[r >> 6]), ~(1ull << (r & 63)));
}

__global__ __launch_bounds__(256) void k_popcount(const uint64_t* __restrict__ vis, int64_t nwords,
                                                  unsigned long long* __restrict__ out) {
    unsigned long long c = 0;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < nwords;
         i += static_cast<int64_t>(gridDim.x) * 256)
        c += __popcll(vis[i]);
    for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off, 64);
    if ((threadIdx.x & 63) == 0 && c) atomicAdd(out, c);
}

void launch_set_bits(uint64_t* vis, int64_t first, int64_t n, hipStream_t stream) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_set_bits, dim3(static_cast<uint32_t>((n + 255) / 256)), dim3(256), 0,
                       stream, vis, first, n);
}
void launch_clear_ids(uint64_t* vis, const int64_t* ids, int64_t n, hipStream_t stream) {
    if (n <= 0) return;
    hipLaunchKernelGGL(k_clear_ids, dim3(static_cast<uint32_t>((n + 255) / 256)), dim3(256), 0,
                       stream, vis, ids, n);
}
void launch_popcount(const uint64_t* vis, int64_t nwords, unsigned long long* out,
                     hipStream_t stream) {
    int64_t g = (nwords + 255) / 256;
    if (g > 1024) g = 1024;
    if (g < 1) g = 1;
    hipLaunchKernelGGL(k_popcount, dim3(static_cast<uint32_t>(g)), dim3(256), 0, stream, vis,
                       nwords, out);
}

}  // namespace pvs
