// Device-side helpers shared by the PVS kernels.
//
// Numerical contract (Sec. 2.3.1, App. A.1) of every kernel of the library:
//  * quantisation: s = fl32(||v||_inf / 127) (IEEE division), smallest
//    positive float32 if that underflows, 1 for a zero vector;
//    z_j = clamp(roundf(fl32(v_j / s)), -127, 127) (roundf: halves away from 0).
//  * norms are float64 sums, inflated by (1 + 2^-40), stored as the smallest
//    float32 not below that.
//  * interval of (q, v), one float32 rounding per operation (all HIP sources
//    are compiled with -ffp-contract=off, so no operation is fused):
//      c = (s_q * s_v) * float(<z_q, z_v>)
//      E = ||e_q|| * ||v|| + ||q_hat|| * ||e_v||
//      G = ((|c| + E) + ||q|| * ||v||) * gamma_m
//      lo = down(c - (E + G)),  hi = up(c + (E + G))   (one ulp outward)
//  * authoritative float32 score: lane l of a wavefront accumulates
//    q_j * v_j with fmaf over j = 256 t + 4 l + i in (t, i) order, then the
//    64 lane sums are combined by an xor butterfly (offsets 32, 16, .., 1).
//    Every path that reports a score uses row_score below.
#pragma once
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "pvs_kernels.h"

namespace pvs {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

// 16-byte streaming load (codes are read once per scan)
__device__ __forceinline__ u32x4 load_nt(const uint4* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// Order-preserving float -> uint32 map (ascending floats give ascending
// keys); -0 maps like +0.
__device__ __forceinline__ uint32_t mono32(float f) {
    const uint32_t b = __float_as_uint(f + 0.0f);
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

// Conservative pre-test of the scans: hi >= tau implies c >= this value
// (wmax bounds E + G over every row with a relative margin; the extra terms
// absorb the float32 rounding of the comparison itself).
__device__ __forceinline__ float center_threshold(const ScanQ& Q) {
    return Q.tau - Q.wmax * 1.001f - 0x1p-20f * (fabsf(Q.tau) + Q.wmax);
}

// The same pre-test for one block, whose visible rows have norms at most nvb
// (||v||) and nevb (||e_v||): E + G over those rows is bounded as wmax is over
// the index (|c| <= ||q_hat|| (||v|| + ||e_v||)), with a 1 % margin that
// absorbs the float32 rounding of the bound.
__device__ __forceinline__ float block_threshold(const ScanQ& Q, float nvb, float nevb,
                                                 float gamma) {
    const float E = Q.neq * nvb + Q.nqh * nevb;
    const float cb = Q.nqh * (nvb + nevb);
    const float G = (cb + E + Q.nq * nvb) * gamma;
    const float w = fminf((E + G) * 1.01f, Q.wmax);
    return Q.tau - w * 1.001f - 0x1p-20f * (fabsf(Q.tau) + w);
}

// Threshold for fl(s_v * dot) equivalent to `thr` for c = fl(fl(s_q s_v) dot),
// loosened so that c >= thr implies fl(s_v * dot) >= the result: the two
// products differ by at most 3 roundings (relative 2^-22), the margin is
// 2^-20 relative plus an absolute term for results near zero.  A tiny s_q
// (or an overflowing quotient) gives -inf: every pair then takes the exact
// test.
__device__ __forceinline__ float scaled_threshold(float thr, float sq) {
    if (!(sq >= 0x1p-20f)) return -INFINITY;
    const float t = thr / sq;
    const float r = t - fabsf(t) * 0x1p-20f - 0x1p-100f;
    return (r > -INFINITY && r < INFINITY) ? r : -INFINITY;
}

// Authoritative float32 score of one row (fixed order, see the file header).
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

template <int J>
__device__ __forceinline__ void load_query_row(const float4* __restrict__ qrows, int32_t qi,
                                               int df4, int lane, float4 (&qv)[J]) {
#pragma unroll
    for (int t = 0; t < J; ++t) {
        const int idx = 64 * t + lane;
        qv[t] = (idx < df4) ? qrows[static_cast<int64_t>(qi) * df4 + idx] : make_float4(0, 0, 0, 0);
    }
}

// Number of float4 chunks per lane for a row of df floats, rounded to the
// instantiated sizes.
inline int row_chunks(int df) {
    const int j = (df / 4 + 63) / 64;
    return j <= 1 ? 1 : j <= 2 ? 2 : j <= 3 ? 3 : j <= 4 ? 4 : j <= 8 ? 8 : 16;
}

}  // namespace pvs
