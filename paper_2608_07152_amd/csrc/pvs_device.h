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
//  * authoritative float32 score: a group of 16 lanes scores one row.  Lane
//    j of the group takes the float4 chunks c = 16 t + j (t = 0, 1, .. while
//    c < df / 4) of the row and of the query and accumulates their products
//    with fmaf in (t, x, y, z, w) order; the 16 lane sums are then added as a
//    balanced pairwise tree: partners j ^ 1, then j ^ 2, j ^ 4, j ^ 8.
//    Every path that reports a score uses group_dot / group_score_seg below.
#pragma once
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <utility>

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

// Sum of the 16 lanes of every row of the wavefront as a pairwise tree:
// partners j ^ 1 and j ^ 2 (quad permutations), then the lane mirrored
// within 8 and within 16 lanes, which after the earlier steps hold the same
// values as j ^ 4 and j ^ 8.  Float addition is commutative, so both
// partners of a pair compute the same bits and every lane of the row ends
// with the row's sum.
__device__ __forceinline__ float sum16(float a) {
    a = a + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(a), 0xB1, 0xF, 0xF, false));
    a = a + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(a), 0x4E, 0xF, 0xF, false));
    a = a + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(a), 0x141, 0xF, 0xF, false));
    a = a + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(a), 0x140, 0xF, 0xF, false));
    return a;
}

// Lane I of every row of 16 lanes, broadcast to its row.
template <int I>
__device__ __forceinline__ int32_t bcast16(int32_t x) {
    return __builtin_amdgcn_update_dpp(0, x, 0x150 + I, 0xF, 0xF, false);
}

// f(integral_constant<int, I>) for I = 0 .. N - 1 (compile-time indices).
template <typename F, int... Is>
__device__ __forceinline__ void static_for(F&& f, std::integer_sequence<int, Is...>) {
    (f(std::integral_constant<int, Is>{}), ...);
}

// Chunks per lane of a 16-lane group for a row of df floats, rounded to the
// instantiated sizes; 0 for rows longer than 16 * kSegChunks chunks, which
// are scored in segments.  FULL instantiations are for df / 4 == 16 * J.
constexpr int kSegChunks = 16;
inline int group_chunks(int df) {
    const int j = (df / 4 + 15) / 16;
    return j <= 1 ? 1 : j <= 2 ? 2 : j <= 3 ? 3 : j <= 4 ? 4 : j <= 6 ? 6 : j <= 8 ? 8 : j <= 12 ? 12 : j <= 16 ? 16 : 0;
}

// The chunks of lane j of a group (zeros past the row's end).
template <int J, bool FULL>
__device__ __forceinline__ void load_chunks(const float4* __restrict__ base, int j, int df4, float4 (&dst)[J]) {
#pragma unroll
    for (int t = 0; t < J; ++t) {
        const int c = 16 * t + j;
        dst[t] = (FULL || c < df4) ? base[c] : make_float4(0, 0, 0, 0);
    }
}

// Authoritative score of a row held by a group (its chunks in v, the
// query's in q), in the fixed order of the file header.
template <int J, bool FULL>
__device__ __forceinline__ float group_dot(const float4 (&v)[J], const float4 (&q)[J], int j, int df4) {
    float acc = 0.0f;
#pragma unroll
    for (int t = 0; t < J; ++t) {
        if (FULL || 16 * t + j < df4) {
            acc = fmaf(q[t].x, v[t].x, acc);
            acc = fmaf(q[t].y, v[t].y, acc);
            acc = fmaf(q[t].z, v[t].z, acc);
            acc = fmaf(q[t].w, v[t].w, acc);
        }
    }
    return sum16(acc);
}

// The same score for rows longer than 16 * kSegChunks chunks: segments of
// kSegChunks chunks per lane, loaded and accumulated one after another.
__device__ __forceinline__ float group_score_seg(const float4* __restrict__ rp, const float4* __restrict__ qp,
                                                 int j, int df4) {
    float acc = 0.0f;
    for (int c0 = 0; c0 < df4; c0 += 16 * kSegChunks) {
        float4 v[kSegChunks], q[kSegChunks];
#pragma unroll
        for (int t = 0; t < kSegChunks; ++t) {
            const int c = c0 + 16 * t + j;
            v[t] = c < df4 ? rp[c] : make_float4(0, 0, 0, 0);
            q[t] = c < df4 ? qp[c] : make_float4(0, 0, 0, 0);
        }
#pragma unroll
        for (int t = 0; t < kSegChunks; ++t) {
            if (c0 + 16 * t + j < df4) {
                acc = fmaf(q[t].x, v[t].x, acc);
                acc = fmaf(q[t].y, v[t].y, acc);
                acc = fmaf(q[t].z, v[t].z, acc);
                acc = fmaf(q[t].w, v[t].w, acc);
            }
        }
    }
    return sum16(acc);
}

}  // namespace pvs
