// Quantisation, visibility, exhaustive float32 scoring and debug kernels of
// the PVS dense channel (Sec. 2.3.1).  The numerical contract is stated in
// pvs_device.h.
#include "pvs_device.h"

namespace pvs {

// ---------------------------------------------------------------- quantise
// One wavefront per row.  Writes codes (chunk-major 64-row blocks when
// `tiled`, row-major otherwise), scale, ||v|| up, ||e_v|| up, ||s z|| up and
// the float32 row; flags[0] |= 1 on a non-finite value, flags[1..2] = max of
// the two norms (as float bits, which order like the values for x >= 0).
__global__ __launch_bounds__(256) void k_quantize(
    const float* __restrict__ src, int64_t nrows, int32_t d, int64_t src_stride, int64_t row0,
    int tiled, int8_t* __restrict__ codes, int32_t dp, float* __restrict__ scale,
    float* __restrict__ vnorm, float* __restrict__ enorm, float* __restrict__ hnorm,
    float* __restrict__ rows, int32_t df, float fixed_s, uint32_t* __restrict__ flags) {
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
    if (fixed_s > 0.0f) s = fixed_s;   // one scale for every row (global scalar quantisation)
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
        const uint4 out = make_uint4(w[0], w[1], w[2], w[3]);
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
                     float* enorm, float* hnorm, float* rows, int32_t df, float fixed_s,
                     uint32_t* flags, hipStream_t stream) {
    if (nrows <= 0) return;
    const int64_t grid = (nrows + 3) / 4;
    hipLaunchKernelGGL(k_quantize, dim3(static_cast<uint32_t>(grid)), dim3(256), 0, stream, src,
                       nrows, d, src_stride, row0, tiled ? 1 : 0, codes, dp, scale, vnorm, enorm,
                       hnorm, rows, df, fixed_s, flags);
}

// Largest |x| over count floats (atomic max of the float's bits into flags[3],
// valid for non-negative floats) and a non-finite flag in flags[0].
__global__ __launch_bounds__(256) void k_maxabs(const float* __restrict__ src, int64_t count,
                                                uint32_t* __restrict__ flags) {
    float mu = 0.0f;
    bool bad = false;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < count; i += stride) {
        const float x = src[i];
        bad |= !isfinite(x);
        mu = fmaxf(mu, fabsf(x));
    }
    mu = wave_max(mu);
    const bool any_bad = __any(bad);
    if ((threadIdx.x & 63) == 0) {
        if (any_bad) atomicOr(&flags[0], 1u);
        atomicMax(&flags[3], __float_as_uint(mu));
    }
}

void launch_maxabs(const float* src, int64_t count, uint32_t* flags, hipStream_t stream) {
    if (count <= 0) return;
    const int64_t blocks = std::min<int64_t>((count + 255) / 256, 4096);
    hipLaunchKernelGGL(k_maxabs, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0, stream, src,
                       count, flags);
}

// ------------------------------------------------------- exhaustive scoring
// The exhaustive float32 generator (the "full float32 scan" alternative of
// Sec. 4.4, Table 4-1): every row of the epoch gets its authoritative score in
// the fixed order of group_dot, so each key equals the one rescoring would
// write; rows not visible get the key ~0, which sorts after every real key.
// One 16-lane group per row (four rows per wavefront, 256 contiguous bytes
// per group and load), the query row in registers; blockIdx.y selects the
// query of the group.
template <int J, bool FULL>
__global__ __launch_bounds__(256) void k_full_keys(const float* __restrict__ rows, int32_t df,
                                                   const uint64_t* __restrict__ vis, int64_t n_rows,
                                                   const float* __restrict__ qrows,
                                                   const int32_t* __restrict__ qidx,
                                                   uint64_t* __restrict__ keys, int64_t ld) {
    const int j = threadIdx.x & 15;
    const int df4 = df / 4;
    const float4* qp = reinterpret_cast<const float4*>(qrows) + static_cast<int64_t>(qidx[blockIdx.y]) * df4;
    float4 q[J > 0 ? J : 1];
    if constexpr (J > 0) load_chunks<J, FULL>(qp, j, df4, q);
    uint64_t* out = keys + static_cast<int64_t>(blockIdx.y) * ld;
    const int64_t ng = static_cast<int64_t>(gridDim.x) * 16;
    for (int64_t r = static_cast<int64_t>(blockIdx.x) * 16 + (threadIdx.x >> 4); r < n_rows; r += ng) {
        if (!((vis[r >> 6] >> (r & 63)) & 1ull)) {   // the same in every lane of the group
            if (j == 0) out[r] = ~0ull;
            continue;
        }
        const float4* rp = reinterpret_cast<const float4*>(rows + r * df);
        float sc;
        if constexpr (J > 0) {
            float4 v[J];
            load_chunks<J, FULL>(rp, j, df4, v);
            sc = group_dot<J, FULL>(v, q, j, df4);
        } else {
            sc = group_score_seg(rp, qp, j, df4);
        }
        if (j == 0) out[r] = (static_cast<uint64_t>(~mono32(sc)) << 32) | static_cast<uint32_t>(r);
    }
}

// Instantiations of a group kernel for the chunk count of df floats.
#define PVS_GROUP_SWITCH(df, CASE)                 \
    do {                                           \
        const int J_ = group_chunks(df);           \
        const bool full_ = J_ > 0 && (df) / 4 == 16 * J_; \
        switch (J_) {                              \
            CASE(1)                                \
            CASE(2)                                \
            CASE(3)                                \
            CASE(4)                                \
            CASE(6)                                \
            CASE(8)                                \
            CASE(12)                               \
            CASE(16)                               \
            default:                               \
                CASE_SEG();                        \
                break;                             \
        }                                          \
    } while (0)

void launch_full_keys(const IndexView& ix, const uint64_t* vis, int64_t n_rows, const float* qrows,
                      const int32_t* qidx, int32_t ng, uint64_t* keys, int64_t ld,
                      hipStream_t stream) {
    if (n_rows <= 0 || ng <= 0) return;
    const int64_t blocks = std::min<int64_t>((n_rows + 15) / 16, 8192);
    const dim3 grid(static_cast<uint32_t>(blocks), static_cast<uint32_t>(ng));
#define PVS_FK(N)                                                                                  \
    case N:                                                                                        \
        if (full_)                                                                                 \
            hipLaunchKernelGGL((k_full_keys<N, true>), grid, dim3(256), 0, stream, ix.rows, ix.df, vis, \
                               n_rows, qrows, qidx, keys, ld);                                     \
        else                                                                                       \
            hipLaunchKernelGGL((k_full_keys<N, false>), grid, dim3(256), 0, stream, ix.rows, ix.df, \
                               vis, n_rows, qrows, qidx, keys, ld);                                \
        break;
#define CASE_SEG()                                                                                 \
    hipLaunchKernelGGL((k_full_keys<0, false>), grid, dim3(256), 0, stream, ix.rows, ix.df, vis,   \
                       n_rows, qrows, qidx, keys, ld)
    PVS_GROUP_SWITCH(ix.df, PVS_FK);
#undef CASE_SEG
#undef PVS_FK
}

// ----------------------------------------------------------- debug paths
// Intervals of one query against listed rows, by the scans' own arithmetic
// (one wavefront per row, lanes split the code chunks, integer sum exact).
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

// Authoritative scores of one query against listed rows: one 16-lane group
// per row, in the fixed order of group_dot.
template <int J, bool FULL>
__global__ __launch_bounds__(256) void k_scores(const float4* __restrict__ rows, int32_t df4,
                                                const float4* __restrict__ qrows, int32_t qi,
                                                const int64_t* __restrict__ ids, int64_t n,
                                                float* __restrict__ out) {
    const int j = threadIdx.x & 15;
    const float4* qp = qrows + static_cast<int64_t>(qi) * df4;
    float4 q[J > 0 ? J : 1];
    if constexpr (J > 0) load_chunks<J, FULL>(qp, j, df4, q);
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 16 + (threadIdx.x >> 4); i < n;
         i += static_cast<int64_t>(gridDim.x) * 16) {
        const float4* rp = rows + ids[i] * df4;
        float s;
        if constexpr (J > 0) {
            float4 v[J];
            load_chunks<J, FULL>(rp, j, df4, v);
            s = group_dot<J, FULL>(v, q, j, df4);
        } else {
            s = group_score_seg(rp, qp, j, df4);
        }
        if (j == 0) out[i] = s;
    }
}

void launch_scores(const IndexView& ix, const float* qrows, int32_t qi, const int64_t* rows,
                   int64_t n, float* out, hipStream_t stream) {
    if (n <= 0) return;
    int64_t g = (n + 15) / 16;
    if (g > 65536) g = 65536;
    const float4* r4 = reinterpret_cast<const float4*>(ix.rows);
    const float4* q4 = reinterpret_cast<const float4*>(qrows);
    const dim3 grid(static_cast<uint32_t>(g));
    const int32_t df4 = ix.df / 4;
#define PVS_SC(N)                                                                                  \
    case N:                                                                                        \
        if (full_)                                                                                 \
            hipLaunchKernelGGL((k_scores<N, true>), grid, dim3(256), 0, stream, r4, df4, q4, qi, rows, n, out); \
        else                                                                                       \
            hipLaunchKernelGGL((k_scores<N, false>), grid, dim3(256), 0, stream, r4, df4, q4, qi, rows, n, out); \
        break;
#define CASE_SEG() \
    hipLaunchKernelGGL((k_scores<0, false>), grid, dim3(256), 0, stream, r4, df4, q4, qi, rows, n, out)
    PVS_GROUP_SWITCH(ix.df, PVS_SC);
#undef CASE_SEG
#undef PVS_SC
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
