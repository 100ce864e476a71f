// Post-communication reorder fused into the following element-wise kernel
// (Section 3.3 Approach, last paragraph: the kernel after communication
// loads by the reordered index; Section 6.6 fuses it with RMSNorm).
//
// One wave per output row, four rows per workgroup. Lane l handles the
// 16-byte chunks l, l+64, ... of the row. A chunk lies inside one tile
// column, so its source is 16 contiguous bytes of one row piece: the row's
// place in that tile's slot (tile pattern), in the slice's destination
// buffer (subtile pattern) or in the row's pool (subtoken pattern), and
// lanes of one tile column read one contiguous tile_n-wide piece.
//
// The workgroup first resolves the reorder map for its rows: for every
// (row, tile column) it writes the offset of the source piece to LDS. After
// that a chunk's source address is one LDS read and an add, so all of a
// lane's loads can be in flight at once.
//
// Two kernels:
//   post_gather_kernel  the plain restore (bit-exact copy): 16 loads per lane
//                       in flight before their stores;
//   post_norm_kernel    bias add and/or RMSNorm: the row is loaded up front
//                       and held in registers between the sum-of-squares and
//                       the scaling (rows up to 8192 wide, bias and gamma
//                       copied to LDS), or read twice for wider rows; which
//                       of bias, RMSNorm and gamma run is a compile-time
//                       choice.
// Sources are read through the caches (the consumer has just written them,
// so part of them is still in the memory-side cache); the output is written
// nontemporal.
#include <hip/hip_runtime.h>

#include "fo_device.h"
#include "fo_internal.h"
#include "post.h"

namespace fo {
namespace {

constexpr int kThreads = 256;
constexpr int kRowsPerBlock = kThreads / 64;
constexpr int kMaxRegChunks = 64 * 16;     // rows held in registers: up to 8192 columns

typedef __attribute__((address_space(3))) char lds_char_t;
typedef __attribute__((address_space(3))) uint32_t lds_u32_t;
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4_t;

template <int DT>
__device__ __forceinline__ void widen8(u32x4_t v, float* f) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        f[2 * e] = to_f32<DT>(v[e] & 0xFFFFu);
        f[2 * e + 1] = to_f32<DT>(v[e] >> 16);
    }
}

// Offset, in 16-byte chunks of the consumer's buffer, of the tile_n-wide
// source piece of output row i in tile column tn.
__device__ __forceinline__ uint32_t piece_offset(const PostArgs& a, int64_t i, int tn) {
    const int64_t tw = a.tile_n;
    if (a.pattern == FO_PATTERN_ROWMAJOR) return (uint32_t)((i * a.N + tn * tw) >> 3);
    const int32_t tm = (int32_t)(i / a.tile_m);
    const int32_t r = (int32_t)(i - (int64_t)tm * a.tile_m);
    const int64_t slot = a.tile_to_slot[(int64_t)tm * a.tiles_n + tn];
    int64_t off;
    if (a.pattern == FO_PATTERN_TILE) {
        off = (slot * a.tile_m + r) * tw;
    } else if (a.pattern == FO_PATTERN_SUBTILE) {
        const int32_t h = a.tile_m / a.num_dest;
        const int32_t k = r / h;
        off = (int64_t)a.dest_perm[k] * a.per_dest + (slot * h + (r - k * h)) * tw;
    } else {
        const int32_t b = a.row_bucket[i];
        off = ((int64_t)a.pool_off[b] + a.pool_base[slot * a.num_dest + b] + a.row_rank[i]) * tw;
    }
    return (uint32_t)(off >> 3);
}

// Source pieces of the workgroup's rows i0 .. i0+3: bases[w * tiles_n + tn].
__device__ __forceinline__ void stage_pieces(const PostArgs& a, lds_u32_t* bases, int64_t i0) {
    const int n = kRowsPerBlock * a.tiles_n;
    for (int idx = threadIdx.x; idx < n; idx += kThreads) {
        const int w = idx / a.tiles_n, tn = idx - (idx / a.tiles_n) * a.tiles_n;
        const int64_t i = i0 + w;
        if (i < a.M) bases[idx] = piece_offset(a, i, tn);
    }
}

// Chunk c of the row whose piece offsets are `bases` (tile_n / 8 is a power
// of two, 1 << cpt_log2).
__device__ __forceinline__ u32x4_t load_chunk(const PostArgs& a, const lds_u32_t* bases, int64_t c) {
    const uint32_t cpt_mask = (1u << a.cpt_log2) - 1u;
    const uint32_t off = bases[(uint32_t)c >> a.cpt_log2] + ((uint32_t)c & cpt_mask);
    return reinterpret_cast<const u32x4_t*>(a.src)[off];
}

template <int DT>
__global__ __launch_bounds__(kThreads) void post_gather_kernel(const PostArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    lds_u32_t* bases = reinterpret_cast<lds_u32_t*>((lds_char_t*)smem);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t i0 = (int64_t)blockIdx.x * kRowsPerBlock;
    stage_pieces(a, bases, i0);
    __syncthreads();
    const int64_t i = i0 + w;
    if (i >= a.M) return;
    const lds_u32_t* rb = bases + w * a.tiles_n;
    const int64_t nch = a.N >> 3;
    u32x4_t* out4 = reinterpret_cast<u32x4_t*>(a.out + i * a.N);
    constexpr int B = 16;
    for (int64_t c0 = lane; c0 < nch; c0 += 64 * B) {
        u32x4_t v[B];
#pragma unroll
        for (int t = 0; t < B; ++t)
            if (c0 + 64 * t < nch) v[t] = load_chunk(a, rb, c0 + 64 * t);
#pragma unroll
        for (int t = 0; t < B; ++t)
            if (c0 + 64 * t < nch) __builtin_nontemporal_store(v[t], out4 + c0 + 64 * t);
    }
}

// y = (x + bias) [* rsqrt(mean((x + bias)^2) + eps) * gamma]. NORM, BIAS and
// GAMMA fix at compile time which parts run (GAMMA only with NORM), so that
// no per-chunk branch and no value of an unused part holds registers.
template <int DT, int CH, bool NORM, bool BIAS, bool GAMMA>
__global__ __launch_bounds__(kThreads) void post_norm_kernel(const PostArgs a) {
    constexpr bool kLdsAffine = (BIAS || GAMMA) && CH > 0;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int64_t nch = a.N >> 3;
    // LDS: [bias chunks][gamma chunks] (with kLdsAffine), then the pieces
    lds_u32x4_t* s_bias = reinterpret_cast<lds_u32x4_t*>((lds_char_t*)smem);
    lds_u32x4_t* s_gamma = s_bias + (kLdsAffine ? nch : 0);
    lds_u32_t* bases = reinterpret_cast<lds_u32_t*>(s_gamma + (kLdsAffine ? nch : 0));
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t i0 = (int64_t)blockIdx.x * kRowsPerBlock;
    const u32x4_t* bias4 = reinterpret_cast<const u32x4_t*>(a.bias);
    const u32x4_t* gamma4 = reinterpret_cast<const u32x4_t*>(a.gamma);
    if constexpr (kLdsAffine) {
        for (int64_t c = threadIdx.x; c < nch; c += kThreads) {
            if constexpr (BIAS) s_bias[c] = bias4[c];
            if constexpr (GAMMA) s_gamma[c] = gamma4[c];
        }
    }
    stage_pieces(a, bases, i0);
    __syncthreads();
    const int64_t i = i0 + w;
    if (i >= a.M) return;
    const lds_u32_t* rb = bases + w * a.tiles_n;
    u32x4_t* out4 = reinterpret_cast<u32x4_t*>(a.out + i * a.N);

    // h = x + bias (fp32, no rounding); sb: where bias chunks are read
    auto shift = [&](u32x4_t xv, int64_t c, const lds_u32x4_t* sb, float* h) {
        widen8<DT>(xv, h);
        if constexpr (BIAS) {
            float bv[8];
            widen8<DT>(kLdsAffine ? sb[c] : bias4[c], bv);
#pragma unroll
            for (int e = 0; e < 8; ++e) h[e] += bv[e];
        }
    };
    auto sumsq = [&](u32x4_t xv, int64_t c, const lds_u32x4_t* sb) {
        float h[8];
        shift(xv, c, sb, h);
        float q = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) q += h[e] * h[e];
        return q;
    };
    auto finish = [&](int64_t c, u32x4_t xv, float inv, const lds_u32x4_t* sb, const lds_u32x4_t* sg, bool live) {
        float h[8], gv[8];
        shift(xv, c, sb, h);
        if constexpr (GAMMA) widen8<DT>(kLdsAffine ? sg[c] : gamma4[c], gv);
        u32x4_t o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float y0 = h[2 * e], y1 = h[2 * e + 1];
            if constexpr (NORM) {
                y0 *= inv;
                y1 *= inv;
                if constexpr (GAMMA) {
                    y0 *= gv[2 * e];
                    y1 *= gv[2 * e + 1];
                }
            }
            o[e] = pack2<DT>(y0, y1);
        }
        if (live) __builtin_nontemporal_store(o, out4 + c);
    };
    auto rsqrt_mean = [&](float ss) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
        return 1.0f / sqrtf(ss / (float)a.N + a.eps);
    };

    if constexpr (CH > 0) {
        // The row is loaded up front. Lanes past the row's end load its last
        // chunk (no branches around the loads: the array stays in registers)
        // and drop the result.
        u32x4_t xc[CH];
#pragma unroll
        for (int t = 0; t < CH; ++t) {
            const int64_t c = lane + 64 * t;
            xc[t] = load_chunk(a, rb, c < nch ? c : nch - 1);
        }
        float inv = 1.0f;
        if constexpr (NORM) {
            float ss = 0.0f;
#pragma unroll
            for (int t = 0; t < CH; ++t) {
                const int64_t c = lane + 64 * t;
                const float q = sumsq(xc[t], c < nch ? c : nch - 1, s_bias);
                ss += c < nch ? q : 0.0f;
                // one bias chunk at a time: the LDS reads are not all hoisted
                // to the top, where their values would hold registers
                if constexpr (kLdsAffine) asm volatile("" ::: "memory");
            }
            inv = rsqrt_mean(ss);
        }
        // The scaling pass widens the chunks again and reads bias and gamma
        // again, through pointers the compiler cannot match with the first
        // pass's, instead of keeping the first pass's values alive.
#pragma unroll
        for (int t = 0; t < CH; ++t) asm volatile("" : "+v"(xc[t]));
        // The lane index is laundered too, so that the second pass's addresses
        // are formed here and not kept live through the first pass.
        const lds_u32x4_t* sb = s_bias;
        const lds_u32x4_t* sg = s_gamma;
        int ln = lane;
        asm volatile("" : "+v"(sb), "+v"(sg), "+v"(ln));
#pragma unroll
        for (int t = 0; t < CH; ++t) {
            const int64_t c = ln + 64 * t;
            finish(c < nch ? c : nch - 1, xc[t], inv, sb, sg, c < nch);
            if constexpr (kLdsAffine) asm volatile("" ::: "memory");
        }
    } else {
        float inv = 1.0f;
        if constexpr (NORM) {
            float ss = 0.0f;
            for (int64_t c = lane; c < nch; c += 64) ss += sumsq(load_chunk(a, rb, c), c, s_bias);
            inv = rsqrt_mean(ss);
        }
        for (int64_t c = lane; c < nch; c += 64) finish(c, load_chunk(a, rb, c), inv, s_bias, s_gamma, true);
    }
}

template <int DT, int CH>
void launch_norm(const PostArgs& a, dim3 g, dim3 b, hipStream_t s) {
    const size_t lds = post_lds_bytes(a);
    const bool bias = a.bias != nullptr, gamma = a.do_norm && a.gamma != nullptr;
    if (!a.do_norm) hipLaunchKernelGGL((post_norm_kernel<DT, CH, false, true, false>), g, b, lds, s, a);
    else if (bias && gamma) hipLaunchKernelGGL((post_norm_kernel<DT, CH, true, true, true>), g, b, lds, s, a);
    else if (bias) hipLaunchKernelGGL((post_norm_kernel<DT, CH, true, true, false>), g, b, lds, s, a);
    else if (gamma) hipLaunchKernelGGL((post_norm_kernel<DT, CH, true, false, true>), g, b, lds, s, a);
    else hipLaunchKernelGGL((post_norm_kernel<DT, CH, true, false, false>), g, b, lds, s, a);
}

template <int DT>
hipError_t launch_dt(const PostArgs& a, hipStream_t s) {
    const int64_t nch = a.N >> 3;
    const dim3 g((unsigned)((a.M + kRowsPerBlock - 1) / kRowsPerBlock)), b(kThreads);
    if (!a.do_norm && !a.bias) hipLaunchKernelGGL((post_gather_kernel<DT>), g, b, post_lds_bytes(a), s, a);
    else if (nch <= 64 * 4) launch_norm<DT, 4>(a, g, b, s);
    else if (nch <= 64 * 8) launch_norm<DT, 8>(a, g, b, s);
    else if (nch <= kMaxRegChunks) launch_norm<DT, 16>(a, g, b, s);
    else launch_norm<DT, 0>(a, g, b, s);
    return hipGetLastError();
}

}  // namespace

size_t post_lds_bytes(const PostArgs& a) {
    const int64_t nch = a.N >> 3;
    const bool norm_path = a.do_norm || a.bias;
    const bool lds_affine = norm_path && (a.bias || (a.do_norm && a.gamma)) && nch <= kMaxRegChunks;
    return (size_t)kRowsPerBlock * a.tiles_n * sizeof(uint32_t) + (lds_affine ? 2 * (size_t)nch * 16 : 0);
}

hipError_t launch_post(int dtype, const PostArgs& a, hipStream_t s) {
    if (a.M == 0 || a.N == 0) return hipSuccess;
    return dtype == FO_FP16 ? launch_dt<FO_FP16>(a, s) : launch_dt<FO_BF16>(a, s);
}

}  // namespace fo
