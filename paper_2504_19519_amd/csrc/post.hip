// Post-communication reorder fused into the following element-wise kernel
// (Section 3.3 Approach, last paragraph: the kernel after communication
// loads by the reordered index; Section 6.6 fuses it with RMSNorm).
//
// One wave per output row, four rows per workgroup. Lane l handles the
// 16-byte chunks l, l+64, ... of the row. A chunk lies inside one tile
// column, so its source address is the row's place in that tile's slot (tile
// pattern), in the slice's destination buffer (subtile pattern) or in the
// row's pool (subtoken pattern); every source read is 16 contiguous bytes
// and lanes of one tile column read one contiguous tile_n-wide row piece.
// The workgroup first copies the slots of its tile row from the reorder map
// into LDS, so a chunk's address needs no dependent global load. Loads are
// issued in batches (16 per lane, or the whole row when it is held for
// RMSNorm) before their stores, so that many reads are in flight. Output
// rows are written fully coalesced; source and output bypass the caches
// (nontemporal). With RMSNorm the row is held in registers between the
// sum-of-squares pass and the scaling pass (rows up to 8192 wide), or read
// twice for wider rows.
#include <hip/hip_runtime.h>

#include "fo_device.h"
#include "fo_internal.h"
#include "post.h"

namespace fo {
namespace {

constexpr int kThreads = 256;
constexpr int kRowsPerBlock = kThreads / 64;

template <int DT>
__device__ __forceinline__ void widen8(u32x4_t v, float* f) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        f[2 * e] = to_f32<DT>(v[e] & 0xFFFFu);
        f[2 * e + 1] = to_f32<DT>(v[e] >> 16);
    }
}

// Slots of one tile row kept in LDS (tile rows up to this many tiles; wider
// tile rows read the map from memory).
constexpr int kSlotCache = 1024;

template <int DT, int CH>
__global__ __launch_bounds__(kThreads, 4) void post_kernel(const PostArgs a) {
    __shared__ int32_t s_slot[kSlotCache];
    const int lane = threadIdx.x & 63;
    const int64_t i0 = (int64_t)blockIdx.x * kRowsPerBlock;
    const int64_t tm0 = i0 / a.tile_m;
    const bool cached = a.pattern != FO_PATTERN_ROWMAJOR && a.tiles_n <= kSlotCache;
    if (cached) {     // uniform over the workgroup
        for (int t = threadIdx.x; t < a.tiles_n; t += kThreads) s_slot[t] = a.tile_to_slot[tm0 * a.tiles_n + t];
        __syncthreads();
    }
    const int64_t i = i0 + (threadIdx.x >> 6);
    if (i >= a.M) return;
    const int64_t nch = a.N >> 3;
    const int64_t tm = i / a.tile_m;
    const int64_t r = i - tm * a.tile_m;
    const int cpt = a.tile_n >> 3;                      // chunks per tile row piece

    // Row-level part of the source address.
    int64_t row_part = 0, dest_base = 0;
    int32_t b = 0;
    if (a.pattern == FO_PATTERN_TILE) {
        row_part = r * a.tile_n;
    } else if (a.pattern == FO_PATTERN_SUBTILE) {
        const int64_t h = a.tile_m / a.num_dest;
        const int64_t k = r / h;
        dest_base = (int64_t)a.dest_perm[k] * a.per_dest;
        row_part = (r - k * h) * a.tile_n;
    } else if (a.pattern == FO_PATTERN_SUBTOKEN) {
        b = a.row_bucket[i];
        row_part = ((int64_t)a.pool_off[b] + a.row_rank[i]) * a.tile_n;
    }
    const bool from_lds = cached && tm == tm0;
    auto src_of = [&](int64_t c) -> int64_t {
        if (a.pattern == FO_PATTERN_ROWMAJOR) return i * a.N + c * 8;
        const int64_t tn = a.cpt_log2 >= 0 ? c >> a.cpt_log2 : c / cpt;
        const int64_t cin = (c - tn * cpt) * 8;
        const int64_t slot = from_lds ? s_slot[tn] : a.tile_to_slot[tm * a.tiles_n + tn];
        if (a.pattern == FO_PATTERN_TILE) return slot * a.tile_m * a.tile_n + row_part + cin;
        if (a.pattern == FO_PATTERN_SUBTILE)
            return dest_base + slot * (a.tile_m / a.num_dest) * a.tile_n + row_part + cin;
        return row_part + (int64_t)a.pool_base[slot * a.num_dest + b] * a.tile_n + cin;
    };
    auto load = [&](int64_t c) -> u32x4_t {
        return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(a.src + src_of(c)));
    };
    const u32x4_t* bias4 = reinterpret_cast<const u32x4_t*>(a.bias);
    const u32x4_t* gamma4 = reinterpret_cast<const u32x4_t*>(a.gamma);
    u32x4_t* out4 = reinterpret_cast<u32x4_t*>(a.out + i * a.N);

    auto finish = [&](int64_t c, u32x4_t xv, float inv) {
        float x[8], bv[8], gv[8];
        widen8<DT>(xv, x);
        if (a.bias) widen8<DT>(bias4[c], bv);
        if (a.do_norm && a.gamma) widen8<DT>(gamma4[c], gv);
        u32x4_t o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float y0 = x[2 * e] + (a.bias ? bv[2 * e] : 0.0f);
            float y1 = x[2 * e + 1] + (a.bias ? bv[2 * e + 1] : 0.0f);
            if (a.do_norm) {
                y0 *= inv;
                y1 *= inv;
                if (a.gamma) {
                    y0 *= gv[2 * e];
                    y1 *= gv[2 * e + 1];
                }
            }
            o[e] = pack2<DT>(y0, y1);
        }
        __builtin_nontemporal_store(o, out4 + c);
    };
    auto sumsq = [&](int64_t c, u32x4_t xv) {
        float x[8], bv[8];
        widen8<DT>(xv, x);
        if (a.bias) widen8<DT>(bias4[c], bv);
        float s = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float h = x[e] + (a.bias ? bv[e] : 0.0f);
            s += h * h;
        }
        return s;
    };

    if (!a.do_norm && !a.bias) {          // plain gather: bit-exact copy
        constexpr int B = 16;
        for (int64_t c0 = lane; c0 < nch; c0 += 64 * B) {
            u32x4_t v[B];
#pragma unroll
            for (int t = 0; t < B; ++t)
                if (c0 + 64 * t < nch) v[t] = load(c0 + 64 * t);
#pragma unroll
            for (int t = 0; t < B; ++t)
                if (c0 + 64 * t < nch) __builtin_nontemporal_store(v[t], out4 + c0 + 64 * t);
        }
        return;
    }
    float ss = 0.0f;
    if constexpr (CH > 0) {
        u32x4_t cache[CH];
#pragma unroll
        for (int t = 0; t < CH; ++t) {
            const int64_t c = lane + 64 * t;
            if (c < nch) cache[t] = load(c);
        }
        if (a.do_norm) {
#pragma unroll
            for (int t = 0; t < CH; ++t) {
                const int64_t c = lane + 64 * t;
                if (c < nch) ss += sumsq(c, cache[t]);
            }
        }
        float inv = 1.0f;
        if (a.do_norm) {
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
            inv = 1.0f / sqrtf(ss / (float)a.N + a.eps);
        }
#pragma unroll
        for (int t = 0; t < CH; ++t) {
            const int64_t c = lane + 64 * t;
            if (c < nch) finish(c, cache[t], inv);
        }
    } else {
        if (a.do_norm) {
            for (int64_t c = lane; c < nch; c += 64)
                ss += sumsq(c, load(c));
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
        }
        const float inv = a.do_norm ? 1.0f / sqrtf(ss / (float)a.N + a.eps) : 1.0f;
        for (int64_t c = lane; c < nch; c += 64)
            finish(c, load(c), inv);
    }
}

template <int DT>
hipError_t launch_dt(const PostArgs& a, hipStream_t s) {
    const int64_t nch = a.N >> 3;
    const dim3 g((unsigned)((a.M + kRowsPerBlock - 1) / kRowsPerBlock)), b(kThreads);
    if (nch <= 64 * 4) hipLaunchKernelGGL((post_kernel<DT, 4>), g, b, 0, s, a);
    else if (nch <= 64 * 8) hipLaunchKernelGGL((post_kernel<DT, 8>), g, b, 0, s, a);
    else if (nch <= 64 * 16) hipLaunchKernelGGL((post_kernel<DT, 16>), g, b, 0, s, a);
    else hipLaunchKernelGGL((post_kernel<DT, 0>), g, b, 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_post(int dtype, const PostArgs& a, hipStream_t s) {
    if (a.M == 0 || a.N == 0) return hipSuccess;
    return dtype == FO_FP16 ? launch_dt<FO_FP16>(a, s) : launch_dt<FO_BF16>(a, s);
}

}  // namespace fo
