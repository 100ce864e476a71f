// GEMM with the reordering, signalling epilogue (gfx950).
//
// C = A x B (Section 2.1.1) with A [M, K] and W = B^T [N, K], both K
// contiguous. One workgroup computes one BM x BN output tile; workgroup p
// takes the tile at dispatch position p (fo_order), so tiles run in waves of
// one tile per compute unit (Section 2.1.1) and position p is the tile's slot
// in the reordered output (Section 3.3 Approach (1)).
//
// Main loop: MFMA v_mfma_f32_32x32x16 (fp16 / bf16 in, fp32 accumulate),
// A and B tiles of BK = 64 double-buffered in LDS with padded rows (conflict
// free 16-byte fragment reads), the next K block prefetched into registers
// while the current one is multiplied. The main loop is the same for every
// output pattern (Section 5: only the epilogue changes).
//
// Epilogue (Section 3.3 Approach; Section 3.2 Approach):
//   1. accumulators -> fp16/bf16 (round to nearest even) -> LDS staging tile;
//   2. every tile row goes out as full-row stores to its destination:
//      row-major C, the tile's slot (tile pattern), the slice's place in its
//      group segment (subtile pattern) or the row's pool position (subtoken
//      pattern);
//   3. once the tile's stores are visible to all chiplets (fo_sync_mode:
//      device-coherent stores + wait, or an agent-scope release), one lane
//      adds 1 to the counter of the group that owns the slot.
#include <hip/hip_runtime.h>

#include "fo_device.h"
#include "fo_internal.h"
#include "gemm.h"

namespace fo {
namespace {

constexpr int kThreads = 256;
constexpr int kBK = 64;
constexpr int kLDK = kBK + 8;       // padded LDS row of an operand tile (halfs)
// s_waitcnt operand with vmcnt = 0 and the other counters at their maximum
// (gfx9 encoding: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8], vmcnt[5:4] at 15:14)
constexpr int kWaitVmcnt0 = 0x0F70;

template <int DT>
__device__ __forceinline__ f32x16_t mfma32(u32x4_t a, u32x4_t b, f32x16_t c) {
    if constexpr (DT == FO_FP16)
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(bit_cast<half8_t>(a), bit_cast<half8_t>(b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(bit_cast<bf16x8_t>(a), bit_cast<bf16x8_t>(b), c, 0, 0, 0);
}

template <int BM, int BN>
struct Smem {
    static constexpr int kStageA = BM * kLDK;          // halfs
    static constexpr int kStageB = BN * kLDK;
    static constexpr int kLDC = BN + 8;
    static constexpr int kOperands = 2 * (kStageA + kStageB);
    static constexpr int kStaging = BM * kLDC;
    static constexpr int kHalfs = kOperands > kStaging ? kOperands : kStaging;
};

template <int DT, int BM, int BN, int WAVES_M, int WAVES_N>
__global__ __launch_bounds__(kThreads, 2) void gemm_signal_kernel(const GemmArgs a) {
    constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
    constexpr int MI = WTM / 32, NJ = WTN / 32;
    constexpr int A_CH = BM * kBK / 8 / kThreads;      // 16-byte chunks per thread
    constexpr int B_CH = BN * kBK / 8 / kThreads;
    constexpr int ROWS_PER_LOAD = kThreads / (kBK / 8);
    using S = Smem<BM, BN>;
    static_assert(WAVES_M * WAVES_N == kThreads / 64, "four waves");
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "32x32 MFMA blocks");
    static_assert(A_CH >= 1 && B_CH >= 1, "tile too small for the loader");

    __shared__ __attribute__((aligned(16))) uint16_t smem[S::kHalfs];
    __shared__ int64_t row_off[BM];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int p = blockIdx.x;
    const int tile = tile_of_position(p, a.tiles_m, a.tiles_n, a.order, a.group_m, a.num_xcds);
    const int tm = tile / a.tiles_n, tn = tile - (tile / a.tiles_n) * a.tiles_n;
    const int64_t K = a.K;

    // Plan lookups needed only by the epilogue: issued now, consumed later.
    const int slot = a.tile_to_slot ? a.tile_to_slot[tile] : p;
    int bucket = 0, rank = 0;
    if (a.pattern == FO_PATTERN_SUBTOKEN && tid < BM) {
        bucket = a.row_bucket[tm * BM + tid];
        rank = a.row_rank[tm * BM + tid];
    }

    const uint16_t* Ag = a.A + (int64_t)tm * BM * K;
    const uint16_t* Wg = a.W + (int64_t)tn * BN * K;
    const int lrow = tid / (kBK / 8), lkc = tid % (kBK / 8);

    u32x4_t ra[A_CH], rb[B_CH];
    auto gload = [&](int kt) {
        const int64_t k0 = (int64_t)kt * kBK + lkc * 8;
#pragma unroll
        for (int i = 0; i < A_CH; ++i)
            ra[i] = *reinterpret_cast<const u32x4_t*>(Ag + (int64_t)(lrow + ROWS_PER_LOAD * i) * K + k0);
#pragma unroll
        for (int i = 0; i < B_CH; ++i)
            rb[i] = *reinterpret_cast<const u32x4_t*>(Wg + (int64_t)(lrow + ROWS_PER_LOAD * i) * K + k0);
    };
    auto sstore = [&](int stage) {
        uint16_t* As = smem + stage * S::kStageA;
        uint16_t* Bs = smem + 2 * S::kStageA + stage * S::kStageB;
#pragma unroll
        for (int i = 0; i < A_CH; ++i)
            *reinterpret_cast<u32x4_t*>(As + (lrow + ROWS_PER_LOAD * i) * kLDK + lkc * 8) = ra[i];
#pragma unroll
        for (int i = 0; i < B_CH; ++i)
            *reinterpret_cast<u32x4_t*>(Bs + (lrow + ROWS_PER_LOAD * i) * kLDK + lkc * 8) = rb[i];
    };

    f32x16_t acc[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    const int KT = (int)(K / kBK);
    if (KT > 0) {
        gload(0);
        sstore(0);
    }
    __syncthreads();

    // Fragment addressing: lane l feeds row (l % 32) of a 32-row block with
    // the 8 consecutive k values starting at 8 * (l / 32) of a 16-wide step.
    const int frag = (lane & 31) * kLDK + (lane >> 5) * 8;
    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < KT) gload(kt + 1);
        const uint16_t* As = smem + cur * S::kStageA + wm * WTM * kLDK + frag;
        const uint16_t* Bs = smem + 2 * S::kStageA + cur * S::kStageB + wn * WTN * kLDK + frag;
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            u32x4_t af[MI], bf[NJ];
#pragma unroll
            for (int i = 0; i < MI; ++i)
                af[i] = *reinterpret_cast<const u32x4_t*>(As + i * 32 * kLDK + kk * 16);
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                bf[j] = *reinterpret_cast<const u32x4_t*>(Bs + j * 32 * kLDK + kk * 16);
            // W fragment as the MFMA's first operand: the 32x32 result block
            // is C^T, so each lane holds 4 consecutive output columns.
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    acc[i][j] = mfma32<DT>(bf[j], af[i], acc[i][j]);
        }
        if (kt + 1 < KT) sstore(cur ^ 1);
        __syncthreads();
    }

    // ---- epilogue -------------------------------------------------------
    // Destination of row `tid` of the tile, by pattern.
    if (tid < BM) {
        const int r = tid;
        int64_t off;
        if (a.pattern == FO_PATTERN_ROWMAJOR) {
            off = ((int64_t)tm * BM + r) * a.N + (int64_t)tn * BN;
        } else if (a.pattern == FO_PATTERN_TILE) {
            off = ((int64_t)slot * BM + r) * BN;
        } else if (a.pattern == FO_PATTERN_SUBTILE) {
            const int h = BM / a.num_dest;
            const int k = r / h, rr = r - (r / h) * h;
            const int j = a.slot_group[slot];
            const int64_t f0 = a.group_first[j];
            const int64_t nj = a.group_first[j + 1] - f0;
            off = f0 * BM * BN + ((int64_t)k * nj + (slot - f0)) * h * BN + (int64_t)rr * BN;
        } else {
            const int B = a.num_dest;
            off = ((int64_t)a.pool_off[bucket] + a.pool_base[(int64_t)slot * B + bucket] + rank) * BN;
        }
        row_off[r] = off;
    }

    // accumulators -> LDS staging [BM][BN + 8] (operand buffers are free:
    // the loop ended with a barrier)
    uint16_t* Cs = smem;
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        const int m = wm * WTM + i * 32 + (lane & 31);
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int n = wn * WTN + j * 32 + q * 8 + (lane >> 5) * 4;
                u32x2_t v;
                v[0] = pack2<DT>(acc[i][j][4 * q + 0], acc[i][j][4 * q + 1]);
                v[1] = pack2<DT>(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
                *reinterpret_cast<u32x2_t*>(Cs + m * S::kLDC + n) = v;
            }
        }
    }
    __syncthreads();

    if (a.counters && a.sync == FO_SYNC_COHERENT) {
        // Device-coherent 8-byte stores (written through to the point all
        // chiplets share), each wave waits until its stores are complete,
        // then one lane counts the tile: no cache write-back is needed.
        constexpr int LPR = BN / 4;             // lanes per row (8 bytes each)
        constexpr int RPI = 64 / LPR;           // rows per wave instruction
        const int lr = lane / LPR, lc = lane % LPR;
#pragma unroll 4
        for (int r = wave * RPI + lr; r < BM; r += 4 * RPI) {
            const uint64_t v = *reinterpret_cast<const uint64_t*>(Cs + r * S::kLDC + lc * 4);
            __hip_atomic_store(reinterpret_cast<uint64_t*>(a.C + row_off[r]) + lc, v, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (tid == 0)
            __hip_atomic_fetch_add(a.counters + a.slot_group[slot], 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        return;
    }

    constexpr int CPR = BN / 8;                 // 16-byte chunks per tile row
    constexpr int RPP = kThreads / CPR;         // rows per pass
    const int c = tid % CPR;
#pragma unroll 4
    for (int r = tid / CPR; r < BM; r += RPP) {
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(Cs + r * S::kLDC + c * 8);
        *reinterpret_cast<u32x4_t*>(a.C + row_off[r] + c * 8) = v;
    }

    if (a.counters) {
        // Section 3.2: count the finished tile for its group once all of the
        // tile's stores are visible to every compute unit.
        if (a.sync == FO_SYNC_FENCE_ALL) {
            // every wave: release fence at agent scope (L2 write-back + wait)
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            __syncthreads();
            if (tid == 0)
                __hip_atomic_fetch_add(a.counters + a.slot_group[slot], 1u, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
        } else {
            // workgroup barrier, then one release increment (one write-back)
            __syncthreads();
            if (tid == 0)
                __hip_atomic_fetch_add(a.counters + a.slot_group[slot], 1u, __ATOMIC_RELEASE,
                                       __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

template <int DT, int BM, int BN, int WM, int WN>
hipError_t launch_t(const GemmArgs& a, int grid, hipStream_t s) {
    hipLaunchKernelGGL((gemm_signal_kernel<DT, BM, BN, WM, WN>), dim3(grid), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(int dtype, int tile_m, int tile_n, const GemmArgs& a, int grid, hipStream_t s) {
    if (tile_m == 256 && tile_n == 128)
        return dtype == FO_FP16 ? launch_t<FO_FP16, 256, 128, 2, 2>(a, grid, s)
                                : launch_t<FO_BF16, 256, 128, 2, 2>(a, grid, s);
    if (tile_m == 64 && tile_n == 64)
        return dtype == FO_FP16 ? launch_t<FO_FP16, 64, 64, 2, 2>(a, grid, s)
                                : launch_t<FO_BF16, 64, 64, 2, 2>(a, grid, s);
    return hipErrorInvalidValue;
}

bool gemm_tile_supported(int tile_m, int tile_n) {
    return (tile_m == 256 && tile_n == 128) || (tile_m == 64 && tile_n == 64);
}

}  // namespace fo
