// Consumer: the one-GPU stand-in for the collective that follows each wave
// group (Section 5: a signalling kernel stalls the communication of a group
// until its count reaches the group's tile count; the communication itself
// is a library call on a contiguous buffer, Section 3.3 Motivation).
//
// One launch handles one contiguous segment: every workgroup waits for the
// group's counter (relaxed agent-scope polls with s_sleep, then one
// agent-scope acquire), then streams the segment:
//   dst = RNE(src + peer)   AllReduce / ReduceScatter of two partials
//   dst = src               All-to-All (copy to the receive buffer)
// The wait is bounded by a wall-clock limit; on timeout the workgroup writes
// nothing and raises bit 0 of the status word, so a missing signal can never
// hang the device.
//
// The grid is capped (kMaxBlocks) and a workgroup holds no LDS and few
// registers, so polling workgroups never take the resources a not yet
// dispatched GEMM workgroup needs (the GEMM holds 110 KB of LDS, four waves
// and about half of each SIMD's registers per CU).
#include <hip/hip_runtime.h>

#include "consume.h"
#include "fo_device.h"
#include "fo_internal.h"

namespace fo {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

__device__ __forceinline__ bool wait_counter(const uint32_t* counter, uint32_t target,
                                             uint32_t* status, uint64_t timeout_ticks) {
    __shared__ int s_ok;
    if (threadIdx.x == 0) {
        int ok = 1;
        if (__hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
            const uint64_t t0 = wall_clock64();
            while (__hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
                __builtin_amdgcn_s_sleep(8);
                if (wall_clock64() - t0 > timeout_ticks) {
                    ok = 0;
                    break;
                }
            }
        }
        if (ok)
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        else if (status)
            __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_ok = ok;
    }
    __syncthreads();
    // every wave invalidates its view before reading the group's data
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    return s_ok != 0;
}

template <int DT>
__device__ __forceinline__ u32x4_t add8(u32x4_t x, u32x4_t y) {
    u32x4_t r;
    if constexpr (DT == FO_FP16) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            r[e] = bit_cast<uint32_t>(bit_cast<half2_t>(x[e]) + bit_cast<half2_t>(y[e]));
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float lo = bf16_bits_to_f32(x[e] & 0xFFFFu) + bf16_bits_to_f32(y[e] & 0xFFFFu);
            const float hi = bf16_bits_to_f32(x[e] >> 16) + bf16_bits_to_f32(y[e] >> 16);
            r[e] = pack2<FO_BF16>(lo, hi);
        }
    }
    return r;
}

template <int DT>
__device__ __forceinline__ uint16_t add1(uint16_t x, uint16_t y) {
    return (uint16_t)from_f32<DT>(to_f32<DT>(x) + to_f32<DT>(y));
}

// 16-byte path: src, peer and dst 16-byte aligned.
template <int DT, bool SUM>
__global__ __launch_bounds__(kThreads) void consume_vec_kernel(
    const uint16_t* __restrict__ src, const uint16_t* __restrict__ peer, uint16_t* __restrict__ dst,
    int64_t len, const uint32_t* counter, uint32_t target, uint32_t* status, uint64_t timeout_ticks) {
    if (counter && !wait_counter(counter, target, status, timeout_ticks)) return;
    const int64_t n16 = len >> 3;
    const u32x4_t* s = reinterpret_cast<const u32x4_t*>(src);
    const u32x4_t* q = reinterpret_cast<const u32x4_t*>(peer);
    u32x4_t* d = reinterpret_cast<u32x4_t*>(dst);
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    for (; i + (kUnroll - 1) * stride < n16; i += kUnroll * stride) {
        u32x4_t x[kUnroll], y[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) x[u] = __builtin_nontemporal_load(s + i + u * stride);
        if constexpr (SUM) {
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) y[u] = __builtin_nontemporal_load(q + i + u * stride);
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) x[u] = add8<DT>(x[u], y[u]);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) __builtin_nontemporal_store(x[u], d + i + u * stride);
    }
    for (; i < n16; i += stride) {
        u32x4_t x = __builtin_nontemporal_load(s + i);
        if constexpr (SUM) x = add8<DT>(x, __builtin_nontemporal_load(q + i));
        __builtin_nontemporal_store(x, d + i);
    }
    // ragged tail (< 8 elements)
    if (blockIdx.x == 0 && threadIdx.x < (len & 7)) {
        const int64_t e = (n16 << 3) + threadIdx.x;
        dst[e] = SUM ? add1<DT>(src[e], peer[e]) : src[e];
    }
}

// Element path for unaligned buffers.
template <int DT, bool SUM>
__global__ __launch_bounds__(kThreads) void consume_elem_kernel(
    const uint16_t* __restrict__ src, const uint16_t* __restrict__ peer, uint16_t* __restrict__ dst,
    int64_t len, const uint32_t* counter, uint32_t target, uint32_t* status, uint64_t timeout_ticks) {
    if (counter && !wait_counter(counter, target, status, timeout_ticks)) return;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < len; i += stride)
        dst[i] = SUM ? add1<DT>(src[i], peer[i]) : src[i];
}

}  // namespace

hipError_t launch_consume(int dtype, const uint16_t* src, const uint16_t* peer, uint16_t* dst,
                          int64_t len, const uint32_t* counter, uint32_t target, uint32_t* status,
                          uint64_t timeout_ticks, hipStream_t s) {
    const bool vec = ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst) |
                       reinterpret_cast<uintptr_t>(peer)) & 15) == 0;
    const int64_t work = vec ? (len >> 3) : len;
    int64_t blocks = (work + (int64_t)kThreads * kUnroll - 1) / ((int64_t)kThreads * kUnroll);
    if (blocks < 1) blocks = 1;
    if (blocks > kMaxConsumeBlocks) blocks = kMaxConsumeBlocks;
    const dim3 g((unsigned)blocks), b(kThreads);
    const bool sum = peer != nullptr;
#define FO_CONSUME(KERN, DT, SUM) \
    hipLaunchKernelGGL((KERN<DT, SUM>), g, b, 0, s, src, peer, dst, len, counter, target, status, timeout_ticks)
    if (vec) {
        if (dtype == FO_FP16) { if (sum) FO_CONSUME(consume_vec_kernel, FO_FP16, true); else FO_CONSUME(consume_vec_kernel, FO_FP16, false); }
        else { if (sum) FO_CONSUME(consume_vec_kernel, FO_BF16, true); else FO_CONSUME(consume_vec_kernel, FO_BF16, false); }
    } else {
        if (dtype == FO_FP16) { if (sum) FO_CONSUME(consume_elem_kernel, FO_FP16, true); else FO_CONSUME(consume_elem_kernel, FO_FP16, false); }
        else { if (sum) FO_CONSUME(consume_elem_kernel, FO_BF16, true); else FO_CONSUME(consume_elem_kernel, FO_BF16, false); }
    }
#undef FO_CONSUME
    return hipGetLastError();
}

}  // namespace fo
