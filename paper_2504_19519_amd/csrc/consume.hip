// Consumer: the one-GPU stand-in for the collective that follows each wave
// group (Section 5: a signalling kernel stalls the communication of a group
// until its count reaches the group's tile count; the communication itself
// is a library call on a contiguous buffer, Section 3.3 Motivation).
//
// One launch handles the contiguous segments of one group (one segment for a
// plain (ptr, len) call; the R or B destination pieces of a group for the
// ReduceScatter and All-to-All stand-ins). As in Section 5 (a signalling
// kernel holds back the communication call of a group until the group's
// count reaches its tile count), a one-wave wait kernel polls the group's
// counter, and the streaming kernel that follows it on the stream takes an
// agent-scope acquire (or reads with device-coherent loads, see
// fo_sync_mode) and streams each segment with a grid-stride loop:
//   dst = RNE(src + peer)   AllReduce / ReduceScatter of two partials
//   dst = src               All-to-All (copy to the receive buffer)
// The wait is bounded by a wall-clock limit; on timeout the streaming
// workgroups write nothing and bit 0 of the status word is raised, so a
// missing signal can never hang the device.
//
// A consumer workgroup holds 4 bytes of LDS and at most 56 registers per
// lane, so it fits beside a GEMM workgroup on the same compute unit (the
// GEMM kernels leave at least 64 registers per SIMD lane and 10 KB of LDS
// free): polling consumers share compute units with the GEMM instead of
// taking them away from it.
#include <hip/hip_runtime.h>

#include "consume.h"
#include "fo_device.h"
#include "fo_internal.h"

namespace fo {
namespace {

constexpr int kMaxThreads = 256;
// buffer resource word 3 for raw byte-addressed loads on gfx9
constexpr int kRsrcWord3 = 0x00020000;
// Accesses in flight per thread and stream: kUnrollFull for launches that
// have the device to themselves (the last group of an overlapped run, a
// serialized run), kUnrollBeside for launches beside the GEMM, whose
// registers must leave room for the GEMM's waves on the same SIMD.
constexpr int kUnrollFull = 4;
constexpr int kUnrollBeside = 2;
// s_waitcnt operand: vmcnt(0), other counters not waited for
constexpr int kWaitVmcnt0 = 0x0F70;

// Destination stores. Nontemporal by default (the next kernel reads the data,
// not this one). WT: device-coherent write-through stores (sc1), used by the
// launch that counts its finished workgroups for a wait on another stream:
// they reach the memory side that every chiplet shares, so once a wave's
// stores are complete (vmcnt 0) they are visible device-wide and no L2
// write-back is needed before the count.
template <bool WT>
__device__ __forceinline__ void put16(u32x4_t* p, u32x4_t v) {
    if constexpr (WT) asm volatile("global_store_dwordx4 %0, %1, off sc1" : : "v"(p), "v"(v) : "memory");
    else __builtin_nontemporal_store(v, p);
}
template <bool WT>
__device__ __forceinline__ void put8(uint64_t* p, uint64_t v) {
    if constexpr (WT) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else __builtin_nontemporal_store(v, p);
}
template <bool WT>
__device__ __forceinline__ void put2(uint16_t* p, uint16_t v) {
    if constexpr (WT) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else *p = v;
}

// The wait of a launch runs in a kernel of its own, one workgroup of one
// wave, ahead of the streaming kernel on the same stream: one lane polls the
// counter with relaxed agent-scope loads (device-coherent, no cache
// invalidation) and sleeps between polls. Polling from every streaming
// workgroup instead (hundreds of pollers on one cache line) measurably slows
// a GEMM running beside it; one poller does not. The streaming kernel starts
// only when the wait kernel has ended. The wait is bounded by a wall-clock
// limit; on timeout bit 0 of the status word is raised.
__global__ __launch_bounds__(64) void wait_kernel(const uint32_t* counter, uint32_t target, uint32_t* status,
                                                  uint64_t timeout_ticks) {
    if (threadIdx.x != 0) return;
    if (__hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target) return;
    const uint64_t t0 = wall_clock64();
    while (__hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        __builtin_amdgcn_s_sleep(8);
        if (wall_clock64() - t0 > timeout_ticks) {
            if (status) __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return;
        }
    }
}

// End handoff of an overlapped run (one wave, on the GEMM stream ahead of the
// post-reorder): lane k < kDoneWords polls done word k until it reaches the
// run's tag plus its share of the final launch's workgroups; the wave ends
// when every lane's word has. Bounded like wait_kernel.
__global__ __launch_bounds__(64) void done_wait_kernel(const uint32_t* done, uint32_t done_tag, int32_t blocks,
                                                       uint32_t* status, uint64_t timeout_ticks) {
    const int k = threadIdx.x;
    const bool mine = k < kDoneWords;
    const uint32_t target = done_tag + done_share(blocks, k);
    const uint32_t* w = done + (mine ? k : 0) * kDoneStride;
    const uint64_t t0 = wall_clock64();
    while (!__all(!mine || __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target)) {
        __builtin_amdgcn_s_sleep(8);
        if (wall_clock64() - t0 > timeout_ticks) {
            if (k == 0 && status) __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return;
        }
    }
}

// Start handoff of an overlapped run (one wave, on the consumer stream ahead
// of the run's first consumer): lane 0 polls the gate word until it holds
// the run's tag, which the run's reset kernel writes with a release once the
// counters are zero and the previous run's post-reorder, ordered before it
// on the GEMM stream, has finished reading the destination buffer. On
// timeout the lane raises bit 0 of the status word and, unless the word
// already holds a later run's tag (which must not be held up), marks the
// word (compare-and-swap, so a tag that arrives meanwhile still wins).
__global__ __launch_bounds__(64) void gate_kernel(uint32_t* gate, uint32_t tag, uint32_t* status,
                                                  uint64_t timeout_ticks) {
    if (threadIdx.x != 0) return;
    uint32_t v = __hip_atomic_load(gate, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t t0 = wall_clock64();
    while (v != tag) {
        __builtin_amdgcn_s_sleep(8);
        v = __hip_atomic_load(gate, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (v != tag && wall_clock64() - t0 > timeout_ticks) {
            // a later run's tag (sequence ahead of ours, modulo 2^30)
            const bool later = (v & (kGateTag | kGateTimedOut)) == kGateTag &&
                               (int32_t)(((v - tag) & kGateSeqMask) << 2) > 0;
            if (later) {
                if (status) __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                return;
            }
            if (__hip_atomic_compare_exchange_strong(gate, &v, tag | kGateTimedOut, __ATOMIC_RELAXED,
                                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                if (status) __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                return;
            }
            // v now holds the word's current value; the loop re-checks it
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

// Start of a streaming workgroup: one read of the counter (the wait kernel
// has returned, so it normally holds the target already; if the wait timed
// out the workgroup raises the status bit and writes nothing), then the
// acquire the mode needs.
// SYNC == FENCE_ALL: thread 0 and then every wave take an agent-scope
// acquire (cache invalidation); FENCE_ONE: thread 0 only (its invalidation
// covers the CU's L1 and the chiplet's L2 that the whole workgroup uses);
// COHERENT: no acquire, the data is then read with device-coherent loads.
template <int SYNC>
__device__ __forceinline__ bool check_counter(const uint32_t* counter, uint32_t target, uint32_t* status) {
    __shared__ int s_ok;
    if (threadIdx.x == 0) {
        const int ok = __hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target;
        if (ok) {
            if constexpr (SYNC != FO_SYNC_COHERENT) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        } else if (status) {
            __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        s_ok = ok;
    }
    __syncthreads();
    if constexpr (SYNC == FO_SYNC_FENCE_ALL) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
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

// The streaming functions take the thread's first unit index in the segment
// in `i0` (below the grid size) and leave there its first index in the next
// segment: the grid-stride sequence runs on across the launch's segments as
// if they were one buffer, so the threads that take a segment's last partial
// round start the next one later and every thread ends up with the same
// share of the group (restarting each segment at the thread's own index left
// the low-numbered threads with one extra, latency-bound round per segment).

// Stream one segment, 16 bytes per lane per access (FENCE_ALL / FENCE_ONE;
// src, peer and dst 16-byte aligned): nontemporal loads and stores.
template <int DT, bool SUM, int kUnroll, bool WT>
__device__ __forceinline__ void stream_vec16(const uint16_t* __restrict__ src, const uint16_t* __restrict__ peer,
                                             uint16_t* __restrict__ dst, int64_t len, uint32_t& i0) {
    int64_t i = i0;
    const int64_t n16 = len >> 3;
    const u32x4_t* s = reinterpret_cast<const u32x4_t*>(src);
    const u32x4_t* q = reinterpret_cast<const u32x4_t*>(peer);
    u32x4_t* d = reinterpret_cast<u32x4_t*>(dst);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
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
        for (int u = 0; u < kUnroll; ++u) put16<WT>(d + i + u * stride, x[u]);
    }
    for (; i < n16; i += stride) {
        u32x4_t x = __builtin_nontemporal_load(s + i);
        if constexpr (SUM) x = add8<DT>(x, __builtin_nontemporal_load(q + i));
        put16<WT>(d + i, x);
    }
    i0 = (uint32_t)(i - n16);
    // ragged tail (< 8 elements)
    if (blockIdx.x == 0 && threadIdx.x < (len & 7)) {
        const int64_t e = (n16 << 3) + threadIdx.x;
        put2<WT>(dst + e, SUM ? add1<DT>(src[e], peer[e]) : src[e]);
    }
}

// Stream one segment with device-coherent 8-byte source loads (COHERENT;
// src, peer and dst 8-byte aligned). Two 8-byte units per lane per
// unrolled step.
template <int DT, bool SUM, int kUnroll, bool WT>
__device__ __forceinline__ void stream_coherent8(const uint16_t* __restrict__ src,
                                                 const uint16_t* __restrict__ peer,
                                                 uint16_t* __restrict__ dst, int64_t len, uint32_t& i0) {
    int64_t i = i0;
    constexpr int U = 2 * kUnroll;
    const int64_t n8 = len >> 2;
    const uint64_t* s = reinterpret_cast<const uint64_t*>(src);
    const uint64_t* q = reinterpret_cast<const uint64_t*>(peer);
    uint64_t* d = reinterpret_cast<uint64_t*>(dst);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    auto add4 = [](uint64_t x, uint64_t y) -> uint64_t {
        u32x4_t a, b;
        a[0] = (uint32_t)x; a[1] = (uint32_t)(x >> 32); a[2] = 0; a[3] = 0;
        b[0] = (uint32_t)y; b[1] = (uint32_t)(y >> 32); b[2] = 0; b[3] = 0;
        const u32x4_t r = add8<DT>(a, b);
        return (uint64_t)r[0] | ((uint64_t)r[1] << 32);
    };
    for (; i + (U - 1) * stride < n8; i += U * stride) {
        uint64_t x[U], y[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            x[u] = __hip_atomic_load(s + i + u * stride, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if constexpr (SUM) {
#pragma unroll
            for (int u = 0; u < U; ++u) y[u] = __builtin_nontemporal_load(q + i + u * stride);
#pragma unroll
            for (int u = 0; u < U; ++u) x[u] = add4(x[u], y[u]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) put8<WT>(d + i + u * stride, x[u]);
    }
    for (; i < n8; i += stride) {
        uint64_t x = __hip_atomic_load(s + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if constexpr (SUM) x = add4(x, __builtin_nontemporal_load(q + i));
        put8<WT>(d + i, x);
    }
    i0 = (uint32_t)(i - n8);
    // ragged tail (< 4 elements): an acquire, then plain 2-byte loads
    if (blockIdx.x == 0 && threadIdx.x < (len & 3)) {
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        const int64_t e = (n8 << 2) + threadIdx.x;
        put2<WT>(dst + e, SUM ? add1<DT>(src[e], peer[e]) : src[e]);
    }
}

// Stream one segment with device-coherent 16-byte source loads (COHERENT;
// src, peer and dst 16-byte aligned, len * 2 < 2^31): buffer loads with the
// sc1 cache policy, which a relaxed agent-scope atomic load also uses, so
// the data the GEMM wrote through to memory is read past this chiplet's L2,
// plus the nontemporal hint: the stream is read once, and without the hint it
// displaces the GEMM's operands from the memory-side cache (measured: the
// GEMM beside the consumers 415 -> 398 us at 8192x8192x3584).
template <int DT, bool SUM, int kUnroll, bool WT>
__device__ __forceinline__ void stream_coherent16(const uint16_t* __restrict__ src,
                                                  const uint16_t* __restrict__ peer,
                                                  uint16_t* __restrict__ dst, int64_t len, uint32_t& i0) {
    int64_t i = i0;
    constexpr int kSc1Nt = 16 | 2;   // cache policy operand: sc1, nt
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void*)src, 0, (int)(len * 2), kRsrcWord3);
    const int64_t n16 = len >> 3;
    const u32x4_t* q = reinterpret_cast<const u32x4_t*>(peer);
    u32x4_t* d = reinterpret_cast<u32x4_t*>(dst);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i + (kUnroll - 1) * stride < n16; i += kUnroll * stride) {
        u32x4_t x[kUnroll], y[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            x[u] = bit_cast<u32x4_t>(__builtin_amdgcn_raw_buffer_load_b128(rs, (int)((i + u * stride) * 16), 0, kSc1Nt));
        if constexpr (SUM) {
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) y[u] = __builtin_nontemporal_load(q + i + u * stride);
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) x[u] = add8<DT>(x[u], y[u]);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) put16<WT>(d + i + u * stride, x[u]);
    }
    for (; i < n16; i += stride) {
        u32x4_t x = bit_cast<u32x4_t>(__builtin_amdgcn_raw_buffer_load_b128(rs, (int)(i * 16), 0, kSc1Nt));
        if constexpr (SUM) x = add8<DT>(x, __builtin_nontemporal_load(q + i));
        put16<WT>(d + i, x);
    }
    i0 = (uint32_t)(i - n16);
    // ragged tail (< 8 elements): an acquire, then plain 2-byte loads
    if (blockIdx.x == 0 && threadIdx.x < (len & 7)) {
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        const int64_t e = (n16 << 3) + threadIdx.x;
        put2<WT>(dst + e, SUM ? add1<DT>(src[e], peer[e]) : src[e]);
    }
}

// Stream one segment element by element (unaligned buffers).
template <int DT, bool SUM, bool WT>
__device__ __forceinline__ void stream_elem(const uint16_t* __restrict__ src, const uint16_t* __restrict__ peer,
                                            uint16_t* __restrict__ dst, int64_t len, uint32_t& i0) {
    int64_t i = i0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < len; i += stride)
        put2<WT>(dst + i, SUM ? add1<DT>(src[i], peer[i]) : src[i]);
    i0 = (uint32_t)(i - len);
}

enum { kPathVec16 = 0, kPathCoherent8 = 1, kPathElem = 2, kPathCoherent16 = 3 };

// SYNC: how the group is published to the workgroup (check_counter).
// PATH: kPathCoherent16 / kPathCoherent8 go with SYNC == COHERENT;
// kPathElem (unaligned buffers) waits with FENCE_ALL in every mode, since
// plain loads follow.
// WT: the launch counts its finished workgroups in *a.done (non-null):
// every workgroup, written or not, writes through (put16 and friends), waits
// until its stores are complete, and adds 1, so a wait for the grid size on
// another stream covers the whole launch.
template <int DT, bool SUM, int SYNC, int PATH, int U, bool WT>
__global__ __launch_bounds__(kMaxThreads) void consume_kernel(const ConsumeArgs a) {
    if (!a.counter || check_counter<SYNC>(a.counter, a.target, a.status)) {
        uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;   // < grid size: fits 32 bits
        for (int k = 0; k < a.nseg; ++k) {
            const ConsumeSegment g = a.seg[k];
            const uint16_t* src = a.src + g.src_off;
            const uint16_t* peer = SUM ? a.peer + g.src_off : nullptr;
            uint16_t* dst = a.dst + g.dst_off;
            if constexpr (PATH == kPathVec16) stream_vec16<DT, SUM, U, WT>(src, peer, dst, g.len, i);
            else if constexpr (PATH == kPathCoherent16) stream_coherent16<DT, SUM, U, WT>(src, peer, dst, g.len, i);
            else if constexpr (PATH == kPathCoherent8) stream_coherent8<DT, SUM, U, WT>(src, peer, dst, g.len, i);
            else stream_elem<DT, SUM, WT>(src, peer, dst, g.len, i);
        }
    }
    if constexpr (WT) {
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (threadIdx.x == 0) {
            // Count only for this launch's own run: once a later run's reset
            // has put its tag into the word, a late workgroup leaves it alone.
            // (A plain add after the check: a compare-and-swap loop would
            // serialise the grid's workgroups on one word, about a
            // microsecond each. A late workgroup can only race with a later
            // run's reset if an earlier wait of the stream pair timed out,
            // which the sticky status bit already reports.)
            uint32_t* w = a.done + (blockIdx.x % kDoneWords) * kDoneStride;
            const uint32_t v = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if ((v & 0xFFFF0000u) == a.done_tag)
                __hip_atomic_fetch_add(w, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// Unroll of the 8-byte coherent path (outputs past a 31-bit byte range): at
// most 4 x 2 units per thread in flight, 2 x 2 for bf16, whose sums need
// more registers (4 x 2 bf16 units took ~87 registers, more than a SIMD
// running a 256x256 GEMM wave leaves free).
template <int DT, int U>
constexpr int kUnit8Unroll = DT == FO_BF16 ? (U < 2 ? U : 2) : (U < 4 ? U : 4);

template <int DT, bool SUM, int U, bool WT>
void launch_variant(int sync, int path, dim3 g, dim3 b, hipStream_t s, const ConsumeArgs& a) {
    if (path == kPathCoherent16)
        hipLaunchKernelGGL((consume_kernel<DT, SUM, FO_SYNC_COHERENT, kPathCoherent16, U, WT>), g, b, 0, s, a);
    else if (path == kPathCoherent8)   // bf16 sums: fewer 8-byte units in flight (the budget of registers)
        hipLaunchKernelGGL((consume_kernel<DT, SUM, FO_SYNC_COHERENT, kPathCoherent8, kUnit8Unroll<DT, U>, WT>), g,
                           b, 0, s, a);
    else if (path == kPathVec16 && sync == FO_SYNC_FENCE_ALL)
        hipLaunchKernelGGL((consume_kernel<DT, SUM, FO_SYNC_FENCE_ALL, kPathVec16, U, WT>), g, b, 0, s, a);
    else if (path == kPathVec16)
        hipLaunchKernelGGL((consume_kernel<DT, SUM, FO_SYNC_FENCE_ONE, kPathVec16, U, WT>), g, b, 0, s, a);
    else
        hipLaunchKernelGGL((consume_kernel<DT, SUM, FO_SYNC_FENCE_ALL, kPathElem, U, WT>), g, b, 0, s, a);
}

// A counting launch (a.done) is the last group's; it takes the unroll its
// `full` flag asks for like any other launch.
// A copy has one load per unit where a sum has two, so it unrolls twice as
// far for the same bytes in flight per thread.
template <int DT, bool SUM>
void launch_unroll(bool full, int sync, int path, dim3 g, dim3 b, hipStream_t s, const ConsumeArgs& a) {
    constexpr int kFull = SUM ? kUnrollFull : 2 * kUnrollFull;
    constexpr int kBeside = SUM ? kUnrollBeside : 2 * kUnrollBeside;
    if (a.done && full) launch_variant<DT, SUM, kFull, true>(sync, path, g, b, s, a);
    else if (a.done) launch_variant<DT, SUM, kBeside, true>(sync, path, g, b, s, a);
    else if (full) launch_variant<DT, SUM, kFull, false>(sync, path, g, b, s, a);
    else launch_variant<DT, SUM, kBeside, false>(sync, path, g, b, s, a);
}

}  // namespace

hipError_t launch_wait(const uint32_t* counter, uint32_t target, uint32_t* status, uint64_t timeout_ticks,
                       hipStream_t s) {
    hipLaunchKernelGGL(wait_kernel, dim3(1), dim3(64), 0, s, counter, target, status, timeout_ticks);
    return hipGetLastError();
}

hipError_t launch_done_wait(const uint32_t* done, uint32_t done_tag, int32_t blocks, uint32_t* status,
                            uint64_t timeout_ticks, hipStream_t s) {
    hipLaunchKernelGGL(done_wait_kernel, dim3(1), dim3(64), 0, s, done, done_tag, blocks, status, timeout_ticks);
    return hipGetLastError();
}

hipError_t launch_gate(uint32_t* gate, uint32_t tag, uint32_t* status, uint64_t timeout_ticks, hipStream_t s) {
    hipLaunchKernelGGL(gate_kernel, dim3(1), dim3(64), 0, s, gate, tag, status, timeout_ticks);
    return hipGetLastError();
}

hipError_t launch_consume(int dtype, int sync, const ConsumeArgs& a, int max_blocks, int threads, bool full,
                          hipStream_t s, int* launched_blocks) {
    // The path is chosen once for the launch: every segment's pointers must
    // allow it.
    uintptr_t bits = 0;
    int64_t total = 0, longest = 0;
    for (int k = 0; k < a.nseg; ++k) {
        bits |= reinterpret_cast<uintptr_t>(a.src + a.seg[k].src_off) |
                reinterpret_cast<uintptr_t>(a.dst + a.seg[k].dst_off);
        if (a.peer) bits |= reinterpret_cast<uintptr_t>(a.peer + a.seg[k].src_off);
        total += a.seg[k].len;
        longest = a.seg[k].len > longest ? a.seg[k].len : longest;
    }
    const bool vec16 = (bits & 15) == 0, vec8 = (bits & 7) == 0;
    // the 16-byte coherent path addresses a segment with 32-bit byte offsets
    const bool fits32 = longest * 2 <= 0x7FFFFFFF;
    const int path = sync == FO_SYNC_COHERENT
                         ? (vec16 && fits32 ? kPathCoherent16 : vec8 ? kPathCoherent8 : kPathElem)
                         : (vec16 ? kPathVec16 : kPathElem);
    // elements one workgroup moves per unrolled round (the unrolls of
    // launch_unroll and kUnit8Unroll), for the grid of a short launch
    const bool sum = a.peer != nullptr;
    const int unroll = (full ? kUnrollFull : kUnrollBeside) * (sum ? 1 : 2);
    const int unroll8 = dtype == FO_BF16 ? (unroll < 2 ? unroll : 2) : (unroll < 4 ? unroll : 4);
    const int64_t per_block = path == kPathCoherent8 ? (int64_t)threads * 2 * unroll8 * 4
                              : path == kPathVec16 || path == kPathCoherent16 ? (int64_t)threads * unroll * 8
                                                                               : (int64_t)threads;
    int64_t blocks = (total + per_block - 1) / per_block;
    if (blocks < 1) blocks = 1;
    if (blocks > max_blocks) blocks = max_blocks;
    const dim3 g((unsigned)blocks), b((unsigned)threads);
    if (launched_blocks) *launched_blocks = (int)blocks;
    if (a.counter) {
        hipLaunchKernelGGL(wait_kernel, dim3(1), dim3(64), 0, s, a.counter, a.target, a.status, a.timeout_ticks);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (dtype == FO_FP16) {
        if (sum) launch_unroll<FO_FP16, true>(full, sync, path, g, b, s, a);
        else launch_unroll<FO_FP16, false>(full, sync, path, g, b, s, a);
    } else {
        if (sum) launch_unroll<FO_BF16, true>(full, sync, path, g, b, s, a);
        else launch_unroll<FO_BF16, false>(full, sync, path, g, b, s, a);
    }
    return hipGetLastError();
}

}  // namespace fo
