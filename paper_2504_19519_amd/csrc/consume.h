// Launch interface of the consumer kernels (internal to libfo).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fo {

// Largest consumer grid: one workgroup per compute unit.
constexpr int kMaxConsumeBlocks = 256;
// Segments one launch can carry (a group has R or B of them).
constexpr int kMaxConsumeSegments = 16;

// One contiguous piece of a group: `len` elements at src + src_off (and
// peer + src_off) go to dst + dst_off.
struct ConsumeSegment {
    int64_t src_off, dst_off, len;
};

struct ConsumeArgs {
    const uint16_t* src;
    const uint16_t* peer;        // nullptr: copy
    uint16_t* dst;
    const uint32_t* counter;     // nullptr: no wait
    uint32_t target;
    uint32_t* status;            // bit 0 set on a timed-out wait (may be nullptr)
    uint64_t timeout_ticks;      // wall-clock ticks
    int32_t nseg;                // 1 .. kMaxConsumeSegments
    ConsumeSegment seg[kMaxConsumeSegments];
};

// One launch: wait once for *counter >= target, then stream every segment.
// max_blocks caps the grid (1 .. kMaxConsumeBlocks); threads per workgroup:
// 64, 128 or 256. full: the launch has the device to itself (more accesses
// in flight per thread); otherwise it runs beside the GEMM and keeps its
// registers within what a SIMD running two GEMM waves has left.
hipError_t launch_consume(int dtype, int sync, const ConsumeArgs& a, int max_blocks, int threads, bool full,
                          hipStream_t s);

}  // namespace fo
