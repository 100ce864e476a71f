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
    uint32_t* done;              // non-null: done word 0; workgroup b adds 1 to word b % kDoneWords
                                 // (kDoneStride words apart) when its stores are visible, while
                                 // that word's high half equals done_tag's
    uint32_t done_tag;           // run tag of the done word (done_tag_of)
    int32_t nseg;                // 1 .. kMaxConsumeSegments
    ConsumeSegment seg[kMaxConsumeSegments];
};

// One launch: wait once for *counter >= target, then stream every segment.
// max_blocks caps the grid (1 .. kMaxConsumeBlocks); threads per workgroup:
// 64, 128 or 256. full: the launch has the device to itself (more accesses
// in flight per thread); otherwise it runs beside the GEMM and keeps its
// registers within what a SIMD running two GEMM waves has left.
// *blocks (if non-null) receives the streaming kernel's grid size.
hipError_t launch_consume(int dtype, int sync, const ConsumeArgs& a, int max_blocks, int threads, bool full,
                          hipStream_t s, int* blocks = nullptr);

// One wave that polls until *counter >= target (bounded by timeout_ticks;
// on timeout bit 0 of *status is raised).
hipError_t launch_wait(const uint32_t* counter, uint32_t target, uint32_t* status, uint64_t timeout_ticks,
                       hipStream_t s);

// Tags of the start handoff of an overlapped run: the run's reset kernel
// writes its tag (bit 31 and 30 bits of the run's sequence number) into the
// gate word once the counters are zero; the gate kernel on the other stream
// waits for that tag. A gate that times out while the word holds an older
// run's tag replaces it by tag | kGateTimedOut, which the reset kernel, if it
// runs later, turns into bit 0 of the status word; a gate that times out
// after a later run's tag has arrived only raises the status bit.
constexpr uint32_t kGateTag = 0x80000000u;
constexpr uint32_t kGateTimedOut = 0x40000000u;
constexpr uint32_t kGateSeqMask = kGateTimedOut - 1;
// Done words of an overlapped run: the low 16 bits of the run's sequence
// number in the high half, a count of finished final-consumer workgroups in
// the low half. The count is spread over kDoneWords words kDoneStride words
// apart (each in a 128-byte line of its own): workgroup b counts in word
// b % kDoneWords, so that at most ceil(grid / kDoneWords) device-scope adds
// meet on one address (256 adds on one word took ~8 us to drain).
constexpr int kDoneWords = 8;
constexpr int kDoneStride = 32;
__host__ __device__ inline uint32_t done_tag_of(uint32_t seq) { return (seq & 0xFFFFu) << 16; }
// Workgroups b < blocks with b % kDoneWords == k.
__host__ __device__ inline uint32_t done_share(int32_t blocks, int k) {
    return blocks > k ? (uint32_t)((blocks - 1 - k) / kDoneWords + 1) : 0u;
}
// One wave that polls the done words until word k reaches done_tag plus
// done_share(blocks, k) for every k (bounded like launch_wait).
hipError_t launch_done_wait(const uint32_t* done, uint32_t done_tag, int32_t blocks, uint32_t* status,
                            uint64_t timeout_ticks, hipStream_t s);
hipError_t launch_gate(uint32_t* gate, uint32_t tag, uint32_t* status, uint64_t timeout_ticks, hipStream_t s);

}  // namespace fo
