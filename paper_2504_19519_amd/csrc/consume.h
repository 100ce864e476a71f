// Launch interface of the consumer kernels (internal to libfo).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fo {

// Largest consumer grid. With 256-thread workgroups this is at most one
// wave per SIMD on average, far from what could keep the GEMM off a CU.
constexpr int kMaxConsumeBlocks = 256;

hipError_t launch_consume(int dtype, int sync, const uint16_t* src, const uint16_t* peer, uint16_t* dst,
                          int64_t len, const uint32_t* counter, uint32_t target, uint32_t* status,
                          uint64_t timeout_ticks, hipStream_t s);

}  // namespace fo
