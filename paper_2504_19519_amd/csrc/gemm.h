// Launch interface of the signalling GEMM kernel (internal to libfo).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fo {

struct GemmArgs {
    const uint16_t* A;          // [M, K]
    const uint16_t* W;          // [N, K]
    uint16_t* C;                // output buffer, layout by pattern
    int64_t M, N, K;
    int32_t tiles_m, tiles_n;
    int32_t order, group_m, num_xcds;
    int32_t pattern, num_dest;
    const int32_t* tile_to_slot;   // device plan tables (may be null for ROWMAJOR)
    const int32_t* slot_group;
    const int32_t* group_first;
    const int32_t* row_bucket;
    const int32_t* row_rank;
    const int32_t* pool_base;
    const int32_t* pool_off;
    uint32_t* counters;            // [P] or null
    uint32_t* dispenser;           // [num_dispensers] zeroed position counters, or null
    int32_t num_dispensers;        // D >= 1 (with a dispenser)
    int32_t sync;                  // fo_sync_mode of the producer side
    int32_t c_rsrc;                // 1: C fits a 31-bit byte range (16-byte buffer stores)
    uint64_t* trace;               // [4 * trace_cap] tile timeline, or null
    int64_t trace_cap;
};

// grid: number of persistent workgroups (at most the number of tiles; with
// a dispenser, a multiple of num_dispensers).
hipError_t launch_gemm(int dtype, int tile_m, int tile_n, const GemmArgs& a, int grid, hipStream_t s);
bool gemm_tile_supported(int tile_m, int tile_n);

}  // namespace fo
