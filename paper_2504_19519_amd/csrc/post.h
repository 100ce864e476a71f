// Launch interface of the post-communication reorder kernel (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fo {

struct PostArgs {
    const uint16_t* src;        // consumer destination buffer
    uint16_t* out;              // [M, N] row-major
    const uint16_t* bias;       // [N] or null
    const uint16_t* gamma;      // [N] or null
    int64_t M, N;
    int32_t tile_m, tile_n, tiles_n, pattern, num_dest;
    int32_t cpt_log2;           // log2(tile_n / 8) for reordered patterns; 31 for row-major
                                // (a row is one piece)
    int64_t per_dest;           // SUBTILE: elements of one destination buffer
    const int32_t* tile_to_slot;
    const int32_t* dest_perm;
    const int32_t* row_bucket;
    const int32_t* row_rank;
    const int32_t* pool_base;
    const int32_t* pool_off;
    float eps;
    int32_t do_norm;
};

// LDS bytes one post-reorder workgroup uses (source piece offsets of its 4
// rows; bias and gamma chunks when the row is normalised in registers).
size_t post_lds_bytes(const PostArgs& a);
hipError_t launch_post(int dtype, const PostArgs& a, hipStream_t s);

}  // namespace fo
