// Internal declarations shared by the planner, the kernels' launchers and the
// runtime glue of libfo. Not part of the public ABI (see include/fo.h).
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "fo.h"

#if defined(__HIPCC__)
#define FO_HD __host__ __device__
#else
#define FO_HD
#endif

namespace fo {

// Tile computed by the workgroup at dispatch position p (fo_order in fo.h).
// The GEMM kernel evaluates this on the device for its blockIdx, the planner
// on the host for the reorder map, so both always agree.
FO_HD inline int32_t tile_of_position(int32_t p, int32_t tiles_m, int32_t tiles_n,
                                      int32_t order, int32_t group_m, int32_t num_xcds) {
    if (order == FO_ORDER_ROWMAJOR) return p;
    const int32_t tiles = tiles_m * tiles_n;
    int32_t q = p;
    if (order == FO_ORDER_XCD) {
        const int32_t per = (tiles + num_xcds - 1) / num_xcds;
        int32_t full = tiles % num_xcds;
        if (full == 0) full = num_xcds;
        const int32_t x = p % num_xcds;
        const int32_t l = p / num_xcds;
        q = x < full ? x * per + l : full * per + (x - full) * (per - 1) + l;
    }
    const int32_t band_tiles = group_m * tiles_n;
    const int32_t band = q / band_tiles;
    const int32_t first = band * group_m;
    const int32_t rows = (tiles_m - first) < group_m ? (tiles_m - first) : group_m;
    const int32_t r = q - band * band_tiles;
    const int32_t tm = first + r % rows;
    const int32_t tn = r / rows;
    return tm * tiles_n + tn;
}

inline int dtype_bytes(int32_t) { return 2; }

// Set the calling thread's last error and return `st`.
fo_status fail(fo_status st, const std::string& msg);
void clear_error();

// Poll timeout in microseconds (runtime.hip).
int64_t poll_timeout_us();

}  // namespace fo

// Word offsets of the tables inside the device image (all int32, each
// section starts on a 16-byte boundary).
struct fo_dev_layout {
    int64_t tile_to_slot = 0;   // [tiles]
    int64_t slot_group = 0;     // [tiles]
    int64_t group_first = 0;    // [P+1]
    int64_t dest_perm = -1;     // [R]          SUBTILE
    int64_t row_bucket = -1;    // [M]          SUBTOKEN
    int64_t row_rank = -1;      // [M]          SUBTOKEN
    int64_t pool_base = -1;     // [(tiles+1)B] SUBTOKEN
    int64_t pool_off = -1;      // [B+1]        SUBTOKEN
    int64_t words = 0;
};

struct fo_plan {
    int64_t M = 0, N = 0, K = 0;
    int32_t dtype = 0, tile_m = 0, tile_n = 0, order = 0, group_m = 1, num_xcds = 1;
    int32_t num_cus = 0, wg_per_cu = 1, reserved_cus = 0, pattern = 0, num_dest = 0;
    int32_t unit = FO_UNIT_WAVES;
    int32_t tiles_m = 0, tiles_n = 0, tiles = 0, W = 0, T = 0, P = 0;
    double predicted_us = 0.0;
    int64_t dest_elems = 0;
    std::vector<int32_t> sizes;         // [P] in `unit`
    std::vector<int32_t> order_tbl;     // [tiles] position -> tile
    std::vector<int32_t> tile_to_slot;  // [tiles]
    std::vector<int32_t> slot_group;    // [tiles]
    std::vector<int32_t> group_first;   // [P+1]
    std::vector<int32_t> targets;       // [P]
    std::vector<int32_t> dest_perm;     // [R]
    std::vector<int32_t> row_bucket;    // [M]
    std::vector<int32_t> row_rank;      // [M]
    std::vector<int32_t> pool_base;     // [(tiles+1)*B]
    std::vector<int32_t> pool_off;      // [B+1]
    std::vector<int64_t> segs;          // [nseg*5]
    fo_dev_layout layout;
    std::vector<int32_t> image;         // device image (layout.words)
};
