// Host planner: tile dispatch order, waves, wave groups (explicit or by the
// predictive search of Algorithm 1), the reorder map, counter targets,
// communication segments and the device image of the tables.
//
// Paper passages: waves (Section 2.1.1), block swizzling (Section 2.1.2),
// group-wise tile counting (Section 3.2 Approach), execution-order-aware
// reordering (Section 3.3 Approach), design space (Section 3.4), predictive
// search (Section 4.1, Algorithm 1; Section 4.2 online stage).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <limits>
#include <new>

#include "fo_internal.h"

namespace {

constexpr int kMaxSearchWaves = 24;

// Piecewise-linear latency of `bytes` on the sampled curve; outside the
// samples the latency scales with size at the end point's bandwidth.
double interp_latency(const double* xs, const double* ys, int n, double bytes) {
    if (bytes <= 0.0) return 0.0;
    if (bytes <= xs[0]) return ys[0] * bytes / xs[0];
    if (bytes >= xs[n - 1]) return ys[n - 1] * bytes / xs[n - 1];
    int i = 1;
    while (bytes > xs[i]) ++i;
    const double x0 = xs[i - 1], x1 = xs[i], y0 = ys[i - 1], y1 = ys[i];
    return y0 + (y1 - y0) * (bytes - x0) / (x1 - x0);
}

// Slot range [f0, f1) of every group of a partition given in waves.
void firsts_from_waves(const std::vector<int32_t>& sizes, int32_t W, int32_t tiles,
                       std::vector<int32_t>& first) {
    first.assign(sizes.size() + 1, 0);
    int64_t acc = 0;
    for (size_t j = 0; j < sizes.size(); ++j) {
        acc += sizes[j];
        first[j + 1] = (int32_t)std::min<int64_t>(acc * W, tiles);
    }
}

// Bytes handed to the communication by slots [f0, f1) (Algorithm 1,
// get_data_size); All-to-All takes its largest per-destination piece unless
// all_dest (then every piece of the group counts).
double range_bytes(const fo_plan& p, int32_t f0, int32_t f1, bool all_dest) {
    const double eb = fo::dtype_bytes(p.dtype);
    if (p.pattern == FO_PATTERN_SUBTOKEN && !all_dest) {
        int64_t mx = 0;
        for (int b = 0; b < p.num_dest; ++b) {
            const int64_t n = (int64_t)p.pool_base[(size_t)f1 * p.num_dest + b] -
                              p.pool_base[(size_t)f0 * p.num_dest + b];
            mx = std::max(mx, n);
        }
        return (double)mx * p.tile_n * eb;
    }
    return (double)(f1 - f0) * p.tile_m * p.tile_n * eb;
}

// Predicted overlapped latency of one partition (Section 4.1, the estimate
// Algorithm 1 ranks candidates by): the GEMM's time is spread evenly over
// its waves, so group g's computation is done at C_g, the time of the waves
// up to and including g; its communication starts once that computation and
// the previous group's communication are both done, and takes the curve's
// latency for the group's bytes: E_g = max(C_g, E_(g-1)) + comm(g), with
// E_(-1) = 0. The partition's latency is the last group's E. The last
// group's latency comes from the grouping's second curve when it has one
// (its communication runs after the GEMM).
double predict(const fo_plan& p, const std::vector<int32_t>& sizes, double gemm_us,
               const fo_grouping& g, std::vector<int32_t>& first_scratch) {
    firsts_from_waves(sizes, p.W, p.tiles, first_scratch);
    auto comm = [&](size_t j) {
        const double bytes = range_bytes(p, first_scratch[j], first_scratch[j + 1], g.all_dest_bytes != 0);
        if (j + 1 == sizes.size() && g.last_curve_len > 0)
            return interp_latency(g.last_curve_bytes, g.last_curve_us, g.last_curve_len, bytes);
        return interp_latency(g.curve_bytes, g.curve_us, g.curve_len, bytes);
    };
    double compute_done = 0.0;   // C_g
    double comm_done = 0.0;      // E_(g-1), then E_g
    for (size_t j = 0; j < sizes.size(); ++j) {
        compute_done += gemm_us / p.T * sizes[j];
        comm_done = std::max(compute_done, comm_done) + comm(j);
    }
    return comm_done;
}

fo_status check_curve(const fo_grouping& g) {
    for (int i = 0; i < g.curve_len; ++i) {
        if (!(g.curve_bytes[i] > 0.0) || !(g.curve_us[i] >= 0.0) ||
            (i > 0 && !(g.curve_bytes[i] > g.curve_bytes[i - 1])))
            return fo::fail(FO_ERR_ARG, "curve bytes must be positive and ascending, latencies >= 0");
    }
    if (g.last_curve_len < 0 || (g.last_curve_len > 0 && (!g.last_curve_bytes || !g.last_curve_us)))
        return fo::fail(FO_ERR_ARG, "last-group curve: length >= 0 and both arrays when it is > 0");
    for (int i = 0; i < g.last_curve_len; ++i) {
        if (!(g.last_curve_bytes[i] > 0.0) || !(g.last_curve_us[i] >= 0.0) ||
            (i > 0 && !(g.last_curve_bytes[i] > g.last_curve_bytes[i - 1])))
            return fo::fail(FO_ERR_ARG, "last-group curve bytes must be positive and ascending, latencies >= 0");
    }
    if (!(g.gemm_us >= 0.0)) return fo::fail(FO_ERR_ARG, "gemm_us must be >= 0");
    if (g.all_dest_bytes != 0 && g.all_dest_bytes != 1) return fo::fail(FO_ERR_ARG, "all_dest_bytes must be 0 or 1");
    return FO_OK;
}

fo_status search(fo_plan& p, const fo_grouping& g) {
    if (p.T == 0) return FO_OK;
    if (p.T > kMaxSearchWaves)
        return fo::fail(FO_ERR_UNSUPPORTED, "predictive search supports at most 24 waves");
    const int32_t s1 = g.s_first > 0 ? g.s_first : p.T;
    const int32_t sp = g.s_last > 0 ? g.s_last : p.T;
    double best_t = std::numeric_limits<double>::infinity();
    std::vector<int32_t> sizes, best, first;
    const uint64_t count = 1ull << (p.T - 1);
    for (uint64_t x = 0; x < count; ++x) {
        // cut after wave i+1 when bit i of x is set; the last wave closes a group
        sizes.clear();
        int32_t run = 0;
        for (int32_t w = 1; w <= p.T; ++w) {
            ++run;
            if (w == p.T || ((x >> (w - 1)) & 1ull)) {
                sizes.push_back(run);
                run = 0;
            }
        }
        if (sizes.front() > s1 || sizes.back() > sp) continue;
        const double t = predict(p, sizes, g.gemm_us, g, first);
        if (t < best_t) {
            best_t = t;
            best = sizes;
        }
    }
    if (best.empty()) return fo::fail(FO_ERR_ARG, "no partition satisfies the pruning bounds");
    p.sizes = best;
    p.predicted_us = best_t;
    return FO_OK;
}

int64_t align4(int64_t w) { return (w + 3) & ~int64_t(3); }

void build_image(fo_plan& p) {
    fo_dev_layout& L = p.layout;
    int64_t w = 0;
    L.tile_to_slot = w; w = align4(w + p.tiles);
    L.slot_group = w;   w = align4(w + p.tiles);
    L.group_first = w;  w = align4(w + p.P + 1);
    if (p.pattern == FO_PATTERN_SUBTILE) { L.dest_perm = w; w = align4(w + p.num_dest); }
    if (p.pattern == FO_PATTERN_SUBTOKEN) {
        L.row_bucket = w; w = align4(w + p.M);
        L.row_rank = w;   w = align4(w + p.M);
        L.pool_base = w;  w = align4(w + (int64_t)(p.tiles + 1) * p.num_dest);
        L.pool_off = w;   w = align4(w + p.num_dest + 1);
    }
    L.words = std::max<int64_t>(w, 4);
    p.image.assign((size_t)L.words, 0);
    auto put = [&](int64_t off, const std::vector<int32_t>& v) {
        std::copy(v.begin(), v.end(), p.image.begin() + off);
    };
    put(L.tile_to_slot, p.tile_to_slot);
    put(L.slot_group, p.slot_group);
    put(L.group_first, p.group_first);
    if (L.dest_perm >= 0) put(L.dest_perm, p.dest_perm);
    if (L.row_bucket >= 0) {
        put(L.row_bucket, p.row_bucket);
        put(L.row_rank, p.row_rank);
        put(L.pool_base, p.pool_base);
        put(L.pool_off, p.pool_off);
    }
}

fo_status build(fo_plan& p, const fo_problem& pr, const fo_grouping& g) {
    if (pr.M < 0 || pr.N < 0 || pr.K < 0) return fo::fail(FO_ERR_SHAPE, "negative dimension");
    if (pr.tile_m < 1 || pr.tile_n < 1) return fo::fail(FO_ERR_ARG, "tile_m and tile_n must be >= 1");
    if (pr.M % pr.tile_m || pr.N % pr.tile_n)
        return fo::fail(FO_ERR_SHAPE, "M and N must be multiples of tile_m and tile_n");
    if (pr.dtype != FO_FP16 && pr.dtype != FO_BF16) return fo::fail(FO_ERR_ARG, "bad dtype");
    if (pr.order < FO_ORDER_ROWMAJOR || pr.order > FO_ORDER_XCD) return fo::fail(FO_ERR_ARG, "bad order");
    if (pr.order != FO_ORDER_ROWMAJOR && pr.group_m < 1) return fo::fail(FO_ERR_ARG, "group_m must be >= 1");
    if (pr.order == FO_ORDER_XCD && pr.num_xcds < 1) return fo::fail(FO_ERR_ARG, "num_xcds must be >= 1");
    if (pr.num_cus < 1 || pr.wg_per_cu < 1 || pr.reserved_cus < 0 || pr.reserved_cus >= pr.num_cus)
        return fo::fail(FO_ERR_ARG, "need num_cus >= 1, wg_per_cu >= 1, 0 <= reserved_cus < num_cus");
    if (pr.pattern < FO_PATTERN_TILE || pr.pattern > FO_PATTERN_ROWMAJOR) return fo::fail(FO_ERR_ARG, "bad pattern");
    const int64_t tiles64 = (pr.M / pr.tile_m) * (pr.N / pr.tile_n);
    if (tiles64 > (int64_t)1 << 30 || pr.M > (int64_t)1 << 30) return fo::fail(FO_ERR_SHAPE, "problem too large");
    if (pr.M * pr.N > ((int64_t)1 << 40)) return fo::fail(FO_ERR_SHAPE, "problem too large");

    p.M = pr.M; p.N = pr.N; p.K = pr.K;
    p.dtype = pr.dtype; p.tile_m = pr.tile_m; p.tile_n = pr.tile_n;
    p.order = pr.order; p.group_m = pr.order == FO_ORDER_ROWMAJOR ? 1 : pr.group_m;
    p.num_xcds = pr.order == FO_ORDER_XCD ? pr.num_xcds : 1;
    p.num_cus = pr.num_cus; p.wg_per_cu = pr.wg_per_cu; p.reserved_cus = pr.reserved_cus;
    p.pattern = pr.pattern;
    p.num_dest = (pr.pattern == FO_PATTERN_SUBTILE || pr.pattern == FO_PATTERN_SUBTOKEN) ? pr.num_dest : 0;
    p.tiles_m = (int32_t)(pr.M / pr.tile_m);
    p.tiles_n = (int32_t)(pr.N / pr.tile_n);
    p.tiles = (int32_t)tiles64;
    p.W = (pr.num_cus - pr.reserved_cus) * pr.wg_per_cu;
    p.T = p.tiles ? (p.tiles + p.W - 1) / p.W : 0;

    // dispatch order and the reorder map: slot = dispatch position
    p.order_tbl.resize(p.tiles);
    p.tile_to_slot.assign(p.tiles, -1);
    for (int32_t q = 0; q < p.tiles; ++q) {
        const int32_t t = fo::tile_of_position(q, p.tiles_m, p.tiles_n, p.order, p.group_m, p.num_xcds);
        if (t < 0 || t >= p.tiles || p.tile_to_slot[t] != -1)
            return fo::fail(FO_ERR_ARG, "dispatch order is not a bijection");
        p.order_tbl[q] = t;
        p.tile_to_slot[t] = q;
    }

    // destination data
    if (p.pattern == FO_PATTERN_SUBTILE) {
        if (p.num_dest < 1) return fo::fail(FO_ERR_ARG, "SUBTILE needs num_dest >= 1");
        if (p.tile_m % p.num_dest) return fo::fail(FO_ERR_SHAPE, "tile_m must be a multiple of num_dest");
        p.dest_perm.resize(p.num_dest);
        std::vector<char> seen(p.num_dest, 0);
        for (int k = 0; k < p.num_dest; ++k) {
            const int32_t d = pr.dest_perm ? pr.dest_perm[k] : k;
            if (d < 0 || d >= p.num_dest || seen[d]) return fo::fail(FO_ERR_ARG, "dest_perm is not a permutation");
            seen[d] = 1;
            p.dest_perm[k] = d;
        }
    }
    if (p.pattern == FO_PATTERN_SUBTOKEN) {
        if (p.num_dest < 1) return fo::fail(FO_ERR_ARG, "SUBTOKEN needs num_dest >= 1");
        if (p.M > 0 && !pr.row_bucket) return fo::fail(FO_ERR_ARG, "SUBTOKEN needs row_bucket");
        const int B = p.num_dest;
        p.row_bucket.resize(p.M);
        p.row_rank.resize(p.M);
        std::vector<int32_t> cnt((size_t)p.tiles_m * B, 0);   // rows of tile row tm bound for b
        for (int64_t i = 0; i < p.M; ++i) {
            const int32_t b = pr.row_bucket[i];
            if (b < 0 || b >= B) return fo::fail(FO_ERR_ARG, "row_bucket value out of range");
            p.row_bucket[i] = b;
            const int64_t tm = i / p.tile_m;
            p.row_rank[i] = cnt[tm * B + b]++;
        }
        p.pool_base.assign((size_t)(p.tiles + 1) * B, 0);
        for (int32_t s = 0; s < p.tiles; ++s) {
            const int32_t tm = p.order_tbl[s] / p.tiles_n;
            for (int b = 0; b < B; ++b)
                p.pool_base[(size_t)(s + 1) * B + b] = p.pool_base[(size_t)s * B + b] + cnt[(size_t)tm * B + b];
        }
        p.pool_off.assign(B + 1, 0);
        for (int b = 0; b < B; ++b)
            p.pool_off[b + 1] = p.pool_off[b] + p.pool_base[(size_t)p.tiles * B + b];
    }

    // partition
    if (g.unit != FO_UNIT_WAVES && g.unit != FO_UNIT_TILES) return fo::fail(FO_ERR_ARG, "bad unit");
    if (g.num_groups < 0) return fo::fail(FO_ERR_ARG, "num_groups must be >= 0");
    p.unit = g.unit;
    if (g.num_groups > 0) {
        if (!g.sizes) return fo::fail(FO_ERR_ARG, "sizes is NULL");
        int64_t sum = 0;
        for (int j = 0; j < g.num_groups; ++j) {
            if (g.sizes[j] < 1) return fo::fail(FO_ERR_ARG, "group sizes must be >= 1");
            sum += g.sizes[j];
        }
        const int64_t want = g.unit == FO_UNIT_WAVES ? p.T : p.tiles;
        if (sum != want) return fo::fail(FO_ERR_ARG, "group sizes must sum to the number of waves (or tiles)");
        p.sizes.assign(g.sizes, g.sizes + g.num_groups);
        // With a latency curve, the given partition gets Algorithm 1's
        // estimate too (no search).
        if (g.unit == FO_UNIT_WAVES && p.T > 0 && g.curve_len >= 1 && g.curve_bytes && g.curve_us) {
            fo_status st = check_curve(g);
            if (st != FO_OK) return st;
            std::vector<int32_t> first;
            p.predicted_us = predict(p, p.sizes, g.gemm_us, g, first);
        }
    } else {
        if (g.unit != FO_UNIT_WAVES) return fo::fail(FO_ERR_ARG, "the search partitions waves");
        if (p.T > 0) {
            if (g.curve_len < 1 || !g.curve_bytes || !g.curve_us)
                return fo::fail(FO_ERR_ARG, "the search needs a latency curve");
            fo_status st = check_curve(g);
            if (st != FO_OK) return st;
        }
        fo_status st = search(p, g);
        if (st != FO_OK) return st;
    }
    p.P = (int32_t)p.sizes.size();
    if (p.unit == FO_UNIT_WAVES) {
        firsts_from_waves(p.sizes, p.W, p.tiles, p.group_first);
    } else {
        p.group_first.assign(p.P + 1, 0);
        for (int j = 0; j < p.P; ++j) p.group_first[j + 1] = p.group_first[j] + p.sizes[j];
    }
    p.targets.resize(p.P);
    p.slot_group.assign(p.tiles, 0);
    for (int j = 0; j < p.P; ++j) {
        p.targets[j] = p.group_first[j + 1] - p.group_first[j];
        for (int32_t s = p.group_first[j]; s < p.group_first[j + 1]; ++s) p.slot_group[s] = j;
    }

    // communication segments
    const int64_t tmn = (int64_t)p.tile_m * p.tile_n;
    p.segs.clear();
    auto seg = [&](int64_t j, int64_t d, int64_t so, int64_t dso, int64_t len) {
        p.segs.insert(p.segs.end(), {j, d, so, dso, len});
    };
    if (p.pattern == FO_PATTERN_ROWMAJOR) {
        if (p.P > 0) seg(p.P - 1, 0, 0, 0, p.M * p.N);
        p.dest_elems = p.M * p.N;
    } else if (p.pattern == FO_PATTERN_TILE) {
        for (int j = 0; j < p.P; ++j)
            seg(j, 0, p.group_first[j] * tmn, p.group_first[j] * tmn, (int64_t)p.targets[j] * tmn);
        p.dest_elems = p.M * p.N;
    } else if (p.pattern == FO_PATTERN_SUBTILE) {
        const int64_t h = p.tile_m / p.num_dest;
        const int64_t per_dest = (int64_t)p.tiles * h * p.tile_n;
        for (int j = 0; j < p.P; ++j) {
            const int64_t f0 = p.group_first[j], n = p.targets[j];
            for (int k = 0; k < p.num_dest; ++k)
                seg(j, k, f0 * tmn + k * n * h * p.tile_n,
                    p.dest_perm[k] * per_dest + f0 * h * p.tile_n, n * h * p.tile_n);
        }
        p.dest_elems = per_dest * p.num_dest;
    } else {
        const int B = p.num_dest;
        for (int j = 0; j < p.P; ++j) {
            const int64_t f0 = p.group_first[j], f1 = p.group_first[j + 1];
            for (int b = 0; b < B; ++b) {
                const int64_t o = ((int64_t)p.pool_off[b] + p.pool_base[f0 * B + b]) * p.tile_n;
                const int64_t l = ((int64_t)p.pool_base[f1 * B + b] - p.pool_base[f0 * B + b]) * p.tile_n;
                seg(j, b, o, o, l);
            }
        }
        p.dest_elems = p.M * p.N;
    }
    build_image(p);
    return FO_OK;
}

// Partition of T_new waves that keeps the relative cut positions of `ref`
// (a partition of T_ref waves): a cut after wave c becomes a cut after wave
// round(c * T_new / T_ref) (halves round up); cuts that fall on 0 or T_new,
// or on an earlier cut, are dropped.
std::vector<int32_t> map_partition(const std::vector<int32_t>& ref, int32_t t_new) {
    int64_t t_ref = 0;
    for (int32_t s : ref) t_ref += s;
    std::vector<int32_t> out;
    if (t_new <= 0) return out;
    if (t_ref <= 0) return {t_new};
    int64_t cut = 0;
    int32_t prev = 0;
    for (size_t j = 0; j + 1 < ref.size(); ++j) {
        cut += ref[j];
        const int32_t c = (int32_t)((2 * cut * t_new + t_ref) / (2 * t_ref));
        if (c <= prev || c >= t_new) continue;
        out.push_back(c - prev);
        prev = c;
    }
    out.push_back(t_new - prev);
    return out;
}

// Everything of a problem but M (and the per-row bucket map, which has M
// entries): problems of one family share cached partitions.
bool same_family(const fo_problem& a, const fo_problem& b) {
    if (a.N != b.N || a.K != b.K || a.dtype != b.dtype || a.tile_m != b.tile_m || a.tile_n != b.tile_n ||
        a.order != b.order || a.num_cus != b.num_cus || a.wg_per_cu != b.wg_per_cu ||
        a.reserved_cus != b.reserved_cus || a.pattern != b.pattern)
        return false;
    if (a.order != FO_ORDER_ROWMAJOR && a.group_m != b.group_m) return false;
    if (a.order == FO_ORDER_XCD && a.num_xcds != b.num_xcds) return false;
    const bool dest = a.pattern == FO_PATTERN_SUBTILE || a.pattern == FO_PATTERN_SUBTOKEN;
    if (dest && a.num_dest != b.num_dest) return false;
    if (a.pattern == FO_PATTERN_SUBTILE) {
        for (int k = 0; k < a.num_dest; ++k) {
            const int32_t x = a.dest_perm ? a.dest_perm[k] : k, y = b.dest_perm ? b.dest_perm[k] : k;
            if (x != y) return false;
        }
    }
    return true;
}

}  // namespace

// One cached partition: the problem it was searched for (dest_perm copied,
// no bucket map) and its wave groups.
struct fo_cached_partition {
    fo_problem problem;
    std::vector<int32_t> dest_perm;
    std::vector<int32_t> sizes;
};

struct fo_plan_cache {
    std::vector<fo_cached_partition> entries;
};

extern "C" {

fo_status fo_plan_groups(const fo_problem* problem, const fo_grouping* grouping, fo_plan** out) {
    fo::clear_error();
    if (!problem || !grouping || !out) return fo::fail(FO_ERR_ARG, "null argument");
    fo_plan* p = new (std::nothrow) fo_plan();
    if (!p) return fo::fail(FO_ERR_ARG, "out of host memory");
    fo_status st;
    try {
        st = build(*p, *problem, *grouping);
    } catch (const std::bad_alloc&) {
        st = fo::fail(FO_ERR_ARG, "out of host memory");
    }
    if (st != FO_OK) {
        delete p;
        return st;
    }
    *out = p;
    return FO_OK;
}

void fo_plan_destroy(fo_plan* plan) { delete plan; }

fo_status fo_plan_cache_create(fo_plan_cache** out) {
    fo::clear_error();
    if (!out) return fo::fail(FO_ERR_ARG, "null argument");
    *out = new (std::nothrow) fo_plan_cache();
    return *out ? FO_OK : fo::fail(FO_ERR_ARG, "out of host memory");
}

void fo_plan_cache_destroy(fo_plan_cache* cache) { delete cache; }

fo_status fo_plan_cache_add(fo_plan_cache* cache, const fo_problem* problem, const fo_grouping* grouping) {
    fo::clear_error();
    if (!cache || !problem || !grouping) return fo::fail(FO_ERR_ARG, "null argument");
    if (grouping->num_groups > 0 && grouping->unit != FO_UNIT_WAVES)
        return fo::fail(FO_ERR_ARG, "cached partitions are given in waves");
    fo_plan* p = nullptr;
    fo_status st = fo_plan_groups(problem, grouping, &p);
    if (st != FO_OK) return st;
    try {
        fo_cached_partition e;
        e.problem = *problem;
        e.problem.row_bucket = nullptr;
        e.dest_perm = p->dest_perm;
        e.problem.dest_perm = nullptr;
        e.sizes = p->sizes;
        delete p;
        for (auto& old : cache->entries) {
            fo_problem q = old.problem;
            q.dest_perm = old.dest_perm.empty() ? nullptr : old.dest_perm.data();
            fo_problem r = e.problem;
            r.dest_perm = e.dest_perm.empty() ? nullptr : e.dest_perm.data();
            if (q.M == r.M && same_family(q, r)) {      // replace the entry of the same size
                old = std::move(e);
                return FO_OK;
            }
        }
        cache->entries.push_back(std::move(e));
    } catch (const std::bad_alloc&) {
        return fo::fail(FO_ERR_ARG, "out of host memory");
    }
    return FO_OK;
}

fo_status fo_plan_cache_lookup(const fo_plan_cache* cache, const fo_problem* problem, fo_plan** out,
                               int64_t* matched_m) {
    fo::clear_error();
    if (!cache || !problem || !out) return fo::fail(FO_ERR_ARG, "null argument");
    const fo_cached_partition* best = nullptr;
    for (const auto& e : cache->entries) {
        fo_problem q = e.problem;
        q.dest_perm = e.dest_perm.empty() ? nullptr : e.dest_perm.data();
        if (!same_family(q, *problem)) continue;
        const int64_t d = std::llabs(q.M - problem->M), db = best ? std::llabs(best->problem.M - problem->M) : 0;
        if (!best || d < db || (d == db && q.M < best->problem.M)) best = &e;
    }
    if (!best) return fo::fail(FO_ERR_ARG, "no cached partition for this problem family");
    if (problem->tile_m < 1 || problem->tile_n < 1 || problem->num_cus <= problem->reserved_cus ||
        problem->wg_per_cu < 1 || problem->M < 0 || problem->N < 0)
        return fo::fail(FO_ERR_ARG, "bad problem");
    const int64_t tiles = (problem->M / problem->tile_m) * (problem->N / problem->tile_n);
    const int64_t W = (int64_t)(problem->num_cus - problem->reserved_cus) * problem->wg_per_cu;
    const int32_t T = (int32_t)((tiles + W - 1) / W);
    std::vector<int32_t> sizes;
    try {
        sizes = map_partition(best->sizes, T);
    } catch (const std::bad_alloc&) {
        return fo::fail(FO_ERR_ARG, "out of host memory");
    }
    fo_grouping g{};
    g.unit = FO_UNIT_WAVES;
    g.num_groups = (int32_t)sizes.size();
    g.sizes = sizes.empty() ? nullptr : sizes.data();     // no tiles: no groups
    const fo_status st = fo_plan_groups(problem, &g, out);
    if (st == FO_OK && matched_m) *matched_m = best->problem.M;
    return st;
}

int32_t fo_plan_cache_size(const fo_plan_cache* cache) { return cache ? (int32_t)cache->entries.size() : 0; }

fo_status fo_plan_cache_entry(const fo_plan_cache* cache, int32_t e, int64_t* M, int32_t* num_groups,
                              const int32_t** sizes) {
    fo::clear_error();
    if (!cache || e < 0 || e >= (int32_t)cache->entries.size()) return fo::fail(FO_ERR_ARG, "no such entry");
    const auto& x = cache->entries[e];
    if (M) *M = x.problem.M;
    if (num_groups) *num_groups = (int32_t)x.sizes.size();
    if (sizes) *sizes = x.sizes.data();
    return FO_OK;
}

int32_t fo_plan_num_tiles(const fo_plan* p) { return p ? p->tiles : 0; }
int32_t fo_plan_wave_width(const fo_plan* p) { return p ? p->W : 0; }
int32_t fo_plan_num_waves(const fo_plan* p) { return p ? p->T : 0; }
int32_t fo_plan_num_groups(const fo_plan* p) { return p ? p->P : 0; }
const int32_t* fo_plan_group_sizes(const fo_plan* p) { return p ? p->sizes.data() : nullptr; }
const int32_t* fo_plan_order(const fo_plan* p) { return p ? p->order_tbl.data() : nullptr; }
const int32_t* fo_plan_tile_to_slot(const fo_plan* p) { return p ? p->tile_to_slot.data() : nullptr; }
const int32_t* fo_plan_group_first(const fo_plan* p) { return p ? p->group_first.data() : nullptr; }
const int32_t* fo_plan_group_targets(const fo_plan* p) { return p ? p->targets.data() : nullptr; }
double fo_plan_predicted_us(const fo_plan* p) { return p ? p->predicted_us : 0.0; }
const int32_t* fo_plan_pool_base(const fo_plan* p) { return p && !p->pool_base.empty() ? p->pool_base.data() : nullptr; }
const int32_t* fo_plan_pool_off(const fo_plan* p) { return p && !p->pool_off.empty() ? p->pool_off.data() : nullptr; }
int32_t fo_plan_num_counters(const fo_plan* p) { return p ? p->P + FO_DISPENSER_WORDS + FO_HANDOFF_WORDS : 0; }
int32_t fo_plan_num_segments(const fo_plan* p) { return p ? (int32_t)(p->segs.size() / 5) : 0; }
const int64_t* fo_plan_segments(const fo_plan* p) { return p ? p->segs.data() : nullptr; }
int64_t fo_plan_dest_elems(const fo_plan* p) { return p ? p->dest_elems : 0; }
size_t fo_plan_device_bytes(const fo_plan* p) { return p ? (size_t)p->layout.words * 4 : 0; }

fo_status fo_plan_to_device(const fo_plan* p, void* dev_buf, size_t bytes, void* stream) {
    fo::clear_error();
    if (!p || !dev_buf) return fo::fail(FO_ERR_ARG, "null argument");
    if (bytes < fo_plan_device_bytes(p)) return fo::fail(FO_ERR_ARG, "device buffer too small");
    if (reinterpret_cast<uintptr_t>(dev_buf) % 16) return fo::fail(FO_ERR_ARG, "device buffer must be 16-byte aligned");
    hipError_t e = hipMemcpyAsync(dev_buf, p->image.data(), fo_plan_device_bytes(p),
                                  hipMemcpyHostToDevice, (hipStream_t)stream);
    if (e != hipSuccess) return fo::fail(FO_ERR_HIP, std::string("hipMemcpyAsync: ") + hipGetErrorString(e));
    return FO_OK;
}

}  // extern "C"
