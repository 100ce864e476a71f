/*
 * fo.h -- C ABI of the signaled + reordered GEMM path (FlashOverlap,
 * "Efficient and Adaptable Overlapping for Computation and Communication via
 * Signaling and Reordering") for AMD Instinct MI355X (gfx950).
 *
 * The path, one GPU:
 *
 *   1. fo_plan_groups          host: tile dispatch order, waves, wave groups,
 *                              the reorder map and the per-group segments
 *                              (Sections 3.2-3.4, Algorithm 1).
 *   2. fo_gemm_signal_reorder  GPU, stream 1: C = A x B whose epilogue stores
 *                              every finished tile into its group-contiguous
 *                              slot and then bumps the group's counter
 *                              (Section 3.2 Approach, Section 3.3 Approach,
 *                              Section 5).
 *   3. fo_consume_group        GPU, stream 2: waits until a group's counter
 *                              reaches the group's tile count, then processes
 *                              the group's contiguous (ptr, len) segment. On
 *                              one GPU this stands in for the collective
 *                              (Section 3.3 Motivation: one library call per
 *                              contiguous buffer).
 *   4. fo_post_reorder         GPU: restores row-major order, fused with bias
 *                              add and RMSNorm (Section 3.3 Approach, last
 *                              paragraph; Section 6.6).
 *
 * Conventions for every call:
 *   - Device buffers are plain device pointers owned by the caller. The
 *     library never allocates, frees or retains device memory.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Launches are asynchronous; no call synchronizes the device.
 *   - Every call returns fo_status and never aborts. On failure nothing is
 *     launched and fo_last_error() returns a message for the calling thread.
 *   - fp16 is IEEE binary16, bf16 is bfloat16; both are stored as 16-bit
 *     words. Accumulation is fp32 (MFMA); results are rounded to nearest-even.
 */
#ifndef FO_H_
#define FO_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FO_OK = 0,
    FO_ERR_ARG = -1,          /* null / inconsistent argument            */
    FO_ERR_SHAPE = -2,        /* a dimension does not fit the tiling      */
    FO_ERR_UNSUPPORTED = -3,  /* no kernel for this dtype / tile / pattern */
    FO_ERR_HIP = -4,          /* a HIP runtime call failed                */
    FO_ERR_TIMEOUT = -5       /* reported through a status word only      */
} fo_status;

typedef enum { FO_FP16 = 0, FO_BF16 = 1 } fo_dtype;

/* Pre-communication reorder pattern (Section 3.3, Approach (1)-(3)). */
typedef enum {
    FO_PATTERN_TILE = 0,      /* AllReduce: tiles, column-of-tiles buffer          */
    FO_PATTERN_SUBTILE = 1,   /* ReduceScatter: each tile cut into R row slices     */
    FO_PATTERN_SUBTOKEN = 2,  /* All-to-All: tile rows into per-destination pools   */
    FO_PATTERN_ROWMAJOR = 3   /* plain GEMM output (no reorder)                     */
} fo_pattern;

/* Dispatch order of tiles (Section 2.1.2, block swizzling). Workgroup p of
 * the GEMM grid computes tile order(p); tiles are numbered row-major over
 * the (M/tile_m) x (N/tile_n) tile grid.
 *   ROWMAJOR: order(p) = p.
 *   GROUPED:  bands of `group_m` tile rows; inside a band the position walks
 *             down a column of the band, then to the next column:
 *               band = q / (group_m*tiles_n), first = band*group_m,
 *               rows = min(tiles_m - first, group_m), r = q % (group_m*tiles_n),
 *               tm = first + r % rows, tn = r / rows          (q = p).
 *   XCD:      position p runs on chiplet x = p % num_xcds; chiplet x's
 *             positions take a contiguous share of the GROUPED order:
 *               per = ceil(tiles/num_xcds), full = tiles % num_xcds (or
 *               num_xcds when 0), l = p / num_xcds,
 *               q = x < full ? x*per + l : full*per + (x-full)*(per-1) + l,
 *             then GROUPED on q. On MI355X (8 chiplets of 32 CUs, each with
 *             its own L2) and group_m = 4 a chiplet's 32 concurrent 256x256
 *             tiles form a 4x8 block: 1024 rows of A, 2048 columns of B. */
typedef enum { FO_ORDER_ROWMAJOR = 0, FO_ORDER_GROUPED = 1, FO_ORDER_XCD = 2 } fo_order;

/* Unit of a wave-group partition (Section 3.2 Insight: a group is >= 1 whole
 * waves; TILES allows tile-wise signalling inside one wave). */
typedef enum { FO_UNIT_WAVES = 0, FO_UNIT_TILES = 1 } fo_unit;

/* The GEMM and its decomposition. Host memory, read during the call only. */
typedef struct {
    int64_t M, N, K;          /* C[M,N] = A[M,K] x B[K,N] (Section 2.1.1)          */
    int32_t dtype;            /* fo_dtype of A, B, C                                */
    int32_t tile_m, tile_n;   /* output tile; GEMM kernels: 256x128, 256x256, 64x64 */
    int32_t order;            /* fo_order                                           */
    int32_t group_m;          /* band height for GROUPED / XCD (>= 1)               */
    int32_t num_xcds;         /* chiplets for XCD (>= 1)                            */
    int32_t num_cus;          /* compute units of the device (256 on MI355X)        */
    int32_t wg_per_cu;        /* GEMM workgroups resident per CU (1 here)           */
    int32_t reserved_cus;     /* CUs left to communication (Algorithm 1)            */
    int32_t pattern;          /* fo_pattern                                         */
    int32_t num_dest;         /* R for SUBTILE (divides tile_m), B for SUBTOKEN    */
    const int32_t* dest_perm; /* SUBTILE: [R], slice k goes to buffer dest_perm[k];
                                 NULL = identity. Must be a permutation.            */
    const int32_t* row_bucket;/* SUBTOKEN: [M], destination of every row, in [0,B) */
} fo_problem;

/* How the waves are grouped (Section 3.4; Section 4 for the search). */
typedef struct {
    int32_t unit;             /* fo_unit of `sizes`                                 */
    int32_t num_groups;       /* > 0: explicit `sizes`; 0: Algorithm 1 search       */
    const int32_t* sizes;     /* [num_groups], each >= 1, summing to T waves (or to
                                 the tile count when unit == TILES)                 */
    double gemm_us;           /* search (or estimate of given waves): measured GEMM
                                 duration                                          */
    const double* curve_bytes;/* sampled communication latency curve (required by  */
    const double* curve_us;   /*   the search; optional with given waves, then the  */
    int32_t curve_len;        /*   plan carries their estimate): ascending bytes,
                                 piecewise-linear in between, end-point bandwidth
                                 outside the samples                               */
    int32_t s_first, s_last;  /* search pruning |G_1| <= s_first, |G_P| <= s_last
                                 (Section 4.1 uses 2 and 4); <= 0 means no bound    */
    int32_t all_dest_bytes;   /* SUBTOKEN data size of a group in the estimate:
                                 0 = its largest per-destination piece (the slowest
                                 link of a real All-to-All, Section 4.2: maximum
                                 across GPUs); 1 = all its pieces (one device moves
                                 every piece, as the one-GPU stand-in consumer
                                 does). Other patterns ignore it.                  */
    const double* last_curve_bytes; /* optional latency curve of the LAST group's */
    const double* last_curve_us;    /*   communication, which runs after the GEMM */
    int32_t last_curve_len;         /*   has ended: same form as `curve`; 0 = the
                                         last group uses `curve` too. (A one-GPU
                                         stand-in of the communication shares the
                                         device with the GEMM until the last group
                                         and has it to itself for that one.)       */
} fo_grouping;

typedef struct fo_plan fo_plan;   /* opaque, library-owned host memory */

/*
 * fo_plan_groups -- build the plan (host only, deterministic, no GPU work).
 *
 * Tiles: tiles = (M/tile_m)(N/tile_n). Waves (Section 2.1.1; Algorithm 1's
 * wave count): W = (num_cus - reserved_cus) * wg_per_cu tiles run together; the
 * tile at dispatch position p runs in wave p / W; T = ceil(tiles / W).
 * Slots (Section 3.3 Approach (1)): the slot of a tile is its dispatch
 * position, so earlier waves come first and a wave's tiles are adjacent.
 * Groups: group j owns slots [first_j, first_{j+1}); with unit WAVES
 * first_j = min(W * (waves before j), tiles). Counter target of group j =
 * first_{j+1} - first_j (Section 3.2: the j-th count fires at |G_j| tiles).
 * With num_groups == 0 the partition is Algorithm 1: every partition of T
 * waves (cut vector x = 0 .. 2^(T-1)-1, bit i = cut after wave i+1, T <= 24)
 * that meets the pruning bounds is scored by the predicted overlapped
 * latency, and the first strictly smallest wins.
 *
 * Errors: FO_ERR_ARG (null pointers, sizes that do not sum, bad enum,
 * missing dest_perm/row_bucket data, bad curve), FO_ERR_SHAPE (M % tile_m,
 * N % tile_n, tile_m % R not zero, negative dims), FO_ERR_UNSUPPORTED
 * (search with T > 24). *out is set only on FO_OK; free with fo_plan_destroy.
 */
fo_status fo_plan_groups(const fo_problem* problem, const fo_grouping* grouping, fo_plan** out);
void fo_plan_destroy(fo_plan* plan);

/*
 * Plan cache for shapes that vary at run time (Section 4.2, online stage: for
 * dynamic tasks the search is run ahead of time for representative GEMM
 * sizes, and an unseen size takes the partition of its nearest neighbour).
 *
 * A family is every fo_problem field but M and row_bucket (dest_perm compared
 * by content). fo_plan_cache_add builds the plan of `problem` with `grouping`
 * (the Algorithm 1 search when num_groups == 0, else the given partition,
 * which must be in waves) and keeps its wave partition, replacing an entry of
 * the same family and M. fo_plan_cache_lookup picks, among the entries of the
 * problem's family, the one whose M is nearest (the smaller M on ties), maps
 * its partition onto the problem's own wave count T (a cut after wave c moves
 * to after wave round(c * T / T_ref), halves rounding up; cuts that land on 0,
 * on T or on an earlier cut are dropped) and returns the plan built with it
 * (free with fo_plan_destroy); *matched_m (may be NULL) receives the entry's M.
 * The cache is host memory owned by the library; lookups do not modify it.
 * Errors: FO_ERR_ARG (null argument, no entry of the family, a partition in
 * tiles), and every error fo_plan_groups reports.
 */
typedef struct fo_plan_cache fo_plan_cache;
fo_status fo_plan_cache_create(fo_plan_cache** out);
void fo_plan_cache_destroy(fo_plan_cache* cache);
fo_status fo_plan_cache_add(fo_plan_cache* cache, const fo_problem* problem, const fo_grouping* grouping);
fo_status fo_plan_cache_lookup(const fo_plan_cache* cache, const fo_problem* problem, fo_plan** out,
                               int64_t* matched_m);
int32_t fo_plan_cache_size(const fo_plan_cache* cache);
/* Entry e (0 <= e < size): its M and wave partition (valid until the cache
 * changes). */
fo_status fo_plan_cache_entry(const fo_plan_cache* cache, int32_t e, int64_t* M, int32_t* num_groups,
                              const int32_t** sizes);

/* Plan accessors. Arrays stay valid until fo_plan_destroy. */
int32_t fo_plan_num_tiles(const fo_plan* plan);
int32_t fo_plan_wave_width(const fo_plan* plan);      /* W                        */
int32_t fo_plan_num_waves(const fo_plan* plan);       /* T                        */
int32_t fo_plan_num_groups(const fo_plan* plan);      /* P                        */
/* Length of the counters array of a signalling run: P group counters, then
 * FO_DISPENSER_WORDS tile-position counters of the GEMM, then
 * FO_HANDOFF_WORDS words that fo_run_overlapped uses to hand work between
 * its two streams (a gate word, then 8 done words 32 words apart, each in a
 * 128-byte line of its own). */
#define FO_DISPENSER_WORDS 8
#define FO_HANDOFF_WORDS 226
int32_t fo_plan_num_counters(const fo_plan* plan);    /* P + FO_DISPENSER_WORDS
                                                         + FO_HANDOFF_WORDS       */
const int32_t* fo_plan_group_sizes(const fo_plan* plan);   /* [P], in the plan's unit */
const int32_t* fo_plan_order(const fo_plan* plan);         /* [tiles] position -> tile */
const int32_t* fo_plan_tile_to_slot(const fo_plan* plan);  /* [tiles] the reorder map  */
const int32_t* fo_plan_group_first(const fo_plan* plan);   /* [P+1] first slot          */
const int32_t* fo_plan_group_targets(const fo_plan* plan); /* [P] tiles = final count   */
double fo_plan_predicted_us(const fo_plan* plan);     /* Algorithm 1 estimate of the
                                                         plan's partition (searched,
                                                         or given in waves with a
                                                         curve); else 0             */
/* SUBTOKEN pools: pool_base[(s * B) + b] = subtokens of pool b in slots < s,
 * s in [0, tiles]; pool_off[b] = first subtoken of pool b, b in [0, B]. */
const int32_t* fo_plan_pool_base(const fo_plan* plan);
const int32_t* fo_plan_pool_off(const fo_plan* plan);

/*
 * Communication segments, in the order a caller issues them: entry e is
 * seg[5e .. 5e+4] = {group j, destination d, src_off, dst_off, len}, in
 * elements. Source = the GEMM output buffer (and the peer partial, laid out
 * the same way); destination = the consumer's buffer of
 * fo_plan_dest_elems() elements.
 *   TILE:     one segment per group: its slots, dst_off = src_off.
 *   SUBTILE:  one per (group j, slice k): h = tile_m/R rows of each of the
 *             group's n_j tiles; src_off = first_j*tile_m*tile_n + k*n_j*h*tile_n;
 *             destination buffer dest_perm[k] (buffers of tiles*h*tile_n
 *             elements laid end to end) at rows first_j*h.
 *   SUBTOKEN: one per (group, pool b); the receive buffer mirrors the pools.
 *   ROWMAJOR: one segment, the whole output, for the last group.
 */
int32_t fo_plan_num_segments(const fo_plan* plan);
const int64_t* fo_plan_segments(const fo_plan* plan);
int64_t fo_plan_dest_elems(const fo_plan* plan);

/*
 * Device image of the plan's tables (int32 words): what the GEMM epilogue
 * and the post-reorder kernel read. fo_plan_to_device copies it into a
 * caller-owned device buffer of at least fo_plan_device_bytes() bytes
 * (16-byte aligned) on `stream` (asynchronous when the copy engine allows;
 * the host plan must stay alive until the copy is complete).
 */
size_t fo_plan_device_bytes(const fo_plan* plan);
fo_status fo_plan_to_device(const fo_plan* plan, void* dev_buf, size_t bytes, void* stream);

/*
 * Per-call options of the GPU entry points (fo_gemm_signal_reorder,
 * fo_consume_group, fo_run_overlapped). Every such call takes a
 * `const fo_options*`; NULL means the process defaults. fo_options_init
 * fills *o with those defaults as they stand at the time of the call (the
 * fo_set_* calls below and their environment variables), so that a caller
 * changes only what it needs and two layers can run with different options
 * in one process. The library reads the struct during the call only.
 */
typedef struct {
    int32_t sync_producer;    /* fo_sync_mode of the GEMM epilogue             */
    int32_t sync_consumer;    /* fo_sync_mode of the consumer launches         */
    int32_t consumer_blocks;  /* grid cap of consumers beside the GEMM, 1..256 */
    int32_t consumer_threads; /* their workgroup size: 64, 128 or 256          */
    int64_t poll_timeout_us;  /* bound of every device-side wait, > 0          */
    /* Benchmark and diagnostic controls; the path itself never needs them. */
    int32_t consumer_limit;   /* cap on the workgroups of EVERY consumer launch
                                 (1..256), 0 = none: a stand-in for a slower
                                 interconnect (the consumer's bandwidth grows
                                 with its workgroups); under a cap every launch
                                 uses the variant that fits beside the GEMM   */
    int32_t reserved0;        /* must be 0                                     */
    uint64_t* tile_trace;     /* tile timeline (device memory, 8-byte aligned),
                                 NULL = none: each GEMM launch writes, for every
                                 dispatch position p < tile_trace_capacity, four
                                 uint64 at tile_trace[4p]: the device wall clock
                                 (fo_device_wall_clock_khz) when the tile
                                 started and when all of its stores had
                                 completed, the chiplet (XCC_ID register, high
                                 32 bits) and hardware id (HW_ID, low 32 bits)
                                 of its compute unit, and the workgroup index.
                                 Tracing adds a store drain and a barrier per
                                 tile (the timeline of Section 2.1.1, Fig. 3) */
    int64_t tile_trace_capacity; /* >= 1 when tile_trace is set               */
} fo_options;

/* Process defaults into *o. FO_ERR_ARG if o is NULL. */
fo_status fo_options_init(fo_options* o);

/*
 * fo_gemm_signal_reorder -- C = A x B with the reordering, signalling
 * epilogue (Section 3.2 Approach; Section 3.3 Approach; Section 5: the
 * reorder sits in the epilogue, the main loop is untouched).
 *
 * A: [M, K] row-major. W: B^T, [N, K] row-major (K contiguous, the weight
 * layout of a linear layer). K must be a multiple of 64 and max(tile_m,
 * tile_n) * K * 2 must not exceed 2^31 - 1; A, W, C_out 16-byte
 * aligned. C_out by pattern:
 *   ROWMAJOR: [M, N] row-major.
 *   TILE:     [tiles*tile_m, tile_n] row-major; slot s holds the tile at rows
 *             [s*tile_m, (s+1)*tile_m).
 *   SUBTILE:  M*N elements, group j at [first_j*tile_m*tile_n, ...) laid out
 *             [R][n_j][h][tile_n]: slice k of the group's i-th slot at
 *             first_j*tile_m*tile_n + (k*n_j + i)*h*tile_n.
 *   SUBTOKEN: M*N elements, pool b at pool_off[b]*tile_n; row r of tile
 *             (tm, tn) in slot s goes to subtoken pool_off[b] +
 *             pool_base[s*B+b] + (rank of row r among rows of tile row tm
 *             bound for b), b = row_bucket[tm*tile_m + r].
 * counters: at least P + FO_DISPENSER_WORDS uint32 (fo_plan_num_counters
 * also counts the words fo_run_overlapped needs); NULL = no signalling.
 * counters[0, P) are the group counters: zeroed by the caller before the
 * launch and before any consumer of this run starts (see fo_reset_counters).
 * When a tile's stores are complete and visible to every chiplet, one
 * agent-scope increment is made on counters[group of its slot]; when the
 * GEMM is done, counters[j] == target_j for every j < P.
 * counters[P, P + FO_DISPENSER_WORDS) hand out tile positions to the GEMM's
 * workgroups: they must be zero before the first launch on the array, and
 * every launch that runs to its end leaves them zero again (the last
 * workgroup to find its position class exhausted clears the class's word),
 * so back-to-back launches need not clear them.
 * The GEMM runs min(tiles, W) persistent workgroups (W = the plan's wave
 * width). With counters, each takes its next dispatch position from an
 * atomic counter when it finishes a tile, so positions start in increasing
 * order and a workgroup that is not yet scheduled (its compute unit busy
 * with other work) holds no tile back; without counters, workgroup b
 * computes positions b, b + grid, b + 2*grid, ...
 * dev_plan: the plan's device image (fo_plan_to_device).
 * Errors: FO_ERR_ARG, FO_ERR_SHAPE (K % 64), FO_ERR_UNSUPPORTED (tile shape
 * other than 256x128 / 256x256 / 64x64), FO_ERR_HIP (launch failure).
 */
fo_status fo_gemm_signal_reorder(const fo_plan* plan, const void* dev_plan,
                                 const void* A, const void* W, void* C_out,
                                 uint32_t* counters, void* stream,
                                 const fo_options* options);

/*
 * fo_consume_group -- the communication stand-in for one contiguous segment
 * (Section 5: a signalling kernel holds the communication of a group until
 * the group's count reaches its size; the communication itself only sees a
 * contiguous buffer).
 *
 * Two launches on `stream`: a one-wave wait kernel that polls until
 * *counter >= target, then the streaming kernel (agent-scope acquire), which
 * for i < len computes:
 *   peer != NULL:  dst[i] = RNE(src[i] + peer[i])   (AllReduce/ReduceScatter
 *                  of this GPU's partial with one peer partial)
 *   peer == NULL:  dst[i] = src[i]                  (All-to-All copy)
 * counter == NULL: no wait (one launch). The wait is bounded
 * (options->poll_timeout_us); on timeout the segment is not written and
 * *status_word (if non-NULL, device uint32) gets bit 0 set; the library
 * never clears it. The launch uses options->consumer_blocks and
 * consumer_threads (capped by consumer_limit) and the consumer sync mode.
 * Buffers must not overlap. Any alignment works; 16-byte-aligned pointers
 * take the vector path.
 * Errors: FO_ERR_ARG (null src/dst with len > 0, len < 0, bad dtype, an
 * option out of range).
 */
fo_status fo_consume_group(const void* src, const void* peer, void* dst, int64_t len,
                           int32_t dtype, const uint32_t* counter, uint32_t target,
                           uint32_t* status_word, void* stream, const fo_options* options);

/*
 * fo_post_reorder -- post-communication reorder fused into the following
 * element-wise op (Section 3.3: loads go by the reordered index; Section 6.6
 * measures it fused with RMSNorm).
 *
 * src: the consumer's destination buffer (fo_plan_dest_elems elements).
 * out: [M, N] row-major, x[i, n] = src[position of (i, n)].
 * Then, row-wise: h = x + bias (bias [N] or NULL), and if do_rmsnorm:
 * y = h / sqrt(mean_n(h^2) + eps) * gamma (gamma [N] or NULL = 1), in fp32,
 * rounded once to the dtype; else y = h.
 * Errors: FO_ERR_ARG, FO_ERR_UNSUPPORTED (N % 8 or tile_n % 8 not zero;
 * a reordered pattern whose tile_n / 8 is not a power of two; more than 64 KB
 * of LDS per workgroup: 16 * tiles_n bytes of source offsets, plus 4 * N bytes
 * of bias and gamma when rows of up to 8192 columns are normalised),
 * FO_ERR_SHAPE (a source buffer of 2^32 or more 16-byte chunks), FO_ERR_HIP.
 */
fo_status fo_post_reorder(const fo_plan* plan, const void* dev_plan, const void* src,
                          void* out, const void* bias, const void* gamma, float eps,
                          int32_t do_rmsnorm, void* stream);

/* ---- orchestration and helpers ----------------------------------------- */

/* Zero n counters with a fill kernel (safe inside captured graphs). */
fo_status fo_reset_counters(uint32_t* counters, int32_t n, void* stream);

/*
 * One overlapped run of the whole path (Section 5: GEMM on one stream, the
 * signalling + communication on another; Figure 5 order):
 *   gemm_stream: reset kernel -> GEMM (signalling) -> done wait
 *                -> fo_post_reorder (if out != NULL)
 *   comm_stream: gate kernel -> one consumer launch per group
 * The two streams hand work to each other on the device, not with events:
 * the reset kernel zeroes counters[0, P + FO_DISPENSER_WORDS), writes the
 * run's tag (a process-wide sequence number) into the 8 done words
 * counters[P + FO_DISPENSER_WORDS + 1 + 32 k] with a count of zero, then
 * writes the tag into the gate word counters[P + FO_DISPENSER_WORDS]; the
 * gate kernel (one wave) holds the consumers until it reads that tag;
 * workgroup b of the final consumer launch adds 1 to done word b % 8 only
 * while that word carries its own run's tag, and the done wait (one wave)
 * holds the post-reorder until every done word has counted its share of the
 * launch's grid (spreading the count keeps the workgroups' adds from queueing
 * on one address). A consumer of an
 * earlier run that finishes late therefore does not count for a later run
 * (it can only race with the later run's reset, the check and the add being
 * two steps, if a wait of the earlier run timed out: then the status bit is
 * already set).
 * Both waits are bounded like a consumer's (options->poll_timeout_us): on
 * timeout bit 0 of the status word is set and the run's dst and out are
 * unspecified. The status word is sticky: the library only sets bits, the
 * caller clears it, so a timeout of one run stays visible after later runs
 * queued behind it. A gate that gives up because a later run's tag has
 * already arrived leaves the word as it is (that run is not delayed).
 * A group's consumer is one wait kernel on the group's counter and one
 * streaming kernel that does what fo_consume_group does for each of the
 * group's plan segments (fo_plan_segments: 1, R or B of them). Every group
 * but the last uses the grid of fo_get_consumer_grid(); the last group,
 * which runs after the GEMM, uses up to 256 workgroups of 256 threads (as do
 * all groups of a serialized run); options->consumer_limit caps them all.
 * With comm_stream == gemm_stream (or NULL) the same work runs serialized
 * on gemm_stream, without the handoffs and without signalling. A plan of one
 * group has nothing to overlap (its consumer can only start after the whole
 * GEMM): with a comm_stream it runs serialized on gemm_stream too, the same
 * way (counters untouched). An overlapped run needs counters and,
 * with more than one group, a created gemm_stream (not the null stream,
 * which would wait for the gate kernel on a blocking comm_stream).
 * The overlap also needs the two streams on different hardware queues: HIP
 * maps streams onto a few queues per device (GPU_MAX_HW_QUEUES, 4 by
 * default), and kernels of streams that share a queue run one after another.
 * The run is then serialized but still correct (each handoff waits only for
 * work enqueued before it); a process that keeps creating streams should
 * reuse one pair for its overlapped runs.
 * Buffers: C_out (GEMM output, see fo_gemm_signal_reorder), peer (NULL for
 * All-to-All; else the peer's partial in C_out's layout), dst
 * (fo_plan_dest_elems), out ([M, N] or NULL), counters
 * [fo_plan_num_counters] (zero when first used: the gate word must not hold
 * another run's tag from an earlier allocation), status_word [1] or NULL.
 * Once gemm_stream has passed the run, every kernel of the run has made its
 * last memory access (comm_stream may still be retiring the final consumer
 * launch's workgroups).
 * gemm_begin_event / gemm_end_event: optional caller-owned hipEvent_t (as
 * void*) recorded on gemm_stream right before and after the GEMM launch, so
 * a caller can time the GEMM inside the overlapped run; NULL = none.
 * options: as for the three calls the run makes (NULL = process defaults).
 * Errors: FO_ERR_ARG (no plan or dst; overlapped without counters or with a
 * null gemm_stream; an option out of range), and those of the three calls
 * the run makes.
 */
fo_status fo_run_overlapped(const fo_plan* plan, const void* dev_plan,
                            const void* A, const void* W, void* C_out,
                            const void* peer, void* dst, void* out,
                            const void* bias, const void* gamma, float eps,
                            int32_t do_rmsnorm, uint32_t* counters,
                            uint32_t* status_word, void* gemm_stream, void* comm_stream,
                            void* gemm_begin_event, void* gemm_end_event,
                            const fo_options* options);

/*
 * fo_run_overlapped_noalloc -- fo_run_overlapped for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same run, with the counters array
 * taken from a static array of FO_NOALLOC_MAX_COUNTERS uint32 words that the
 * library holds on every device it runs on until the process ends. The call
 * allocates nothing and calls no allocating routine; the caller passes the
 * inputs and outputs as for fo_run_overlapped (status_word included: it is
 * an output, sticky as there), no events. Each run's reset kernel clears what
 * must start at zero (the group and position counters); the gate word keeps
 * the last run's tag. Every call on one device shares that device's array:
 * calls that may overlap on one device (other streams, other threads) race
 * and must not be issued; calls queued on the same pair of streams are
 * ordered by the streams and are fine.
 * Errors: FO_ERR_ARG when the plan needs more than FO_NOALLOC_MAX_COUNTERS
 * counter words (fo_plan_num_counters), before any device work; FO_ERR_HIP
 * when the array's address cannot be had; and those of fo_run_overlapped.
 */
#define FO_NOALLOC_MAX_COUNTERS 1024
fo_status fo_run_overlapped_noalloc(const fo_plan* plan, const void* dev_plan,
                                    const void* A, const void* W, void* C_out,
                                    const void* peer, void* dst, void* out,
                                    const void* bias, const void* gamma, float eps,
                                    int32_t do_rmsnorm, uint32_t* status_word,
                                    void* gemm_stream, void* comm_stream,
                                    const fo_options* options);

/*
 * How the producer (GEMM epilogue) publishes a finished tile and how the
 * consumer reads a signalled group. All modes are correct; they differ in
 * the cache maintenance they cost (MI355X has one L2 per chiplet):
 *   FO_SYNC_FENCE_ALL: producer: every wave makes its stores visible with an
 *     agent-scope release fence (L2 write-back), then one lane increments;
 *     consumer: every wave invalidates its caches with an agent-scope acquire.
 *   FO_SYNC_FENCE_ONE: producer: workgroup barrier, then one agent-scope
 *     release increment; consumer: one acquire (wave 0) before a workgroup
 *     barrier.
 *   FO_SYNC_COHERENT: producer: the tile is written with device-coherent
 *     stores that go through to the memory side shared by all chiplets, every
 *     wave waits for their completion, then one lane increments (no
 *     write-back); consumer: the group is read with device-coherent loads
 *     after the counter is seen (no invalidation).
 * Default: FO_SYNC_COHERENT for both; env FO_SYNC_PRODUCER / FO_SYNC_CONSUMER
 * (0, 1, 2) override at load time. Process default of fo_options.sync_producer
 * and sync_consumer (fo_options_init).
 */
typedef enum { FO_SYNC_FENCE_ALL = 0, FO_SYNC_FENCE_ONE = 1, FO_SYNC_COHERENT = 2 } fo_sync_mode;
fo_status fo_set_sync_mode(int32_t producer, int32_t consumer);
void fo_get_sync_mode(int32_t* producer, int32_t* consumer);

/* Grid of a consumer launch that runs beside the GEMM (every
 * fo_consume_group call, and every group but the last in fo_run_overlapped):
 * at most max_blocks workgroups (1 .. 256) of `threads` threads (64, 128 or
 * 256); default 256 x 64, one wave per compute unit. A smaller grid streams
 * a group more slowly and spreads its memory traffic over more of the GEMM's
 * run. Env
 * FO_CONSUMER_BLOCKS / FO_CONSUMER_THREADS override at load time.
 * Process default of fo_options.consumer_blocks / consumer_threads;
 * FO_ERR_ARG outside the ranges. */
fo_status fo_set_consumer_grid(int32_t max_blocks, int32_t threads);
void fo_get_consumer_grid(int32_t* max_blocks, int32_t* threads);

/* Upper bound of one device-side wait, in microseconds (default 2 s; env
 * FO_POLL_TIMEOUT_US overrides at load time): the process default of
 * fo_options.poll_timeout_us. */
void fo_set_poll_timeout_us(int64_t us);
int64_t fo_get_poll_timeout_us(void);

/* Ticks per millisecond of the device wall clock of the current device. */
fo_status fo_device_wall_clock_khz(int32_t* khz);

/* Compute units of HIP device `device` (for fo_problem.num_cus). */
fo_status fo_device_num_cus(int32_t device, int32_t* num_cus);

const char* fo_status_string(fo_status status);
const char* fo_last_error(void);   /* thread-local; "" when none */

#ifdef __cplusplus
}  /* extern "C" */
#endif

#endif  /* FO_H_ */
