// C ABI entry points of libfo: argument checks, device-plan addressing,
// kernel launches and the two-stream orchestration of one overlapped run.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "consume.h"
#include "fo_internal.h"
#include "gemm.h"
#include "post.h"

namespace fo {

namespace {
thread_local std::string t_last_error;
std::atomic<int64_t> g_timeout_us{[] {
    const char* e = std::getenv("FO_POLL_TIMEOUT_US");
    if (e && *e) {
        char* end = nullptr;
        const long long v = std::strtoll(e, &end, 10);
        if (end && *end == '\0' && v > 0) return (int64_t)v;
    }
    return (int64_t)2000000;
}()};

int env_mode(const char* name, int dflt) {
    const char* e = std::getenv(name);
    if (e && e[0] >= '0' && e[0] <= '2' && e[1] == '\0') return e[0] - '0';
    return dflt;
}
std::atomic<int> g_sync_producer{env_mode("FO_SYNC_PRODUCER", FO_SYNC_COHERENT)};
std::atomic<int> g_sync_consumer{env_mode("FO_SYNC_CONSUMER", FO_SYNC_COHERENT)};
int env_int(const char* name, int lo, int hi, int dflt) {
    const char* e = std::getenv(name);
    if (e && *e) {
        char* end = nullptr;
        const long v = std::strtol(e, &end, 10);
        if (end && *end == '\0' && v >= lo && v <= hi) return (int)v;
    }
    return dflt;
}
bool valid_threads(long t) { return t == 64 || t == 128 || t == 256; }
// Grid of the consumers that run beside the GEMM (default: one workgroup of
// one wave per compute unit; beside the 256x256 GEMM, one wave per compute
// unit costs the GEMM about half of what a wave on each SIMD costs, and the
// group still streams well inside the compute of the groups after it).
std::atomic<int> g_consumer_blocks{env_int("FO_CONSUMER_BLOCKS", 1, kMaxConsumeBlocks, kMaxConsumeBlocks)};
std::atomic<int> g_consumer_threads{[] {
    const int t = env_int("FO_CONSUMER_THREADS", 64, 256, 64);
    return valid_threads(t) ? t : 64;
}()};

fo_options defaults() {
    fo_options o{};
    o.sync_producer = g_sync_producer.load(std::memory_order_relaxed);
    o.sync_consumer = g_sync_consumer.load(std::memory_order_relaxed);
    o.consumer_blocks = g_consumer_blocks.load(std::memory_order_relaxed);
    o.consumer_threads = g_consumer_threads.load(std::memory_order_relaxed);
    o.poll_timeout_us = poll_timeout_us();
    return o;
}

// The options of one call: the caller's, checked, or the process defaults.
fo_status resolve(const fo_options* in, fo_options* out) {
    if (!in) {
        *out = defaults();
        return FO_OK;
    }
    const fo_options& o = *in;
    if (o.sync_producer < FO_SYNC_FENCE_ALL || o.sync_producer > FO_SYNC_COHERENT ||
        o.sync_consumer < FO_SYNC_FENCE_ALL || o.sync_consumer > FO_SYNC_COHERENT)
        return fail(FO_ERR_ARG, "options: sync modes are 0, 1 or 2");
    if (o.consumer_blocks < 1 || o.consumer_blocks > kMaxConsumeBlocks)
        return fail(FO_ERR_ARG, "options: consumer_blocks must be in [1, 256]");
    if (!valid_threads(o.consumer_threads)) return fail(FO_ERR_ARG, "options: consumer_threads must be 64, 128 or 256");
    if (o.poll_timeout_us <= 0) return fail(FO_ERR_ARG, "options: poll_timeout_us must be > 0");
    if (o.consumer_limit < 0 || o.consumer_limit > kMaxConsumeBlocks)
        return fail(FO_ERR_ARG, "options: consumer_limit must be 0 (no cap) or in [1, 256]");
    if (o.reserved0 != 0) return fail(FO_ERR_ARG, "options: reserved0 must be 0");
    if (o.tile_trace && o.tile_trace_capacity < 1) return fail(FO_ERR_ARG, "options: tile_trace_capacity must be >= 1");
    if (o.tile_trace && (reinterpret_cast<uintptr_t>(o.tile_trace) & 7))
        return fail(FO_ERR_ARG, "options: tile_trace must be 8-byte aligned");
    *out = o;
    return FO_OK;
}

// Workgroups of a consumer launch under the options' cap (0 = none).
int limited(const fo_options& o, int blocks) {
    return o.consumer_limit > 0 && o.consumer_limit < blocks ? o.consumer_limit : blocks;
}

constexpr int kMaxDevices = 64;
std::atomic<int64_t> g_clock_khz[kMaxDevices];   // 0 = unknown

fo_status hip_fail(const char* what, hipError_t e) {
    return fail(FO_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Ticks of the device wall clock (s_memrealtime) per microsecond x 1000.
fo_status clock_khz(int64_t* out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail("hipGetDevice", e);
    if (dev < 0 || dev >= kMaxDevices) return fail(FO_ERR_ARG, "device index out of range");
    int64_t k = g_clock_khz[dev].load(std::memory_order_relaxed);
    if (k == 0) {
        int rate = 0;
        e = hipDeviceGetAttribute(&rate, hipDeviceAttributeWallClockRate, dev);
        if (e != hipSuccess || rate <= 0) rate = 100000;   // 100 MHz constant clock
        k = rate;
        g_clock_khz[dev].store(k, std::memory_order_relaxed);
    }
    *out = k;
    return FO_OK;
}

static_assert(FO_HANDOFF_WORDS == 2 + (kDoneWords - 1) * kDoneStride,
              "handoff words: the gate word, then kDoneWords done words kDoneStride apart");

__global__ void fill_u32_kernel(uint32_t* p, int32_t n, uint32_t v) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

// Start of an overlapped run, one workgroup on the GEMM stream: zero the
// group and position counters (n words), set the kDoneWords done words to
// the run's done tag with a count of zero, make both visible device-wide, then
// exchange the gate word for the run's tag (the start handoff that the gate
// kernel on the consumer stream waits for). If a gate of this run timed out
// before, the word holds the tag's timed-out mark: the status word then gets
// bit 0 (the status word is never cleared here: its bits are sticky).
// gate == NULL: only the zeroing.
__global__ __launch_bounds__(256) void reset_run_kernel(uint32_t* counters, int32_t n, uint32_t* done,
                                                        uint32_t done_tag, uint32_t* status, uint32_t* gate,
                                                        uint32_t tag) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) counters[i] = 0u;
    if (done && threadIdx.x < kDoneWords) done[threadIdx.x * kDoneStride] = done_tag;
    if (!gate) return;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t old = __hip_atomic_exchange(gate, tag, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        if (old == (tag | kGateTimedOut) && status)
            __hip_atomic_fetch_or(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Counters array of fo_run_overlapped_noalloc, one copy per device (a
// file-scope device array, zero when the code object is loaded). Host code
// never passes the array's name to a kernel: the address of this device's
// copy comes from hipGetSymbolAddress, once per device.
__device__ __align__(256) uint32_t scratch[FO_NOALLOC_MAX_COUNTERS];
std::mutex g_scratch_mu;
uint32_t* g_scratch_ptr[kMaxDevices];

fo_status scratch_of_current_device(uint32_t** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail("hipGetDevice", e);
    if (dev < 0 || dev >= kMaxDevices) return fail(FO_ERR_ARG, "device index out of range");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return hip_fail("hipGetSymbolAddress(scratch)", e);
        g_scratch_ptr[dev] = static_cast<uint32_t*>(p);
    }
    *out = g_scratch_ptr[dev];
    return FO_OK;
}

// Tags of overlapped runs, unique per process (30 bits of sequence).
std::atomic<uint32_t> g_run_seq{0};

template <typename T>
const T* dev_table(const void* dev_plan, int64_t word_off) {
    if (word_off < 0) return nullptr;
    return reinterpret_cast<const T*>(static_cast<const int32_t*>(dev_plan) + word_off);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Common fields of a consumer launch; the wait limit in device clock ticks.
fo_status consume_args(const uint16_t* src, const uint16_t* peer, uint16_t* dst, const uint32_t* counter,
                       uint32_t target, uint32_t* status, const fo_options& o, ConsumeArgs* a) {
    int64_t khz = 0;
    fo_status st = clock_khz(&khz);
    if (st != FO_OK) return st;
    a->src = src;
    a->peer = peer;
    a->dst = dst;
    a->counter = counter;
    a->target = target;
    a->status = status;
    a->timeout_ticks = (uint64_t)o.poll_timeout_us * (uint64_t)khz / 1000u;
    return FO_OK;
}

}  // namespace

fo_status fail(fo_status st, const std::string& msg) {
    t_last_error = msg;
    return st;
}
void clear_error() { t_last_error.clear(); }
int64_t poll_timeout_us() { return g_timeout_us.load(std::memory_order_relaxed); }

}  // namespace fo

extern "C" {

const char* fo_status_string(fo_status s) {
    switch (s) {
        case FO_OK: return "ok";
        case FO_ERR_ARG: return "invalid argument";
        case FO_ERR_SHAPE: return "shape does not fit the tiling";
        case FO_ERR_UNSUPPORTED: return "unsupported configuration";
        case FO_ERR_HIP: return "HIP runtime error";
        case FO_ERR_TIMEOUT: return "consumer wait timed out";
    }
    return "unknown status";
}

const char* fo_last_error(void) { return fo::t_last_error.c_str(); }

void fo_set_poll_timeout_us(int64_t us) {
    if (us > 0) fo::g_timeout_us.store(us, std::memory_order_relaxed);
}
int64_t fo_get_poll_timeout_us(void) { return fo::poll_timeout_us(); }

fo_status fo_set_sync_mode(int32_t producer, int32_t consumer) {
    fo::clear_error();
    if (producer < FO_SYNC_FENCE_ALL || producer > FO_SYNC_COHERENT || consumer < FO_SYNC_FENCE_ALL ||
        consumer > FO_SYNC_COHERENT)
        return fo::fail(FO_ERR_ARG, "sync modes are 0, 1 or 2");
    fo::g_sync_producer.store(producer);
    fo::g_sync_consumer.store(consumer);
    return FO_OK;
}

void fo_get_sync_mode(int32_t* producer, int32_t* consumer) {
    if (producer) *producer = fo::g_sync_producer.load();
    if (consumer) *consumer = fo::g_sync_consumer.load();
}

fo_status fo_set_consumer_grid(int32_t max_blocks, int32_t threads) {
    fo::clear_error();
    if (max_blocks < 1 || max_blocks > fo::kMaxConsumeBlocks)
        return fo::fail(FO_ERR_ARG, "max_blocks must be in [1, 256]");
    if (!fo::valid_threads(threads)) return fo::fail(FO_ERR_ARG, "threads must be 64, 128 or 256");
    fo::g_consumer_blocks.store(max_blocks);
    fo::g_consumer_threads.store(threads);
    return FO_OK;
}

void fo_get_consumer_grid(int32_t* max_blocks, int32_t* threads) {
    if (max_blocks) *max_blocks = fo::g_consumer_blocks.load();
    if (threads) *threads = fo::g_consumer_threads.load();
}

fo_status fo_options_init(fo_options* o) {
    fo::clear_error();
    if (!o) return fo::fail(FO_ERR_ARG, "options is NULL");
    *o = fo::defaults();
    return FO_OK;
}

fo_status fo_device_wall_clock_khz(int32_t* khz) {
    fo::clear_error();
    if (!khz) return fo::fail(FO_ERR_ARG, "khz is NULL");
    int64_t k = 0;
    fo_status st = fo::clock_khz(&k);
    if (st != FO_OK) return st;
    *khz = (int32_t)k;
    return FO_OK;
}

fo_status fo_device_num_cus(int32_t device, int32_t* num_cus) {
    fo::clear_error();
    if (!num_cus) return fo::fail(FO_ERR_ARG, "num_cus is NULL");
    int v = 0;
    hipError_t e = hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return fo::hip_fail("hipDeviceGetAttribute", e);
    *num_cus = v;
    return FO_OK;
}

fo_status fo_reset_counters(uint32_t* counters, int32_t n, void* stream) {
    fo::clear_error();
    if (n < 0 || (n > 0 && !counters)) return fo::fail(FO_ERR_ARG, "bad counters");
    if (n == 0) return FO_OK;
    hipLaunchKernelGGL(fo::fill_u32_kernel, dim3((n + 255) / 256), dim3(256), 0,
                       (hipStream_t)stream, counters, n, 0u);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? FO_OK : fo::hip_fail("fill kernel launch", e);
}

fo_status fo_gemm_signal_reorder(const fo_plan* plan, const void* dev_plan, const void* A,
                                 const void* W, void* C_out, uint32_t* counters, void* stream,
                                 const fo_options* options) {
    fo::clear_error();
    if (!plan) return fo::fail(FO_ERR_ARG, "plan is NULL");
    fo_options o;
    fo_status st = fo::resolve(options, &o);
    if (st != FO_OK) return st;
    if (plan->tiles == 0) return FO_OK;
    if (!A || !W || !C_out) return fo::fail(FO_ERR_ARG, "null operand");
    if (!dev_plan && (plan->pattern != FO_PATTERN_ROWMAJOR || counters))
        return fo::fail(FO_ERR_ARG, "dev_plan is NULL");
    if (!fo::gemm_tile_supported(plan->tile_m, plan->tile_n))
        return fo::fail(FO_ERR_UNSUPPORTED, "GEMM kernels exist for 256x128, 256x256 and 64x64 tiles");
    if (plan->K % 64) return fo::fail(FO_ERR_SHAPE, "K must be a multiple of 64");
    // operand row blocks are addressed with 32-bit byte offsets
    if ((int64_t)std::max(plan->tile_m, plan->tile_n) * plan->K * 2 > INT32_MAX)
        return fo::fail(FO_ERR_SHAPE, "tile rows x K x 2 bytes must fit in 31 bits");
    if (!fo::aligned16(A) || !fo::aligned16(W) || !fo::aligned16(C_out))
        return fo::fail(FO_ERR_ARG, "A, W and C_out must be 16-byte aligned");
    if (dev_plan && !fo::aligned16(dev_plan)) return fo::fail(FO_ERR_ARG, "dev_plan must be 16-byte aligned");
    const fo_dev_layout& L = plan->layout;
    fo::GemmArgs a{};
    a.A = static_cast<const uint16_t*>(A);
    a.W = static_cast<const uint16_t*>(W);
    a.C = static_cast<uint16_t*>(C_out);
    a.M = plan->M; a.N = plan->N; a.K = plan->K;
    a.tiles_m = plan->tiles_m; a.tiles_n = plan->tiles_n;
    a.order = plan->order; a.group_m = plan->group_m; a.num_xcds = plan->num_xcds;
    a.pattern = plan->pattern; a.num_dest = plan->num_dest;
    if (dev_plan) {
        a.tile_to_slot = fo::dev_table<int32_t>(dev_plan, L.tile_to_slot);
        a.slot_group = fo::dev_table<int32_t>(dev_plan, L.slot_group);
        a.group_first = fo::dev_table<int32_t>(dev_plan, L.group_first);
        a.row_bucket = fo::dev_table<int32_t>(dev_plan, L.row_bucket);
        a.row_rank = fo::dev_table<int32_t>(dev_plan, L.row_rank);
        a.pool_base = fo::dev_table<int32_t>(dev_plan, L.pool_base);
        a.pool_off = fo::dev_table<int32_t>(dev_plan, L.pool_off);
    }
    a.counters = plan->P > 0 ? counters : nullptr;
    a.sync = o.sync_producer;
    a.c_rsrc = plan->M * plan->N * 2 <= INT32_MAX ? 1 : 0;
    a.trace = o.tile_trace;
    a.trace_cap = a.trace ? o.tile_trace_capacity : 0;
    // Persistent grid: one workgroup per tile of a wave. Position classes
    // follow the chiplet of the XCD dispatch order.
    const int grid = std::min(plan->tiles, std::max(plan->W, 1));
    if (a.counters) {
        a.dispenser = counters + plan->P;
        a.num_dispensers = plan->order == FO_ORDER_XCD ? std::min(plan->num_xcds, FO_DISPENSER_WORDS) : 1;
        a.num_dispensers = std::max(1, std::min(a.num_dispensers, grid));
    }
    hipError_t e = fo::launch_gemm(plan->dtype, plan->tile_m, plan->tile_n, a, grid, (hipStream_t)stream);
    return e == hipSuccess ? FO_OK : fo::hip_fail("GEMM launch", e);
}

fo_status fo_consume_group(const void* src, const void* peer, void* dst, int64_t len,
                           int32_t dtype, const uint32_t* counter, uint32_t target,
                           uint32_t* status_word, void* stream, const fo_options* options) {
    fo::clear_error();
    fo_options o;
    fo_status st = fo::resolve(options, &o);
    if (st != FO_OK) return st;
    if (len < 0) return fo::fail(FO_ERR_ARG, "len < 0");
    if (dtype != FO_FP16 && dtype != FO_BF16) return fo::fail(FO_ERR_ARG, "bad dtype");
    if (len == 0 && !counter) return FO_OK;
    if (len > 0 && (!src || !dst)) return fo::fail(FO_ERR_ARG, "null src or dst");
    fo::ConsumeArgs a{};
    st = fo::consume_args(static_cast<const uint16_t*>(src), static_cast<const uint16_t*>(peer),
                          static_cast<uint16_t*>(dst), counter, target, status_word, o, &a);
    if (st != FO_OK) return st;
    a.nseg = 1;
    a.seg[0] = fo::ConsumeSegment{0, 0, len};
    hipError_t e = fo::launch_consume(dtype, o.sync_consumer, a, fo::limited(o, o.consumer_blocks),
                                      o.consumer_threads, false, (hipStream_t)stream);
    return e == hipSuccess ? FO_OK : fo::hip_fail("consumer launch", e);
}

fo_status fo_post_reorder(const fo_plan* plan, const void* dev_plan, const void* src, void* out,
                          const void* bias, const void* gamma, float eps, int32_t do_rmsnorm,
                          void* stream) {
    fo::clear_error();
    if (!plan) return fo::fail(FO_ERR_ARG, "plan is NULL");
    if (plan->M == 0 || plan->N == 0) return FO_OK;
    if (!src || !out) return fo::fail(FO_ERR_ARG, "null src or out");
    if (!dev_plan && plan->pattern != FO_PATTERN_ROWMAJOR) return fo::fail(FO_ERR_ARG, "dev_plan is NULL");
    if (plan->N % 8 || plan->tile_n % 8) return fo::fail(FO_ERR_UNSUPPORTED, "N and tile_n must be multiples of 8");
    if (!fo::aligned16(src) || !fo::aligned16(out) || (bias && !fo::aligned16(bias)) ||
        (gamma && !fo::aligned16(gamma)))
        return fo::fail(FO_ERR_ARG, "src, out, bias and gamma must be 16-byte aligned");
    if (do_rmsnorm && !(eps >= 0.0f)) return fo::fail(FO_ERR_ARG, "eps must be >= 0");
    const fo_dev_layout& L = plan->layout;
    fo::PostArgs a{};
    a.src = static_cast<const uint16_t*>(src);
    a.out = static_cast<uint16_t*>(out);
    a.bias = static_cast<const uint16_t*>(bias);
    a.gamma = static_cast<const uint16_t*>(gamma);
    a.M = plan->M; a.N = plan->N;
    a.tile_m = plan->tile_m; a.tile_n = plan->tile_n; a.tiles_n = plan->tiles_n;
    {
        const int cpt = plan->tile_n / 8;
        a.cpt_log2 = -1;
        for (int l = 0; l < 31; ++l)
            if ((1 << l) == cpt) a.cpt_log2 = l;
        if (plan->pattern != FO_PATTERN_ROWMAJOR && (plan->tile_n % 8 || a.cpt_log2 < 0))
            return fo::fail(FO_ERR_UNSUPPORTED, "post-reorder needs tile_n / 8 to be a power of two");
        // row-major source: chunk c of a row lies at the row's first piece + c
        if (plan->pattern == FO_PATTERN_ROWMAJOR) a.cpt_log2 = 31;
    }
    a.pattern = plan->pattern; a.num_dest = plan->num_dest;
    a.per_dest = plan->pattern == FO_PATTERN_SUBTILE
                     ? (int64_t)plan->tiles * (plan->tile_m / plan->num_dest) * plan->tile_n : 0;
    if (dev_plan) {
        a.tile_to_slot = fo::dev_table<int32_t>(dev_plan, L.tile_to_slot);
        a.dest_perm = fo::dev_table<int32_t>(dev_plan, L.dest_perm);
        a.row_bucket = fo::dev_table<int32_t>(dev_plan, L.row_bucket);
        a.row_rank = fo::dev_table<int32_t>(dev_plan, L.row_rank);
        a.pool_base = fo::dev_table<int32_t>(dev_plan, L.pool_base);
        a.pool_off = fo::dev_table<int32_t>(dev_plan, L.pool_off);
    }
    a.eps = eps;
    a.do_norm = do_rmsnorm ? 1 : 0;
    // source pieces are addressed in 16-byte chunks with 32-bit offsets
    if (std::max<int64_t>(plan->dest_elems, plan->M * plan->N) / 8 > (int64_t)UINT32_MAX)
        return fo::fail(FO_ERR_SHAPE, "post-reorder source buffer too large for 32-bit chunk offsets");
    if (fo::post_lds_bytes(a) > 64 * 1024)
        return fo::fail(FO_ERR_UNSUPPORTED, "post-reorder: too many tile columns or too wide a row for LDS");
    hipError_t e = fo::launch_post(plan->dtype, a, (hipStream_t)stream);
    return e == hipSuccess ? FO_OK : fo::hip_fail("post-reorder launch", e);
}


fo_status fo_run_overlapped(const fo_plan* plan, const void* dev_plan, const void* A, const void* W,
                            void* C_out, const void* peer, void* dst, void* out, const void* bias,
                            const void* gamma, float eps, int32_t do_rmsnorm, uint32_t* counters,
                            uint32_t* status_word, void* gemm_stream, void* comm_stream,
                            void* gemm_begin_event, void* gemm_end_event, const fo_options* options) {
    fo::clear_error();
    if (!plan) return fo::fail(FO_ERR_ARG, "plan is NULL");
    fo_options o;
    fo_status st = fo::resolve(options, &o);
    if (st != FO_OK) return st;
    if (plan->tiles == 0) return FO_OK;
    if (!dst) return fo::fail(FO_ERR_ARG, "dst is NULL");
    // An overlapped run with one group has nothing to overlap (its consumer
    // can only start once the whole GEMM is done): it runs on the GEMM stream
    // alone, as a serialized run does (no handoffs, no signalling).
    const bool requested = comm_stream && comm_stream != gemm_stream;
    const bool overlap = requested && plan->P > 1;
    if (requested && !counters) return fo::fail(FO_ERR_ARG, "an overlapped run needs counters");
    // The null stream waits for work on other blocking streams, which would
    // hold its reset kernel behind the gate kernel that waits for it.
    if (overlap && !gemm_stream) return fo::fail(FO_ERR_ARG, "an overlapped run needs a created GEMM stream");
    hipStream_t s1 = (hipStream_t)gemm_stream, s2 = (hipStream_t)comm_stream;
    hipError_t e;
    fo::ConsumeArgs a{};
    // consume_args also yields the wait limit in device clock ticks
    if ((st = fo::consume_args(static_cast<const uint16_t*>(C_out), static_cast<const uint16_t*>(peer),
                               static_cast<uint16_t*>(dst), nullptr, 0, status_word, o, &a)) != FO_OK)
        return st;
    const uint64_t ticks = a.timeout_ticks;
    // Handoff words after the group and position counters.
    uint32_t* gate = overlap ? counters + plan->P + FO_DISPENSER_WORDS : nullptr;
    uint32_t* done = overlap ? gate + 1 : nullptr;      // done word 0; word k at done + k * kDoneStride
    const uint32_t seq = fo::g_run_seq.fetch_add(1, std::memory_order_relaxed);
    const uint32_t tag = fo::kGateTag | (seq & fo::kGateSeqMask);
    const uint32_t done_tag = fo::done_tag_of(seq);
    if (overlap) {
        hipLaunchKernelGGL(fo::reset_run_kernel, dim3(1), dim3(256), 0, s1, counters, plan->P + FO_DISPENSER_WORDS,
                           done, done_tag, status_word, gate, tag);
        if ((e = hipGetLastError()) != hipSuccess) return fo::hip_fail("reset kernel launch", e);
    }
    if (overlap && (e = fo::launch_gate(gate, tag, status_word, ticks, s2)) != hipSuccess)
        return fo::hip_fail("gate kernel launch", e);
    if (gemm_begin_event && (e = hipEventRecord((hipEvent_t)gemm_begin_event, s1)) != hipSuccess)
        return fo::hip_fail("hipEventRecord", e);
    if ((st = fo_gemm_signal_reorder(plan, dev_plan, A, W, C_out, overlap ? counters : nullptr, s1, &o)) !=
        FO_OK)
        return st;
    if (gemm_end_event && (e = hipEventRecord((hipEvent_t)gemm_end_event, s1)) != hipSuccess)
        return fo::hip_fail("hipEventRecord", e);
    // One consumer launch per group (more if a group has more pieces than a
    // launch carries), as a collective library would take one call per
    // group. Groups before the last one share the device with the GEMM and
    // use the configured grid cap; the last group runs once the GEMM is
    // done and takes the full grid. The final launch counts its finished
    // workgroups in the done words, for which the GEMM stream waits before
    // the post-reorder.
    const int64_t* seg = plan->segs.data();
    const int nseg = (int)(plan->segs.size() / 5);
    const int sync = o.sync_consumer;
    const int cap = o.consumer_blocks;
    const int cap_threads = o.consumer_threads;
    struct Launch {
        fo::ConsumeArgs args;
        bool last;
    };
    std::vector<Launch> launches;
    for (int i = 0; i < nseg;) {
        const int64_t j = seg[5 * i];
        Launch l{a, j + 1 == plan->P || !overlap};
        l.args.counter = overlap ? counters + j : nullptr;
        l.args.target = (uint32_t)plan->targets[j];
        l.args.nseg = 0;
        for (; i < nseg && seg[5 * i] == j && l.args.nseg < fo::kMaxConsumeSegments; ++i)
            if (seg[5 * i + 4] > 0)
                l.args.seg[l.args.nseg++] = fo::ConsumeSegment{seg[5 * i + 2], seg[5 * i + 3], seg[5 * i + 4]};
        if (l.args.nseg > 0) launches.push_back(l);
    }
    int final_blocks = 0;
    for (size_t k = 0; k < launches.size(); ++k) {
        fo::ConsumeArgs& c = launches[k].args;
        const bool final_launch = overlap && k + 1 == launches.size();
        c.done = final_launch ? done : nullptr;
        c.done_tag = done_tag;
        // Under a consumer limit every launch takes the variant that runs
        // beside the GEMM, so that the emulated link has one speed in
        // overlapped and serialized runs alike.
        const bool capped = o.consumer_limit > 0;
        const bool last = launches[k].last;
        const int blocks = fo::limited(o, last ? fo::kMaxConsumeBlocks : cap);
        const int threads = last ? 256 : cap_threads;
        if ((e = fo::launch_consume(plan->dtype, sync, c, blocks, threads, last && !capped, overlap ? s2 : s1,
                                    final_launch ? &final_blocks : nullptr)) != hipSuccess)
            return fo::hip_fail("consumer launch", e);
    }
    // the done words reach the run's tag plus their shares of the launch's
    // grid only through this run's final consumer (a late consumer of an
    // earlier run finds another tag in them and does not count)
    if (final_blocks > 0 &&
        (e = fo::launch_done_wait(done, done_tag, final_blocks, status_word, ticks, s1)) != hipSuccess)
        return fo::hip_fail("wait kernel launch", e);
    if (out) return fo_post_reorder(plan, dev_plan, dst, out, bias, gamma, eps, do_rmsnorm, s1);
    return FO_OK;
}

fo_status fo_run_overlapped_noalloc(const fo_plan* plan, const void* dev_plan, const void* A, const void* W,
                                    void* C_out, const void* peer, void* dst, void* out, const void* bias,
                                    const void* gamma, float eps, int32_t do_rmsnorm, uint32_t* status_word,
                                    void* gemm_stream, void* comm_stream, const fo_options* options) {
    fo::clear_error();
    if (!plan) return fo::fail(FO_ERR_ARG, "plan is NULL");
    const int32_t need = fo_plan_num_counters(plan);
    if (need > FO_NOALLOC_MAX_COUNTERS)
        return fo::fail(FO_ERR_ARG, "fo_run_overlapped_noalloc: the plan needs " + std::to_string(need) +
                                        " counter words, the library's static array holds " +
                                        std::to_string(FO_NOALLOC_MAX_COUNTERS));
    fo_options o;
    fo_status st = fo::resolve(options, &o);
    if (st != FO_OK) return st;
    if (plan->tiles == 0) return FO_OK;
    uint32_t* counters = nullptr;
    if ((st = fo::scratch_of_current_device(&counters)) != FO_OK) return st;
    return fo_run_overlapped(plan, dev_plan, A, W, C_out, peer, dst, out, bias, gamma, eps, do_rmsnorm, counters,
                             status_word, gemm_stream, comm_stream, nullptr, nullptr, &o);
}

}  // extern "C"
