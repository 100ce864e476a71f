// GEMM with the reordering, signalling epilogue (gfx950).
//
// C = A x B (Section 2.1.1) with A [M, K] and W = B^T [N, K], both K
// contiguous. The grid is persistent: one workgroup per compute unit, each
// computing BM x BN output tiles one after another. Tiles are taken by
// dispatch position p (fo_order) in increasing order, so they run in waves
// of one tile per compute unit (Section 2.1.1) and position p is the tile's
// slot in the reordered output (Section 3.3 Approach (1)).
//
// Main loop, k steps of 64, A and W tiles moving from memory straight into an
// LDS ring of STAGES stages (direct global-to-LDS loads, XOR-swizzled rows for
// conflict-free 16-byte fragment reads); fragments of the next MFMA k step are
// read while the MFMAs of the current one run, and every LDS read and load
// issue sits in the shadow of an MFMA. Two forms:
//   256x256 and 256x128 tiles: 4 waves of 128 x 128 (128 x 64), one per
//     SIMD, v_mfma_f32_16x16x32 in inline asm with the accumulators tied in
//     place, two stages; a wave of 128 x 128 reads 2/3 of the LDS bytes per
//     flop that 8 waves of 128 x 64 read, which lets the power-limited clock
//     run higher. A substep's MFMAs carry the fragment reads of the next
//     substep and, after the step's barrier, the load issues of the stage
//     just freed, one every 4 (256x128: 2) MFMAs (bunched issues stall the
//     single wave of a SIMD on the memory pipeline).
//   64x64 tiles: 4 waves of 32 x 32, v_mfma_f32_32x32x16 from the compiler's
//     builtin, loads issued STAGES steps ahead.
// The main loop is the same for every output pattern (Section 5: only the
// epilogue changes).
//
// Epilogue (Section 3.3 Approach; Section 3.2 Approach):
//   0. (256x256 form) each row's destination is looked up while the tile's
//      main loop runs, and the next position is claimed a few k steps
//      before its end;
//   1. accumulators -> fp16/bf16 (round to nearest even) -> LDS staging tile
//      (in two passes of half the rows when the tile does not fit);
//   2. every tile row goes out as full-row stores to its destination:
//      row-major C, the tile's slot (tile pattern), the slice's place in its
//      group segment (subtile pattern) or the row's pool position (subtoken
//      pattern);
//   3. once the tile's stores are visible to all chiplets (fo_sync_mode:
//      device-coherent stores + wait, or an agent-scope release), one lane
//      adds 1 to the counter of the group that owns the slot.
#include <hip/hip_runtime.h>

#include <type_traits>
#include <utility>

#include "fo_device.h"
#include "fo_internal.h"
#include "gemm.h"

namespace fo {
namespace {

// s_waitcnt operand for vmcnt = vm and lgkmcnt = lgkm, expcnt at its maximum
// (gfx9 encoding: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8], vmcnt[5:4] at 15:14)
constexpr int wait_imm(int vm, int lgkm) {
    return (vm & 15) | (7 << 4) | ((lgkm & 15) << 8) | (((vm >> 4) & 3) << 14);
}
constexpr int kWaitVmcnt0 = wait_imm(0, 15);
// buffer resource word 3 for raw byte-addressed loads on gfx9
constexpr int kRsrcWord3 = 0x00020000;
// cache-policy operand of a buffer store: sc1 (device-coherent write-through)
constexpr int kCachePolicySc1 = 16;

typedef __attribute__((address_space(3))) void lds_void_t;

// 16x16x32 MFMA in inline asm with the accumulator tied in place (dst =
// srcC): with 256 accumulator registers per wave the compiler's own MFMAs
// get copied between register files every step. KEEP_V: the accumulator is
// held in VGPRs instead of AGPRs. The compiler does not track the hazards of
// these instructions: accumulators are never written by VALU right before
// one (the first MFMA of a tile takes srcC = 0 instead of a zeroed
// accumulator) and are read only after the wait that ends the main loop.
template <int DT, bool KEEP_V, typename C>
__device__ __forceinline__ void mfma16_tied(C& c, const u32x4_t& a, const u32x4_t& b) {
    if constexpr (DT == FO_FP16 && KEEP_V)
        asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b));
    else if constexpr (DT == FO_FP16)
        asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
    else if constexpr (KEEP_V)
        asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b));
    else
        asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}
// The same with srcC = 0: the first MFMA of a tile starts its accumulator.
template <int DT, bool KEEP_V, typename C>
__device__ __forceinline__ void mfma16_first(C& c, const u32x4_t& a, const u32x4_t& b) {
    if constexpr (DT == FO_FP16 && KEEP_V)
        asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, 0" : "=v"(c) : "v"(a), "v"(b));
    else if constexpr (DT == FO_FP16)
        asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, 0" : "=a"(c) : "v"(a), "v"(b));
    else if constexpr (KEEP_V)
        asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=v"(c) : "v"(a), "v"(b));
    else
        asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=a"(c) : "v"(a), "v"(b));
}

// Calls f(std::integral_constant<int, I>{}) for I = 0 .. N-1 (indices known
// at compile time, so the arrays they index stay in registers).
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
    (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

template <int DT>
__device__ __forceinline__ f32x16_t mfma32(u32x4_t a, u32x4_t b, f32x16_t c) {
    if constexpr (DT == FO_FP16)
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(bit_cast<half8_t>(a), bit_cast<half8_t>(b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(bit_cast<bf16x8_t>(a), bit_cast<bf16x8_t>(b), c, 0, 0, 0);
}

// LDS plan of one workgroup. An operand tile row holds the BK k values of
// one row of A (or of W): BK * 2 bytes = BK / 8 chunks of 16 bytes; chunk c
// of row r is stored at slot c ^ ((r >> kSwz) % (BK / 8)). The gfx950 LDS
// serves a 16-byte read for 16 lanes per cycle across 64 banks (256 bytes):
// 256 / (BK * 2) consecutive rows share a 256-byte bank line, so the 16 rows
// read together at one k position must land in 16 different (row within the
// line, slot) pairs, which this swizzle gives for any 16 consecutive rows
// (BK = 64: pairs of rows, shift 1; BK = 32: quads of rows, shift 2).
template <int BM, int BN, int STAGES, int NW, int BK>
struct Tiles {
    static constexpr int kBK = BK;                       // k values per main-loop step
    static constexpr int kRow = BK * 2;                  // bytes per operand row
    static constexpr int kCh = BK / 8;                   // 16-byte chunks per row
    static constexpr int kSwz = BK == 64 ? 1 : 2;        // log2(rows per bank line)
    static constexpr int kRowsPerBlk = 1024 / kRow;      // rows per 1 KB load block
    static constexpr int kA = BM * kRow, kB = BN * kRow;
    static constexpr int kStage = kA + kB;
    // Output staging reuses the operand stages: a staging row holds BN halfs
    // (BN / 8 chunks of 16 bytes); chunk c of row r is stored at chunk
    // c ^ (r % (BN / 8)), so that the 32 rows a half-wave writes at one
    // column land on different banks. kRowsPerStage staging rows per
    // stage, a pass stages as many tile rows as fit
    static constexpr int kLDC = BN;                      // staging row (halfs)
    static constexpr int kCCh = BN / 8;                  // staging chunks per row
    static constexpr int kRowsPerStage = kStage / (kLDC * 2);
    static constexpr int kCap = STAGES * kRowsPerStage;
    static constexpr int kRowsPerPass = BM <= kCap ? BM : BM / 2 <= kCap ? BM / 2 : BM / 4;
    static constexpr int kPasses = BM / kRowsPerPass;
    static constexpr int kAI = kA / 1024 / NW;           // 1 KB load blocks per wave
    static constexpr int kBI = kB / 1024 / NW;
    static constexpr int kLoads = kAI + kBI;
};

// Start loading one k step of this workgroup's A rows (into the first KA
// bytes of `st`) and W rows (after them) with direct global-to-LDS loads:
// each instruction moves 64 x 16 bytes into one 1 KB block. The rows are
// addressed through buffer resources over the tile's row blocks (a_bytes and
// w_bytes long; the host checks they fit in 32 bits): a read past them
// returns zero instead of faulting, and a resource of length 0 loads zeros
// without touching memory.
template <int AI, int BI, int KA, bool OPAQUE = true>
__device__ __forceinline__ void issue_tile(const uint16_t* Ablk, const uint16_t* Wblk, uint32_t a_bytes,
                                           uint32_t w_bytes, const uint32_t* voffA, const uint32_t* voffB,
                                           uint32_t soff, char* st, int wave) {
    const __amdgpu_buffer_rsrc_t rA =
        __builtin_amdgcn_make_buffer_rsrc((void*)Ablk, 0, (int)a_bytes, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t rW =
        __builtin_amdgcn_make_buffer_rsrc((void*)Wblk, 0, (int)w_bytes, kRsrcWord3);
    // The LDS block addresses (one scalar register each, M0 of the load) are
    // formed here from an opaque copy of the wave index, so that they are
    // not all kept live through the main loop (OPAQUE; the 4-wave kernel
    // takes the uniform index directly).
    int w = wave;
    if constexpr (OPAQUE) asm volatile("" : "+s"(w));
    else w = __builtin_amdgcn_readfirstlane(wave);
#pragma unroll
    for (int i = 0; i < AI; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_void_t*)(st + (w * AI + i) * 1024), 16, voffA[i],
                                                 soff, 0, 0);
#pragma unroll
    for (int i = 0; i < BI; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rW, (lds_void_t*)(st + KA + (w * BI + i) * 1024), 16,
                                                 voffB[i], soff, 0, 0);
}

// Load instruction idx (0 .. AI + BI - 1) of issue_tile alone, so that a
// step's loads can be spread over its MFMAs.
template <int AI, int BI, int KA>
__device__ __forceinline__ void issue_one(int idx, const uint16_t* Ablk, const uint16_t* Wblk, uint32_t a_bytes,
                                          uint32_t w_bytes, const uint32_t* voffA, const uint32_t* voffB,
                                          uint32_t soff, char* st, int wave) {
    const int w = __builtin_amdgcn_readfirstlane(wave);
    if (idx < AI) {
        const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc((void*)Ablk, 0, (int)a_bytes, kRsrcWord3);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (lds_void_t*)(st + (w * AI + idx) * 1024), 16, voffA[idx], soff,
                                                 0, 0);
    } else {
        const __amdgpu_buffer_rsrc_t rW = __builtin_amdgcn_make_buffer_rsrc((void*)Wblk, 0, (int)w_bytes, kRsrcWord3);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rW, (lds_void_t*)(st + KA + (w * BI + idx - AI) * 1024), 16,
                                                 voffB[idx - AI], soff, 0, 0);
    }
}

// Instruction order inside one k-step phase of the main loop: each MFMA
// (32 cycles of matrix work) carries up to R LDS fragment reads and V
// direct-to-LDS load issues in its shadow, so the matrix pipe does not
// drain while they are issued.
template <int MFMA, int R, int V>
__device__ __forceinline__ void interleave_phase() {
    constexpr int r1 = (R + MFMA - 1) / MFMA, v1 = (V + MFMA - 1) / MFMA;
#pragma unroll
    for (int i = 0; i < MFMA; ++i) {
        if (i * r1 < R) __builtin_amdgcn_sched_group_barrier(0x100, r1, 0);   // LDS read
        if (i * v1 < V) __builtin_amdgcn_sched_group_barrier(0x020, v1, 0);   // global load
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                    // MFMA
    }
}

// One main-loop synchronization: this wave waits until at most `vm` of its
// vector memory operations are in flight (its part of the next tile has
// landed in LDS) and until all of its LDS reads have returned (the stage it
// read last can be refilled), then the workgroup meets at a barrier. The
// empty asm statements keep the compiler from moving memory accesses (and
// so the load issue order that the vmcnt count relies on) across this
// point; the fence of __syncthreads() is not used because it would wait for
// every in-flight operand load.
template <int VM>
__device__ __forceinline__ void wait_and_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(wait_imm(VM, 0));
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// The kernel body; MF = 32 (v_mfma_f32_32x32x16, compiler builtin) or 16
// (v_mfma_f32_16x16x32 in tied inline asm, two stages of 64-wide k steps).
template <int DT, int BM, int BN, int WAVES_M, int WAVES_N, int STAGES, int BK, int MF>
__device__ __forceinline__ void gemm_body(const GemmArgs& a) {
    constexpr int NW = WAVES_M * WAVES_N, NT = 64 * NW;
    constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
    constexpr int MI = WTM / MF, NJ = WTN / MF;
    constexpr int KPM = 512 / MF;                        // k per MFMA: 16 (32x32) or 32 (16x16)
    using AccT = typename std::conditional<MF == 32, f32x16_t, f32x4_t>::type;
    constexpr int NACC = MF == 32 ? 16 : 4;              // accumulator registers per block and lane
    constexpr int kVRows = MF == 16 ? 2 : 0;             // accumulator block rows held in VGPRs
    using T = Tiles<BM, BN, STAGES, NW, BK>;
    constexpr int kBK = T::kBK;
    constexpr int P = kBK / KPM;                         // MFMA k steps per main-loop step
    static_assert(NW == 4 || NW == 8, "four or eight waves");
    static_assert(NT >= BM, "one thread per tile row in the epilogue set-up");
    static_assert(MF == 32 || MF == 16, "32x32x16 or 16x16x32 MFMAs");
    static_assert(WTM % MF == 0 && WTN % MF == 0, "whole MFMA blocks");
    static_assert(MF == 32 || (STAGES == 2 && P == 2), "the 16x16x32 form runs two stages of 64-wide k steps");
    static_assert(STAGES >= 2 && STAGES <= 4, "two to four LDS stages");
    static_assert(BK == 32 || BK == 64, "k steps of 32 or 64");
    static_assert(T::kAI >= 1 && T::kBI >= 1 && T::kA % (1024 * NW) == 0 && T::kB % (1024 * NW) == 0,
                  "each wave loads whole 1 KB blocks");
    static_assert(T::kRowsPerPass <= T::kCap, "output staging fits in the stages");
    static_assert(T::kRowsPerPass % WTM == 0, "a staging pass holds whole wave rows");

    // The stages live in separate arrays, so that the compiler can tell the
    // stage being read from the stages being filled.
    __shared__ __attribute__((aligned(1024))) char st0[T::kStage];
    __shared__ __attribute__((aligned(1024))) char st1[T::kStage];
    __shared__ __attribute__((aligned(STAGES >= 3 ? 1024 : 16))) char st2[STAGES >= 3 ? T::kStage : 16];
    __shared__ __attribute__((aligned(STAGES >= 4 ? 1024 : 16))) char st3[STAGES >= 4 ? T::kStage : 16];
    __shared__ int64_t row_off[BM];
    __shared__ int s_pos;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar registers
    const int wm = wave / WAVES_N, wn = wave % WAVES_N;
    const int64_t K = a.K;
    const int tiles = a.tiles_m * a.tiles_n;

    // Persistent workgroups. Positions are handed out in increasing order:
    // with a dispenser, workgroup b takes positions d, d + D, d + 2D, ... of
    // its class d = b % D from an atomic counter shared by the class (so a
    // position always runs on the chiplet the dispatch order meant it for,
    // and a workgroup that is never scheduled holds no position back);
    // without one, workgroup b takes b, b + grid, b + 2 grid, ...
    // Every workgroup of a class makes exactly one claim past the class's
    // positions (its last), so the claims of one launch return 0 .. n_cls +
    // w_cls - 1; the workgroup that gets the last value is the word's last
    // user in this launch and leaves it zero for the next launch. A value
    // past the class's positions (also one left over from elsewhere) ends
    // the workgroup's loop.
    const int D = a.num_dispensers;
    const int cls = a.dispenser ? (int)(blockIdx.x % (unsigned)D) : 0;
    const uint32_t n_cls = a.dispenser ? (uint32_t)((tiles - cls + D - 1) / D) : 0u;
    const uint32_t w_cls = a.dispenser ? (uint32_t)(((int)gridDim.x - cls + D - 1) / D) : 0u;
    auto claim = [&]() -> int {
        const uint32_t v = __hip_atomic_fetch_add(a.dispenser + cls, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (v == n_cls + w_cls - 1u)
            __hip_atomic_store(a.dispenser + cls, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return v < n_cls ? cls + D * (int)v : tiles;
    };
    const bool coherent = a.counters && a.sync == FO_SYNC_COHERENT;
    auto signal = [&](int group) {
        if (tid == 0)
            __hip_atomic_fetch_add(a.counters + group, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    int p = (int)blockIdx.x;
    if (a.dispenser) {
        if (tid == 0) s_pos = claim();
        __syncthreads();
        p = __builtin_amdgcn_readfirstlane(s_pos);   // uniform: scalar registers
    }

    // A load instruction fills one 1 KB block of kRowsPerBlk rows: lane l
    // writes slot l % kCh of row r = kRowsPerBlk * block + l / kCh, so it
    // fetches chunk (l % kCh) ^ ((r >> kSwz) % kCh) of that row.
    auto voff = [&](int blk) -> uint32_t {
        const int r = blk * T::kRowsPerBlk + lane / T::kCh;
        return (uint32_t)(r * K * 2) +
               16u * (uint32_t)((lane % T::kCh) ^ ((r >> T::kSwz) & (T::kCh - 1)));
    };
    uint32_t voffA[T::kAI], voffB[T::kBI];
#pragma unroll
    for (int i = 0; i < T::kAI; ++i) voffA[i] = voff(wave * T::kAI + i);
#pragma unroll
    for (int i = 0; i < T::kBI; ++i) voffB[i] = voff(wave * T::kBI + i);
    const int KT = (int)(K / kBK);
    const uint16_t* Ablk = a.A;
    const uint16_t* Wblk = a.W;
    // Tiles past the last k step are "loaded" through empty resources: the
    // loads return zeros without touching memory, so every step issues the
    // same loads and the wait counts stay uniform (no branches).
    auto issue = [&](int kt, char* st) {
        const bool live = kt < KT;
        issue_tile<T::kAI, T::kBI, T::kA, MF == 32>(Ablk, Wblk, live ? (uint32_t)(BM * K * 2) : 0u,
                                         live ? (uint32_t)(BN * K * 2) : 0u, voffA, voffB,
                                         live ? (uint32_t)kt * (kBK * 2) : 0u, st, wave);
    };

    AccT acc[MI][NJ];

    // Fragment addressing: lane l feeds row (l % MF) of an MF-row block with
    // the 8 consecutive k values of chunk (KPM/8)*kk + l/MF of MFMA k step kk
    // (blocks start on multiples of MF, so the row's swizzle depends on l
    // only).
    const int a_row = (wm * WTM + (lane & (MF - 1))) * T::kRow;
    const int b_row = T::kA + (wn * WTN + (lane & (MF - 1))) * T::kRow;
    int cslot[P];
#pragma unroll
    for (int kk = 0; kk < P; ++kk)
        cslot[kk] = 16 * (((KPM / 8) * kk + lane / MF) ^ ((lane >> T::kSwz) & (T::kCh - 1)));

    // Two fragment register sets: the fragments of k step kk+1 are read from
    // LDS while the MFMAs of k step kk run.
    u32x4_t fa0[MI], fb0[NJ], fa1[MI], fb1[NJ];
    auto load_frags = [&](const char* st, int kk, u32x4_t (&fa)[MI], u32x4_t (&fb)[NJ]) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
            fa[i] = *reinterpret_cast<const u32x4_t*>(st + a_row + i * MF * T::kRow + cslot[kk]);
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            fb[j] = *reinterpret_cast<const u32x4_t*>(st + b_row + j * MF * T::kRow + cslot[kk]);
    };
    // W fragment as the MFMA's first operand: the result block is C^T, so
    // each lane holds 4 consecutive output columns.
    auto mma = [&](const u32x4_t (&fa)[MI], const u32x4_t (&fb)[NJ]) {
        if constexpr (MF == 32) {
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    acc[i][j] = mfma32<DT>(fb[j], fa[i], acc[i][j]);
        }
    };

    constexpr int kMfma = MI * NJ, kReads = MI + NJ;
    // 16x16x32 form: destination of tile row `tid` (element offset), looked
    // up at the start of the tile and written to row_off after the first
    // main-loop barrier, so that the lookups' latency hides under the loop
    // (the previous tile's epilogue is done with row_off by then).
    int64_t my_off = 0;
    // Group of the previous tile whose count is still to be sent (or -1):
    // with device-coherent stores and two stages, a tile's count goes out at
    // the first main-loop barrier of the workgroup's next tile, so that the
    // stores complete while the next tile's first loads are in flight.
    int pend = -1;
    constexpr std::true_type kYes{};
    constexpr std::false_type kNo{};
    const bool defer = STAGES == 2 && coherent && !a.trace;
    // Step kt multiplies the tile in stage `cur` (its k step 0 fragments are
    // already in fa0/fb0; tile kt+1 is in stage `nxt`). Before its last k
    // step, every wave has read all of `cur` and tile kt+1 has landed (tiles
    // up to kt+STAGES-1 may still be loading): after the barrier, tile
    // kt+STAGES goes into `cur`, and the first fragments of tile kt+1 are read
    // while the last MFMAs of tile kt run.
    // 16x16x32 form: MFMA m of a substep (block row m / NJ, column m % NJ)
    // carries fragment read m of the next substep (m < MI + NJ: A0, B0 ..
    // B(NJ-1), A1 .. A(MI-1), the order the next substep needs them) and, in
    // the substep after the barrier, every 4th MFMA one load issue of the
    // stage just freed (step lkt; `loads`). sched_barrier keeps this order.
    // The first substep of a tile (FIRST) starts the accumulators.
    auto mma_rd = [&](const u32x4_t (&fa)[MI], const u32x4_t (&fb)[NJ], const char* rst, int rkk,
                      u32x4_t (&ra)[MI], u32x4_t (&rb)[NJ], int lkt, char* lst, bool loads,
                      auto first_c) __attribute__((always_inline)) {
        const bool live = lkt < KT;
        const uint32_t ab = live ? (uint32_t)(BM * K * 2) : 0u, wb = live ? (uint32_t)(BN * K * 2) : 0u;
        const uint32_t so = live ? (uint32_t)lkt * (kBK * 2) : 0u;
        constexpr int kGap = (MI * NJ) / T::kLoads >= 4 ? 4 : (MI * NJ) / T::kLoads;
        static_assert(kGap >= 1, "a load issue at least every MFMA");
        static_for<MI * NJ>([&](auto mc) __attribute__((always_inline)) {
            constexpr int m = decltype(mc)::value;
            constexpr int i = m / NJ, j = m % NJ;
            if constexpr (m < MI + NJ) {
                if constexpr (m == 0)
                    ra[0] = *reinterpret_cast<const u32x4_t*>(rst + a_row + cslot[rkk]);
                else if constexpr (m <= NJ)
                    rb[m - 1] = *reinterpret_cast<const u32x4_t*>(rst + b_row + (m - 1) * MF * T::kRow + cslot[rkk]);
                else
                    ra[m - NJ] = *reinterpret_cast<const u32x4_t*>(rst + a_row + (m - NJ) * MF * T::kRow + cslot[rkk]);
            }
            if constexpr (m % kGap == 0 && m / kGap < T::kLoads)
                if (loads)
                    issue_one<T::kAI, T::kBI, T::kA>(m / kGap, Ablk, Wblk, ab, wb, voffA, voffB, so, lst, wave);
            constexpr bool kV = i >= MI - kVRows;
            if constexpr (decltype(first_c)::value) mfma16_first<DT, kV>(acc[i][j], fb[j], fa[i]);
            else mfma16_tied<DT, kV>(acc[i][j], fb[j], fa[i]);
            __builtin_amdgcn_sched_barrier(0);
        });
    };
    auto step = [&](int kt, char* cur, const char* nxt, auto first_c) __attribute__((always_inline)) {
        if constexpr (MF == 16) {
            mma_rd(fa0, fb0, cur, 1, fa1, fb1, 0, cur, false, first_c);
            wait_and_barrier<0>();
            if constexpr (decltype(first_c)::value) {
                // the previous tile's stores are complete in every wave (this
                // barrier follows a vmcnt(0) wait): its deferred count goes out
                if (pend >= 0) {
                    if (tid == 0)
                        __hip_atomic_fetch_add(a.counters + pend, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    pend = -1;
                }
                if (tid < BM) row_off[tid] = my_off;
            }
            mma_rd(fa1, fb1, nxt, 0, fa0, fb0, kt + STAGES, cur, true, std::false_type{});
            return;
        }
        load_frags(cur, 1, fa1, fb1);
        mma(fa0, fb0);
        interleave_phase<kMfma, kReads, 0>();
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (P == 4) {
            load_frags(cur, 2, fa0, fb0);
            mma(fa1, fb1);
            interleave_phase<kMfma, kReads, 0>();
            __builtin_amdgcn_sched_barrier(0);
            load_frags(cur, 3, fa1, fb1);
            mma(fa0, fb0);
            interleave_phase<kMfma, kReads, 0>();
            __builtin_amdgcn_sched_barrier(0);
        }
        wait_and_barrier<(STAGES - 2) * T::kLoads>();
        if constexpr (STAGES == 2 && decltype(first_c)::value) {
            // The previous tile's stores are complete in every wave (this
            // barrier follows a vmcnt(0) wait): its deferred count goes out.
            if (pend >= 0) {
                if (tid == 0)
                    __hip_atomic_fetch_add(a.counters + pend, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                pend = -1;
            }
        }
        issue(kt + STAGES, cur);
        load_frags(nxt, 0, fa0, fb0);
        mma(fa1, fb1);
        interleave_phase<kMfma, kReads, T::kLoads>();
        __builtin_amdgcn_sched_barrier(0);
    };

    // Column n (a multiple of 4 halfs) of staging row r of an output pass
    // ([0, kRowsPerPass)): row r % RPS of stage r / RPS, RPS = kRowsPerStage,
    // chunk (n / 8) ^ (r % kCCh).
    auto cptr = [&](int r, int n) -> uint16_t* {
        constexpr int RPS = T::kRowsPerStage;
        const int si = r / RPS, rr = r - (r / RPS) * RPS;
        char* base = si == 0 ? st0 : si == 1 ? st1 : si == 2 ? st2 : st3;
        const int chunk = (n >> 3) ^ (r & (T::kCCh - 1));
        return reinterpret_cast<uint16_t*>(base + rr * T::kLDC * 2 + chunk * 16 + (n & 7) * 2);
    };
    while (p < tiles) {
        const uint64_t t_start = a.trace ? wall_clock64() : 0;
        const int tile = tile_of_position(p, a.tiles_m, a.tiles_n, a.order, a.group_m, a.num_xcds);
        const int tm = tile / a.tiles_n, tn = tile - (tile / a.tiles_n) * a.tiles_n;
        Ablk = a.A + (int64_t)tm * BM * K;
        Wblk = a.W + (int64_t)tn * BN * K;

        // Plan lookups needed only by the epilogue: issued now, consumed later.
        const int slot = a.tile_to_slot ? a.tile_to_slot[tile] : p;
        const int group = a.counters ? a.slot_group[slot] : 0;
        int bucket = 0, rank = 0;
        if (a.pattern == FO_PATTERN_SUBTOKEN && tid < BM) {
            bucket = a.row_bucket[tm * BM + tid];
            rank = a.row_rank[tm * BM + tid];
        }

        // Destination (element offset) of row r of the tile, by pattern.
        auto row_dest = [&](int r) -> int64_t {
            int64_t off;
            if (a.pattern == FO_PATTERN_ROWMAJOR) {
                off = ((int64_t)tm * BM + r) * a.N + (int64_t)tn * BN;
            } else if (a.pattern == FO_PATTERN_TILE) {
                off = ((int64_t)slot * BM + r) * BN;
            } else if (a.pattern == FO_PATTERN_SUBTILE) {
                const int h = BM / a.num_dest;
                const int k = r / h, rr = r - (r / h) * h;
                const int j = a.slot_group[slot];
                const int64_t f0 = a.group_first[j];
                const int64_t nj = a.group_first[j + 1] - f0;
                off = f0 * BM * BN + ((int64_t)k * nj + (slot - f0)) * h * BN + (int64_t)rr * BN;
            } else {
                const int B = a.num_dest;
                off = ((int64_t)a.pool_off[bucket] + a.pool_base[(int64_t)slot * B + bucket] + rank) * BN;
            }
            return off;
        };
        if constexpr (MF == 32) {      // (the 16x16x32 form starts them with srcC = 0)
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
#pragma unroll
                    for (int r = 0; r < NACC; ++r) acc[i][j][r] = 0.0f;
        }

        issue(0, st0);
        issue(1, st1);
        if constexpr (MF == 16)
            if (tid < BM) my_off = row_dest(tid);
        if constexpr (STAGES >= 3) issue(2, st2);
        if constexpr (STAGES >= 4) issue(3, st3);
        wait_and_barrier<(STAGES - 1) * T::kLoads>();
        load_frags(st0, 0, fa0, fb0);
        int kt = 0;
        bool claimed = false;
        int next = p + (int)gridDim.x;
        if constexpr (STAGES == 4) {
            for (; kt + 4 <= KT; kt += 4) {      // tile t lives in stage t % 4
                step(kt, st0, st1, kNo);
                step(kt + 1, st1, st2, kNo);
                step(kt + 2, st2, st3, kNo);
                step(kt + 3, st3, st0, kNo);
            }
            if (kt < KT) step(kt, st0, st1, kNo);
            if (kt + 1 < KT) step(kt + 1, st1, st2, kNo);
            if (kt + 2 < KT) step(kt + 2, st2, st3, kNo);
        } else if constexpr (STAGES == 3) {
            for (; kt + 3 <= KT; kt += 3) {      // tile t lives in stage t % 3
                step(kt, st0, st1, kNo);
                step(kt + 1, st1, st2, kNo);
                step(kt + 2, st2, st0, kNo);
            }
            if (kt < KT) step(kt, st0, st1, kNo);
            if (kt + 1 < KT) step(kt + 1, st1, st2, kNo);
        } else {                                 // tile t lives in stage t % 2
            // the first step sends the previous tile's deferred count
            step(0, st0, st1, kYes);
            for (kt = 1; kt + 2 <= KT; kt += 2) {
                // 16x16x32 form: the next position is claimed two to three
                // steps before the end of this tile, so that the atomic's
                // latency hides under them
                if (MF == 16 && a.dispenser && !claimed && kt + 4 >= KT) {
                    claimed = true;
                    if (tid == 0) next = claim();
                }
                step(kt, st1, st0, kNo);
                step(kt + 1, st0, st1, kNo);
            }
            if (kt < KT) step(kt, st1, st0, kNo);
        }
        // inline-asm MFMAs: the accumulators are read only once the last
        // MFMA's result is written (the compiler inserts no wait for them)
        if constexpr (MF == 16) asm volatile("s_nop 7\n s_nop 7\n s_nop 7\n s_nop 7" ::: "memory");
        wait_and_barrier<0>();    // no load may still be writing LDS
        __syncthreads();          // operand stages are reused for the output tile

        // ---- epilogue ---------------------------------------------------
        // The epilogue's thread coordinates go through an opaque copy, so
        // that its address arithmetic stays here instead of being hoisted
        // out of the tile loop (where it would hold registers through the
        // main loop).
        int tid_e = tid;
        asm volatile("" : "+v"(tid_e));
        const int lane_e = tid_e & 63, wave_e = __builtin_amdgcn_readfirstlane(tid_e >> 6);
        const int wm_e = wave_e / WAVES_N, wn_e = wave_e % WAVES_N;
        // Destination of row `tid` of the tile, by pattern.
        if (MF != 16 && tid < BM) row_off[tid] = row_dest(tid);

        // Otherwise the next position is claimed now; the atomic's latency
        // hides behind this tile's stores.
        if (a.dispenser && !claimed && tid == 0) next = claim();

#pragma unroll
        for (int pass = 0; pass < T::kPasses; ++pass) {
            const int r0 = pass * T::kRowsPerPass;
            // accumulators of the waves whose rows are in this pass -> staging
            if constexpr (MF == 16 && BN == 256) {
                // 256 x 256 tile, 4 waves of 128 x 128, one pass: the
                // addresses of cptr in closed form. Lane l of block (i, j)
                // holds tile row wm*128 + i*16 + l%16, columns wn*128 + j*16 +
                // 4*(l/16) .. +3: staging row i*16 + l%16 of stage wm, chunk
                // (wn*16 + 2j + l/32) ^ (row % 32) = 16*(wn ^ (i%2)) +
                // ((l/32 ^ l%16) ^ 2j), byte 8*((l/16) % 2) of it.
                static_assert(T::kPasses == 1 && T::kRowsPerStage == WTM && WAVES_M == 2 && WAVES_N == 2 &&
                              T::kLDC == 256 && T::kCCh == 32 && NT == 256 && NACC == 4,
                              "the 256 x 256 four-wave tile");
                const int lr = lane_e & 15, lh = (lane_e >> 4) & 1, lq = lane_e >> 5;
                char* const sb = wm_e == 0 ? st0 : st1;
                const uint32_t base_e = (uint32_t)(lr * 512 + lh * 8);
                const uint32_t tx = (uint32_t)((lq ^ lr) << 4);
                uint32_t o[2][NJ];
#pragma unroll
                for (int q = 0; q < 2; ++q)
#pragma unroll
                    for (int j = 0; j < NJ; ++j)
                        o[q][j] = base_e + 256u * (uint32_t)(wn_e ^ q) + (tx ^ (uint32_t)(j << 5));
                static_for<MI>([&](auto ic) __attribute__((always_inline)) {
                    constexpr int i = decltype(ic)::value;
                    static_for<NJ>([&](auto jc) __attribute__((always_inline)) {
                        constexpr int j = decltype(jc)::value;
                        u32x2_t v;
                        v[0] = pack2<DT>(acc[i][j][0], acc[i][j][1]);
                        v[1] = pack2<DT>(acc[i][j][2], acc[i][j][3]);
                        *reinterpret_cast<u32x2_t*>(sb + o[i & 1][j] + i * 8192) = v;
                    });
                });
            } else if (wm_e * WTM >= r0 && wm_e * WTM < r0 + T::kRowsPerPass) {
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    const int m = wm_e * WTM - r0 + i * MF + (lane_e & (MF - 1));
#pragma unroll
                    for (int j = 0; j < NJ; ++j) {
#pragma unroll
                        for (int q = 0; q < NACC / 4; ++q) {
                            const int n = wn_e * WTN + j * MF + q * 8 + (lane_e / MF) * 4;
                            u32x2_t v;
                            v[0] = pack2<DT>(acc[i][j][4 * q + 0], acc[i][j][4 * q + 1]);
                            v[1] = pack2<DT>(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
                            *reinterpret_cast<u32x2_t*>(cptr(m, n)) = v;
                        }
                    }
                }
            }
            __syncthreads();
            if (coherent && a.c_rsrc) {
                // Device-coherent 16-byte stores (cache policy sc1: written
                // through to the point all chiplets share), addressed through
                // a buffer resource over C: no cache write-back is needed
                // before the signal.
                const __amdgpu_buffer_rsrc_t rC =
                    __builtin_amdgcn_make_buffer_rsrc((void*)a.C, 0, 0x7FFFFFFF, kRsrcWord3);
                constexpr int CPR = BN / 8;             // 16-byte chunks per tile row
                constexpr int RPP = NT / CPR;           // rows per pass of the workgroup
                const int c = tid_e % CPR;
                if constexpr (MF == 16 && BN == 256) {
                    // thread t stores chunk c of tile rows r = t/32 + 8k
                    // (k < 32): stage k/16, staging row r % 128, chunk
                    // c ^ (r % 32) = c ^ (t/32 + 8 (k % 4))
                    const int r0t = tid_e / CPR;
                    uint32_t y[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) y[q] = (uint32_t)(((c ^ (r0t + 8 * q)) << 4) + r0t * 512);
                    static_for<32>([&](auto kc) __attribute__((always_inline)) {
                        constexpr int k = decltype(kc)::value;
                        const char* sb = k < 16 ? st0 : st1;
                        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(sb + y[k & 3] + 4096 * (k & 15));
                        __builtin_amdgcn_raw_buffer_store_b128(v, rC, (uint32_t)((row_off[r0t + 8 * k] + c * 8) * 2),
                                                               0, kCachePolicySc1);
                    });
                } else {
#pragma unroll 4
                    for (int r = tid_e / CPR; r < T::kRowsPerPass; r += RPP) {
                        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(cptr(r, c * 8));
                        __builtin_amdgcn_raw_buffer_store_b128(v, rC, (uint32_t)((row_off[r0 + r] + c * 8) * 2), 0,
                                                               kCachePolicySc1);
                    }
                }
            } else if (coherent) {
                // Device-coherent 8-byte stores for outputs past a 31-bit
                // byte range (written through to the point all chiplets
                // share): no cache write-back is needed before the signal.
                constexpr int LPR = BN / 4;             // lanes per row (8 bytes each)
                constexpr int RPI = LPR >= 64 ? 1 : 64 / LPR;   // rows per wave_e instruction
                constexpr int CPL = LPR >= 64 ? LPR / 64 : 1;   // 8-byte columns per lane_e
                const int lr = LPR >= 64 ? 0 : lane_e / LPR;
                const int lc = LPR >= 64 ? lane_e : lane_e % LPR;
#pragma unroll 4
                for (int r = wave_e * RPI + lr; r < T::kRowsPerPass; r += NW * RPI) {
#pragma unroll
                    for (int cc = 0; cc < CPL; ++cc) {
                        const int col = lc + cc * 64;
                        const uint64_t v = *reinterpret_cast<const uint64_t*>(cptr(r, col * 4));
                        __hip_atomic_store(reinterpret_cast<uint64_t*>(a.C + row_off[r0 + r]) + col, v,
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
                }
            } else {
                constexpr int CPR = BN / 8;             // 16-byte chunks per tile row
                constexpr int RPP = NT / CPR;           // rows per pass of the workgroup
                const int c = tid_e % CPR;
#pragma unroll 4
                for (int r = tid_e / CPR; r < T::kRowsPerPass; r += RPP) {
                    const u32x4_t v = *reinterpret_cast<const u32x4_t*>(cptr(r, c * 8));
                    *reinterpret_cast<u32x4_t*>(a.C + row_off[r0 + r] + c * 8) = v;
                }
            }
            if (pass + 1 < T::kPasses) __syncthreads();   // staging is refilled
        }

        if (a.counters && !defer) {
            // Section 3.2: count the finished tile for its group once all of
            // the tile's stores are visible to every compute unit.
            if (coherent) {
                // each wave waits until its write-through stores are complete
                __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
                __syncthreads();
                signal(group);
            } else if (a.sync == FO_SYNC_FENCE_ALL) {
                // every wave: release fence at agent scope (L2 write-back + wait)
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                __syncthreads();
                if (tid == 0)
                    __hip_atomic_fetch_add(a.counters + a.slot_group[slot], 1u, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
            } else {
                // workgroup barrier, then one release increment (one write-back)
                __syncthreads();
                if (tid == 0)
                    __hip_atomic_fetch_add(a.counters + a.slot_group[slot], 1u, __ATOMIC_RELEASE,
                                           __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        if (a.trace && p < a.trace_cap) {
            // tile timeline: start, completion of every store of the tile,
            // chiplet and compute unit (hardware id registers), workgroup
            __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
            __syncthreads();
            if (tid == 0) {
                uint64_t* t = a.trace + 4 * (int64_t)p;
                t[0] = t_start;
                t[1] = wall_clock64();
                t[2] = ((uint64_t)__builtin_amdgcn_s_getreg((31 << 11) | 20) << 32) |
                       (uint32_t)__builtin_amdgcn_s_getreg((31 << 11) | 4);
                t[3] = blockIdx.x;
            }
        }
        // Every wave is done with the staging tile (the next tile's loads
        // overwrite it) before the next position is published; the tile's
        // stores may still be in flight.
        wait_and_barrier<63>();
        if (a.dispenser) {
            if (tid == 0) s_pos = next;
            wait_and_barrier<63>();
            next = s_pos;
        }
        p = __builtin_amdgcn_readfirstlane(next);
        if (a.counters && defer) {
            // Section 3.2 as above: this tile's count is sent once all of its
            // stores are complete -- after the next tile's first main-loop
            // barrier, or now if this was the workgroup's last tile.
            if (p < tiles) {
                pend = group;
            } else {
                __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
                __syncthreads();
                signal(group);
            }
        }
    }
}

template <int DT, int BM, int BN, int WM, int WN, int ST, int BK>
__global__ __launch_bounds__(64 * WM * WN, 1) void gemm_signal_kernel(const GemmArgs a) {
    gemm_body<DT, BM, BN, WM, WN, ST, BK, 32>(a);
}

// 256x256 tiles, 4 waves of 128x128 (16x16x32 MFMAs). At most 216 VGPRs
// (two accumulator block rows among them, the rest of the accumulators in
// AGPRs): the wave leaves 64 of the SIMD's 512 registers per lane to a
// consumer wave, which can therefore run beside it.
template <int DT>
__global__ __launch_bounds__(256, 1) __attribute__((amdgpu_num_vgpr(216))) void gemm_w4_kernel(const GemmArgs a) {
    gemm_body<DT, 256, 256, 2, 2, 2, 64, 16>(a);
}

// 256x128 tiles, 4 waves of 128x64 (16x16x32 MFMAs; 128 accumulator
// registers per lane, no register cap needed).
template <int DT>
__global__ __launch_bounds__(256, 1) void gemm_w4n_kernel(const GemmArgs a) {
    gemm_body<DT, 256, 128, 2, 2, 2, 64, 16>(a);
}

template <int DT, int BM, int BN, int WM, int WN, int ST, int BK>
hipError_t launch_t(const GemmArgs& a, int grid, hipStream_t s) {
    hipLaunchKernelGGL((gemm_signal_kernel<DT, BM, BN, WM, WN, ST, BK>), dim3(grid), dim3(64 * WM * WN), 0, s, a);
    return hipGetLastError();
}

template <int DT>
hipError_t launch_w4(const GemmArgs& a, int grid, hipStream_t s) {
    hipLaunchKernelGGL((gemm_w4_kernel<DT>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(int dtype, int tile_m, int tile_n, const GemmArgs& a, int grid, hipStream_t s) {
    if (tile_m == 256 && tile_n == 128) {
        if (dtype == FO_FP16) hipLaunchKernelGGL(gemm_w4n_kernel<FO_FP16>, dim3(grid), dim3(256), 0, s, a);
        else hipLaunchKernelGGL(gemm_w4n_kernel<FO_BF16>, dim3(grid), dim3(256), 0, s, a);
        return hipGetLastError();
    }
    if (tile_m == 256 && tile_n == 256)
        return dtype == FO_FP16 ? launch_w4<FO_FP16>(a, grid, s) : launch_w4<FO_BF16>(a, grid, s);
    if (tile_m == 64 && tile_n == 64)
        return dtype == FO_FP16 ? launch_t<FO_FP16, 64, 64, 2, 2, 3, 64>(a, grid, s)
                                : launch_t<FO_BF16, 64, 64, 2, 2, 3, 64>(a, grid, s);
    return hipErrorInvalidValue;
}

bool gemm_tile_supported(int tile_m, int tile_n) {
    return (tile_m == 256 && tile_n == 128) || (tile_m == 256 && tile_n == 256) ||
           (tile_m == 64 && tile_n == 64);
}

}  // namespace fo
