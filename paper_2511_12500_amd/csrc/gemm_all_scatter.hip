// One rank's share of GEMM + All-Scatter (Section 4 of the paper), on gfx950.
//
// Problem (Section 4, case study): rank r holds A [M, K] and the column
// shard B_r [K, N] (N = N_local) of a column-parallel GEMM.  It computes
// C_r = A * B_r and makes it the column block [r*N, (r+1)*N) of the
// gathered output [M, w*N] in every rank's heap.
//
// Kernel structure (this file's design, not the paper's Triton code):
//   * persistent grid; producer workgroup g takes tiles g, g+G, g+2G, ...
//     (the persistent tile loop of Sections 4.1.1 and 4.2.1);
//   * tile -> (tile row, tile column): an XCD-aware remap (workgroups are
//     dispatched round-robin over the 8 XCDs, so the tiles in flight on one
//     XCD are made spatial neighbours) followed by a GROUP_M swizzle
//     (Section 3.4, swizzling);
//   * main loop (Section 4, GEMM main-loop listing): 8 waves (two per SIMD;
//     4 for 64x64 tiles), each owning a block of 32x32 MFMA accumulators
//     (v_mfma_f32_32x32x16_{bf16,f16}, fp32 accumulate; 16x16x32 for the
//     256x224 tile); A and B stages of BK = 32 go through a 4-stage LDS ring,
//     loaded 3 stages ahead, with XOR swizzles that keep both the staging
//     writes and the fragment reads free of bank conflicts.  Both tiles go
//     global -> LDS directly
//     (buffer loads into LDS), A as [m][k] rows read with 16-byte LDS reads,
//     B as [k][n] rows, whose MFMA operands (8 consecutive k of one column)
//     come from two transposing LDS reads (ds_read_b64_tr_b16);
//   * epilogue (Section 4.2.1): the accumulators are rounded to the output
//     type (nearest even), restaged through LDS as row-major 16-byte
//     chunks and written with coalesced 128-bit stores to each destination
//     heap (value-based store through the translated address), then the
//     per-tile counters are released at agent scope.
//   * workgroup specialisation (Section 4.2.2): with variant WG_SPEC the
//     first gemm_wgs workgroups produce into the local heap and release a
//     per-tile ready counter; the remaining copy_wgs workgroups acquire it
//     and put the tile into the other w-1 heaps (pointer-based put).
//   * bulk-synchronous (Section 4.1.1): producers store locally, and a
//     second kernel on the same stream puts every tile to the other heaps.
//   * split-K (an addition to the paper's schedules, for shapes with fewer
//     tiles than CUs): with split > 1 a work unit is one K slice of a tile;
//     the slices meet through fp32 partial tiles in a caller workspace, and
//     the last slice to arrive sums them in slice order and runs the
//     epilogue above.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <string>
#include <type_traits>
#include <utility>

#include "symtile.h"
#include "symtile_device.h"
#include "symtile_internal.h"

namespace {

using symtile::u32x4;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));

constexpr int BK = 32;                 // K depth of one pipeline stage
constexpr int kRowBytes = BK * 2;      // LDS bytes per staged A row (4 chunks of 16 B)
constexpr int NS = 4;                  // pipeline stages (LDS ring)
constexpr int PD = 3;                  // prefetch distance in stages (< NS)

enum KernelRole : int { ROLE_LOCAL_ONLY = 0, ROLE_FUSED = 1, ROLE_WG_SPEC = 2, ROLE_WAVE_SPEC = 3,
                        ROLE_REDUCE = 4 };
// (UNFUSED_PC runs gas_kernel as WG_SPEC producers only, and consumer_kernel.
// ROLE_REDUCE runs gas_kernel<..., RED = true>, the second kernel of the
// split-K reduction-kernel mode: no K loop, unit = (tile, band of rows), the
// band's sum of the partials, then the epilogue.)

struct GasParams {
    const uint16_t* A;
    const uint16_t* B;
    uint16_t* C;            // gathered output, column 0, in slot `rank`
    uint32_t* arrived;      // [world][tiles_m][tiles_n] in slot `rank`
    uint32_t* ready;        // [tiles_m * tiles_n], WG_SPEC only
    const uint64_t* bases;
    uint32_t* err;
    int M, N, K;
    int lda, ldb, ldc;
    int rank, world;
    int tiles_m, tiles_n, num_tiles;
    int role;
    int gemm_wgs, copy_wgs;
    int group_m;
    uint32_t epoch, spin_limit;
    int nontemporal;
    uint64_t* trace;        // [num_tiles][8] per-tile timeline, or nullptr
    // Split-K: each tile is `split` work units, unit s covering stages
    // [s*KT/split, (s+1)*KT/split) of the KT stages of K; units = tiles * split.
    int split, units;
    uint32_t* sk_cnt;       // [num_tiles][2]: arrival ticket, partials written
    float* sk_part;         // [num_tiles][split][BM*BN] fp32 partial tiles
    // Banded reduction (every unit has its own co-resident workgroup): slice
    // s sums and stores tile rows [s*BM/split, (s+1)*BM/split); 0 = the last
    // slice to arrive sums and stores the whole tile; 2 = every slice only
    // writes its partial (the first kernel of the reduction-kernel mode).
    int sk_band;
    // ROLE_REDUCE: bands of rows per tile (units = tiles * reduce_bands), and
    // whether the tile goes to every slot (fused) or the local one (bulk).
    int reduce_bands, reduce_all;
};

// Trace record of tile (tm, tn), or nullptr when tracing is off.
__device__ __forceinline__ uint64_t* tile_trace(const GasParams& p, int tm, int tn) {
    return p.trace ? p.trace + ((size_t)tm * p.tiles_n + tn) * SYMTILE_TRACE_WORDS : nullptr;
}

// s_waitcnt immediate that waits until at most n LDS (lgkm) operations of
// this wave are outstanding; vmcnt and expcnt are left at their no-wait
// maxima (gfx9 encoding: vmcnt 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
constexpr int lgkm_wait(int n) { return 15 | (3 << 14) | (7 << 4) | ((n & 15) << 8); }

// Wait until at most N LDS reads of this wave are outstanding, with scheduling
// fences on both sides so no instruction is moved across the wait.
template <int N>
__device__ __forceinline__ void wait_lds() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(lgkm_wait(N));
    __builtin_amdgcn_sched_barrier(0);
}

// s_waitcnt immediate that waits until at most n vector-memory operations
// of this wave are outstanding (lgkmcnt and expcnt not waited).
constexpr int vm_wait(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Workgroup barrier for the LDS hand-off inside the pipelined loop.  The
// caller has already waited for its own LDS reads (lgkmcnt) and its loads
// into LDS (vmcnt); unlike __syncthreads() this adds no wait for the loads
// still in flight for later stages.  The empty asm statements keep the
// compiler from moving memory accesses across the barrier.
__device__ __forceinline__ void ring_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Ask the scheduler to interleave the LDS reads and MFMAs of the current
// scheduling region one by one (R reads, M MFMAs; reads first when
// READS_FIRST), so the reads issue in the shadow of the MFMAs instead of as
// one burst.  The compiler's own waits before each MFMA stay exact (it tracks
// which registers each read fills).
template <int R, int M, bool READS_FIRST>
__device__ __forceinline__ void interleave_reads_mfmas() {
    constexpr int Q = R > M ? R : M;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        if (READS_FIRST && q < R) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
        if (q < M) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);               // MFMA
        if (!READS_FIRST && q < R) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
}

// XOR swizzle of the 16-byte chunk index inside a 64-byte staged A row.  A
// fragment read has 16 consecutive rows per 256-byte bank window: the row's
// bits 0-1 pick the 64-byte quarter, bits 2-3 permute the chunk within it.
__device__ __forceinline__ int swz(int row) { return (row >> 2) & 3; }

// XOR swizzle of the 16-byte chunk index inside a staged B row (k fixed,
// CPR chunks of 8 consecutive n).  A transposing fragment read touches rows
// k..k+3 and k+8..k+11 (k a multiple of 4) and four adjacent chunks; the
// swizzle spreads each half-wave's 16 (row, chunk) pairs over distinct
// 16-byte bank groups.  With 8 chunks per row (128-byte rows) the row parity
// already selects the bank half, so bit 1 of k takes the place of bit 0.
template <int CPR>
__device__ __forceinline__ int swz_b(int k) {
    const int lo = (CPR >= 16) ? ((k & 3) << 2) : (((k >> 1) & 1) << 2);
    return lo ^ (((k >> 3) & 1) << 1);
}

// Producer-order work unit u -> (tile row, tile column, K slice).  The XCD
// remap makes consecutive units land on one XCD, and the slices of a tile are
// consecutive units, so with split-K they share that XCD's L2 (and the
// partial tiles they exchange stay there).  Without split-K a unit is a tile.
__device__ __forceinline__ void unit_coords(int u, int G, const GasParams& p, int& tm, int& tn,
                                            int& s) {
    int L = u;
    const int round = u / G;
    if ((G & 7) == 0 && (round + 1) * G <= p.units) {
        const int pos = u - round * G;
        L = round * G + (pos & 7) * (G >> 3) + (pos >> 3);
    }
    if (p.split > 1) {
        s = L % p.split;
        L /= p.split;
    } else {
        s = 0;
    }
    const int width = p.group_m * p.tiles_n;
    const int group = L / width;
    const int first_m = group * p.group_m;
    const int gsize = min(p.tiles_m - first_m, p.group_m);
    const int in = L - group * width;
    tm = first_m + in % gsize;
    tn = in / gsize;
}

// Producer-order tile index t -> (tile row, tile column), for schedules
// without split-K (units == tiles).
__device__ __forceinline__ void tile_coords(int t, int G, const GasParams& p, int& tm, int& tn) {
    int s;
    unit_coords(t, G, p, tm, tn, s);
}

template <bool BF16>
__device__ __forceinline__ f32x16_t mfma32(u32x4 a, u32x4 b, f32x16_t c) {
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                       __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a),
                                                      __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

// The 32x32x16 MFMA as an ordered statement: accumulating in place in
// AGPRs, and a memory clobber, so the compiler keeps every memory access on
// the side of it where the source puts it (the 4-wave loop lays out its own
// interleaving of MFMAs, LDS accesses and loads this way).  The compiler
// does not see the MFMA: its hazard wait states before the first use and
// after the last are the caller's.
template <bool BF16>
__device__ __forceinline__ void mfma32_ordered(f32x16_t& acc, const u32x4& a, const u32x4& b) {
    if constexpr (BF16)
        asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b) : "memory");
    else
        asm volatile("v_mfma_f32_32x32x16_f16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b) : "memory");
}

template <bool BF16>
__device__ __forceinline__ f32x4_t mfma16(u32x4 a, u32x4 b, f32x4_t c) {
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                       __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a),
                                                      __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

// Round two fp32 values to the 16-bit output type (nearest even) and pack.
template <bool BF16>
__device__ __forceinline__ uint32_t cvt_pack(float x, float y) {
    uint16_t a, b;
    if constexpr (BF16) {
        a = __builtin_bit_cast(uint16_t, (__bf16)x);
        b = __builtin_bit_cast(uint16_t, (__bf16)y);
    } else {
        a = __builtin_bit_cast(uint16_t, (_Float16)x);
        b = __builtin_bit_cast(uint16_t, (_Float16)y);
    }
    return (uint32_t)a | ((uint32_t)b << 16);
}

// ---------------------------------------------------------------------------
// Tile widths are staged and moved as BN rounded up to a power of two (64,
// 128 or 256 columns); chunks past the tile's columns are masked.
constexpr int staged_width(int bn) { return bn <= 64 ? 64 : bn <= 128 ? 128 : 256; }

// Geometry of one output tile for 16-byte row chunks: CPR chunks per staged
// tile row, RP tile rows per pass of the THREADS threads.  Thread t always
// handles chunk column t % CPR, rows t / CPR + RP * i.
template <int BM, int BN, int THREADS>
struct TileIO {
    static constexpr int CPR = staged_width(BN) / 8;
    static constexpr int RP = THREADS / CPR;
    static constexpr int PASSES = BM / RP;
    static constexpr int U = PASSES < 8 ? PASSES : 8;
    static_assert(THREADS % CPR == 0 && BM % RP == 0 && PASSES % U == 0, "tile split");
};

// Bytes of the destination resource of one tile (rows_valid x cols_valid,
// row stride ldc elements); rows beyond rows_valid fall outside it.
__device__ __forceinline__ uint32_t tile_span(int rows_valid, int cols_valid, int ldc) {
    return (uint32_t)(((size_t)(rows_valid - 1) * ldc + cols_valid) * 2);
}

// Store policy of the output (GasParams::nontemporal): 0 default, 1
// non-temporal (streaming), 2 write-through (the L2 keeps no dirty line, so
// the release fence that follows finds nothing of these stores to write
// back).  Calls f with the cache-policy bits as a compile-time constant.
template <typename F>
__device__ __forceinline__ void with_store_policy(int mode, F&& f) {
    if (mode == 1)
        f(std::integral_constant<int, symtile::kStoreNonTemporal>{});
    else if (mode == 2)
        f(std::integral_constant<int, symtile::kStoreWriteThrough>{});
    else
        f(std::integral_constant<int, symtile::kStoreDefault>{});
}

// Release of this workgroup's output stores before their counters move
// (agent scope): stores written through need only their acknowledgement,
// the other policies the L2 write-back of a release fence.
template <int POLICY>
__device__ __forceinline__ void release_output() {
    if constexpr (POLICY == symtile::kStoreWriteThrough)
        symtile::release_written_through();
    else
        symtile::fence_release<__HIP_MEMORY_SCOPE_AGENT>();
}

__device__ __forceinline__ void release_output(int mode) {
    if (mode == 2)
        symtile::release_written_through();
    else
        symtile::fence_release<__HIP_MEMORY_SCOPE_AGENT>();
}

// Geometry of output tile (tm, tn) for the tile verbs: 16-bit elements, so
// 8 per 16-byte chunk; THREADS threads cover CPR chunk columns per pass.
template <int BM, int BN, int THREADS>
__device__ __forceinline__ symtile::TileGeom out_tile(const GasParams& p, int tm, int tn) {
    using IO = TileIO<BM, BN, THREADS>;
    symtile::TileGeom g;
    g.rows = min(BM, p.M - tm * BM);
    g.chunks = min(BN, p.N - tn * BN) / 8;
    g.ld_bytes = (uint32_t)p.ldc * 2;
    g.lg_w = __builtin_ctz(IO::CPR);
    return g;
}

// Address of tile (tm, tn) of this rank's column block in the local heap.
__device__ __forceinline__ uint16_t* out_tile_ptr(const GasParams& p, int BM, int BN, int tm, int tn) {
    return p.C + (size_t)p.rank * p.N + (size_t)tm * BM * p.ldc + (size_t)tn * BN;
}

// Copy one finished tile from the local heap to every other heap (the put of
// Sections 4.1.1 and 4.2.2) and release its counters there.  LOAD is the
// policy of the tile's loads (coherent after a flag_wait_coherent).
template <int BM, int BN, int THREADS, int POLICY, int LOAD = symtile::kLoadDefault>
__device__ void put_tile_to_peers(const GasParams& p, int tm, int tn) {
    using IO = TileIO<BM, BN, THREADS>;
    const int tid = threadIdx.x;
    symtile::put_ranks<POLICY, IO::U, LOAD>(out_tile_ptr(p, BM, BN, tm, tn),
                                            out_tile<BM, BN, THREADS>(p, tm, tn), p.rank, 1,
                                            p.world, p.world, p.bases, tid, THREADS);
    symtile::wg_stores_done();
    if (tid < 64) {            // wave 0: one release, then lane d counts slot rank + d
        release_output<POLICY>();
        uint32_t* flag = p.arrived + ((size_t)p.rank * p.tiles_m + tm) * p.tiles_n + tn;
        const int d = tid + 1;
        if (d < p.world)
            symtile::flag_signal(symtile::translate(flag, p.rank, (p.rank + d) % p.world, p.bases));
    }
}

// Consumer loop of the producer-consumer schedules (Sections 4.1.2 and
// 4.2.2): consumer `cid` of `ncons` takes tiles cid, cid + ncons, ... in the
// producers' tile order, waits (bounded) until the producer's ready counter
// reaches the epoch, acquires, and puts the tile to the other heaps.  A
// timed-out wait records ERR_TIMEOUT and ends this consumer.  With the
// write-through output policy the producers' tiles are read back with
// coherent loads, so the acquire needs no L2 invalidate.
template <int BM, int BN, int THREADS>
__device__ void consume_tiles(const GasParams& p, int cid, int ncons) {
    __shared__ int s_ok;
    const int tid = threadIdx.x;
    for (int t = cid; t < p.num_tiles; t += ncons) {
        int tm, tn;
        tile_coords(t, p.gemm_wgs, p, tm, tn);
        uint64_t* tr = tile_trace(p, tm, tn);
        if (tid == 0) {
            if (tr) tr[SYMTILE_TRACE_COPY_WAIT] = symtile::clock_now();
            const uint32_t* rdy = p.ready + tm * p.tiles_n + tn;
            const bool ok = p.nontemporal == 2
                                ? symtile::flag_wait_coherent(rdy, p.epoch, p.spin_limit)
                                : symtile::flag_wait(rdy, p.epoch, p.spin_limit);
            if (!ok) symtile::raise_error(p.err, symtile::ERR_TIMEOUT);
            if (tr) tr[SYMTILE_TRACE_COPY_GO] = symtile::clock_now();
            s_ok = ok;
        }
        __syncthreads();
        if (!s_ok) return;
        with_store_policy(p.nontemporal, [&](auto pol) {
            constexpr int P = decltype(pol)::value;
            put_tile_to_peers<BM, BN, THREADS, P,
                              P == symtile::kStoreWriteThrough ? symtile::kLoadCoherent
                                                               : symtile::kLoadDefault>(p, tm, tn);
        });
        if (tr && tid == 0) tr[SYMTILE_TRACE_COPY_DONE] = symtile::clock_now();
    }
}

// Copy wave of the wave-specialised schedule (Section 4.2.3).  The compute
// waves of the workgroup store each tile into the local slot only (except
// the workgroup's last tile, which they store everywhere); this extra wave
// copies the previous tile from the local slot to the w-1 other slots while
// the compute waves run the next tile's K loop, then releases its counters
// there.  s_barrier counts every wave of the workgroup, so the copy wave
// takes part in exactly the compute waves' barriers: KT ring barriers and 3
// epilogue barriers per tile, and copies a slice of the tile between them.
// A slice must not hold the wave at a barrier waiting for memory (that would
// stretch the compute waves' stage): row groups are loaded two intervals
// before they are stored, into two register sets used alternately, and the
// counters are published two intervals after the last store, when the
// stores have been acknowledged.  Loads and stores share one in-order
// counter, so each interval issues its load before its stores.  With fewer
// barriers than that needs (small K) the wave stores each group as soon as
// it is loaded.
template <int BM, int BN, int POLICY>
__device__ void copy_wave_tiles(const GasParams& p, int KT) {
    constexpr int CPR = staged_width(BN) / 8;   // 16-byte chunks per tile row
    constexpr int RPI = 64 / CPR;               // tile rows per wave-wide access
    constexpr int GROUPS = BM / RPI;
    constexpr int MAXW = SYMTILE_MAX_WORLD;
    static_assert(64 % CPR == 0 && BM % RPI == 0 && GROUPS % 2 == 0, "copy wave split");
    const int lane = threadIdx.x & 63;
    const int G = p.gemm_wgs;
    const int intervals = KT + 3;
    const bool piped = intervals >= GROUPS + 4;
    const uint32_t group_bytes = (uint32_t)RPI * p.ldc * 2;
    int ptm = -1, ptn = -1;                     // tile waiting to be copied
    for (int t = blockIdx.x; t < p.num_tiles; t += G) {
        if (ptm >= 0) {
            // the compute waves' local stores of this tile were released at
            // workgroup scope before the barrier that ended it
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
            if (p.trace && lane == 0) {
                uint64_t* tr = tile_trace(p, ptm, ptn);
                tr[SYMTILE_TRACE_COPY_WAIT] = tr[SYMTILE_TRACE_COPY_GO] = symtile::clock_now();
            }
        }
        const int m0 = max(ptm, 0) * BM, n0 = max(ptn, 0) * BN;
        const int rows = min(BM, p.M - m0), cols = min(BN, p.N - n0);
        const uint16_t* src = p.C + (size_t)p.rank * p.N + (size_t)m0 * p.ldc + n0;
        const uint32_t span = ptm >= 0 ? tile_span(rows, cols, p.ldc) : 0u;
        const symtile::rsrc_t rs = symtile::make_rsrc(src, span);
        symtile::rsrc_t rd[MAXW - 1];
#pragma unroll
        for (int d = 1; d < MAXW; ++d)
            rd[d - 1] = symtile::make_rsrc(
                symtile::translate(src, p.rank, (p.rank + d) % p.world, p.bases),
                d < p.world ? span : 0u);
        const int c = lane % CPR;
        const uint32_t voff =
            (8 * c < cols) ? (uint32_t)((lane / CPR) * p.ldc * 2 + c * 16) : symtile::kOOB;
        auto store_group = [&](const symtile::u32x4& v, int g) {
#pragma unroll
            for (int d = 0; d < MAXW - 1; ++d)       // dropped past the world (empty resource)
                symtile::buf_st16p<POLICY>(v, rd[d], voff, (uint32_t)g * group_bytes);
        };
        auto publish = [&]() {
            __builtin_amdgcn_s_waitcnt(vm_wait(0));
            release_output<POLICY>();                 // one release; lane d counts slot rank + d
            uint32_t* flag = p.arrived + ((size_t)p.rank * p.tiles_m + ptm) * p.tiles_n + ptn;
            if (lane >= 1 && lane < p.world)
                symtile::flag_signal(symtile::translate(flag, p.rank, (p.rank + lane) % p.world,
                                                        p.bases));
            if (lane == 0 && p.trace)
                tile_trace(p, ptm, ptn)[SYMTILE_TRACE_COPY_DONE] = symtile::clock_now();
        };
        if (ptm >= 0 && piped) {
            // interval b loads group b (b < GROUPS) and stores group b-2
            symtile::u32x4 x = symtile::buf_ld16(rs, voff, 0u);
            ring_barrier();
            symtile::u32x4 y = symtile::buf_ld16(rs, voff, group_bytes);
            ring_barrier();
            for (int b = 2; b < GROUPS + 2; b += 2) {
                const symtile::u32x4 x2 = b < GROUPS ? symtile::buf_ld16(rs, voff, b * group_bytes) : x;
                store_group(x, b - 2);
                x = x2;
                ring_barrier();
                const symtile::u32x4 y2 =
                    b + 1 < GROUPS ? symtile::buf_ld16(rs, voff, (b + 1) * group_bytes) : y;
                store_group(y, b - 1);
                y = y2;
                ring_barrier();
            }
            ring_barrier();                          // interval GROUPS + 2
            publish();
            ring_barrier();                          // interval GROUPS + 3
            for (int b = GROUPS + 4; b < intervals; ++b) ring_barrier();
        } else {
            bool published = ptm < 0;
            int g = 0;
            const int per = (GROUPS + intervals - 1) / intervals;
            for (int b = 0; b < intervals; ++b) {
                if (!published) {
                    for (int q = 0; q < per && g < GROUPS; ++q, ++g)
                        store_group(symtile::buf_ld16(rs, voff, (uint32_t)g * group_bytes), g);
                    if (g == GROUPS) {
                        publish();
                        published = true;
                    }
                }
                ring_barrier();                      // the compute waves' barrier b
            }
        }
        int tm, tn;
        tile_coords(t, G, p, tm, tn);
        if (t + G < p.num_tiles) {
            ptm = tm;
            ptn = tn;
        } else {
            ptm = -1;                                // the compute waves store the last tile everywhere
        }
    }
}

// ---------------------------------------------------------------------------
// Producer tile shapes.  MF = 32: v_mfma_f32_32x32x16, waves in a 2 x (NW/2)
// grid, each stage read as two k16 substeps.  MF = 16: v_mfma_f32_16x16x32
// (same rate per flop), waves in a 4 x (NW/4) grid, one k32 substep per
// stage; it allows tile widths that are a multiple of 16 but not of 64 (a
// 256 x 224 tile covers N = 3584 in 16 columns).  B is staged BNS = BN
// rounded up to a power of two wide, so direct-to-LDS loads stay whole rows;
// staged columns past BN are loaded but never read.  With NW = 8 two waves
// share each SIMD, so one wave's MFMAs run while the other waits on LDS,
// global loads or the barrier.
template <int BM, int BN, bool BF16, int NW, int MF, bool CW = false, bool RED = false>
__global__ __launch_bounds__(64 * (NW + CW))
__attribute__((amdgpu_waves_per_eu(NW / 4 + CW, NW / 4 + CW)))
void gas_kernel(const GasParams p) {
    constexpr int THREADS = 64 * NW;
    constexpr int WGM = (MF == 32) ? 2 : 4, WGN = NW / WGM;   // wave grid
    constexpr int WM = BM / WGM, WN = BN / WGN;               // wave tile
    constexpr int MI = WM / MF, NI = WN / MF;                 // MFMA blocks per wave
    constexpr int BNS = staged_width(BN);
    constexpr int A_BYTES = BM * kRowBytes, B_BYTES = BK * BNS * 2;
    constexpr int STAGE = A_BYTES + B_BYTES;
    constexpr int CROW = BNS * 2;                             // bytes per staged C row
    constexpr int C_BYTES = BM * CROW;
    constexpr int LDS_BYTES = (NS * STAGE > C_BYTES) ? NS * STAGE : C_BYTES;
    constexpr int A_RPI = 1024 / kRowBytes;     // A rows per 1 KiB direct-to-LDS load
    constexpr int A_INSTR = BM / A_RPI / NW;    // direct-to-LDS A loads per wave per stage
    constexpr int ROWB = BNS * 2;               // bytes per staged B row (one k)
    constexpr int CPR = BNS / 8;                // 16-byte chunks per staged B row
    constexpr int RPI = 1024 / ROWB;            // B rows per 1 KiB direct-to-LDS load
    constexpr int B_INSTR = BK / RPI / NW;      // direct-to-LDS B loads per wave per stage
    static_assert(NW == 4 || NW == 8, "4 or 8 waves");
    static_assert(MF == 32 || MF == 16, "MFMA shape");
    static_assert(MI >= 1 && NI >= 1 && WM % MF == 0 && WN % MF == 0, "unsupported tile");
    static_assert(A_INSTR >= 1 && (BM / A_RPI) % NW == 0, "A staging split");
    static_assert(RPI >= 1 && B_INSTR >= 1 && (BK / RPI) % NW == 0, "B staging split");
    using IO = TileIO<BM, BN, THREADS>;
    using acc_t = std::conditional_t<MF == 32, f32x16_t, f32x4_t>;
    constexpr int ACC_N = (MF == 32) ? 16 : 4;
    // 256 x 256 tiles with 4 waves: one wave per SIMD holds a 128 x 128 block
    // and the K loop stages 64 k at a time through registers (see below).
    constexpr bool V4 = BM == 256 && BN == 256 && NW == 4 && MF == 32 && !CW && !RED;

    __shared__ __attribute__((aligned(16))) uint8_t smem[LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    const int pid = blockIdx.x;

    // ---------------- consumer workgroups (Section 4.2.2) -----------------
    if (p.role == ROLE_WG_SPEC && pid >= p.gemm_wgs) {
        consume_tiles<BM, BN, THREADS>(p, pid - p.gemm_wgs, p.copy_wgs);
        return;
    }

    // ---------------- producer workgroups ---------------------------------
    const int G = p.gemm_wgs;
    const int KT_all = (p.K + BK - 1) / BK;    // stages of the whole K
    if constexpr (CW) {
        // the copy wave (Section 4.2.3); the test is made visibly uniform so
        // that the compiler keeps the copy wave's addressing scalar
        if (__builtin_amdgcn_readfirstlane(wave) == NW) {
            with_store_policy(p.nontemporal, [&](auto pol) {
                copy_wave_tiles<BM, BN, decltype(pol)::value>(p, KT_all);
            });
            return;
        }
    }

    // A: wave w, load u fills staged rows A_RPI*(NW*u + w) .. +A_RPI-1; lane
    // l lands at chunk l % 4 of row A_RPI*(NW*u + w) + l / 4 and fetches the
    // global chunk the swizzle maps there (the swizzle reads row bits 2-3,
    // which only depend on the lane).
    const int a_rr = lane >> 2;
    const int a_chunk = (lane & 3) ^ swz(a_rr);
    const uint32_t a_row_off = (uint32_t)((A_RPI * wave + a_rr) * p.lda * 2);
    const uint32_t a_u_bytes = (uint32_t)(A_RPI * NW * p.lda * 2);
    // B: wave w, load u fills staged rows RPI*(NW*u + w) .. +RPI-1; lane l
    // lands at chunk l % CPR of row RPI*(NW*u + w) + l / CPR and fetches the
    // global chunk the swizzle maps there.  The swizzle reads bits 0, 1 and 3
    // of the row, so it depends on u only through its parity.
    const int b_rr = lane / CPR, b_pc = lane % CPR;
    const int b_k_even = wave * RPI + b_rr, b_k_odd = (NW + wave) * RPI + b_rr;
    const uint32_t b_row_off = (uint32_t)((wave * RPI + b_rr) * p.ldb * 2);
    const uint32_t b_v_even = b_row_off + (uint32_t)((b_pc ^ swz_b<CPR>(b_k_even)) * 16);
    const uint32_t b_v_odd = b_row_off + (uint32_t)((b_pc ^ swz_b<CPR>(b_k_odd)) * 16);
    const uint32_t b_u_bytes = (uint32_t)(NW * RPI * p.ldb * 2);
    const uint32_t b_row_bytes = (uint32_t)(p.ldb * 2);
    // Fragment reads.  A operand (second MFMA source): lane l holds 8
    // consecutive k of row (l % MF).  B operand (first source) from two
    // transposing reads: in each 16-lane group, lane s addresses row
    // kq + s / 4 and columns 4 * (s % 4) .. +3 of a 16-column block, and
    // receives 4 consecutive k of column (s of that block).
    const int a_row_lane = lane % MF;
    const int tr_row = ((MF == 32) ? 8 * (lane >> 5) : 8 * (lane >> 4)) + ((lane & 15) >> 2);
    const int tr_col = ((MF == 32) ? 16 * ((lane >> 4) & 1) : 0) + 4 * (lane & 3);

    // (the reduction kernel is an instantiation of its own, so its code
    // leaves the register allocation of the K-loop kernels alone)
    constexpr bool reducer = RED;
    for (int t = pid; t < p.units; t += G) {
        int tm, tn, ks;
        if (reducer) {
            // unit = (tile, band); ks is the band (no K slice: KT = 0 below)
            const int tile = t / p.reduce_bands;
            ks = t - tile * p.reduce_bands;
            tm = tile / p.tiles_n;
            tn = tile - tm * p.tiles_n;
        } else {
            unit_coords(t, G, p, tm, tn, ks);
        }
        // this unit's K slice: stages [kt0, kt0 + KT)
        const int kt0 = reducer ? 0 : ks * KT_all / p.split;
        const int KT = reducer ? 0 : (ks + 1) * KT_all / p.split - kt0;
        // (the trace record's address is recomputed at each event so that
        // nothing extra stays live across the K loop)
        if (p.trace && tid == 0 && ks == 0 && !reducer) {
            uint64_t* tr = tile_trace(p, tm, tn);
            tr[SYMTILE_TRACE_START] = symtile::clock_now();
            tr[SYMTILE_TRACE_WHERE] = symtile::trace_location();
        }
        const int m0 = tm * BM, n0 = tn * BN;
        const int rows_a = min(BM, p.M - m0);
        // The resources start at the slice's first k, so the loop indexes
        // stages from 0 and sees kend = the K left from there.
        const int kbeg = kt0 * BK, kend = p.K - kbeg;
        const symtile::i32x4_t rA = symtile::make_rsrc_words(
            p.A + (size_t)m0 * p.lda + kbeg, (uint32_t)(rows_a * p.lda * 2 - kbeg * 2));
        // B's resource ends at the shard's last element (row K-1, column
        // N-1), so with ldb > N the staged columns past N of the last row
        // read zero instead of touching memory past a tightly sized B.
        const symtile::i32x4_t rB = symtile::make_rsrc_words(
            p.B + (size_t)kbeg * p.ldb + n0,
            kend > 0 ? (uint32_t)(((size_t)(kend - 1) * p.ldb + p.N - n0) * 2) : 0u);

        acc_t acc[MI][NI];
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NI; ++j)
#pragma unroll
                for (int e = 0; e < ACC_N; ++e) acc[i][j][e] = 0.0f;

        // A and B straight into LDS stage `buf` (k relative to the slice).
        // A chunks at k >= K read zero: bit 31 (kOOB) is set in their offset,
        // taken from the sign of K - 1 - k (arithmetic rather than a select,
        // which would keep the constant in a vector register), so it lies
        // past the resource; B rows at k >= K lie past the end of B's
        // resource and read zero too.
        auto load_tile = [&](int kt, int buf) {
            const int k0 = kt * BK;
            uint8_t* As = smem + buf * STAGE;
            const uint32_t va = (a_row_off + a_chunk * 16) |
                                ((uint32_t)(kend - 1 - k0 - 8 * a_chunk) & symtile::kOOB);
#pragma unroll
            for (int u = 0; u < A_INSTR; ++u)
                symtile::buf_ld16_lds_async(rA, symtile::lds_addr(As + (NW * u + wave) * 1024),
                                            va, u * a_u_bytes + k0 * 2);
            uint8_t* Bs = As + A_BYTES;
            const uint32_t kb = (uint32_t)k0 * b_row_bytes;
#pragma unroll
            for (int u = 0; u < B_INSTR; ++u)
                symtile::buf_ld16_lds_async(rB, symtile::lds_addr(Bs + (NW * u + wave) * 1024),
                                            (u & 1) ? b_v_odd : b_v_even, u * b_u_bytes + kb);
        };

        // Fragment of A block i (rows wm*WM + i*MF ..) at 16-byte chunk c,
        // and of B block j (columns wn*WN + j*MF ..) at k offset kbase.
        auto read_a = [&](int buf, int i, int c) {
            const uint8_t* As = smem + buf * STAGE;
            const int row = wm * WM + i * MF + a_row_lane;
            return *reinterpret_cast<const symtile::u32x4*>(As + row * kRowBytes +
                                                           ((c ^ swz(row)) << 4));
        };
        auto read_b = [&](int buf, int j, int kbase) {
            const uint8_t* Bs = smem + buf * STAGE + A_BYTES;
            const int col = wn * WN + j * MF + tr_col;
            u32x2_t h[2];
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int k = kbase + tr_row + 4 * half;
                const uint8_t* q = Bs + k * ROWB + (((col >> 3) ^ swz_b<CPR>(k)) << 4) +
                                   ((col & 4) << 1);
                h[half] = __builtin_bit_cast(
                    u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                 (__attribute__((address_space(3))) s16x4_t*)(q)));
            }
            return symtile::u32x4{h[0][0], h[0][1], h[1][0], h[1][1]};
        };
        // Operands are swapped (B fragment as the first source) so each
        // lane's accumulators hold 4 consecutive columns of one row of C,
        // which makes the epilogue restage cheap.
        auto mma = [&](int i, int j, const symtile::u32x4& a, const symtile::u32x4& b) {
            if constexpr (MF == 32)
                acc[i][j] = mfma32<BF16>(b, a, acc[i][j]);
            else
                acc[i][j] = mfma16<BF16>(b, a, acc[i][j]);
        };

        if constexpr (V4) {
            // Four waves, one per SIMD, each a 128 x 128 block of 4 x 4 MFMA
            // blocks.  A stage is 64 k: A as 256 rows of 128 bytes (whole cache
            // lines, half the L2 requests of the ring loop's 64-byte rows), B
            // as 64 rows of 512 bytes, both loaded into registers (no
            // direct-to-LDS loads) and written to one of two LDS buffers by
            // the waves during the stage before their reads, a whole stage
            // after the load.  Within a stage the four k16 substeps are
            // rotated like the ring loop: a substep's MFMAs use the fragments
            // read in the substep before, and the last substep's MFMAs run
            // after the next barrier.  With one wave per SIMD nothing else
            // issues while the wave waits, so the MFMAs are ordered
            // statements, one per slot, with the substep's fragment reads, LDS
            // writes and loads placed in the slots between them.  Loads past
            // the slice read zero (A through the offset bit, B past its
            // resource), so every stage runs the same code.
            constexpr int BK2 = 2 * BK;
            constexpr int A2_BYTES = BM * BK2 * 2, B2_BYTES = BK2 * ROWB;
            constexpr int BUF2 = A2_BYTES + B2_BYTES;
            constexpr int LU = 8;                      // A (and B) loads per wave per stage
            static_assert(2 * BUF2 <= LDS_BYTES && BM * BK2 * 2 == LU * NW * 1024 &&
                          B2_BYTES == LU * NW * 1024 && MI == 4 && NI == 4 && ROWB == 512,
                          "4-wave 256 x 256 staging");
            const int S2 = (KT + 1) / 2;               // 64-k stages of the slice
            const int kend2 = min(KT * BK, kend);      // k of the slice
            const symtile::rsrc_t rA2 = symtile::make_rsrc(
                p.A + (size_t)m0 * p.lda + kbeg, (uint32_t)(rows_a * p.lda * 2 - kbeg * 2));
            const symtile::rsrc_t rB2 = symtile::make_rsrc(
                p.B + (size_t)kbeg * p.ldb + n0,
                kend2 > 0 ? (uint32_t)(((size_t)(kend2 - 1) * p.ldb + p.N - n0) * 2) : 0u);
            // A: load u of wave w brings rows 32u + 8w + l/8, lane l chunk l%8;
            // in LDS a row's chunk c sits at (c ^ ((row >> 1) & 7)), which for
            // these rows is (4w + l/16) & 7 whatever u is.
            const int a2g = lane & 7;
            const uint32_t a2v = (uint32_t)((8 * wave + (lane >> 3)) * p.lda * 2 + a2g * 16);
            const uint32_t a2u = (uint32_t)(32 * p.lda * 2);
            // B: load u of wave w brings k-rows 8u + 2w + l/32, lane l chunk
            // l%32, swizzled in LDS by bits 0, 1 and 3 of the row (bit 3 is
            // u's parity).
            const uint32_t b2v = (uint32_t)((2 * wave + (lane >> 5)) * p.ldb * 2 + (lane & 31) * 16);
            const uint32_t b2u = (uint32_t)(8 * p.ldb * 2);
            const uint32_t kb2 = (uint32_t)(BK2 * p.ldb * 2);

            symtile::u32x4 P[2 * LU];                  // x < LU: A, else B
            auto load_part = [&](int st, int u0, int u1) {
                const int k0 = st * BK2;
                const uint32_t va = a2v | ((uint32_t)(kend2 - 1 - k0 - 8 * a2g) & symtile::kOOB);
#pragma unroll
                for (int x = u0; x < u1; ++x) {
                    if (x < LU)
                        P[x] = symtile::buf_ld16p<symtile::kLoadDefault>(rA2, va, x * a2u + k0 * 2);
                    else
                        P[x] = symtile::buf_ld16p<symtile::kLoadDefault>(
                            rB2, b2v, (x - LU) * b2u + (uint32_t)st * kb2);
                }
            };
            // (The LDS addresses below are recomputed from `ln` in every stage:
            // kept live across the loop they would not fit in registers.)
            auto write_part = [&](int ln, int buf, int u0, int u1) {
                uint8_t* As = smem + buf * BUF2;
                uint8_t* Bs = As + A2_BYTES;
                const uint32_t aw = (uint32_t)((8 * wave + (ln >> 3)) * (BK2 * 2) +
                                               (((ln & 7) ^ ((4 * wave + (ln >> 4)) & 7)) << 4));
                const int bk = 2 * wave + (ln >> 5), bc = ln & 31;
#pragma unroll
                for (int x = u0; x < u1; ++x) {
                    if (x < LU) {
                        *reinterpret_cast<symtile::u32x4*>(As + aw + x * 4096) = P[x];
                    } else {
                        const int u = x - LU;
                        const uint32_t bw = (uint32_t)(bk * ROWB +
                                                       ((bc ^ swz_b<CPR>(bk + 8 * (u & 1))) << 4));
                        *reinterpret_cast<symtile::u32x4*>(Bs + bw + u * 4096) = P[x];
                    }
                }
            };
            symtile::u32x4 fa0[MI], fb0[NI], fa1[MI], fb1[NI];
#pragma unroll
            for (int i = 0; i < MI; ++i) fa1[i] = symtile::u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int j = 0; j < NI; ++j) fb1[j] = symtile::u32x4{0u, 0u, 0u, 0u};
            // (wait states between the VALU writes above and the first MFMA)
            asm volatile("s_nop 7\n\ts_nop 7" ::: "memory");
            // One substep: its 16 MFMAs on the fragments read in the substep
            // before (fa, fb), one per slot; the slots also carry this
            // substep's 12 fragment reads (slots 0-5, into na, nb), a quarter
            // of P to LDS and its reloads (alternating, slots 6-13), so that
            // the wave issues something between any two MFMAs.
            auto substep = [&](int ln, int buf, int t, int st,
                               const symtile::u32x4 (&fa)[MI], const symtile::u32x4 (&fb)[NI],
                               symtile::u32x4 (&na)[MI], symtile::u32x4 (&nb)[NI]) {
                const uint8_t* As = smem + buf * BUF2;
                const uint8_t* Bs = As + A2_BYTES;
                const int c = 2 * t + (ln >> 5);
                const int trr = 8 * (ln >> 5) + ((ln & 15) >> 2);
                const int trc = 16 * ((ln >> 4) & 1) + 4 * (ln & 3);
                u32x2_t h[NI][2];
#pragma unroll
                for (int q = 0; q < MI * NI; ++q) {
                    mfma32_ordered<BF16>(acc[q / NI][q % NI], fb[q % NI], fa[q / NI]);
                    // slots 0-5: two fragment reads each; slots 6, 8, 10, 12:
                    // the LDS writes, each followed in the next slot by the
                    // reload of the same registers
                    const int r0 = q < 6 ? 2 * q : 12, r1 = q < 6 ? 2 * q + 2 : 12;
                    if (q >= 6 && q < 14 && !(q & 1))
                        write_part(ln, buf ^ 1, 4 * t + (q - 6) / 2, 4 * t + (q - 6) / 2 + 1);
                    if (q >= 7 && q < 14 && (q & 1))
                        load_part(st + 2, 4 * t + (q - 7) / 2, 4 * t + (q - 7) / 2 + 1);
                    if (r0 < r1) {
                        // reads r0 .. r1-1 of a0..a3, b0 (two halves), .. b3
#pragma unroll
                        for (int r = r0; r < r1; ++r) {
                            if (r < MI) {
                                const int row = wm * WM + r * MF + (ln & 31);
                                na[r] = *reinterpret_cast<const symtile::u32x4*>(
                                    As + row * (BK2 * 2) + ((c ^ ((row >> 1) & 7)) << 4));
                            } else {
                                const int j = (r - MI) / 2, half = (r - MI) % 2;
                                const int col = wn * WN + j * MF + trc;
                                const int k = 16 * t + trr + 4 * half;
                                const uint8_t* qa = Bs + k * ROWB +
                                                    (((col >> 3) ^ swz_b<CPR>(k)) << 4) +
                                                    ((col & 4) << 1);
                                h[j][half] = __builtin_bit_cast(
                                    u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                                 (__attribute__((address_space(3))) s16x4_t*)(qa)));
                            }
                        }
                    }
                }
#pragma unroll
                for (int j = 0; j < NI; ++j)
                    nb[j] = symtile::u32x4{h[j][0][0], h[j][0][1], h[j][1][0], h[j][1][1]};
            };
            // One stage: its fragments from buffer `buf`.  P holds stage st + 1
            // (loaded during the stage before); in each substep a quarter of
            // its registers goes to the other buffer (free since the barrier)
            // and is reloaded at once with stage st + 2, so loads lead their
            // LDS writes by a whole stage.
            auto stage = [&](int st, int buf) {
                int ln = lane;
                asm volatile("" : "+v"(ln));
                wait_lds<0>();
                ring_barrier();
                substep(ln, buf, 0, st, fa1, fb1, fa0, fb0);
                substep(ln, buf, 1, st, fa0, fb0, fa1, fb1);
                substep(ln, buf, 2, st, fa1, fb1, fa0, fb0);
                substep(ln, buf, 3, st, fa0, fb0, fa1, fb1);
            };
            if (S2 > 0) {
                load_part(0, 0, 2 * LU);
                write_part(lane, 0, 0, 2 * LU);
                load_part(1, 0, 2 * LU);
                // (pairs of stages without a branch between them, so that the
                // compiler's load waits stay exact across the loop's back edge)
                int st = 0;
                for (; st + 1 < S2; st += 2) {
                    stage(st, 0);
                    stage(st + 1, 1);
                }
                if (st < S2) stage(st, 0);
                wait_lds<0>();
#pragma unroll
                for (int q = 0; q < MI * NI; ++q)     // last stage, substep 3
                    mfma32_ordered<BF16>(acc[q / NI][q % NI], fb1[q % NI], fa1[q / NI]);
            }
            // (wait states between the last MFMA and reads of its result)
            asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
        } else {
        // Pipeline over an LDS ring of NS stages of BK = 32, loads issued PD
        // stages ahead.  Each stage's fragment reads form two groups; the
        // loop is rotated so that the MFMAs of stage kt-1's second group
        // issue right after the barrier, interleaved with the reads of stage
        // kt's first group: no wave waits on LDS after a barrier.  Loads into LDS are not tracked by
        // the compiler: each wave waits for its own with vmcnt, leaving the
        // later stages' loads in flight, and the barrier then publishes the
        // stage.
        constexpr int LPS = A_INSTR + B_INSTR;    // loads per wave per stage
        static_assert((PD - 1) * LPS <= 63 && NS > PD, "pipeline depth");
        auto stage_ready = [&](int kt) {
            // this wave's loads of stage kt are done; those of the stages
            // after it (at most PD-1 of them) may still be in flight
            if (kt + 2 < KT) {
                __builtin_amdgcn_s_waitcnt(vm_wait((PD - 1) * LPS));
            } else if (kt + 1 < KT) {
                __builtin_amdgcn_s_waitcnt(vm_wait(LPS));
            } else {
                __builtin_amdgcn_s_waitcnt(vm_wait(0));
            }
            wait_lds<0>();         // the previous stage's last fragments are in registers
            ring_barrier();
            __builtin_amdgcn_sched_barrier(0);
        };
        // After the barrier every wave is past stage kt-1, so its ring slot
        // can take stage kt+PD.  The loads are issued between the two MFMA
        // groups of stage kt rather than right after the barrier, where they
        // would delay the first MFMAs.
        auto prefetch = [&](int kt) {
            if (kt + PD < KT) load_tile(kt + PD, (kt + PD) % NS);
            __builtin_amdgcn_sched_barrier(0);
        };

#pragma unroll
        for (int d = 0; d < PD; ++d)
            if (d < KT) load_tile(d, d);

        if constexpr (MF == 32) {
            // group 0 = k16 substep 0 (A and B), group 1 = substep 1.
            constexpr int RD = MI + 2 * NI;       // LDS reads per group
            symtile::u32x4 a0[MI], b0[NI], a1[MI], b1[NI];
#pragma unroll
            for (int i = 0; i < MI; ++i) a1[i] = symtile::u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int j = 0; j < NI; ++j) b1[j] = symtile::u32x4{0u, 0u, 0u, 0u};
            auto read_group = [&](int buf, int s, symtile::u32x4 (&a)[MI], symtile::u32x4 (&b)[NI]) {
#pragma unroll
                for (int i = 0; i < MI; ++i) a[i] = read_a(buf, i, 2 * s + (lane >> 5));
#pragma unroll
                for (int j = 0; j < NI; ++j) b[j] = read_b(buf, j, 16 * s);
            };
            auto mfmas = [&](const symtile::u32x4 (&a)[MI], const symtile::u32x4 (&b)[NI]) {
#pragma unroll
                for (int i = 0; i < MI; ++i)
#pragma unroll
                    for (int j = 0; j < NI; ++j) mma(i, j, a[i], b[j]);
            };
            for (int kt = 0; kt < KT; ++kt) {
                const int buf = kt % NS;
                stage_ready(kt);
                // substep-0 reads of stage kt interleaved with the MFMAs of
                // stage kt-1's substep 1 (zeros when kt = 0) ...
                read_group(buf, 0, a0, b0);
                mfmas(a1, b1);
                interleave_reads_mfmas<RD, MI * NI, true>();
                prefetch(kt);
                // ... then substep-1 reads behind the substep-0 MFMAs (the
                // reads overwrite a1/b1 only after the MFMAs that use them)
                read_group(buf, 1, a1, b1);
                mfmas(a0, b0);
                interleave_reads_mfmas<RD, MI * NI, false>();
            }
            wait_lds<0>();
            mfmas(a1, b1);         // last stage, substep 1
        } else {
            // One k32 substep per stage.  Group 0 = the A fragments and B
            // blocks [0, NJ0); group 1 = B blocks [NJ0, NI).  The MFMAs of
            // group 1 need the A fragments of their own stage, kept in aprev
            // while the next stage's A fragments are read.
            constexpr int NJ0 = (NI + 1) / 2, NJ1 = NI - NJ0;
            constexpr int RD1 = 2 * NJ1;          // LDS reads of group 1
            symtile::u32x4 acur[MI], aprev[MI], b0[NJ0], b1[NJ1 > 0 ? NJ1 : 1];
#pragma unroll
            for (int i = 0; i < MI; ++i) aprev[i] = symtile::u32x4{0u, 0u, 0u, 0u};
#pragma unroll
            for (int j = 0; j < NJ1; ++j) b1[j] = symtile::u32x4{0u, 0u, 0u, 0u};
            auto mfmas1 = [&]() {
#pragma unroll
                for (int i = 0; i < MI; ++i)
#pragma unroll
                    for (int j = 0; j < NJ1; ++j) mma(i, NJ0 + j, aprev[i], b1[j]);
            };
            for (int kt = 0; kt < KT; ++kt) {
                const int buf = kt % NS;
                stage_ready(kt);
#pragma unroll
                for (int i = 0; i < MI; ++i) acur[i] = read_a(buf, i, lane >> 4);
#pragma unroll
                for (int j = 0; j < NJ0; ++j) b0[j] = read_b(buf, j, 0);
                mfmas1();          // stage kt-1, group 1 (zeros when kt = 0)
                interleave_reads_mfmas<MI + 2 * NJ0, MI * NJ1, true>();
                prefetch(kt);
#pragma unroll
                for (int j = 0; j < NJ1; ++j) b1[j] = read_b(buf, NJ0 + j, 0);
#pragma unroll
                for (int i = 0; i < MI; ++i)
#pragma unroll
                    for (int j = 0; j < NJ0; ++j) mma(i, j, acur[i], b0[j]);
                interleave_reads_mfmas<RD1, MI * NJ0, false>();
#pragma unroll
                for (int i = 0; i < MI; ++i) aprev[i] = acur[i];
            }
            wait_lds<0>();
            mfmas1();              // last stage, group 1
        }
        }  // V4
        __syncthreads();           // every wave is done with the ring
        if (p.trace && tid == 0 && ks == 0 && !reducer)
            tile_trace(p, tm, tn)[SYMTILE_TRACE_MAINLOOP] = symtile::clock_now();

        // ---- split-K: combine the K slices of the tile ------------------
        // Every slice takes an arrival ticket (counter 0 of the tile).
        //  * Last-arriver protocol (p.sk_band == 0): a slice that is not the
        //    last to arrive writes its fp32 partial tile, releases it and
        //    counts it as written (counter 1), and moves on.  The last one
        //    waits until the others' partials are written: they all took
        //    their tickets before it, so they are running and wait for
        //    nothing themselves (no deadlock, and no co-residency is
        //    assumed).  It acquires them, forms the sum in slice order, and
        //    runs the epilogue for the whole tile.
        //  * Banded protocol (p.sk_band == 1, chosen by the host only when
        //    every work unit has a workgroup of its own and all of them are
        //    resident at once): the tile's rows form split bands; slice s
        //    writes its partial for the rows of the other bands, counts
        //    itself, waits until every slice has, and then sums band s in
        //    slice order and stores band s.  The reduction and the stores are
        //    shared by all slices instead of falling on the last one.
        //  * Reduction-kernel mode (p.sk_band == 2 here, then the RED
        //    instantiation): every slice writes its whole partial and moves
        //    on, taking no ticket; the second kernel sums each (tile, band of
        //    rows) and stores it, and its bands take the tickets that decide
        //    which one publishes the tile.
        // Every way the sum is p0 + p1 + ... in slice order, so all give the
        // same bits, whichever slice came last.  (Not built into the
        // copy-wave kernel: wave specialisation has no split-K, and its
        // third wave per SIMD leaves no registers for it.)
        const bool banded = !CW && p.split > 1 &&
                            (reducer ? p.reduce_bands > 1 : p.sk_band == 1);
        const int band_rows = banded ? BM / (reducer ? p.reduce_bands : p.split) : BM;
        // band of accumulator block row i of this wave (blocks are MF rows)
        auto block_band = [&](int i) { return (wm * WM + i * MF) / band_rows; };
        // reduction kernel: counter 1 of the tile as the band found it (read
        // before the sums, so its round trip overlaps them)
        [[maybe_unused]] uint32_t red_cnt1 = 0;
        if (!CW && p.split > 1) {
            __shared__ uint32_t s_ticket, s_ok;
            const int tile = tm * p.tiles_n + tn;
            uint32_t* cnt = p.sk_cnt + 2 * tile;
            // (the reduction-kernel mode takes no ticket: the kernel boundary
            // orders its two kernels)
            const bool ticketed = !reducer && p.sk_band != 2;
            if (tid == 0 && ticketed)
                s_ticket = symtile::atomic_add<__ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT>(cnt, 1u);
            __syncthreads();
            const uint32_t ticket = ticketed ? __builtin_amdgcn_readfirstlane(s_ticket) : 0u;
            if (ticket >= (uint32_t)p.split) {
                // more arrivals than slices: the counters were not zero at
                // the start of this call (a timed-out call leaves them so);
                // nothing of this tile can be trusted, so report and skip it
                if (tid == 0) symtile::raise_error(p.err, symtile::ERR_WORKSPACE);
                continue;
            }
            const bool last = !banded && ticketed && ticket + 1 == (uint32_t)p.split;
            // Partial tile of slice q: each thread's accumulators, 16 bytes
            // per (i, j, 4-value group), so a wave's access is 1 KiB contiguous.
            auto slot = [&](int q) {
                return symtile::make_rsrc(p.sk_part + ((size_t)tile * p.split + q) * (BM * BN),
                                          (uint32_t)(BM * BN * 4));
            };
            // Blocks of this thread's accumulators that a step covers: all of
            // them, or (banded) the ones in this slice's band (`own`) or
            // outside it.
            auto covered = [&](int i, bool own) {
                return !banded || ((block_band(i) == ks) == own);
            };
            // With large accumulators and more than two slices the reducing
            // slice sums every partial from memory, its own included, so
            // its own rows go to memory too.
            constexpr bool kBig = MI * NI * ACC_N > 64;
            const bool own_to_memory = kBig && p.split > 2;
            auto put_partial = [&](int q) {
                const symtile::rsrc_t rs = slot(q);
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    if (!own_to_memory && !covered(i, false)) continue;
#pragma unroll
                    for (int j = 0; j < NI; ++j)
#pragma unroll
                        for (int g = 0; g < ACC_N / 4; ++g) {
                            // (element copies first: this compiler's bit_cast of
                            // a vector element reads the vector's element 0)
                            const f32x4_t f{acc[i][j][4 * g], acc[i][j][4 * g + 1],
                                            acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
                            const symtile::u32x4 v = __builtin_bit_cast(symtile::u32x4, f);
                            symtile::buf_st16p<symtile::kStoreWriteThrough>(
                                v, rs, (uint32_t)tid * 16,
                                (uint32_t)(((i * NI + j) * (ACC_N / 4) + g) * THREADS * 16));
                        }
                }
            };
            // dst = partial q (first) or dst + partial q, in batches of 8
            // loads (32 registers): scheduling fences keep the compiler from
            // hoisting every load at once, which would need 4 registers per
            // accumulator register.  Blocks outside the covered set are not
            // touched.
            auto add_partial = [&](acc_t (&dst)[MI][NI], int q, bool first) {
                const symtile::rsrc_t rs = slot(q);
                constexpr int GPA = ACC_N / 4;                 // 4-value groups per accumulator
                constexpr int NG = MI * NI * GPA;
                constexpr int BATCH = NG % 8 == 0 ? 8 : NG % 4 == 0 ? 4 : 1;
                static_assert(NG % BATCH == 0, "batch split");
#pragma unroll
                for (int b = 0; b < NG; b += BATCH) {
                    symtile::u32x4 v[BATCH];
#pragma unroll
                    for (int x = 0; x < BATCH; ++x) {
                        const int i = (b + x) / (NI * GPA);
                        v[x] = symtile::buf_ld16p<symtile::kLoadCoherent>(
                            rs, covered(i, true) ? (uint32_t)tid * 16 : symtile::kOOB,
                            (uint32_t)((b + x) * THREADS * 16));
                    }
#pragma unroll
                    for (int x = 0; x < BATCH; ++x) {
                        const int n = b + x, i = n / (NI * GPA), j = (n / GPA) % NI, g = n % GPA;
                        if (!covered(i, true)) continue;
                        const f32x4_t y = __builtin_bit_cast(f32x4_t, v[x]);   // whole vector
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            dst[i][j][4 * g + e] = first ? y[e] : dst[i][j][4 * g + e] + y[e];
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            };
            if constexpr (RED) {
                // Second kernel: this band's p0 + p1 + ... in slice order,
                // rounded straight into the LDS staging of the epilogue (the
                // first kernel's partials were completed by the kernel
                // boundary).  Every wave shares the band: chunk x is 16 bytes
                // of a partial (4 consecutive columns of one row), taken in
                // memory order, so a wave reads 1 KiB runs; CH chunks of QB
                // slices are in flight per thread at once.
                constexpr int GPA = ACC_N / 4;
                constexpr int PER_BR = NI * GPA * WGN * 64;    // chunks per block row
                constexpr int CH = 4, QB = 4;
                const int total = band_rows / MF * PER_BR;
                const int br0 = ks * (band_rows / MF);
                if (tid == 0)
                    red_cnt1 = __hip_atomic_load(symtile::global_ptr(cnt + 1), __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
                uint8_t* Cs = smem;
#pragma unroll 1
                for (int x0 = 0; x0 < total; x0 += THREADS * CH) {
                    float sum[CH][4];
#pragma unroll 1
                    for (int q0 = 0; q0 < p.split; q0 += QB) {
                        symtile::u32x4 v[CH][QB];
#pragma unroll
                        for (int c = 0; c < CH; ++c) {
                            const int x = x0 + c * THREADS + tid;
                            const int br = br0 + x / PER_BR, rem = x % PER_BR;
                            const int jg = rem / (WGN * 64), wl = rem % (WGN * 64);
                            const uint32_t off =
                                (uint32_t)(((((br % MI) * NI + jg / GPA) * GPA + jg % GPA) * THREADS +
                                            ((br / MI) * WGN + wl / 64) * 64 + wl % 64) * 16);
#pragma unroll
                            for (int qq = 0; qq < QB; ++qq) {
                                const int q = min(q0 + qq, p.split - 1);
                                v[c][qq] = symtile::buf_ld16p<symtile::kLoadCoherent>(
                                    slot(q), x < total && q0 + qq < p.split ? off : symtile::kOOB, 0);
                            }
                        }
#pragma unroll
                        for (int c = 0; c < CH; ++c)
#pragma unroll
                            for (int qq = 0; qq < QB; ++qq) {
                                if (q0 + qq >= p.split) continue;      // uniform
                                const f32x4_t y = __builtin_bit_cast(f32x4_t, v[c][qq]);
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    sum[c][e] = q0 + qq == 0 ? y[e] : sum[c][e] + y[e];
                            }
                    }
#pragma unroll
                    for (int c = 0; c < CH; ++c) {
                        const int x = x0 + c * THREADS + tid;
                        if (x >= total) continue;
                        const int br = br0 + x / PER_BR, rem = x % PER_BR;
                        const int jg = rem / (WGN * 64), wl = rem % (WGN * 64);
                        const int ln = wl % 64, j = jg / GPA, g = jg % GPA;
                        // the accumulator layout of the K-loop kernel (see the
                        // epilogue below)
                        const int row = br * MF + (ln % MF);
                        const int col = (wl / 64) * WN + j * MF +
                                        ((MF == 32) ? 8 * g + 4 * (ln >> 5) : 4 * (ln >> 4));
                        uint2 w;
                        w.x = cvt_pack<BF16>(sum[c][0], sum[c][1]);
                        w.y = cvt_pack<BF16>(sum[c][2], sum[c][3]);
                        const int chunk = col >> 3, half = (col >> 2) & 1;
                        *reinterpret_cast<uint2*>(Cs + row * CROW + ((chunk ^ (row & 7)) << 4) +
                                                  (half << 3)) = w;
                    }
                }
            } else {
                // 1. partials: every slice but the last-arriving one (banded:
                // every slice, for the other bands' rows), and the reducing
                // slice's own rows when it sums from memory
                // (the first kernel of the reduction-kernel mode, which takes
                // no ticket and so is never last, writes its whole partial and
                // moves on: the second kernel sums them; one call site of
                // put_partial, as two spill inside the K loop)
                if (!last || own_to_memory) put_partial(ks);
                if (p.sk_band == 2) continue;
                if (!last) {
                    symtile::wg_stores_done();
                    // (partials are always stored write-through)
                    if (tid == 0) symtile::flag_publish_written_through(cnt + 1);
                    if (!banded) continue;
                } else if (own_to_memory) {
                    __builtin_amdgcn_s_waitcnt(vm_wait(0));
                }
                // 2. wait for the others' partials (bounded); they were written
                // through and are read with coherent loads, so the wait needs
                // no L2 invalidate
                if (tid == 0) {
                    const uint32_t target = banded ? (uint32_t)p.split : (uint32_t)p.split - 1;
                    const bool ok = symtile::flag_wait_coherent(cnt + 1, target, p.spin_limit);
                    if (ok && !banded) {
                        // every slice of this call has counted itself: the next
                        // call starts again from zero (banded: reset by the last
                        // slice to store its band, below)
                        symtile::atomic_xchg<__ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT>(cnt, 0u);
                        symtile::atomic_xchg<__ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT>(cnt + 1, 0u);
                    } else if (!ok) {
                        // a slice that holds a ticket may still count itself
                        // later, so the counters are left as they are: the next
                        // call that uses this workspace then draws tickets past
                        // the slice count and reports ERR_WORKSPACE instead of
                        // summing stale partials, until the caller zeroes them
                        symtile::raise_error(p.err, symtile::ERR_TIMEOUT);
                    }
                    s_ok = ok;
                }
                __syncthreads();
                if (!s_ok) continue;
                // 3. the sum in slice order over the covered blocks
                if constexpr (!kBig) {
                    // Small accumulators fold in registers:
                    // tmp = p0 + ... + p(ks-1), acc = tmp + acc, which is
                    // (p0 + ... + p(ks-1)) + p(ks) since addition commutes, then
                    // acc += p(ks+1), ... in slice order.
                    acc_t tmp[MI][NI];
                    for (int q = 0; q < ks; ++q) add_partial(tmp, q, q == 0);
                    if (ks > 0) {
    #pragma unroll
                        for (int i = 0; i < MI; ++i)
    #pragma unroll
                            for (int j = 0; j < NI; ++j)
    #pragma unroll
                                for (int e = 0; e < ACC_N; ++e)
                                    if (covered(i, true)) acc[i][j][e] = tmp[i][j][e] + acc[i][j][e];
                    }
                    for (int q = ks + 1; q < p.split; ++q) add_partial(acc, q, false);
                } else {
                    // Two slices: acc + the other partial, which is p0 + p1 either
                    // way (fp32 addition commutes).  More: this slice's partial
                    // joined the others in memory and the sum is formed
                    // p0 + p1 + ... in slice order.  (One call site of
                    // add_partial: with two, the compiler spills inside the K
                    // loop.)
                    const int nq = p.split == 2 ? 1 : p.split;
                    for (int n = 0; n < nq; ++n)
                        add_partial(acc, p.split == 2 ? 1 - ks : n, p.split != 2 && n == 0);
                }
            }
        }

        // ---- epilogue: round, restage row-major, store, release --------
        // (banded split-K: only this slice's band is restaged and stored)
        // (the reduction kernel staged its band above)
        uint8_t* Cs = smem;
        // (4-wave 256 x 256: the staging offsets are recomputed here from a
        // lane value the compiler cannot hoist; computed before the K loop
        // they were spilled and reloaded one at a time)
        int lane_e = lane;
        if constexpr (V4) asm volatile("" : "+v"(lane_e));
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            if (RED || (banded && block_band(i) != ks)) continue;
#pragma unroll
            for (int j = 0; j < NI; ++j) {
                // (4-wave 256 x 256: the block leaves its AGPRs only here, one
                // block at a time; all at once they would not fit in VGPRs)
                acc_t blk = acc[i][j];
                if constexpr (V4) asm volatile("" : "+v"(blk));
#pragma unroll
                for (int g = 0; g < ACC_N / 4; ++g) {
                    // MF = 32: lane l, registers 4g..4g+3 hold row l % 32,
                    // columns 8g + 4 * (l / 32) .. +3 of the block; MF = 16:
                    // row l % 16, columns 4 * (l / 16) .. +3.
                    const int row = wm * WM + i * MF + (lane_e % MF);
                    const int col = wn * WN + j * MF +
                                    ((MF == 32) ? 8 * g + 4 * (lane_e >> 5) : 4 * (lane_e >> 4));
                    uint2 w;
                    w.x = cvt_pack<BF16>(blk[4 * g + 0], blk[4 * g + 1]);
                    w.y = cvt_pack<BF16>(blk[4 * g + 2], blk[4 * g + 3]);
                    const int chunk = col >> 3, half = (col >> 2) & 1;
                    *reinterpret_cast<uint2*>(Cs + row * CROW + ((chunk ^ (row & 7)) << 4) +
                                              (half << 3)) = w;
                }
            }
        }
        __syncthreads();

        // FUSED: every slot.  WAVE_SPEC: the local slot (the copy wave does the
        // rest during the next tile), except for this workgroup's last tile.
        const int n_dst = (p.role == ROLE_FUSED || (reducer && p.reduce_all) ||
                           (CW && t + G >= p.num_tiles))
                              ? p.world
                              : 1;
        const uint16_t* tile_local = out_tile_ptr(p, BM, BN, tm, tn);
        const symtile::TileGeom geom = out_tile<BM, BN, THREADS>(p, tm, tn);
        const symtile::TileLanes lanes = symtile::tile_lanes(geom, tid, THREADS);
        const int c = tid % IO::CPR, r0 = tid / IO::CPR;
        const uint32_t voff = lanes.voff;
        const uint32_t pass_bytes = lanes.pass_bytes;
        const uint8_t* crow = Cs + r0 * CROW + ((c ^ (r0 & 7)) << 4);
        // passes [pass_lo, pass_hi) hold the rows to store: the whole tile,
        // or this slice's band (the host checks that a band is a whole
        // number of passes)
        const int pass_lo = banded ? ks * (band_rows / IO::RP) : 0;
        const int pass_hi = banded ? pass_lo + band_rows / IO::RP : IO::PASSES;
#pragma unroll 1
        for (int b = pass_lo; b < pass_hi; b += IO::U) {
            symtile::u32x4 v[IO::U];
#pragma unroll
            for (int u = 0; u < IO::U; ++u)
                v[u] = *reinterpret_cast<const symtile::u32x4*>(
                    crow + min(b + u, IO::PASSES - 1) * IO::RP * CROW);
            for (int d = 0; d < n_dst; ++d) {
                const symtile::rsrc_t rd =
                    symtile::tile_rsrc(tile_local, geom, p.rank, (p.rank + d) % p.world, p.bases);
                with_store_policy(p.nontemporal, [&](auto pol) {
#pragma unroll
                    for (int u = 0; u < IO::U; ++u)
                        if (b + u < pass_hi)       // uniform: a band may be one pass
                            symtile::buf_st16p<decltype(pol)::value>(v[u], rd, voff,
                                                                     (b + u) * pass_bytes);
                });
            }
        }
        symtile::wg_stores_done();     // also orders the LDS reads above before reuse
        if (tid < 64) {                // wave 0: one release, then lane d counts slot rank + d
            bool publish = true;
            if (reducer) {
                // Reduction kernel: the tile is whole once every band is
                // stored; each band releases its stores and takes a ticket,
                // and the one that draws the last resets the counter and
                // publishes the tile's counters.  This mode leaves counter 1
                // alone, so a non-zero counter 1 (read above) or a ticket
                // past the band count means the workspace was not zero when
                // the call started: the data stored is this call's, but the
                // tile is not published, and the error is reported.
                release_output(p.nontemporal);
                uint32_t* cnt = p.sk_cnt + 2 * (tm * p.tiles_n + tn);
                uint32_t u = 0;
                if (tid == 0) {
                    u = symtile::atomic_add<__ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT>(cnt, 1u);
                    if (red_cnt1 != 0 || u >= (uint32_t)p.reduce_bands)
                        symtile::raise_error(p.err, symtile::ERR_WORKSPACE);
                }
                u = __shfl(u, 0);
                const uint32_t w1 = __shfl(red_cnt1, 0);
                publish = w1 == 0 && u == (uint32_t)p.reduce_bands - 1u;
                if (publish) {
                    if (p.nontemporal != 2) symtile::fence_acquire<__HIP_MEMORY_SCOPE_AGENT>();
                    if (tid == 0)
                        symtile::atomic_xchg<__ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT>(cnt, 0u);
                }
            } else if (banded) {
                // Banded: the tile is whole once every slice has stored its
                // band.  Each slice releases its stores and takes a second
                // ticket on counter 0 (the first round of tickets left it at
                // split); the one that draws 2*split - 1 acquires the others'
                // stores, resets the counters for the next call and publishes
                // the tile's counters behind a release of its own.
                release_output(p.nontemporal);
                uint32_t* cnt = p.sk_cnt + 2 * (tm * p.tiles_n + tn);
                uint32_t u2 = 0;
                if (tid == 0)
                    u2 = symtile::atomic_add<__ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT>(cnt, 1u);
                u2 = __shfl(u2, 0);
                publish = u2 == 2u * (uint32_t)p.split - 1u;
                if (publish) {
                    // the other slices' band stores happen before the counters
                    // move: written through, they were in memory before their
                    // slices' tickets; otherwise acquire their releases
                    if (p.nontemporal != 2) symtile::fence_acquire<__HIP_MEMORY_SCOPE_AGENT>();
                    if (tid == 0) {
                        symtile::atomic_xchg<__ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT>(cnt, 0u);
                        symtile::atomic_xchg<__ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT>(cnt + 1, 0u);
                    }
                }
            }
            if (publish) {
                if (p.trace && tid == 0) tile_trace(p, tm, tn)[SYMTILE_TRACE_STORED] = symtile::clock_now();
                release_output(p.nontemporal);
                uint32_t* flag = p.arrived + ((size_t)p.rank * p.tiles_m + tm) * p.tiles_n + tn;
                if (tid < n_dst)
                    symtile::flag_signal(symtile::translate(flag, p.rank, (p.rank + tid) % p.world, p.bases));
                if (tid == 0 && p.role == ROLE_WG_SPEC) symtile::flag_signal(p.ready + tm * p.tiles_n + tn);
                if (p.trace && tid == 0) tile_trace(p, tm, tn)[SYMTILE_TRACE_RELEASED] = symtile::clock_now();
            }
        }
    }
}

// Copy kernels of the bulk-synchronous and unfused producer-consumer
// schedules run on CUs of their own, so their workgroups are wide (16 waves
// keep many loads and stores in flight per CU).
template <int BM>
constexpr int copy_threads() { return BM >= 128 ? 1024 : 256; }

// Second kernel of the bulk-synchronous schedule (Section 4.1.1).
template <int BM, int BN>
__global__ __launch_bounds__(copy_threads<BM>()) void scatter_kernel(const GasParams p) {
    for (int t = blockIdx.x; t < p.num_tiles; t += gridDim.x) {
        const int tm = t / p.tiles_n, tn = t % p.tiles_n;
        uint64_t* tr = tile_trace(p, tm, tn);
        if (tr && threadIdx.x == 0)
            tr[SYMTILE_TRACE_COPY_WAIT] = tr[SYMTILE_TRACE_COPY_GO] = symtile::clock_now();
        with_store_policy(p.nontemporal, [&](auto pol) {
            put_tile_to_peers<BM, BN, copy_threads<BM>(), decltype(pol)::value>(p, tm, tn);
        });
        if (tr && threadIdx.x == 0) tr[SYMTILE_TRACE_COPY_DONE] = symtile::clock_now();
    }
}

// Copy kernel of the unfused producer-consumer schedule (Section 4.1.2):
// runs on its own stream next to the producer grid of gas_kernel.
template <int BM, int BN>
__global__ __launch_bounds__(copy_threads<BM>()) void consumer_kernel(const GasParams p) {
    consume_tiles<BM, BN, copy_threads<BM>()>(p, blockIdx.x, gridDim.x);
}

// ---------------------------------------------------------------------------
struct Variant {
    int bm, bn;
    bool bf16;
    int waves;
    const void* gas;
    const void* scatter;
    const void* consumer;
    int copy_threads;            // workgroup size of scatter_kernel and consumer_kernel
    const void* gas_ws;          // wave-specialised kernel (NW compute waves + 1), or null
    const void* reduce;          // second kernel of the split-K reduction-kernel mode
    int band_q;                  // banded split-K: a band's rows must be a multiple of this
};

// Rows of a banded split-K reduction band must cover whole MFMA accumulator
// blocks (MF rows) and whole passes of the epilogue's row stores.
template <int BM, int BN, int NW, int MF>
constexpr int band_quantum() {
    constexpr int rp = TileIO<BM, BN, 64 * NW>::RP;
    return rp > MF ? rp : MF;
}

// The copy-wave kernel is instantiated only for the shapes that use it.
template <int BM, int BN, bool BF16, int NW, int MF, bool WS>
const void* wave_spec_kernel() {
    if constexpr (WS)
        return reinterpret_cast<const void*>(&gas_kernel<BM, BN, BF16, NW, MF, true>);
    else
        return nullptr;
}

template <int BM, int BN, bool BF16, int NW, int MF = 32, bool WS = false>
Variant make_variant() {
    return Variant{BM, BN, BF16, NW,
                   reinterpret_cast<const void*>(&gas_kernel<BM, BN, BF16, NW, MF>),
                   reinterpret_cast<const void*>(&scatter_kernel<BM, BN>),
                   reinterpret_cast<const void*>(&consumer_kernel<BM, BN>),
                   copy_threads<BM>(), wave_spec_kernel<BM, BN, BF16, NW, MF, WS>(),
                   reinterpret_cast<const void*>(&gas_kernel<BM, BN, BF16, NW, MF, false, true>),
                   band_quantum<BM, BN, NW, MF>()};
}

// waves == 0 picks the first entry of the shape (the default wave count).
const Variant* find_variant(int bm, int bn, bool bf16, int waves) {
    static const Variant table[] = {
        make_variant<64, 64, false, 4>(),    make_variant<64, 64, true, 4>(),
        make_variant<128, 128, false, 8>(),  make_variant<128, 128, true, 8>(),
        make_variant<128, 128, false, 4>(),  make_variant<128, 128, true, 4>(),
        make_variant<256, 128, false, 8, 32, true>(), make_variant<256, 128, true, 8, 32, true>(),
        make_variant<256, 128, false, 4>(),  make_variant<256, 128, true, 4>(),
        make_variant<256, 256, false, 8>(),  make_variant<256, 256, true, 8>(),
        make_variant<256, 256, false, 4>(),  make_variant<256, 256, true, 4>(),
        make_variant<256, 224, false, 8, 16>(), make_variant<256, 224, true, 8, 16>(),
    };
    for (const Variant& v : table)
        if (v.bm == bm && v.bn == bn && v.bf16 == bf16 && (waves == 0 || v.waves == waves))
            return &v;
    return nullptr;
}

// The shape's build with a copy wave, or null.
const Variant* find_wave_spec_variant(int bm, int bn, bool bf16) {
    for (int w : {8, 4}) {
        const Variant* v = find_variant(bm, bn, bf16, w);
        if (v && v->gas_ws) return v;
    }
    return nullptr;
}

symtile_status coresident_limit(const Variant* v, int device, int* cus, int* limit) {
    int n_cu = symtile_host::cu_count(device);
    if (n_cu <= 0) return symtile_host::fail(SYMTILE_EHIP, "cannot read the CU count");
    // workgroups of a kernel per CU: fixed for the process, so asked once per
    // (kernel, device) (the query costs microseconds on every call's path)
    static std::mutex mu;
    static std::map<std::pair<const void*, int>, int> per_cu_known;
    int per_cu = 0;
    {
        std::lock_guard<std::mutex> lock(mu);
        auto it = per_cu_known.find({v->gas, device});
        if (it != per_cu_known.end()) per_cu = it->second;
    }
    if (per_cu == 0) {
        SYMTILE_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, v->gas, 64 * v->waves, 0));
        std::lock_guard<std::mutex> lock(mu);
        per_cu_known[{v->gas, device}] = per_cu;
    }
    *cus = n_cu;
    *limit = per_cu * n_cu;
    return SYMTILE_OK;
}

// Split-K workspace: two counters per tile, rounded up to 256 bytes, then
// `split` fp32 partial tiles per tile.
constexpr int kMaxSplit = 64;
size_t sk_counter_bytes(size_t tiles) { return (tiles * 8 + 255) / 256 * 256; }
size_t sk_workspace_bytes(size_t tiles, int bm, int bn, int split) {
    return split <= 1 ? 0 : sk_counter_bytes(tiles) + tiles * split * (size_t)bm * bn * 4;
}

// ---------------------------------------------------------------------------
// Scratch of the allocation-free entry point: the split-K workspace (tile
// counters, then fp32 partial tiles) in a static device array, one copy per
// GPU, held from the library's first use on that GPU until the process ends.
// Host code never passes this name to a kernel or a copy (on the host it is
// only a stand-in for the symbol): its device address comes from
// hipGetSymbolAddress, once per device, with that device current.
static __device__ __align__(256) uint8_t g_noalloc_scratch[SYMTILE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

symtile_status noalloc_scratch(int device, void** out) {
    if (device < 0 || device >= kMaxDevices)
        return symtile_host::fail(SYMTILE_EINVAL, "device index beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        int prev = -1;
        SYMTILE_HIP(hipGetDevice(&prev));
        SYMTILE_HIP(hipSetDevice(device));
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(g_noalloc_scratch));
        (void)hipSetDevice(prev);
        if (e != hipSuccess) return symtile_host::hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!ptr) return symtile_host::fail(SYMTILE_EHIP, "scratch symbol has no device address");
        g_scratch_ptr[device] = ptr;
    }
    *out = g_scratch_ptr[device];
    return SYMTILE_OK;
}

// Zero n 32-bit words (the split-K counters) with a kernel, so the call adds
// no memset node when a caller captures it into a graph.
__global__ __launch_bounds__(256) void zero_words_kernel(uint32_t* p, int n) {
    for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0u;
}

}  // namespace

extern "C" symtile_status symtile_gas_workspace_bytes(int M, int N_local, int tile_m, int tile_n,
                                                      int split_k, size_t* bytes) {
    using symtile_host::fail;
    if (!bytes) return fail(SYMTILE_EINVAL, "bytes is NULL");
    if (M < 0 || N_local < 0) return fail(SYMTILE_EINVAL, "negative size");
    if (tile_m == 0 && tile_n == 0) tile_m = tile_n = 256;
    if (!find_variant(tile_m, tile_n, true, 0)) return fail(SYMTILE_EINVAL, "tile shape not built");
    if (split_k < 0 || split_k > kMaxSplit) return fail(SYMTILE_EINVAL, "split_k must be 0..64");
    const size_t tiles = (size_t)((M + tile_m - 1) / tile_m) * ((N_local + tile_n - 1) / tile_n);
    *bytes = sk_workspace_bytes(tiles, tile_m, tile_n, split_k);
    return SYMTILE_OK;
}

extern "C" symtile_status symtile_device_info(int device, int tile_m, int tile_n, int* cu_count,
                                              int* max_coresident_wgs) {
    if (tile_m == 0 && tile_n == 0) tile_m = tile_n = 256;
    const Variant* v = find_variant(tile_m, tile_n, true, 0);
    if (!v) return symtile_host::fail(SYMTILE_EUNSUPPORTED, "tile shape not built");
    int cus = 0, lim = 0;
    if (symtile_status st = coresident_limit(v, device, &cus, &lim)) return st;
    if (cu_count) *cu_count = cus;
    if (max_coresident_wgs) *max_coresident_wgs = lim;
    return SYMTILE_OK;
}

extern "C" symtile_status symtile_gemm_all_scatter(
    symtile_heap* h, const void* A, const void* B_shard, void* C_gathered_local,
    uint32_t* arrived_local, uint32_t* ready, int M, int N_local, int K, int lda, int ldb,
    int dtype, int rank, int world_size, const symtile_gas_config* cfg_in, symtile_stream s) {
    using symtile_host::fail;
    if (!h) return fail(SYMTILE_EINVAL, "heap is NULL");
    symtile_gas_config cfg{};
    if (cfg_in) cfg = *cfg_in;
    if (cfg.tile_m == 0 && cfg.tile_n == 0) cfg.tile_m = cfg.tile_n = 256;
    if (cfg.epoch == 0) cfg.epoch = 1;
    if (cfg.spin_limit == 0) cfg.spin_limit = 1u << 22;
    if (cfg.group_m <= 0) cfg.group_m = 4;
    if (cfg.variant < SYMTILE_BULK_SYNC || cfg.variant > SYMTILE_WAVE_SPEC)
        return fail(SYMTILE_EINVAL, "unknown variant");
    if (dtype != SYMTILE_F16 && dtype != SYMTILE_BF16)
        return fail(SYMTILE_EUNSUPPORTED, "dtype must be SYMTILE_F16 or SYMTILE_BF16");
    if (world_size != h->world) return fail(SYMTILE_EINVAL, "world_size differs from the heap's");
    if (rank < 0 || rank >= world_size) return fail(SYMTILE_EINVAL, "rank out of range");
    if (M < 0 || N_local < 0 || K < 0) return fail(SYMTILE_EINVAL, "negative size");
    if (lda == 0) lda = K;
    if (ldb == 0) ldb = N_local;
    if (lda < K || ldb < N_local) return fail(SYMTILE_EINVAL, "lda < K or ldb < N_local");
    if (K % 8 || N_local % 8 || lda % 8 || ldb % 8)
        return fail(SYMTILE_EINVAL, "K, N_local, lda and ldb must be multiples of 8");
    if (cfg.waves_per_wg != 0 && cfg.waves_per_wg != 4 && cfg.waves_per_wg != 8)
        return fail(SYMTILE_EINVAL, "waves_per_wg must be 0, 4 or 8");
    if (cfg.split_k < 0 || cfg.split_k > kMaxSplit) return fail(SYMTILE_EINVAL, "split_k must be 0..64");
    if (cfg.split_reduce < SYMTILE_SPLIT_REDUCE_AUTO || cfg.split_reduce > SYMTILE_SPLIT_REDUCE_KERNEL)
        return fail(SYMTILE_EINVAL, "split_reduce must be 0, 1, 2 or 3");
    const int split = cfg.split_k > 1 ? cfg.split_k : 1;
    if (split > 1 && cfg.variant != SYMTILE_FUSED_SEQ && cfg.variant != SYMTILE_BULK_SYNC)
        return fail(SYMTILE_EUNSUPPORTED, "split_k > 1 is built for BULK_SYNC and FUSED_SEQ");
    // Default wave count: the shape's first build, except that unsplit
    // 256 x 256 fused and bulk-synchronous calls run the 4-wave kernel (its
    // register-staged loop is faster there; 8 waves stay for split-K, whose
    // banded exchange favours them, and for the schedules with consumer
    // workgroups, which take the producers' workgroup size).
    int waves = cfg.waves_per_wg;
    if (waves == 0 && cfg.tile_m == 256 && cfg.tile_n == 256 && split == 1 &&
        (cfg.variant == SYMTILE_FUSED_SEQ || cfg.variant == SYMTILE_BULK_SYNC))
        waves = 4;
    const Variant* v = find_variant(cfg.tile_m, cfg.tile_n, dtype == SYMTILE_BF16, waves);
    if (!v) return fail(SYMTILE_EUNSUPPORTED, "tile shape / wave count not built");
    // Buffer resources span one tile row band of A or C and the whole of B;
    // each must stay below 2 GiB.
    const size_t kMaxSpan = size_t(1) << 31;
    if ((size_t)world_size * N_local * 2 * cfg.tile_m >= kMaxSpan ||
        (size_t)lda * 2 * cfg.tile_m >= kMaxSpan || (size_t)K * ldb * 2 >= kMaxSpan)
        return fail(SYMTILE_EINVAL, "a tile band of A or C, or B, exceeds 2 GiB");
    if (M == 0 || N_local == 0) return SYMTILE_OK;   // no tiles, nothing to publish
    if ((K > 0 && (!A || !B_shard)) || !C_gathered_local || !arrived_local)
        return fail(SYMTILE_EINVAL, "NULL pointer argument");
    if (reinterpret_cast<uintptr_t>(A) % 16 || reinterpret_cast<uintptr_t>(B_shard) % 16 ||
        reinterpret_cast<uintptr_t>(C_gathered_local) % 16 ||
        reinterpret_cast<uintptr_t>(arrived_local) % 4)
        return fail(SYMTILE_EINVAL, "A, B_shard and C_gathered_local must be 16-byte aligned");

    const int tiles_m = (M + cfg.tile_m - 1) / cfg.tile_m;
    const int tiles_n = (N_local + cfg.tile_n - 1) / cfg.tile_n;
    const size_t num_tiles = (size_t)tiles_m * tiles_n;
    const size_t ldc = (size_t)world_size * N_local;
    const size_t c_bytes = ((size_t)(M - 1) * ldc + ldc) * 2;
    const size_t flag_bytes = (size_t)world_size * num_tiles * 4;
    if (!symtile_host::in_slot(h, C_gathered_local, c_bytes, rank))
        return fail(SYMTILE_EINVAL, "C_gathered_local [M, w*N_local] is not inside slot `rank`");
    if (!symtile_host::in_slot(h, arrived_local, flag_bytes, rank))
        return fail(SYMTILE_EINVAL, "arrived_local [w, tiles_m, tiles_n] is not inside slot `rank`");
    {
        const uint64_t c0 = reinterpret_cast<uint64_t>(C_gathered_local);
        const uint64_t f0 = reinterpret_cast<uint64_t>(arrived_local);
        if (f0 < c0 + c_bytes && c0 < f0 + flag_bytes)
            return fail(SYMTILE_EINVAL, "arrived_local overlaps C_gathered_local");
    }
    if ((cfg.variant == SYMTILE_WG_SPEC || cfg.variant == SYMTILE_UNFUSED_PC) && !ready)
        return fail(SYMTILE_EINVAL, "WG_SPEC and UNFUSED_PC need a ready counter array");
    if (reinterpret_cast<uintptr_t>(cfg.trace) % 8)
        return fail(SYMTILE_EINVAL, "trace must be 8-byte aligned");
    if (split > 1) {
        if (split > (K + BK - 1) / BK)
            return fail(SYMTILE_EINVAL, "split_k " + std::to_string(split) +
                                            " exceeds the ceil(K/32) stages of K");
        if (num_tiles * split > (size_t)INT32_MAX) return fail(SYMTILE_EINVAL, "too many work units");
        const size_t need = sk_workspace_bytes(num_tiles, cfg.tile_m, cfg.tile_n, split);
        if (!cfg.workspace || cfg.workspace_bytes < need)
            return fail(SYMTILE_EINVAL, "split_k needs a workspace of " + std::to_string(need) +
                                            " bytes");
        if (reinterpret_cast<uintptr_t>(cfg.workspace) % 16)
            return fail(SYMTILE_EINVAL, "workspace must be 16-byte aligned");
        const uint64_t w0 = reinterpret_cast<uint64_t>(cfg.workspace);
        const uint64_t c0 = reinterpret_cast<uint64_t>(C_gathered_local);
        const uint64_t f0 = reinterpret_cast<uint64_t>(arrived_local);
        for (int s = 0; s < world_size; ++s) {   // the output and counters of every slot
            const uint64_t cs = c0 + (uint64_t)s * h->slot_stride - (uint64_t)rank * h->slot_stride;
            const uint64_t fs = f0 + (uint64_t)s * h->slot_stride - (uint64_t)rank * h->slot_stride;
            if ((w0 < cs + c_bytes && cs < w0 + need) || (w0 < fs + flag_bytes && fs < w0 + need))
                return fail(SYMTILE_EINVAL, "workspace overlaps the output or the counters");
        }
    }

    int cus = 0, limit = 0;
    if (symtile_status st = coresident_limit(v, h->device, &cus, &limit)) return st;

    GasParams p;
    p.A = static_cast<const uint16_t*>(A);
    p.B = static_cast<const uint16_t*>(B_shard);
    p.C = static_cast<uint16_t*>(C_gathered_local);
    p.arrived = arrived_local;
    p.ready = ready;
    p.bases = h->dev_bases;
    p.err = h->dev_err;
    p.M = M;
    p.N = N_local;
    p.K = K;
    p.lda = lda;
    p.ldb = ldb;
    p.ldc = (int)ldc;
    p.rank = rank;
    p.world = world_size;
    p.tiles_m = tiles_m;
    p.tiles_n = tiles_n;
    p.num_tiles = (int)num_tiles;
    p.group_m = cfg.group_m;
    p.epoch = cfg.epoch;
    p.spin_limit = cfg.spin_limit;
    p.nontemporal = cfg.nontemporal;
    if (cfg.nontemporal < 0 || cfg.nontemporal > 2)
        return fail(SYMTILE_EINVAL, "nontemporal must be 0, 1 or 2");
    p.trace = cfg.trace;
    p.copy_wgs = 0;
    p.split = split;
    p.units = (int)(num_tiles * split);
    p.sk_cnt = split > 1 ? static_cast<uint32_t*>(cfg.workspace) : nullptr;
    p.sk_part = split > 1 ? reinterpret_cast<float*>(static_cast<uint8_t*>(cfg.workspace) +
                                                     sk_counter_bytes(num_tiles))
                          : nullptr;

    hipStream_t stream = static_cast<hipStream_t>(s);
    int prev = -1;
    if (symtile_status st = symtile_host::set_device(h, &prev)) return st;
    struct Restore {
        int d;
        ~Restore() {
            if (d >= 0) (void)hipSetDevice(d);
        }
    } restore{prev};

    const int ntiles = (int)num_tiles;
    p.sk_band = 0;
    p.reduce_bands = 1;
    p.reduce_all = 0;
    if (cfg.variant == SYMTILE_FUSED_SEQ || cfg.variant == SYMTILE_BULK_SYNC) {
        int g = cfg.gemm_wgs > 0 ? cfg.gemm_wgs : std::min(p.units, cus);
        g = std::min(g, p.units);
        p.gemm_wgs = g;
        if (split > 1) {
            // Banded reduction: every slice waits for all the others, so
            // every work unit needs a workgroup of its own, all resident at
            // once; a band covers whole accumulator blocks and store passes.
            const bool fits = g == p.units && g <= limit && cfg.tile_m % split == 0 &&
                              (cfg.tile_m / split) % v->band_q == 0;
            if (cfg.split_reduce == SYMTILE_SPLIT_REDUCE_BANDED && !fits)
                return fail(SYMTILE_EUNSUPPORTED,
                            "banded split-K reduction needs one resident workgroup per K slice "
                            "(tiles * split_k <= " + std::to_string(limit) +
                                ") and tile_m / split_k a multiple of " +
                                std::to_string(v->band_q));
            // AUTO: for two slices banded where it fits (each slice reduces
            // half the tile, with the last-arriver's round trips), else the
            // last arriver, both ahead of a second kernel; with more slices
            // the reduction kernel, which spreads the sum and the stores over
            // every CU instead of one slice per tile (banded: every slice
            // then pays a partial write, a wait and a second ticket)
            const bool automatic = cfg.split_reduce == SYMTILE_SPLIT_REDUCE_AUTO;
            p.sk_band = cfg.split_reduce == SYMTILE_SPLIT_REDUCE_BANDED ||
                        (automatic && fits && split == 2);
            if (cfg.split_reduce == SYMTILE_SPLIT_REDUCE_KERNEL || (automatic && split > 2))
                p.sk_band = 2;
        }
        p.role = cfg.variant == SYMTILE_FUSED_SEQ ? ROLE_FUSED : ROLE_LOCAL_ONLY;
        void* args[] = {&p};
        SYMTILE_HIP(hipLaunchKernel(v->gas, dim3(g), dim3(64 * v->waves), args, 0, stream));
        if (p.sk_band == 2) {
            // Reduction kernel: every (tile, band of rows) sums its rows of
            // the partials in slice order and stores them.  Bands: the most
            // (a power of two, whole accumulator blocks and store passes)
            // that keep the grid within the CU count.
            GasParams r = p;
            int nb = 1;
            while (cfg.tile_m % (2 * nb) == 0 && (cfg.tile_m / (2 * nb)) % v->band_q == 0 &&
                   (size_t)ntiles * 2 * nb <= (size_t)cus)
                nb *= 2;
            r.role = ROLE_REDUCE;
            r.sk_band = 0;
            r.reduce_bands = nb;
            r.reduce_all = cfg.variant == SYMTILE_FUSED_SEQ;
            r.units = ntiles * nb;
            r.gemm_wgs = std::min(r.units, cus);
            void* rargs[] = {&r};
            SYMTILE_HIP(hipLaunchKernel(v->reduce, dim3(r.gemm_wgs), dim3(64 * v->waves), rargs, 0,
                                        stream));
        }
        if (cfg.variant == SYMTILE_BULK_SYNC && world_size > 1) {
            int c = cfg.copy_wgs > 0 ? cfg.copy_wgs : cus;
            c = std::min(c, ntiles);
            p.copy_wgs = c;
            SYMTILE_HIP(hipLaunchKernel(v->scatter, dim3(c), dim3(v->copy_threads), args, 0, stream));
        }
        return SYMTILE_OK;
    }

    if (cfg.variant == SYMTILE_WAVE_SPEC) {
        // One extra wave per workgroup copies finished tiles (Section 4.2.3).
        const Variant* ws = find_wave_spec_variant(cfg.tile_m, cfg.tile_n, dtype == SYMTILE_BF16);
        if (!ws)
            return fail(SYMTILE_EUNSUPPORTED, "wave specialisation is built for 256x128 tiles");
        int g = cfg.gemm_wgs > 0 ? cfg.gemm_wgs : std::min(ntiles, cus);
        g = std::min(g, ntiles);
        p.gemm_wgs = g;
        p.role = ROLE_WAVE_SPEC;
        void* args[] = {&p};
        SYMTILE_HIP(hipLaunchKernel(ws->gas_ws, dim3(g), dim3(64 * (ws->waves + 1)), args, 0,
                                    stream));
        return SYMTILE_OK;
    }

    if (cfg.variant == SYMTILE_UNFUSED_PC) {
        // Two grids side by side (Section 4.1.2): producers on `stream`,
        // consumers on the copy stream.  With g + c <= CU count the consumers
        // occupy at most c CUs, so g CUs stay free for the producers and the
        // consumers' waits always end.  Fork/join events keep the call's
        // stream semantics: the copy kernel starts after earlier work on
        // `stream`, and later work on `stream` waits for it.
        int c = cfg.copy_wgs > 0 ? cfg.copy_wgs : std::max(1, cus / 8);
        int g = cfg.gemm_wgs > 0 ? cfg.gemm_wgs : cus - c;
        if (g <= 0 || c <= 0)
            return fail(SYMTILE_EINVAL, "UNFUSED_PC needs gemm_wgs > 0 and copy_wgs > 0");
        if (g + c > cus)
            return fail(SYMTILE_EUNSUPPORTED,
                        "gemm_wgs + copy_wgs = " + std::to_string(g + c) + " exceeds the " +
                            std::to_string(cus) + " CUs the two grids partition");
        hipStream_t cs = static_cast<hipStream_t>(cfg.copy_stream);
        if (symtile_status st = symtile_host::aux_stream(h)) return st;
        if (!cs) cs = h->aux_stream;
        if (cs == stream) return fail(SYMTILE_EINVAL, "copy_stream is the call's stream");
        p.gemm_wgs = g;
        p.copy_wgs = std::min(c, ntiles);
        p.role = ROLE_WG_SPEC;
        void* args[] = {&p};
        SYMTILE_HIP(hipEventRecord(h->ev_fork, stream));
        SYMTILE_HIP(hipStreamWaitEvent(cs, h->ev_fork, 0));
        SYMTILE_HIP(hipLaunchKernel(v->gas, dim3(g), dim3(64 * v->waves), args, 0, stream));
        SYMTILE_HIP(hipLaunchKernel(v->consumer, dim3(p.copy_wgs), dim3(v->copy_threads),
                                    args, 0, cs));
        SYMTILE_HIP(hipEventRecord(h->ev_join, cs));
        SYMTILE_HIP(hipStreamWaitEvent(stream, h->ev_join, 0));
        return SYMTILE_OK;
    }

    // WG_SPEC: producers and consumers must all be resident at once.
    int c = cfg.copy_wgs > 0 ? cfg.copy_wgs : std::max(1, cus / 8);
    int g = cfg.gemm_wgs > 0 ? cfg.gemm_wgs : cus - c;
    if (g <= 0 || c <= 0) return fail(SYMTILE_EINVAL, "WG_SPEC needs gemm_wgs > 0 and copy_wgs > 0");
    if (g + c > limit)
        return fail(SYMTILE_EUNSUPPORTED,
                    "gemm_wgs + copy_wgs = " + std::to_string(g + c) +
                        " exceeds the co-resident limit " + std::to_string(limit));
    if (world_size == 1) c = std::min(c, ntiles);
    p.gemm_wgs = g;
    p.copy_wgs = c;
    p.role = ROLE_WG_SPEC;
    void* args[] = {&p};
    SYMTILE_HIP(hipLaunchKernel(v->gas, dim3(g + c), dim3(64 * v->waves), args, 0, stream));
    return SYMTILE_OK;
}

extern "C" symtile_status symtile_gemm_all_scatter_noalloc(
    symtile_heap* h, const void* A, const void* B_shard, void* C_gathered_local,
    uint32_t* arrived_local, uint32_t* ready, int M, int N_local, int K, int lda, int ldb,
    int dtype, int rank, int world_size, const symtile_gas_config* cfg_in, symtile_stream s) {
    using symtile_host::fail;
    if (!h) return fail(SYMTILE_EINVAL, "heap is NULL");
    symtile_gas_config cfg{};
    if (cfg_in) cfg = *cfg_in;
    if (cfg.workspace || cfg.workspace_bytes)
        return fail(SYMTILE_EINVAL, "the allocation-free call takes no workspace (it uses the "
                                    "library's scratch)");
    if (cfg.variant == SYMTILE_UNFUSED_PC)
        return fail(SYMTILE_EUNSUPPORTED, "UNFUSED_PC creates a stream and events on first use; "
                                          "the allocation-free call does not run it");
    if (cfg.split_k <= 1)
        return symtile_gemm_all_scatter(h, A, B_shard, C_gathered_local, arrived_local, ready, M,
                                        N_local, K, lda, ldb, dtype, rank, world_size, &cfg, s);
    if (cfg.tile_m == 0 && cfg.tile_n == 0) cfg.tile_m = cfg.tile_n = 256;
    size_t need = 0;
    if (symtile_status st =
            symtile_gas_workspace_bytes(M, N_local, cfg.tile_m, cfg.tile_n, cfg.split_k, &need))
        return st;
    if (need > (size_t)SYMTILE_NOALLOC_SCRATCH_BYTES)
        return fail(SYMTILE_EINVAL, "split-K workspace of " + std::to_string(need) +
                                        " bytes exceeds the scratch of " +
                                        std::to_string((size_t)SYMTILE_NOALLOC_SCRATCH_BYTES) +
                                        " bytes");
    if (need == 0)   // no tiles
        return symtile_gemm_all_scatter(h, A, B_shard, C_gathered_local, arrived_local, ready, M,
                                        N_local, K, lda, ldb, dtype, rank, world_size, &cfg, s);
    void* scratch = nullptr;
    if (symtile_status st = noalloc_scratch(h->device, &scratch)) return st;
    // the counters start at zero on every call, whatever an earlier call left
    const size_t tiles = (size_t)((M + cfg.tile_m - 1) / cfg.tile_m) *
                         ((N_local + cfg.tile_n - 1) / cfg.tile_n);
    const int words = (int)(sk_counter_bytes(tiles) / 4);
    int prev = -1;
    if (symtile_status st = symtile_host::set_device(h, &prev)) return st;
    hipLaunchKernelGGL(zero_words_kernel, dim3(std::min((words + 255) / 256, 1024)), dim3(256), 0,
                       static_cast<hipStream_t>(s), static_cast<uint32_t*>(scratch), words);
    const hipError_t e = hipGetLastError();
    if (prev >= 0) (void)hipSetDevice(prev);
    if (e != hipSuccess) return symtile_host::hip_fail(e, "zero_words_kernel launch");
    cfg.workspace = scratch;
    cfg.workspace_bytes = SYMTILE_NOALLOC_SCRATCH_BYTES;
    return symtile_gemm_all_scatter(h, A, B_shard, C_gathered_local, arrived_local, ready, M,
                                    N_local, K, lda, ldb, dtype, rank, world_size, &cfg, s);
}
