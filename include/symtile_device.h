// Device-side API of the symmetric heap for gfx950 (header-only).
//
// The device verbs of Section 3.3 (device API table), for kernels that work
// on the heap; every verb takes the device array of per-rank heap bases:
//   * translate (3.3.1): the same offset in another rank's heap;
//   * value-based load / store (3.3.2) of 16-byte vectors and of tile rows;
//   * pointer-based put / get / copy (3.3.2) of whole tiles, performed by
//     the threads of one workgroup together;
//   * atomic_{add,xchg,cas,and,or,xor,min,max}<SEM, SCOPE> (3.3.3);
//   * per-tile flags (the producer/consumer handshake of Section 4.2.2):
//     flag_publish (release, then +1) and flag_wait (bounded wait, then
//     acquire).
//
// Memory-model notes (LLVM AMDGPU memory model for gfx9.4/9.5 family):
// the L2 is private to each XCD, so publishing data to a workgroup on any
// other XCD needs agent-scope release (the compiler emits the L2 write-back)
// and the reader needs agent-scope acquire (L2 invalidate).  Everything
// here goes through __hip_atomic_* and __builtin_amdgcn_fence; no cache
// maintenance is written by hand.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace symtile {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---- translation (Section 3.3.1) -----------------------------------------
// p points into the slot of from_rank; the result is the same offset inside
// the slot of to_rank: bases[to] + (p - bases[from]), in bytes.
__device__ __forceinline__ uint64_t translate_addr(uint64_t p, int from_rank, int to_rank,
                                                   const uint64_t* __restrict__ bases) {
    return bases[to_rank] + (p - bases[from_rank]);
}

template <class T>
__device__ __forceinline__ T* translate(T* p, int from_rank, int to_rank,
                                        const uint64_t* __restrict__ bases) {
    return reinterpret_cast<T*>(
        translate_addr(reinterpret_cast<uint64_t>(p), from_rank, to_rank, bases));
}

// ---- value-based 16-byte access (Section 3.3.2) ----------------------------
__device__ __forceinline__ u32x4 ld16(const void* p) {
    return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ void st16(void* p, u32x4 v, bool nontemporal) {
    if (nontemporal)
        __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
    else
        *reinterpret_cast<u32x4*>(p) = v;
}

// load: read 16 bytes at p's counterpart in the heap of `remote`.
__device__ __forceinline__ u32x4 load(const void* p, int cur, int remote,
                                      const uint64_t* __restrict__ bases) {
    return ld16(translate(p, cur, remote, bases));
}

// store: write 16 bytes to p's counterpart in the heap of `remote`.
__device__ __forceinline__ void store(void* p, u32x4 v, int cur, int remote,
                                      const uint64_t* __restrict__ bases, bool nt) {
    st16(translate(p, cur, remote, bases), v, nt);
}

// ---- buffer resources ----------------------------------------------------
// A raw buffer resource covers [base, base + bytes); a load whose offset
// falls outside returns zero and a store there is dropped.  The kernels use
// this instead of branches for ragged edges: an invalid lane gets kOOB as
// its offset.  All resources here stay below 2^31 bytes, so kOOB plus any
// scalar offset used is outside every resource.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;

// The resource must be the same for every lane of the wave (all uses here
// are per tile and per slot).  Its base and size are read through
// readfirstlane so the descriptor lives in scalar registers even when the
// compiler cannot prove uniformity (e.g. a base loaded from the bases array);
// a descriptor in vector registers would turn every buffer access into a
// loop over distinct descriptor values.
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    void* ub = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
    // dword 3 = 0x00020000: 32-bit data format, no swizzle, no index stride
    return __builtin_amdgcn_make_buffer_rsrc(ub, (short)0,
                                             (int)__builtin_amdgcn_readfirstlane(bytes),
                                             0x00020000);
}

// The scalar offset `soff` must be the same in every lane of the wave (it is
// an SGPR operand); it is made uniform explicitly so that the compiler never
// wraps the access in a per-lane loop when it cannot prove it.
__device__ __forceinline__ u32x4 buf_ld16(rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, voff, __builtin_amdgcn_readfirstlane(soff), 0);
}

// Store cache policies (the cache-policy bits of the gfx9.4/9.5 store):
//   kStoreDefault      write-back in the L2;
//   kStoreNonTemporal  nt: streaming hint, the line is a preferred victim;
//   kStoreWriteThrough sc0 sc1: system-scope coherence, written through the
//                      L2 to memory (measured best for the cold heap copy,
//                      where the destination is not read again soon).
enum : int { kStoreDefault = 0, kStoreNonTemporal = 2, kStoreWriteThrough = 17 };

// Load cache policies: kLoadDefault may hit a line this XCD's L2 holds from
// before; kLoadCoherent (sc0 sc1, the encoding the memory model gives a
// system-scope relaxed atomic load) reads the value that is coherent for
// every XCD, not a copy the L2 kept.
enum : int { kLoadDefault = 0, kLoadCoherent = 17 };

template <int POLICY>
__device__ __forceinline__ u32x4 buf_ld16p(rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, voff, __builtin_amdgcn_readfirstlane(soff),
                                                 POLICY);
}

template <int POLICY>
__device__ __forceinline__ void buf_st16p(u32x4 v, rsrc_t r, uint32_t voff, uint32_t soff) {
    __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, __builtin_amdgcn_readfirstlane(soff),
                                           POLICY);
}

// Descriptor words of the same buffer resource, for inline assembly.
typedef int i32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4_t make_rsrc_words(const void* base, uint32_t bytes) {
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    return i32x4_t{(int)__builtin_amdgcn_readfirstlane((uint32_t)b),
                   (int)(__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32)) & 0xFFFFu),
                   (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000};
}

// 16 bytes per lane from the buffer straight into LDS (lane l writes
// lds_addr + 16 * l), issued from inline assembly so that the compiler does
// not track it.  The compiler cannot tell which LDS bytes a direct-to-LDS
// load writes, so for a tracked one it drains every such load before any
// later LDS read, including reads of other pipeline stages; with this form
// the caller orders the load itself: s_waitcnt vmcnt, then a barrier, before
// any wave reads the bytes.  M0 carries the LDS address; it is an input
// operand, so the compiler writes it and knows it is in use.  The compiler's
// hazard recognizer does not look inside inline assembly, so the statement
// provides the wait states itself: a VALU write of an SGPR (readfirstlane,
// or readlane when the compiler reloads a spilled SGPR) needs 5 wait states
// before a vector memory instruction reads that SGPR (offset or descriptor),
// and writing M0 needs 1 before the load reads it; s_nop 4 gives 5.
__device__ __forceinline__ void buf_ld16_lds_async(const i32x4_t& r, uint32_t lds_addr,
                                                   uint32_t voff, uint32_t soff) {
    asm volatile(
        "s_nop 4\n\t"
        "buffer_load_dwordx4 %0, %1, %2 offen lds"
        :
        : "v"(voff), "s"(r), "s"(__builtin_amdgcn_readfirstlane(soff)),
          "{m0}"(__builtin_amdgcn_readfirstlane(lds_addr))
        : "memory");
}

// LDS byte address of a pointer into __shared__ memory.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Every pointer in the heap is device (global) memory.  Atomics through a
// generic pointer compile to flat instructions, which count on both the
// vector-memory and the LDS counters; while one is outstanding the compiler
// can only wait for LDS reads with a full drain.  Casting to the global
// address space keeps LDS waits exact.
template <typename T>
__device__ __forceinline__ __attribute__((address_space(1))) T* global_ptr(T* p) {
    return (__attribute__((address_space(1))) T*)p;
}

// ---- atomics with ordering and scope (Section 3.3.3) ----------------------
// SEM is a __ATOMIC_* order, SCOPE a __HIP_MEMORY_SCOPE_* constant.
template <int SEM, int SCOPE>
__device__ __forceinline__ uint32_t atomic_add(uint32_t* p, uint32_t v) {
    return __hip_atomic_fetch_add(global_ptr(p), v, SEM, SCOPE);
}
template <int SEM, int SCOPE>
__device__ __forceinline__ uint32_t atomic_xchg(uint32_t* p, uint32_t v) {
    return __hip_atomic_exchange(global_ptr(p), v, SEM, SCOPE);
}
template <int SEM, int SCOPE>
__device__ __forceinline__ uint32_t atomic_cas(uint32_t* p, uint32_t expected, uint32_t desired) {
    // failure order: the strongest of relaxed/acquire not above SEM
    constexpr int FAIL = (SEM == __ATOMIC_ACQUIRE || SEM == __ATOMIC_ACQ_REL) ? __ATOMIC_ACQUIRE
                                                                              : __ATOMIC_RELAXED;
    __hip_atomic_compare_exchange_strong(global_ptr(p), &expected, desired, SEM, FAIL, SCOPE);
    return expected;   // the value observed
}
template <int SEM, int SCOPE>
__device__ __forceinline__ uint32_t atomic_and(uint32_t* p, uint32_t v) {
    return __hip_atomic_fetch_and(global_ptr(p), v, SEM, SCOPE);
}
template <int SEM, int SCOPE>
__device__ __forceinline__ uint32_t atomic_or(uint32_t* p, uint32_t v) {
    return __hip_atomic_fetch_or(global_ptr(p), v, SEM, SCOPE);
}
template <int SEM, int SCOPE>
__device__ __forceinline__ uint32_t atomic_xor(uint32_t* p, uint32_t v) {
    return __hip_atomic_fetch_xor(global_ptr(p), v, SEM, SCOPE);
}
template <int SEM, int SCOPE>
__device__ __forceinline__ uint32_t atomic_min(uint32_t* p, uint32_t v) {
    return __hip_atomic_fetch_min(global_ptr(p), v, SEM, SCOPE);
}
template <int SEM, int SCOPE>
__device__ __forceinline__ uint32_t atomic_max(uint32_t* p, uint32_t v) {
    return __hip_atomic_fetch_max(global_ptr(p), v, SEM, SCOPE);
}

// ---- fences at a scope (Section 3.3.3, memory model) ----------------------
// SCOPE is a __HIP_MEMORY_SCOPE_* constant (WORKGROUP = the paper's block,
// AGENT = gpu, SYSTEM = sys).
template <int SCOPE>
__device__ __forceinline__ void fence_release() {
    if constexpr (SCOPE == __HIP_MEMORY_SCOPE_WORKGROUP)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    else if constexpr (SCOPE == __HIP_MEMORY_SCOPE_AGENT)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    else
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
}

template <int SCOPE>
__device__ __forceinline__ void fence_acquire() {
    if constexpr (SCOPE == __HIP_MEMORY_SCOPE_WORKGROUP)
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    else if constexpr (SCOPE == __HIP_MEMORY_SCOPE_AGENT)
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    else
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
}

// ---- per-tile flags (Section 4.2.2 handshake, Section 3.3.3 orderings) -----
// Flags are uint32 counters rather than locks: a publication adds 1, a
// waiter waits until the counter reaches the value it expects (the call's
// epoch), and nothing resets them inside a kernel, so a tile published twice
// reads 2.
//
// flag_publish<SCOPE>(flag), by one thread: a release fence at SCOPE, then a
// relaxed +1 at SCOPE.  A release fence followed by an atomic write
// synchronises with an acquire that reads the value written, so whatever
// was visible to the thread before the fence is visible to the waiter after
// its acquire.
//
// A workgroup publishing its stores: every thread calls wg_stores_done()
// (each wave waits for the acknowledgement of its own stores, i.e. they have
// reached this XCD's L2, then the workgroup meets at a barrier), then one
// thread calls flag_publish.  Further counters covered by the same release
// take flag_signal (the relaxed +1 alone; the lanes of one wave may signal
// different counters together), so a workgroup pays one L2 write-back however
// many counters it publishes.  An agent-scope release per wave, or a
// release-ordered increment per counter, would each cost another write-back.
__device__ __forceinline__ void wg_stores_done() {
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0); expcnt and lgkmcnt not waited
    __syncthreads();
}

// Release of write-through stores.  An agent- or system-scope release fence
// writes back the XCD's L2 (buffer_wbl2), because ordinary stores may sit
// dirty in it; that write-back costs about as much whether or not anything
// is dirty, and the write-backs of one XCD's workgroups run one after
// another.  Stores issued with kStoreWriteThrough carry the system-coherence
// bits (sc0 sc1), the same encoding the memory model gives a system-scope
// relaxed atomic store: they leave no dirty line, and their acknowledgement
// (vmcnt) comes back once they are coherent for every XCD.  For data written
// only that way, waiting for the acknowledgements is the whole release: the
// caller has already waited for them (wg_stores_done), and this adds the
// compiler barrier that keeps the counter update after the stores.  The
// reader still acquires (flag_wait), which invalidates its own L2's copies.
// Covers only stores this workgroup made with kStoreWriteThrough; any other
// store that the reader must see needs fence_release.  The message-passing
// litmus test exercises exactly this form (symtile_litmus_mp, SYMTILE_MP_WT).
__device__ __forceinline__ void release_written_through() {
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    asm volatile("" ::: "memory");
}

template <int SCOPE = __HIP_MEMORY_SCOPE_AGENT>
__device__ __forceinline__ void flag_signal(uint32_t* flag) {
    __hip_atomic_fetch_add(global_ptr(flag), 1u, __ATOMIC_RELAXED, SCOPE);
}

template <int SCOPE = __HIP_MEMORY_SCOPE_AGENT>
__device__ __forceinline__ void flag_publish(uint32_t* flag) {
    fence_release<SCOPE>();
    flag_signal<SCOPE>(flag);
}

// Acquire for data read with kLoadCoherent only, the mirror of
// release_written_through: an agent- or system-scope acquire fence
// invalidates the XCD's L2 (and the CU's L1) so that later ordinary loads
// miss copies of lines that another XCD has since rewritten; like the
// write-back, the invalidate costs about the same whatever the L2 holds, and
// one XCD's run one after another.  Loads issued with kLoadCoherent do not
// take such copies, so after a poll that saw the counter the acquire needs
// only the order of the accesses: the poll's value is waited for (its
// result decides the branch) and the compiler barrier keeps the data loads
// after it.  Covers only loads made with kLoadCoherent; other loads of the
// published data need fence_acquire.  Litmus: SYMTILE_MP_WT_COHERENT.
__device__ __forceinline__ void acquire_coherent_reads() {
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): the poll has returned
    asm volatile("" ::: "memory");
}

// flag_publish for data written with kStoreWriteThrough only (see
// release_written_through).
template <int SCOPE = __HIP_MEMORY_SCOPE_AGENT>
__device__ __forceinline__ void flag_publish_written_through(uint32_t* flag) {
    release_written_through();
    flag_signal<SCOPE>(flag);
}

// Bounded poll by one thread until *flag >= target: relaxed loads at SCOPE
// with a short sleep between them.  Returns false when spin_limit polls pass
// without success.  Orders nothing by itself.
template <int SCOPE = __HIP_MEMORY_SCOPE_AGENT>
__device__ __forceinline__ bool flag_poll(const uint32_t* flag, uint32_t target,
                                          uint32_t spin_limit) {
    for (uint32_t n = 0; n < spin_limit; ++n) {
        const uint32_t v = __hip_atomic_load(global_ptr(flag), __ATOMIC_RELAXED, SCOPE);
        if (v >= target) return true;
        __builtin_amdgcn_s_sleep(1);
    }
    return false;
}

// flag_wait: flag_poll, then on success an acquire fence at SCOPE, so the
// publisher's data is visible to the caller.  Returns false (and acquires
// nothing) on timeout; callers record ERR_TIMEOUT and give up on the tile.
// Other threads of the workgroup see the data after a barrier that follows.
template <int SCOPE = __HIP_MEMORY_SCOPE_AGENT>
__device__ __forceinline__ bool flag_wait(const uint32_t* flag, uint32_t target,
                                          uint32_t spin_limit) {
    if (!flag_poll<SCOPE>(flag, target, spin_limit)) return false;
    fence_acquire<SCOPE>();
    return true;
}

// flag_wait for data read with kLoadCoherent only: flag_poll, then on
// success acquire_coherent_reads instead of the L2-invalidating fence.
template <int SCOPE = __HIP_MEMORY_SCOPE_AGENT>
__device__ __forceinline__ bool flag_wait_coherent(const uint32_t* flag, uint32_t target,
                                                   uint32_t spin_limit) {
    if (!flag_poll<SCOPE>(flag, target, spin_limit)) return false;
    acquire_coherent_reads();
    return true;
}

// ---- pointer-based tile moves (Section 3.3.2: get, put, copy) ---------------
// A tile is `rows` rows of `chunks` 16-byte chunks with a row stride of
// ld_bytes, named by its address in the heap of the executing rank (cur).
// The threads of one workgroup move it together: a pass covers
// `threads >> lg_w` rows, and inside a pass 1 << lg_w consecutive threads
// take the consecutive 16-byte chunks of one row (1 << lg_w >= chunks; the
// threads of columns past the row stay idle), so every wave access covers
// whole cache lines.  The tile's bytes lie in one buffer resource, so a
// tile spans less than 2 GiB; rows past the last one lie outside it.
struct TileGeom {
    int rows;            // rows of the tile
    int chunks;          // 16-byte chunks per row
    uint32_t ld_bytes;   // row stride in bytes (>= 16 * chunks)
    int lg_w;            // log2 of the threads per row in a pass
};

// Bytes from the tile's first byte to one past its last.
__device__ __forceinline__ uint32_t tile_bytes(const TileGeom& g) {
    return g.rows > 0 ? (uint32_t)((size_t)(g.rows - 1) * g.ld_bytes + (size_t)g.chunks * 16) : 0u;
}

// This thread's part of a tile move.
struct TileLanes {
    uint32_t voff;        // byte offset of the thread's chunk in pass 0, or kOOB
    uint32_t pass_bytes;  // bytes between passes
    int passes;           // passes that cover the rows
};

__device__ __forceinline__ TileLanes tile_lanes(const TileGeom& g, int tid, int threads) {
    const int c = tid & ((1 << g.lg_w) - 1);
    const int rp = threads >> g.lg_w;
    TileLanes L;
    L.voff = c < g.chunks ? (uint32_t)((tid >> g.lg_w) * g.ld_bytes + c * 16) : kOOB;
    L.pass_bytes = (uint32_t)rp * g.ld_bytes;
    L.passes = (g.rows + rp - 1) / rp;
    return L;
}

// A buffer resource over the tile at p (an address in cur's heap) as it lies
// in the heap of `rank`: the target of value-based loads and stores of tile
// rows (Section 3.3.2, load and store), one resource per tile and rank.
__device__ __forceinline__ rsrc_t tile_rsrc(const void* p, const TileGeom& g, int cur, int rank,
                                            const uint64_t* __restrict__ bases) {
    return make_rsrc(translate(p, cur, rank, bases), tile_bytes(g));
}

// Move every pass of a tile from resource rs to rd, BATCH passes per batch,
// software-pipelined: the loads of batch i+1 are issued before the stores of
// batch i.  Loads and stores share one in-order completion counter, so in
// the plain order (load i, store i, load i+1) the wait for batch i+1's data
// would also wait for batch i's store acknowledgements; in this order the
// wait before storing batch i leaves the newer loads and stores in flight.
// Passes past the last one lie outside the resources (zero loads, dropped
// stores).  The loop body has no branch, so the compiler's waits stay exact.
template <int POLICY, int BATCH>
__device__ __forceinline__ void move_tile(rsrc_t rs, rsrc_t rd, const TileLanes& L) {
    const int nb = (L.passes + BATCH - 1) / BATCH;
    if (nb <= 0) return;
    u32x4 x[BATCH], y[BATCH];      // batches alternate between x and y (no register moves)
    auto load = [&](u32x4 (&v)[BATCH], int batch) {
#pragma unroll
        for (int u = 0; u < BATCH; ++u)
            v[u] = buf_ld16(rs, L.voff, (uint32_t)(batch * BATCH + u) * L.pass_bytes);
    };
    auto store = [&](const u32x4 (&v)[BATCH], int batch) {
#pragma unroll
        for (int u = 0; u < BATCH; ++u)
            buf_st16p<POLICY>(v[u], rd, L.voff, (uint32_t)(batch * BATCH + u) * L.pass_bytes);
    };
    load(x, 0);
    int i = 0;
    for (; i + 2 < nb; i += 2) {     // batch i in x; batches i+1, i+2 exist
        load(y, i + 1);
        store(x, i);
        load(x, i + 2);
        store(y, i + 1);
    }
    if (i + 1 < nb) {
        load(y, i + 1);
        store(x, i);
        store(y, i + 1);
    } else {
        store(x, i);
    }
}

// copy: the tile at src as it lies in from_rank's heap, to the tile at dst
// as it lies in to_rank's heap (both addresses named in cur's heap).  Every
// thread of the workgroup (threads of them) calls it; it returns when this
// thread's stores are issued, not acknowledged (see wg_stores_done).
template <int POLICY = kStoreDefault, int BATCH = 8>
__device__ __forceinline__ void copy(const void* src, void* dst, const TileGeom& g, int from_rank,
                                     int to_rank, int cur, const uint64_t* __restrict__ bases,
                                     int tid, int threads) {
    move_tile<POLICY, BATCH>(tile_rsrc(src, g, cur, from_rank, bases),
                             tile_rsrc(dst, g, cur, to_rank, bases), tile_lanes(g, tid, threads));
}

// put: from the executing rank's own heap to `remote`'s (the write is remote).
template <int POLICY = kStoreDefault, int BATCH = 8>
__device__ __forceinline__ void put(const void* src, void* dst, const TileGeom& g, int cur,
                                    int remote, const uint64_t* __restrict__ bases, int tid,
                                    int threads) {
    copy<POLICY, BATCH>(src, dst, g, cur, remote, cur, bases, tid, threads);
}

// get: from `remote`'s heap into the executing rank's own (the read is remote).
template <int POLICY = kStoreDefault, int BATCH = 8>
__device__ __forceinline__ void get(const void* src, void* dst, const TileGeom& g, int cur,
                                    int remote, const uint64_t* __restrict__ bases, int tid,
                                    int threads) {
    copy<POLICY, BATCH>(src, dst, g, remote, cur, cur, bases, tid, threads);
}

// put to several ranks: the tile at p in the executing rank's heap, read
// once, is written to the same place in the heaps of ranks (cur + d) mod
// world for d in [d0, d1) -- the consumer copy of the producer/consumer
// schedules, which sends a finished tile to every other rank.  U passes are
// loaded (with load policy LOAD), then stored to each rank in turn.
template <int POLICY, int U, int LOAD = kLoadDefault>
__device__ __forceinline__ void put_ranks(const void* p, const TileGeom& g, int cur, int d0,
                                          int d1, int world, const uint64_t* __restrict__ bases,
                                          int tid, int threads) {
    const TileLanes L = tile_lanes(g, tid, threads);
    const rsrc_t rs = make_rsrc(p, tile_bytes(g));
#pragma unroll 1
    for (int b = 0; b < L.passes; b += U) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            v[u] = buf_ld16p<LOAD>(rs, L.voff, (uint32_t)(b + u) * L.pass_bytes);
        for (int d = d0; d < d1; ++d) {
            const rsrc_t rd = tile_rsrc(p, g, cur, (cur + d) % world, bases);
#pragma unroll
            for (int u = 0; u < U; ++u)
                buf_st16p<POLICY>(v[u], rd, L.voff, (uint32_t)(b + u) * L.pass_bytes);
        }
    }
}

// ---- per-tile trace (Section 3.4, instrumentation) -----------------------
// Timestamps come from the device's constant-rate realtime counter (100 MHz
// on this GPU family; the rate is the HIP wall-clock rate attribute), which
// every CU reads from the same source, so times taken by different
// workgroups compare directly.
__device__ __forceinline__ uint64_t clock_now() { return __builtin_amdgcn_s_memrealtime(); }

// Where the calling wave runs: the raw HW_ID register in the high 32 bits,
// XCC_ID in bits 16-31 and the workgroup id in bits 0-15.
__device__ __forceinline__ uint64_t trace_location() {
    const uint32_t hw = __builtin_amdgcn_s_getreg(4 | (31 << 11));    // HW_REG_HW_ID
    const uint32_t xcc = __builtin_amdgcn_s_getreg(20 | (15 << 11));  // HW_REG_XCC_ID
    return ((uint64_t)hw << 32) | ((uint64_t)(xcc & 0xFFFFu) << 16) | (blockIdx.x & 0xFFFFu);
}

// Device error word codes (OR-ed into the heap's error word).
//   ERR_TIMEOUT    a bounded wait expired;
//   ERR_WORKSPACE  a split-K slice (or band of the reduction kernel) drew a
//                  ticket beyond its count, or found the other counter
//                  non-zero: the workspace counters were not zero when the
//                  call started (a timed-out call leaves them so).
enum : uint32_t { ERR_TIMEOUT = 1u, ERR_WORKSPACE = 2u };

__device__ __forceinline__ void raise_error(uint32_t* err, uint32_t code) {
    __hip_atomic_fetch_or(global_ptr(err), code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

}  // namespace symtile
