// Device-side primitives of the symmetric heap for gfx950 (header-only).
//
// These are the device verbs of Section 3.3 (device API table): pointer
// translation (3.3.1), value-based load/store and pointer-based tile copies
// (3.3.2), and atomics with an ordering and a scope (3.3.3).  Every verb
// takes the device array of per-rank heap bases.
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

// ---- per-tile flags ------------------------------------------------------
// Publication of a workgroup's stores, with one L2 write-back per workgroup:
//  1. wg_stores_done(), by every thread: the wave waits until its own
//     earlier memory operations are acknowledged (vmcnt 0, i.e. the stores
//     have reached the L2), then the workgroup meets at a barrier;
//  2. release_agent(), by one thread afterwards: an agent-scope release
//     fence, whose L2 write-back covers the stores of every wave of the
//     workgroup (they are all in this XCD's L2 by step 1);
//  3. flag_add(), by the same thread: relaxed agent-scope increments.  A
//     release fence followed by an atomic write synchronises with an
//     acquire that reads the written value.
// An agent-scope release per wave, or a release-ordered increment per
// counter, would each cost another full L2 write-back.
__device__ __forceinline__ void wg_stores_done() {
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0); expcnt and lgkmcnt not waited
    __syncthreads();
}

__device__ __forceinline__ void release_agent() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
}

__device__ __forceinline__ void flag_add(uint32_t* flag) {
    __hip_atomic_fetch_add(global_ptr(flag), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Bounded wait by one thread until *flag >= target.  Polls with relaxed
// agent-scope loads and a short sleep between polls; the caller follows a
// successful wait with an agent-scope acquire fence.  Returns false when
// spin_limit polls pass without success.
__device__ __forceinline__ bool flag_wait_geq(const uint32_t* flag, uint32_t target,
                                              uint32_t spin_limit) {
    for (uint32_t n = 0; n < spin_limit; ++n) {
        uint32_t v = __hip_atomic_load(global_ptr(flag), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (v >= target) return true;
        __builtin_amdgcn_s_sleep(1);
    }
    return false;
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
enum : uint32_t { ERR_TIMEOUT = 1u };

__device__ __forceinline__ void raise_error(uint32_t* err, uint32_t code) {
    __hip_atomic_fetch_or(global_ptr(err), code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

}  // namespace symtile
