// Symmetric heap, translation, barrier, fill and the atomic exercise kernel.
//
// The heap follows the constructor of Section 3.2 for one process on one
// GPU: step 3 (allocate the heap on the device) and step 6 (a device array
// of every rank's heap base).  Steps 1, 2, 4 and 5 (process group, device
// per rank, IPC handle exchange and opening) have nothing to do when every
// rank's heap is a slot of one allocation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdio>
#include <cstring>
#include <string>

#include "symtile.h"
#include "symtile_device.h"
#include "symtile_internal.h"

namespace {

thread_local std::string g_last_error;

constexpr size_t kSlotAlign = size_t(2) << 20;   // 2 MiB
constexpr size_t kControlBytes = 256;            // bases[8] + error word + spare

struct DeviceGuard {
    int prev = -1;
    bool ok = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) return;
        ok = hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

__global__ void translate_kernel(const uint64_t* __restrict__ in, int n, int from_rank,
                                 int to_rank, const uint64_t* __restrict__ bases,
                                 uint64_t* __restrict__ out) {
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) out[i] = symtile::translate_addr(in[i], from_rank, to_rank, bases);
}

__global__ void fill16_kernel(symtile::u32x4* __restrict__ p, size_t n16, uint32_t word) {
    symtile::u32x4 v = {word, word, word, word};
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n16;
         i += (size_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void fill1_kernel(uint8_t* __restrict__ p, size_t n, uint8_t value) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x)
        p[i] = value;
}

// Value verbs (Section 3.3.2): one 16-byte vector per thread.  `own` is the
// executing rank's slot base; the remote side is reached by translation.
__global__ void value_exercise_kernel(char* own, const uint64_t* __restrict__ bases, int op,
                                      int cur, int remote, uint64_t src_off, uint64_t dst_off,
                                      size_t n16, int nontemporal) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n16;
         i += (size_t)gridDim.x * blockDim.x) {
        char* src = own + src_off + 16 * i;
        char* dst = own + dst_off + 16 * i;
        if (op == SYMTILE_LOAD) {
            symtile::st16(dst, symtile::load(src, cur, remote, bases), nontemporal != 0);
        } else {
            symtile::store(dst, symtile::ld16(src), cur, remote, bases, nontemporal != 0);
        }
    }
}

// One atomic verb with compile-time order and scope.
template <int SEM, int SCOPE>
__device__ uint32_t apply_atomic(int op, uint32_t* p, uint32_t v, uint32_t cmp) {
    switch (op) {
        case SYMTILE_ATOMIC_ADD: return symtile::atomic_add<SEM, SCOPE>(p, v);
        case SYMTILE_ATOMIC_XCHG: return symtile::atomic_xchg<SEM, SCOPE>(p, v);
        case SYMTILE_ATOMIC_CAS: return symtile::atomic_cas<SEM, SCOPE>(p, cmp, v);
        case SYMTILE_ATOMIC_AND: return symtile::atomic_and<SEM, SCOPE>(p, v);
        case SYMTILE_ATOMIC_OR: return symtile::atomic_or<SEM, SCOPE>(p, v);
        case SYMTILE_ATOMIC_XOR: return symtile::atomic_xor<SEM, SCOPE>(p, v);
        case SYMTILE_ATOMIC_MIN: return symtile::atomic_min<SEM, SCOPE>(p, v);
        default: return symtile::atomic_max<SEM, SCOPE>(p, v);
    }
}

template <int SCOPE>
__device__ uint32_t apply_sem(int op, int sem, uint32_t* p, uint32_t v, uint32_t cmp) {
    switch (sem) {
        case SYMTILE_RELAXED: return apply_atomic<__ATOMIC_RELAXED, SCOPE>(op, p, v, cmp);
        case SYMTILE_ACQUIRE: return apply_atomic<__ATOMIC_ACQUIRE, SCOPE>(op, p, v, cmp);
        case SYMTILE_RELEASE: return apply_atomic<__ATOMIC_RELEASE, SCOPE>(op, p, v, cmp);
        default: return apply_atomic<__ATOMIC_ACQ_REL, SCOPE>(op, p, v, cmp);
    }
}

__global__ void atomic_exercise_kernel(uint32_t* local_word, int from_rank, int to_rank,
                                       const uint64_t* __restrict__ bases, int op, int sem,
                                       int scope, int n, uint32_t operand, uint32_t compare,
                                       uint32_t* __restrict__ old_out) {
    int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n) return;
    uint32_t* p = symtile::translate(local_word, from_rank, to_rank, bases);
    uint32_t v = operand + (uint32_t)t;
    uint32_t old;
    switch (scope) {
        case SYMTILE_SCOPE_BLOCK:
            old = apply_sem<__HIP_MEMORY_SCOPE_WORKGROUP>(op, sem, p, v, compare);
            break;
        case SYMTILE_SCOPE_GPU:
            old = apply_sem<__HIP_MEMORY_SCOPE_AGENT>(op, sem, p, v, compare);
            break;
        default:
            old = apply_sem<__HIP_MEMORY_SCOPE_SYSTEM>(op, sem, p, v, compare);
            break;
    }
    if (old_out) old_out[t] = old;
}

symtile_status check_heap(const symtile_heap* h) {
    if (!h) return symtile_host::fail(SYMTILE_EINVAL, "heap is NULL");
    return SYMTILE_OK;
}

symtile_status build_heap(int device, int world, size_t slot_bytes, void* base,
                          size_t total_bytes, bool owns, symtile_heap** out) {
    if (!out) return symtile_host::fail(SYMTILE_EINVAL, "out is NULL");
    *out = nullptr;
    if (world < 1 || world > SYMTILE_MAX_WORLD)
        return symtile_host::fail(SYMTILE_EINVAL, "world_size must be in [1, 8]");
    if (slot_bytes == 0) return symtile_host::fail(SYMTILE_EINVAL, "slot_bytes is 0");
    int ndev = 0;
    SYMTILE_HIP(hipGetDeviceCount(&ndev));
    if (device < 0 || device >= ndev)
        return symtile_host::fail(SYMTILE_EINVAL, "device " + std::to_string(device) +
                                                      " out of range");
    DeviceGuard guard(device);
    if (!guard.ok) return symtile_host::fail(SYMTILE_EHIP, "hipSetDevice failed");
    if (slot_bytes > (SIZE_MAX - kSlotAlign) / SYMTILE_MAX_WORLD)
        return symtile_host::fail(SYMTILE_EINVAL, "slot_bytes too large");
    const size_t stride = (slot_bytes + kSlotAlign - 1) / kSlotAlign * kSlotAlign;
    const size_t need = stride * (size_t)world;

    uint8_t* mem = static_cast<uint8_t*>(base);
    if (owns) {
        hipError_t e = hipMalloc(reinterpret_cast<void**>(&mem), need);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return symtile_host::fail(SYMTILE_ENOMEM, "hipMalloc of " + std::to_string(need) +
                                                          " bytes failed: " +
                                                          hipGetErrorString(e));
        }
        e = hipMemset(mem, 0, need);
        if (e != hipSuccess) {
            (void)hipFree(mem);
            return symtile_host::hip_fail(e, "hipMemset(heap)");
        }
    } else {
        if (!mem) return symtile_host::fail(SYMTILE_EINVAL, "base is NULL");
        if (reinterpret_cast<uintptr_t>(mem) % 256)
            return symtile_host::fail(SYMTILE_EINVAL, "base must be 256-byte aligned");
        if (total_bytes < need)
            return symtile_host::fail(SYMTILE_EINVAL,
                                      "external memory smaller than world * slot stride (" +
                                          std::to_string(need) + " bytes)");
    }
    void* control = nullptr;
    hipError_t e = hipMalloc(&control, kControlBytes);
    if (e != hipSuccess) {
        if (owns) (void)hipFree(mem);
        (void)hipGetLastError();
        return symtile_host::fail(SYMTILE_ENOMEM, "hipMalloc(control block) failed");
    }
    symtile_heap* h = new symtile_heap();
    h->device = device;
    h->world = world;
    h->slot_stride = stride;
    h->used = 0;
    h->owns_memory = owns;
    h->base = mem;
    std::memset(h->host_bases, 0, sizeof h->host_bases);
    for (int r = 0; r < world; ++r)
        h->host_bases[r] = reinterpret_cast<uint64_t>(mem) + (uint64_t)r * stride;
    h->control = control;
    h->dev_bases = static_cast<uint64_t*>(control);
    h->dev_err = reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(control) + 64);
    unsigned char host_control[kControlBytes];
    std::memset(host_control, 0, sizeof host_control);
    std::memcpy(host_control, h->host_bases, sizeof h->host_bases);
    e = hipMemcpy(control, host_control, kControlBytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        symtile_heap_destroy(h);
        return symtile_host::hip_fail(e, "hipMemcpy(control block)");
    }
    *out = h;
    return symtile_host::ok();
}

}  // namespace

namespace symtile_host {

symtile_status fail(symtile_status st, const std::string& msg) {
    g_last_error = msg;
    return st;
}

symtile_status ok() { return SYMTILE_OK; }

symtile_status hip_fail(hipError_t e, const char* what) {
    g_last_error = std::string(what) + ": " + hipGetErrorString(e);
    return SYMTILE_EHIP;
}

bool in_slot(const symtile_heap* h, const void* p, size_t bytes, int rank) {
    if (!h || rank < 0 || rank >= h->world) return false;
    const uint64_t a = reinterpret_cast<uint64_t>(p);
    const uint64_t lo = h->host_bases[rank];
    const uint64_t hi = lo + h->slot_stride;
    return a >= lo && a <= hi && bytes <= hi - a;
}

symtile_status set_device(const symtile_heap* h, int* previous) {
    int cur = -1;
    SYMTILE_HIP(hipGetDevice(&cur));
    if (previous) *previous = cur == h->device ? -1 : cur;
    if (cur != h->device) SYMTILE_HIP(hipSetDevice(h->device));
    return SYMTILE_OK;
}

symtile_status aux_stream(symtile_heap* h) {
    if (!h->aux_stream)
        SYMTILE_HIP(hipStreamCreateWithFlags(&h->aux_stream, hipStreamNonBlocking));
    if (!h->ev_fork) SYMTILE_HIP(hipEventCreateWithFlags(&h->ev_fork, hipEventDisableTiming));
    if (!h->ev_join) SYMTILE_HIP(hipEventCreateWithFlags(&h->ev_join, hipEventDisableTiming));
    return SYMTILE_OK;
}

int cu_count(int device) {
    // a device's CU count does not change: read once per device
    static std::atomic<int> known[64];
    if (device >= 0 && device < 64) {
        const int n = known[device].load(std::memory_order_relaxed);
        if (n > 0) return n;
    }
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess)
        return 0;
    if (device >= 0 && device < 64) known[device].store(n, std::memory_order_relaxed);
    return n;
}

}  // namespace symtile_host


// Message-passing litmus test of the flag protocol (Section 3.3.3, memory
// model): pair p = workgroups 2p (writer, rank p % w) and 2p+1 (reader, rank
// (p + 1) % w); consecutive workgroup ids land on different XCDs, whose L2s
// are not coherent with each other.  Round i: the writer waits until
// ack == i-1, writes the round's pattern into the reader's slot, waits for its
// stores and publishes ready = i; the reader waits until ready == i, checks
// every word, counts mismatches, and publishes ack = i in the writer's slot.
// The data words are plain loads, and plain stores except in the WT form.  How the counters publish and wait is the form:
//   RELAXED  relaxed +1, relaxed polls, no fences: the unsynchronised form
//            the protocol exists to prevent;
//   FENCES   release fence at SCOPE then relaxed +1; relaxed polls then an
//            acquire fence at SCOPE (the kernels' protocol);
//   RMW      the ordering carried by the read-modify-writes themselves:
//            fetch_add(+1, release, SCOPE) publishes, fetch_add(0, acquire,
//            SCOPE) polls;
//   CAS      the lock handshake of the workgroup-specialised listing:
//            cas(i-1 -> i, release, SCOPE) publishes, cas(i -> i, acquire,
//            SCOPE) polls until it observes i;
//   WT       the data stored write-through (kStoreWriteThrough), released by
//            the stores' acknowledgement alone (release_written_through, no
//            L2 write-back), relaxed +1; relaxed polls then an acquire fence
//            at SCOPE (the kernels' publication of write-through data);
//   ACK      the same release after ordinary write-back stores: the control,
//            which needs the write-back the fence performs;
//   WT_COHERENT  WT's writer; the reader polls, then reads the data with
//            coherent loads (kLoadCoherent) after acquire_coherent_reads, no
//            acquire fence (the kernels' reads of published partials);
//   WT_PLAIN WT's writer; the reader polls and reads with ordinary loads and
//            no acquire fence: the control, which needs the L2 invalidate.
// In RELAXED and FENCES the counters themselves are updated and polled at
// agent scope or wider, so that only the data's ordering depends on SCOPE;
// in RMW and CAS the counters take SCOPE too.  Compiler barriers keep
// program order in every form, so what the test sees is the hardware's.  A
// wait that exceeds spin_limit polls records ETIMEOUT and ends that
// workgroup; its partner then times out too, so the kernel always ends.
__device__ __forceinline__ uint32_t litmus_word(uint32_t round, uint32_t j) {
    return (round * 0x9E3779B1u) ^ (j * 0x85EBCA77u) ^ 0x5bd1e995u;
}

template <int SCOPE>
constexpr int at_least_agent() {
    return SCOPE == __HIP_MEMORY_SCOPE_SYSTEM ? __HIP_MEMORY_SCOPE_SYSTEM : __HIP_MEMORY_SCOPE_AGENT;
}

// Wait (one thread) until the counter reaches `target` (== target for CAS).
template <int SCOPE>
__device__ bool mp_wait(int form, uint32_t* flag, uint32_t target, uint32_t spin_limit) {
    constexpr int WIDE = at_least_agent<SCOPE>();
    if (form == SYMTILE_MP_RELAXED) return symtile::flag_poll<WIDE>(flag, target, spin_limit);
    if (form == SYMTILE_MP_WT_COHERENT || form == SYMTILE_MP_WT_PLAIN) {
        if (!symtile::flag_poll<WIDE>(flag, target, spin_limit)) return false;
        if (form == SYMTILE_MP_WT_COHERENT) symtile::acquire_coherent_reads();
        return true;
    }
    if (form == SYMTILE_MP_FENCES || form == SYMTILE_MP_WT || form == SYMTILE_MP_ACK) {
        if (!symtile::flag_poll<WIDE>(flag, target, spin_limit)) return false;
        symtile::fence_acquire<SCOPE>();
        return true;
    }
    for (uint32_t n = 0; n < spin_limit; ++n) {
        if (form == SYMTILE_MP_RMW) {
            if (symtile::atomic_add<__ATOMIC_ACQUIRE, SCOPE>(flag, 0u) >= target) return true;
        } else if (symtile::atomic_cas<__ATOMIC_ACQUIRE, SCOPE>(flag, target, target) == target) {
            return true;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    return false;
}

// Publish round i (one thread, after the workgroup's accesses are done).
template <int SCOPE>
__device__ void mp_publish(int form, uint32_t* flag, uint32_t i) {
    constexpr int WIDE = at_least_agent<SCOPE>();
    if (form == SYMTILE_MP_RELAXED) {
        symtile::flag_signal<WIDE>(flag);
    } else if (form == SYMTILE_MP_FENCES) {
        symtile::fence_release<SCOPE>();
        symtile::flag_signal<WIDE>(flag);
    } else if (form == SYMTILE_MP_WT || form == SYMTILE_MP_ACK || form == SYMTILE_MP_WT_COHERENT ||
               form == SYMTILE_MP_WT_PLAIN) {
        symtile::flag_publish_written_through<WIDE>(flag);
    } else if (form == SYMTILE_MP_RMW) {
        symtile::atomic_add<__ATOMIC_RELEASE, SCOPE>(flag, 1u);
    } else {
        symtile::atomic_cas<__ATOMIC_RELEASE, SCOPE>(flag, i - 1, i);
    }
}

template <int SCOPE>
__global__ __launch_bounds__(256) void litmus_mp_kernel(const uint64_t* bases, uint32_t* err,
                                                        int world, uint64_t data_off,
                                                        uint64_t flag_off, int rounds, int words,
                                                        int form, uint32_t spin_limit,
                                                        uint32_t* result) {
    __shared__ int s_ok;
    __shared__ uint32_t s_bad;
    const int pair = blockIdx.x >> 1;
    const bool writer = (blockIdx.x & 1) == 0;
    const int wr = pair % world, rd = (pair + 1) % world;
    const int me = writer ? wr : rd;
    // every address is named in rank `me`'s heap and translated
    uint32_t* data_me = reinterpret_cast<uint32_t*>(bases[me] + data_off) + (size_t)pair * words;
    uint32_t* ready_me = reinterpret_cast<uint32_t*>(bases[me] + flag_off) + 2 * pair;
    uint32_t* ack_me = ready_me + 1;
    uint32_t* data = symtile::translate(data_me, me, rd, bases);   // the reader's buffer
    uint32_t* ready = symtile::translate(ready_me, me, rd, bases);  // in the reader's slot
    uint32_t* ack = symtile::translate(ack_me, me, wr, bases);      // in the writer's slot
    const int tid = threadIdx.x;
    if (tid == 0) s_bad = 0;
    int done = 0;
    for (int i = 1; i <= rounds; ++i) {
        if (tid == 0) {
            const bool ok = writer ? mp_wait<SCOPE>(form, ack, (uint32_t)(i - 1), spin_limit)
                                   : mp_wait<SCOPE>(form, ready, (uint32_t)i, spin_limit);
            if (!ok) symtile::raise_error(err, symtile::ERR_TIMEOUT);
            s_ok = ok;
        }
        __syncthreads();
        if (!s_ok) break;
        asm volatile("" ::: "memory");
        const bool wt = form == SYMTILE_MP_WT || form == SYMTILE_MP_WT_COHERENT ||
                        form == SYMTILE_MP_WT_PLAIN;
        if (writer && wt) {
            const symtile::rsrc_t rd = symtile::make_rsrc(data, (uint32_t)words * 4u);
            for (int j = tid; j < words; j += blockDim.x)
                __builtin_amdgcn_raw_buffer_store_b32(litmus_word(i, j), rd, (uint32_t)j * 4u, 0,
                                                      symtile::kStoreWriteThrough);
            symtile::wg_stores_done();
            if (tid == 0) mp_publish<SCOPE>(form, ready, (uint32_t)i);
        } else if (writer) {
            for (int j = tid; j < words; j += blockDim.x)
                *symtile::global_ptr(data + j) = litmus_word(i, j);
            symtile::wg_stores_done();
            if (tid == 0) mp_publish<SCOPE>(form, ready, (uint32_t)i);
        } else if (form == SYMTILE_MP_WT_COHERENT) {
            const symtile::rsrc_t rs = symtile::make_rsrc(data, (uint32_t)words * 4u);
            uint32_t bad = 0;
            for (int j = tid; j < words; j += blockDim.x)
                bad += __builtin_amdgcn_raw_buffer_load_b32(rs, (uint32_t)j * 4u, 0,
                                                            symtile::kLoadCoherent) !=
                       litmus_word(i, j);
            if (bad) atomicAdd(&s_bad, bad);
            __syncthreads();                 // every word read before the ack
            if (tid == 0) mp_publish<SCOPE>(form, ack, (uint32_t)i);
        } else {
            uint32_t bad = 0;
            for (int j = tid; j < words; j += blockDim.x)
                bad += *symtile::global_ptr(data + j) != litmus_word(i, j);
            if (bad) atomicAdd(&s_bad, bad);
            __syncthreads();                 // every word read before the ack
            if (tid == 0) mp_publish<SCOPE>(form, ack, (uint32_t)i);
        }
        done = i;
    }
    __syncthreads();
    if (tid == 0 && !writer) {
        __hip_atomic_fetch_add(symtile::global_ptr(result), s_bad, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_add(symtile::global_ptr(result + 1), (uint32_t)done,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Store-buffering litmus test (Section 3.3.3, memory model): pair p =
// workgroups 2p (side 0, rank p % w) and 2p+1 (side 1, rank (p + 1) % w), one
// thread each, on different XCDs.  Round i uses fresh zeroed words x, y (x in
// side 1's slot, y in side 0's) and an arrival counter: both sides arrive and
// wait for each other (bounded, agent scope), then side 0 writes x = 1 and
// reads y, side 1 writes y = 1 and reads x, and each records what it read.
// Forms: RELAXED = relaxed atomic store and load at SCOPE; ACQ_REL = an
// exchange and a fetch_add(0), both acq_rel at SCOPE (read-modify-writes
// read the latest value, and a release RMW read by an acquire RMW
// synchronises, so both reading 0 is forbidden); SEQ_CST = seq_cst store and
// load at SCOPE (both reading 0 is forbidden).  out[(p * rounds + i) * 2 +
// side] receives the value read, or 2 when the round was not run (timeout).
template <int SCOPE>
__global__ __launch_bounds__(64) void litmus_sb_kernel(const uint64_t* bases, uint32_t* err,
                                                       int world, uint64_t flag_off, int rounds,
                                                       int form, uint32_t spin_limit,
                                                       uint32_t* out) {
    if (threadIdx.x != 0) return;
    const int pair = blockIdx.x >> 1, side = blockIdx.x & 1;
    const int r0 = pair % world, r1 = (pair + 1) % world;
    const int me = side ? r1 : r0;
    bool ok = true;
    for (int i = 0; i < rounds; ++i) {
        uint32_t* base_me =
            reinterpret_cast<uint32_t*>(bases[me] + flag_off) + ((size_t)pair * rounds + i) * 4;
        uint32_t* x = symtile::translate(base_me, me, r1, bases);         // side 1's slot
        uint32_t* y = symtile::translate(base_me, me, r0, bases) + 1;     // side 0's slot
        uint32_t* arrive = symtile::translate(base_me, me, r0, bases) + 2;
        uint32_t* mine = side ? y : x;
        uint32_t* other = side ? x : y;
        uint32_t seen = 2;
        if (ok) {
            symtile::flag_signal(arrive);
            ok = symtile::flag_poll(arrive, 2u, spin_limit);
            if (!ok) symtile::raise_error(err, symtile::ERR_TIMEOUT);
        }
        if (ok) {
            if (form == SYMTILE_SB_RELAXED) {
                __hip_atomic_store(symtile::global_ptr(mine), 1u, __ATOMIC_RELAXED, SCOPE);
                seen = __hip_atomic_load(symtile::global_ptr(other), __ATOMIC_RELAXED, SCOPE);
            } else if (form == SYMTILE_SB_ACQ_REL) {
                symtile::atomic_xchg<__ATOMIC_ACQ_REL, SCOPE>(mine, 1u);
                seen = symtile::atomic_add<__ATOMIC_ACQ_REL, SCOPE>(other, 0u);
            } else {
                __hip_atomic_store(symtile::global_ptr(mine), 1u, __ATOMIC_SEQ_CST, SCOPE);
                seen = __hip_atomic_load(symtile::global_ptr(other), __ATOMIC_SEQ_CST, SCOPE);
            }
        }
        out[((size_t)pair * rounds + i) * 2 + side] = seen;
    }
}

extern "C" {

const char* symtile_last_error(void) { return g_last_error.c_str(); }

const char* symtile_version(void) { return "symtile 0.2 (gfx950)"; }

symtile_status symtile_clock_rate_khz(int device, int* khz) {
    if (!khz) return symtile_host::fail(SYMTILE_EINVAL, "khz is NULL");
    int n = 0;
    SYMTILE_HIP(hipGetDeviceCount(&n));
    if (device < 0 || device >= n) return symtile_host::fail(SYMTILE_EINVAL, "bad device");
    SYMTILE_HIP(hipDeviceGetAttribute(khz, hipDeviceAttributeWallClockRate, device));
    return SYMTILE_OK;
}

symtile_status symtile_heap_create(int device, int world_size, size_t slot_bytes,
                                   symtile_heap** out) {
    return build_heap(device, world_size, slot_bytes, nullptr, 0, true, out);
}

symtile_status symtile_heap_create_on(int device, int world_size, size_t slot_bytes,
                                      void* base, size_t total_bytes, symtile_heap** out) {
    return build_heap(device, world_size, slot_bytes, base, total_bytes, false, out);
}

symtile_status symtile_heap_destroy(symtile_heap* h) {
    if (!h) return SYMTILE_OK;
    DeviceGuard guard(h->device);
    symtile_status st = SYMTILE_OK;
    if (hipDeviceSynchronize() != hipSuccess) st = symtile_host::fail(SYMTILE_EHIP, "sync failed");
    if (h->owns_memory && h->base) (void)hipFree(h->base);
    if (h->control) (void)hipFree(h->control);
    if (h->ev_fork) (void)hipEventDestroy(h->ev_fork);
    if (h->ev_join) (void)hipEventDestroy(h->ev_join);
    if (h->ev_t0) (void)hipEventDestroy(h->ev_t0);
    if (h->ev_t1) (void)hipEventDestroy(h->ev_t1);
    if (h->aux_stream) (void)hipStreamDestroy(h->aux_stream);
    delete h;
    return st;
}

symtile_status symtile_heap_alloc(symtile_heap* h, size_t bytes, size_t align,
                                  size_t* offset_out) {
    if (symtile_status st = check_heap(h)) return st;
    if (!offset_out) return symtile_host::fail(SYMTILE_EINVAL, "offset_out is NULL");
    if (align == 0) align = 256;
    if (align & (align - 1)) return symtile_host::fail(SYMTILE_EINVAL, "align not a power of 2");
    if (align > h->slot_stride) return symtile_host::fail(SYMTILE_EINVAL, "align too large");
    const size_t off = (h->used + align - 1) & ~(align - 1);
    if (off > h->slot_stride || bytes > h->slot_stride - off)
        return symtile_host::fail(SYMTILE_ENOMEM, "symmetric heap slot exhausted: " +
                                                      std::to_string(bytes) + " bytes requested, " +
                                                      std::to_string(h->slot_stride - h->used) +
                                                      " free");
    h->used = off + bytes;
    *offset_out = off;
    return SYMTILE_OK;
}

symtile_status symtile_heap_ptr(const symtile_heap* h, int rank, size_t offset, void** out) {
    if (symtile_status st = check_heap(h)) return st;
    if (!out) return symtile_host::fail(SYMTILE_EINVAL, "out is NULL");
    if (rank < 0 || rank >= h->world) return symtile_host::fail(SYMTILE_EINVAL, "rank out of range");
    if (offset > h->slot_stride) return symtile_host::fail(SYMTILE_EINVAL, "offset beyond slot");
    *out = reinterpret_cast<void*>(h->host_bases[rank] + offset);
    return SYMTILE_OK;
}

symtile_status symtile_heap_info(const symtile_heap* h, int* world_size, size_t* slot_stride,
                                 size_t* used, int* device) {
    if (symtile_status st = check_heap(h)) return st;
    if (world_size) *world_size = h->world;
    if (slot_stride) *slot_stride = h->slot_stride;
    if (used) *used = h->used;
    if (device) *device = h->device;
    return SYMTILE_OK;
}

symtile_status symtile_heap_bases(const symtile_heap* h, const uint64_t** dev_bases,
                                  uint64_t* host_bases) {
    if (symtile_status st = check_heap(h)) return st;
    if (dev_bases) *dev_bases = h->dev_bases;
    if (host_bases) std::memcpy(host_bases, h->host_bases, sizeof(uint64_t) * h->world);
    return SYMTILE_OK;
}

symtile_status symtile_translate(const symtile_heap* h, const void* p, int from_rank,
                                 int to_rank, void** out) {
    if (symtile_status st = check_heap(h)) return st;
    if (!out) return symtile_host::fail(SYMTILE_EINVAL, "out is NULL");
    if (from_rank < 0 || from_rank >= h->world || to_rank < 0 || to_rank >= h->world)
        return symtile_host::fail(SYMTILE_EINVAL, "rank out of range");
    if (!symtile_host::in_slot(h, p, 1, from_rank))
        return symtile_host::fail(SYMTILE_EINVAL, "pointer is not inside the slot of from_rank");
    const uint64_t a = reinterpret_cast<uint64_t>(p);
    *out = reinterpret_cast<void*>(h->host_bases[to_rank] + (a - h->host_bases[from_rank]));
    return SYMTILE_OK;
}

symtile_status symtile_translate_device(const symtile_heap* h, const uint64_t* in, int n,
                                        int from_rank, int to_rank, uint64_t* out,
                                        symtile_stream s) {
    if (symtile_status st = check_heap(h)) return st;
    if (n < 0 || (n > 0 && (!in || !out)))
        return symtile_host::fail(SYMTILE_EINVAL, "bad array arguments");
    if (from_rank < 0 || from_rank >= h->world || to_rank < 0 || to_rank >= h->world)
        return symtile_host::fail(SYMTILE_EINVAL, "rank out of range");
    if (n == 0) return SYMTILE_OK;
    DeviceGuard guard(h->device);
    hipLaunchKernelGGL(translate_kernel, dim3((n + 255) / 256), dim3(256), 0,
                       static_cast<hipStream_t>(s), in, n, from_rank, to_rank, h->dev_bases, out);
    SYMTILE_HIP(hipGetLastError());
    return SYMTILE_OK;
}

symtile_status symtile_barrier(symtile_heap* h, symtile_stream s) {
    if (symtile_status st = check_heap(h)) return st;
    DeviceGuard guard(h->device);
    if (s)
        SYMTILE_HIP(hipStreamSynchronize(static_cast<hipStream_t>(s)));
    else
        SYMTILE_HIP(hipDeviceSynchronize());
    uint32_t err = 0;
    SYMTILE_HIP(hipMemcpy(&err, h->dev_err, sizeof err, hipMemcpyDeviceToHost));
    if (err) {
        const uint32_t zero = 0;
        SYMTILE_HIP(hipMemcpy(h->dev_err, &zero, sizeof zero, hipMemcpyHostToDevice));
        if (err & symtile::ERR_TIMEOUT)
            return symtile_host::fail(
                SYMTILE_ETIMEOUT,
                std::string("a device-side wait exceeded its spin limit") +
                    ((err & symtile::ERR_WORKSPACE) ? "; a split-K workspace was not zeroed" : ""));
        if (err & symtile::ERR_WORKSPACE)
            return symtile_host::fail(
                SYMTILE_EINVAL,
                "split-K workspace counters were not zero when a call started (zero the "
                "workspace after an ETIMEOUT); the affected tiles were not written");
        return symtile_host::fail(SYMTILE_EHIP, "device error word " + std::to_string(err));
    }
    return SYMTILE_OK;
}

symtile_status symtile_heap_fill(symtile_heap* h, int rank, size_t offset, size_t bytes,
                                 int value, symtile_stream s) {
    if (symtile_status st = check_heap(h)) return st;
    if (rank >= h->world) return symtile_host::fail(SYMTILE_EINVAL, "rank out of range");
    if (offset > h->slot_stride || bytes > h->slot_stride - offset)
        return symtile_host::fail(SYMTILE_EINVAL, "fill range beyond the slot");
    if (bytes == 0) return SYMTILE_OK;
    DeviceGuard guard(h->device);
    const uint8_t v = static_cast<uint8_t>(value);
    const uint32_t word = v * 0x01010101u;
    const int r0 = rank < 0 ? 0 : rank, r1 = rank < 0 ? h->world : rank + 1;
    hipStream_t st = static_cast<hipStream_t>(s);
    for (int r = r0; r < r1; ++r) {
        uint8_t* p = reinterpret_cast<uint8_t*>(h->host_bases[r] + offset);
        if (reinterpret_cast<uintptr_t>(p) % 16 == 0 && bytes % 16 == 0) {
            size_t n16 = bytes / 16;
            unsigned grid = (unsigned)std::min<size_t>((n16 + 255) / 256, 4096);
            hipLaunchKernelGGL(fill16_kernel, dim3(grid), dim3(256), 0, st,
                               reinterpret_cast<symtile::u32x4*>(p), n16, word);
        } else {
            unsigned grid = (unsigned)std::min<size_t>((bytes + 255) / 256, 4096);
            hipLaunchKernelGGL(fill1_kernel, dim3(grid), dim3(256), 0, st, p, bytes, v);
        }
        SYMTILE_HIP(hipGetLastError());
    }
    return SYMTILE_OK;
}

symtile_status symtile_litmus_mp(symtile_heap* h, size_t data_off, size_t flag_off, int pairs,
                                 int rounds, int words, int form, int scope, uint32_t spin_limit,
                                 uint32_t* result, symtile_stream s) {
    if (symtile_status st = check_heap(h)) return st;
    if (pairs < 1 || pairs > 256 || rounds < 1 || words < 1 || words > (1 << 20))
        return symtile_host::fail(SYMTILE_EINVAL, "pairs in [1, 256], rounds >= 1, words in [1, 2^20]");
    if (form < SYMTILE_MP_RELAXED || form > SYMTILE_MP_WT_PLAIN)
        return symtile_host::fail(SYMTILE_EINVAL, "unknown message-passing form");
    if (scope < SYMTILE_SCOPE_BLOCK || scope > SYMTILE_SCOPE_SYS)
        return symtile_host::fail(SYMTILE_EINVAL, "unknown scope");
    if (!result) return symtile_host::fail(SYMTILE_EINVAL, "result is NULL");
    const size_t data_bytes = (size_t)pairs * words * 4, flag_bytes = (size_t)pairs * 8;
    if (data_off % 4 || flag_off % 4 || data_off > h->slot_stride ||
        data_bytes > h->slot_stride - data_off || flag_off > h->slot_stride ||
        flag_bytes > h->slot_stride - flag_off ||
        (data_off < flag_off + flag_bytes && flag_off < data_off + data_bytes))
        return symtile_host::fail(SYMTILE_EINVAL, "data or flags misaligned, outside the slot, or overlapping");
    if (2 * pairs > symtile_host::cu_count(h->device))
        return symtile_host::fail(SYMTILE_EUNSUPPORTED, "more workgroups than CUs (all must be resident)");
    DeviceGuard guard(h->device);
    auto launch = [&](auto kernel) {
        hipLaunchKernelGGL(kernel, dim3(2 * pairs), dim3(256), 0, static_cast<hipStream_t>(s),
                           h->dev_bases, h->dev_err, h->world, (uint64_t)data_off,
                           (uint64_t)flag_off, rounds, words, form,
                           spin_limit ? spin_limit : (1u << 22), result);
    };
    if (scope == SYMTILE_SCOPE_BLOCK) launch(litmus_mp_kernel<__HIP_MEMORY_SCOPE_WORKGROUP>);
    else if (scope == SYMTILE_SCOPE_GPU) launch(litmus_mp_kernel<__HIP_MEMORY_SCOPE_AGENT>);
    else launch(litmus_mp_kernel<__HIP_MEMORY_SCOPE_SYSTEM>);
    SYMTILE_HIP(hipGetLastError());
    return SYMTILE_OK;
}

symtile_status symtile_litmus_sb(symtile_heap* h, size_t flag_off, int pairs, int rounds,
                                 int form, int scope, uint32_t spin_limit, uint32_t* out,
                                 symtile_stream s) {
    if (symtile_status st = check_heap(h)) return st;
    if (pairs < 1 || pairs > 256 || rounds < 1 || rounds > (1 << 16))
        return symtile_host::fail(SYMTILE_EINVAL, "pairs in [1, 256], rounds in [1, 65536]");
    if (form < SYMTILE_SB_RELAXED || form > SYMTILE_SB_SEQ_CST)
        return symtile_host::fail(SYMTILE_EINVAL, "unknown store-buffering form");
    if (scope < SYMTILE_SCOPE_BLOCK || scope > SYMTILE_SCOPE_SYS)
        return symtile_host::fail(SYMTILE_EINVAL, "unknown scope");
    if (!out) return symtile_host::fail(SYMTILE_EINVAL, "out is NULL");
    const size_t bytes = (size_t)pairs * rounds * 16;
    if (flag_off % 16 || flag_off > h->slot_stride || bytes > h->slot_stride - flag_off)
        return symtile_host::fail(SYMTILE_EINVAL, "words misaligned or outside the slot");
    if (2 * pairs > symtile_host::cu_count(h->device))
        return symtile_host::fail(SYMTILE_EUNSUPPORTED, "more workgroups than CUs (all must be resident)");
    DeviceGuard guard(h->device);
    auto launch = [&](auto kernel) {
        hipLaunchKernelGGL(kernel, dim3(2 * pairs), dim3(64), 0, static_cast<hipStream_t>(s),
                           h->dev_bases, h->dev_err, h->world, (uint64_t)flag_off, rounds, form,
                           spin_limit ? spin_limit : (1u << 22), out);
    };
    if (scope == SYMTILE_SCOPE_BLOCK) launch(litmus_sb_kernel<__HIP_MEMORY_SCOPE_WORKGROUP>);
    else if (scope == SYMTILE_SCOPE_GPU) launch(litmus_sb_kernel<__HIP_MEMORY_SCOPE_AGENT>);
    else launch(litmus_sb_kernel<__HIP_MEMORY_SCOPE_SYSTEM>);
    SYMTILE_HIP(hipGetLastError());
    return SYMTILE_OK;
}

symtile_status symtile_value_exercise(symtile_heap* h, int op, size_t src_off, size_t dst_off,
                                      size_t bytes, int cur_rank, int remote_rank,
                                      int nontemporal, symtile_stream s) {
    if (symtile_status st = check_heap(h)) return st;
    if (op != SYMTILE_LOAD && op != SYMTILE_STORE)
        return symtile_host::fail(SYMTILE_EINVAL, "op must be SYMTILE_LOAD or SYMTILE_STORE");
    if (cur_rank < 0 || cur_rank >= h->world || remote_rank < 0 || remote_rank >= h->world)
        return symtile_host::fail(SYMTILE_EINVAL, "rank out of range");
    if (nontemporal != 0 && nontemporal != 1)
        return symtile_host::fail(SYMTILE_EINVAL, "nontemporal must be 0 or 1");
    if (src_off % 16 || dst_off % 16 || bytes % 16)
        return symtile_host::fail(SYMTILE_EINVAL, "offsets and bytes must be multiples of 16");
    if (src_off > h->slot_stride || bytes > h->slot_stride - src_off ||
        dst_off > h->slot_stride || bytes > h->slot_stride - dst_off)
        return symtile_host::fail(SYMTILE_EINVAL, "region outside the slot");
    if (cur_rank == remote_rank && src_off < dst_off + bytes && dst_off < src_off + bytes)
        return symtile_host::fail(SYMTILE_EINVAL, "source and destination overlap in one slot");
    if (bytes == 0) return SYMTILE_OK;
    DeviceGuard guard(h->device);
    const size_t n16 = bytes / 16;
    unsigned grid = (unsigned)std::min<size_t>((n16 + 255) / 256, 4096);
    hipLaunchKernelGGL(value_exercise_kernel, dim3(grid), dim3(256), 0,
                       static_cast<hipStream_t>(s),
                       reinterpret_cast<char*>(h->host_bases[cur_rank]), h->dev_bases, op,
                       cur_rank, remote_rank, (uint64_t)src_off, (uint64_t)dst_off, n16,
                       nontemporal);
    SYMTILE_HIP(hipGetLastError());
    return SYMTILE_OK;
}

symtile_status symtile_atomic_exercise(symtile_heap* h, int op, int sem, int scope,
                                       size_t offset, int from_rank, int to_rank,
                                       int n_threads, uint32_t operand, uint32_t compare,
                                       uint32_t* old_out, symtile_stream s) {
    if (symtile_status st = check_heap(h)) return st;
    if (op < SYMTILE_ATOMIC_ADD || op > SYMTILE_ATOMIC_MAX)
        return symtile_host::fail(SYMTILE_EINVAL, "unknown atomic op");
    if (sem < SYMTILE_RELAXED || sem > SYMTILE_ACQ_REL)
        return symtile_host::fail(SYMTILE_EINVAL, "unknown ordering");
    if (scope < SYMTILE_SCOPE_BLOCK || scope > SYMTILE_SCOPE_SYS)
        return symtile_host::fail(SYMTILE_EINVAL, "unknown scope");
    if (from_rank < 0 || from_rank >= h->world || to_rank < 0 || to_rank >= h->world)
        return symtile_host::fail(SYMTILE_EINVAL, "rank out of range");
    if (offset % 4 || offset > h->slot_stride - 4)
        return symtile_host::fail(SYMTILE_EINVAL, "offset must be a 4-byte aligned slot offset");
    if (n_threads < 0 || n_threads > (1 << 24))
        return symtile_host::fail(SYMTILE_EINVAL, "n_threads out of range");
    if (n_threads == 0) return SYMTILE_OK;
    DeviceGuard guard(h->device);
    uint32_t* word = reinterpret_cast<uint32_t*>(h->host_bases[from_rank] + offset);
    hipLaunchKernelGGL(atomic_exercise_kernel, dim3((n_threads + 255) / 256), dim3(256), 0,
                       static_cast<hipStream_t>(s), word, from_rank, to_rank, h->dev_bases, op,
                       sem, scope, n_threads, operand, compare, old_out);
    SYMTILE_HIP(hipGetLastError());
    return SYMTILE_OK;
}

}  // extern "C"
