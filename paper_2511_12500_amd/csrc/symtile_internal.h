// Internal host-side definitions shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>

#include "symtile.h"

#define SYMTILE_MAX_WORLD 8

struct symtile_heap {
    int device;
    int world;
    size_t slot_stride;          // bytes between slot bases (multiple of 2 MiB)
    size_t used;                 // bump pointer, same in every slot
    bool owns_memory;
    uint8_t* base;               // slot 0 base
    uint64_t host_bases[SYMTILE_MAX_WORLD];
    uint64_t* dev_bases;         // device copy of host_bases (control block)
    uint32_t* dev_err;           // device error word (control block)
    void* control;               // the control allocation
    // Second stream and fork/join events of the unfused producer-consumer
    // schedule, created on first use (default priority) and destroyed with
    // the heap.
    hipStream_t aux_stream;
    hipEvent_t ev_fork, ev_join;
    // Events bracketing one kernel of a timed call (symtile_tile_copy_timed),
    // created on first use and destroyed with the heap.
    hipEvent_t ev_t0, ev_t1;
};

namespace symtile_host {

// Record `msg` as this thread's last error and return `st`.
symtile_status fail(symtile_status st, const std::string& msg);
symtile_status ok();

// Map a HIP error to EHIP with a message naming `what`.
symtile_status hip_fail(hipError_t e, const char* what);

#define SYMTILE_HIP(call)                                              \
    do {                                                               \
        hipError_t e_ = (call);                                        \
        if (e_ != hipSuccess) return symtile_host::hip_fail(e_, #call); \
    } while (0)

// True when [p, p + bytes) lies inside slot `rank` of h.
bool in_slot(const symtile_heap* h, const void* p, size_t bytes, int rank);

// Make h's device current for the calling thread; *previous = the device to
// restore afterwards, or -1 when h's device already was current.
symtile_status set_device(const symtile_heap* h, int* previous);

int cu_count(int device);

// The heap's second stream and its fork/join events, created on first use on
// the heap's device (which must be current).
symtile_status aux_stream(symtile_heap* h);

}  // namespace symtile_host
