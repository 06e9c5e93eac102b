// Symmetric-heap tile copy: the pointer-based put and get of Section 3.3.2
// applied to every tile of a matrix, every emulated rank r taking part in one
// launch.  Put: rank r copies its own buffer into rank (r + shift) mod w's.
// Get: rank r copies rank (r - shift) mod w's buffer into its own.  Either
// way one release-published counter per tile lands in the destination slot,
// and the post-state is the same; what differs is which side's addresses are
// translated (the remote read of a get, the remote write of a put).
//
// Data path: HBM-bound.  Each workgroup owns a run of tiles_per_wg
// consecutive (rank, tile) items; every thread moves 16-byte chunks,
// issuing a batch of loads before the matching stores so many requests are
// in flight per wave.  Consecutive lanes take consecutive chunks of a tile
// row, so each wave instruction covers whole cache lines.  After its run the
// workgroup publishes all of its counters behind one agent-scope release:
// the release is an L2 write-back, serialised per XCD, so its count (not the
// data path) bounds the kernel when every tile pays for one.  A run of
// adjacent tiles of one tile row is copied as one rectangle, row by row, so
// the memory sees long row segments instead of many short ones.  Stores are
// written through to memory (cold copies measured fastest that way).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <string>

#include "symtile.h"
#include "symtile_device.h"
#include "symtile_internal.h"

namespace {

using symtile::u32x4;

// Workgroup shape: one wide workgroup per CU keeps the number of releases
// (one per workgroup) small while 16 waves per CU keep enough loads in
// flight to cover HBM latency.
#ifndef SYMTILE_COPY_THREADS
#define SYMTILE_COPY_THREADS 1024
#endif
#ifndef SYMTILE_COPY_BATCH
#define SYMTILE_COPY_BATCH 8
#endif
constexpr int kThreads = SYMTILE_COPY_THREADS;
constexpr int kBatch = SYMTILE_COPY_BATCH;   // chunks in flight per thread

struct CopyParams {
    const uint64_t* bases;
    int world, shift, only_rank;
    int mode;                // SYMTILE_PUT or SYMTILE_GET
    uint64_t src_off, dst_off, flag_off;
    int rows;                // matrix rows
    int row_chunks;          // 16-byte chunks per matrix row
    int ld_bytes;            // row stride in bytes
    int tile_r;              // tile rows
    int tile_chunks;         // 16-byte chunks per tile row
    int tiles_c;             // tiles per matrix row of tiles
    int ntiles;              // tiles per rank
    int nitems;              // (rank, tile) items of this launch
    int per_wg;              // consecutive items per workgroup
    int band_lg_w;           // >= 0: each run is one rectangle, 1 << band_lg_w chunks wide
};

// Source and destination ranks of executing rank r.
__device__ __forceinline__ void copy_ranks(const CopyParams& p, int r, int& src, int& dst) {
    const int peer_up = ((r + p.shift) % p.world + p.world) % p.world;
    const int peer_down = ((r - p.shift) % p.world + p.world) % p.world;
    src = (p.mode == SYMTILE_GET) ? peer_down : r;
    dst = (p.mode == SYMTILE_GET) ? r : peer_up;
}

// Copy the nrows x nchunks block at (row0, chunk0) of the matrix from rank
// src_rank to rank dst with the tile verb `copy`: both buffers are symmetric
// objects named by their address in rank r's heap, and the verb translates
// them.  With lg_w >= 0 a pass covers 1 << lg_w chunk columns of
// kThreads >> lg_w rows, so a run of horizontally adjacent tiles streams
// whole row segments (up to 8 KiB); lg_w < 0 (a tile width that is not a
// power of two of chunks) numbers the chunks row-major through the block.
template <int POLICY>
__device__ __forceinline__ void copy_block(const CopyParams& p, int r, int src_rank, int dst,
                                           int row0, int chunk0, int nrows, int nchunks,
                                           int lg_w) {
    const uint8_t* src = reinterpret_cast<const uint8_t*>(p.bases[r] + p.src_off) +
                         (size_t)row0 * p.ld_bytes + (size_t)chunk0 * 16;
    uint8_t* dst_local = reinterpret_cast<uint8_t*>(p.bases[r] + p.dst_off) +
                         (size_t)row0 * p.ld_bytes + (size_t)chunk0 * 16;
    symtile::TileGeom g;
    g.rows = nrows;
    g.chunks = nchunks;
    g.ld_bytes = (uint32_t)p.ld_bytes;
    g.lg_w = lg_w;
    if (lg_w >= 0) {
        symtile::copy<POLICY, kBatch>(src, dst_local, g, src_rank, dst, r, p.bases, threadIdx.x,
                                      kThreads);
        return;
    }
    const symtile::rsrc_t rs = symtile::tile_rsrc(src, g, r, src_rank, p.bases);
    const symtile::rsrc_t rd = symtile::tile_rsrc(dst_local, g, r, dst, p.bases);
    const int total = nrows * p.tile_chunks;
    for (int base = threadIdx.x; base < total; base += kThreads * kBatch) {
        u32x4 v[kBatch];
        uint32_t off[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int q = base + u * kThreads;
            const int row = q / p.tile_chunks, c = q - row * p.tile_chunks;
            off[u] = (q < total && c < nchunks) ? (uint32_t)(row * p.ld_bytes + c * 16)
                                                : symtile::kOOB;
            v[u] = symtile::buf_ld16(rs, off[u], 0);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) symtile::buf_st16p<POLICY>(v[u], rd, off[u], 0);
    }
}

// Copy tile `tile` of rank r (TC = 16-byte chunks per tile row when that is a
// power of two dividing the thread count, else 0).
template <int TC, int POLICY>
__device__ __forceinline__ void copy_one_tile(const CopyParams& p, int r, int src_rank, int dst,
                                              int tile) {
    const int tr = tile / p.tiles_c, tc = tile - tr * p.tiles_c;
    const int row0 = tr * p.tile_r;
    const int chunk0 = tc * p.tile_chunks;
    copy_block<POLICY>(p, r, src_rank, dst, row0, chunk0, min(p.tile_r, p.rows - row0),
                       min(p.tile_chunks, p.row_chunks - chunk0),
                       TC > 0 ? __builtin_ctz(TC) : -1);
}

template <int TC, int POLICY>
__global__ __launch_bounds__(kThreads) void tile_copy_kernel(const CopyParams p) {
    const int first = blockIdx.x * p.per_wg;
    const int last = min(first + p.per_wg, p.nitems);
    if (p.band_lg_w >= 0) {
        // The run is per_wg adjacent tiles of one tile row: one rectangle.
        const int r = p.only_rank >= 0 ? p.only_rank : first / p.ntiles;
        int src, dst;
        copy_ranks(p, r, src, dst);
        const int t0 = first % p.ntiles;
        const int tr = t0 / p.tiles_c, tc = t0 - tr * p.tiles_c;
        const int row0 = tr * p.tile_r, chunk0 = tc * p.tile_chunks;
        copy_block<POLICY>(p, r, src, dst, row0, chunk0, min(p.tile_r, p.rows - row0),
                           min(p.per_wg * p.tile_chunks, p.row_chunks - chunk0), p.band_lg_w);
    } else {
        for (int it = first; it < last; ++it) {
            const int r = p.only_rank >= 0 ? p.only_rank : it / p.ntiles;
            int src, dst;
            copy_ranks(p, r, src, dst);
            copy_one_tile<TC, POLICY>(p, r, src, dst, it % p.ntiles);
        }
    }
    // Publish: every tile of the run is in its destination heap before any
    // of its counters moves.  Wave 0 releases once, then its lanes increment
    // the run's counters together (one tile per lane), rather than one
    // thread issuing them one after another into the same cache lines.
    symtile::wg_stores_done();
    if (threadIdx.x < 64) {
        if constexpr (POLICY == symtile::kStoreWriteThrough)
            symtile::release_written_through();   // nothing of the run sits dirty in the L2
        else
            symtile::fence_release<__HIP_MEMORY_SCOPE_AGENT>();
        for (int it = first + (int)threadIdx.x; it < last; it += 64) {
            const int r = p.only_rank >= 0 ? p.only_rank : it / p.ntiles;
            int src, dst;
            copy_ranks(p, r, src, dst);
            uint32_t* flag_local =
                reinterpret_cast<uint32_t*>(p.bases[r] + p.flag_off) + it % p.ntiles;
            symtile::flag_signal(symtile::translate(flag_local, r, dst, p.bases));
        }
    }
}

}  // namespace

// The checks and launch of symtile_tile_copy; with t0 and t1 set the kernel
// is launched with hipExtLaunchKernel, which records the two events as part
// of the kernel's dispatch.
static symtile_status tile_copy_launch(symtile_heap* h, size_t src_off, size_t dst_off, int rows,
                                       int cols, int ld, int dtype, int tile_r, int tile_c,
                                       int shift, int only_rank, size_t flag_off,
                                       int tiles_per_wg, int mode, symtile_stream s,
                                       hipEvent_t t0, hipEvent_t t1) {

    using symtile_host::fail;
    if (!h) return fail(SYMTILE_EINVAL, "heap is NULL");
    int esize = 0;
    if (dtype == SYMTILE_F16 || dtype == SYMTILE_BF16) esize = 2;
    else if (dtype == SYMTILE_F32) esize = 4;
    else return fail(SYMTILE_EINVAL, "unknown dtype");
    if (rows < 0 || cols < 0 || tile_r <= 0 || tile_c <= 0 || ld < cols)
        return fail(SYMTILE_EINVAL, "bad matrix or tile extents");
    if ((size_t)cols * esize % 16 || (size_t)tile_c * esize % 16 || (size_t)ld * esize % 16)
        return fail(SYMTILE_EINVAL, "cols, tile_c and ld must span multiples of 16 bytes");
    if (src_off % 16 || dst_off % 16 || flag_off % 4)
        return fail(SYMTILE_EINVAL, "offsets misaligned (16 bytes for data, 4 for flags)");
    if (only_rank >= h->world) return fail(SYMTILE_EINVAL, "only_rank out of range");
    if (tiles_per_wg < 0) return fail(SYMTILE_EINVAL, "tiles_per_wg < 0");
    if (mode != SYMTILE_PUT && mode != SYMTILE_GET)
        return fail(SYMTILE_EINVAL, "mode must be SYMTILE_PUT or SYMTILE_GET");
    if (rows == 0 || cols == 0) return SYMTILE_OK;
    const size_t ld_bytes = (size_t)ld * esize;
    const size_t span = (size_t)(rows - 1) * ld_bytes + (size_t)cols * esize;
    const int tiles_r = (rows + tile_r - 1) / tile_r;
    const int tiles_c = (cols + tile_c - 1) / tile_c;
    const size_t ntiles = (size_t)tiles_r * tiles_c;
    if (ld_bytes * (size_t)tile_r >= (size_t(1) << 31) || ntiles > INT32_MAX)
        return fail(SYMTILE_EINVAL, "a tile row band exceeds 2 GiB or too many tiles");
    if (src_off > h->slot_stride || span > h->slot_stride - src_off ||
        dst_off > h->slot_stride || span > h->slot_stride - dst_off ||
        flag_off > h->slot_stride || ntiles * 4 > h->slot_stride - flag_off)
        return fail(SYMTILE_EINVAL, "source, destination or flags exceed the slot");
    if (src_off < dst_off + span && dst_off < src_off + span)
        return fail(SYMTILE_EINVAL, "source and destination regions overlap");
    if ((flag_off < src_off + span && src_off < flag_off + ntiles * 4) ||
        (flag_off < dst_off + span && dst_off < flag_off + ntiles * 4))
        return fail(SYMTILE_EINVAL, "flags overlap the data");

    CopyParams p;
    p.bases = h->dev_bases;
    p.world = h->world;
    p.shift = shift;
    p.only_rank = only_rank;
    p.mode = mode;
    p.src_off = src_off;
    p.dst_off = dst_off;
    p.flag_off = flag_off;
    p.rows = rows;
    p.row_chunks = (int)((size_t)cols * esize / 16);
    p.ld_bytes = (int)ld_bytes;
    p.tile_r = tile_r;
    p.tile_chunks = (int)((size_t)tile_c * esize / 16);
    p.tiles_c = tiles_c;
    p.ntiles = (int)ntiles;
    const size_t nitems = ntiles * (only_rank >= 0 ? 1 : (size_t)h->world);
    if (nitems > INT32_MAX) return fail(SYMTILE_EINVAL, "too many tiles");
    p.nitems = (int)nitems;
    if (tiles_per_wg == 0) {
        // about one workgroup per CU: enough waves to fill the chip while
        // keeping the number of L2 write-backs (one per workgroup) small;
        // rounded to a power of two that divides the tiles of a tile row so
        // that every run is one rectangle
        const size_t target = (size_t)std::max(1, symtile_host::cu_count(h->device));
        size_t per = std::max<size_t>(1, (nitems + target - 1) / target);
        size_t pow2 = 1;
        while (pow2 * 2 <= per && tiles_c % (pow2 * 2) == 0) pow2 *= 2;
        tiles_per_wg = (int)pow2;
    }
    p.per_wg = tiles_per_wg;
    // Rectangle mode: runs never straddle a tile row and the run width
    // (rounded up to a power of two) fits the workgroup.
    p.band_lg_w = -1;
    if (tiles_c % tiles_per_wg == 0) {
        const size_t width = (size_t)tiles_per_wg * p.tile_chunks;
        int lg = 0;
        while (((size_t)1 << lg) < width) ++lg;
        if (((size_t)1 << lg) <= (size_t)kThreads) p.band_lg_w = lg;
    }
    // Buffer offsets are 32-bit: a tile's rows plus the out-of-range passes
    // that complete its last batch must stay below 2 GiB (the out-of-range
    // offset marker), or an offset could wrap back into the tile.
    {
        size_t rows_per_pass = 0;
        if (p.band_lg_w >= 0)
            rows_per_pass = (size_t)kThreads >> p.band_lg_w;
        else if (p.tile_chunks == 16 || p.tile_chunks == 32 || p.tile_chunks == 64)
            rows_per_pass = (size_t)kThreads / p.tile_chunks;
        if (rows_per_pass &&
            ((size_t)tile_r + rows_per_pass * kBatch) * ld_bytes >= (size_t(1) << 31))
            return fail(SYMTILE_EINVAL, "row stride too large for this tile shape");
    }

    int prev = -1;
    if (symtile_status st = symtile_host::set_device(h, &prev)) return st;
    const dim3 grid((unsigned)((nitems + p.per_wg - 1) / p.per_wg));
    hipStream_t stream = static_cast<hipStream_t>(s);
    const void* kernel;
    switch (p.tile_chunks) {
        case 16: kernel = reinterpret_cast<const void*>(&tile_copy_kernel<16, symtile::kStoreWriteThrough>); break;
        case 32: kernel = reinterpret_cast<const void*>(&tile_copy_kernel<32, symtile::kStoreWriteThrough>); break;
        case 64: kernel = reinterpret_cast<const void*>(&tile_copy_kernel<64, symtile::kStoreWriteThrough>); break;
        default: kernel = reinterpret_cast<const void*>(&tile_copy_kernel<0, symtile::kStoreWriteThrough>); break;
    }
    void* args[] = {&p};
    hipError_t e = t0 ? hipExtLaunchKernel(kernel, grid, dim3(kThreads), args, 0, stream, t0, t1, 0)
                      : hipLaunchKernel(kernel, grid, dim3(kThreads), args, 0, stream);
    if (e == hipSuccess) e = hipGetLastError();
    if (prev >= 0) (void)hipSetDevice(prev);
    if (e != hipSuccess) return symtile_host::hip_fail(e, "tile_copy_kernel launch");
    return SYMTILE_OK;
}

extern "C" symtile_status symtile_tile_copy(symtile_heap* h, size_t src_off, size_t dst_off,
                                            int rows, int cols, int ld, int dtype, int tile_r,
                                            int tile_c, int shift, int only_rank,
                                            size_t flag_off, int tiles_per_wg, int mode,
                                            symtile_stream s) {
    return tile_copy_launch(h, src_off, dst_off, rows, cols, ld, dtype, tile_r, tile_c, shift,
                            only_rank, flag_off, tiles_per_wg, mode, s, nullptr, nullptr);
}

extern "C" symtile_status symtile_tile_copy_timed(symtile_heap* h, size_t src_off,
                                                  size_t dst_off, int rows, int cols, int ld,
                                                  int dtype, int tile_r, int tile_c, int shift,
                                                  int only_rank, size_t flag_off,
                                                  int tiles_per_wg, int mode, symtile_stream s,
                                                  float* kernel_ms) {
    using symtile_host::fail;
    if (!h) return fail(SYMTILE_EINVAL, "heap is NULL");
    if (!kernel_ms) return fail(SYMTILE_EINVAL, "kernel_ms is NULL");
    *kernel_ms = 0.0f;
    int prev = -1;
    if (symtile_status st = symtile_host::set_device(h, &prev)) return st;
    struct Restore {
        int d;
        ~Restore() {
            if (d >= 0) (void)hipSetDevice(d);
        }
    } restore{prev};
    if (!h->ev_t0) SYMTILE_HIP(hipEventCreate(&h->ev_t0));
    if (!h->ev_t1) SYMTILE_HIP(hipEventCreate(&h->ev_t1));
    if (symtile_status st = tile_copy_launch(h, src_off, dst_off, rows, cols, ld, dtype, tile_r,
                                             tile_c, shift, only_rank, flag_off, tiles_per_wg,
                                             mode, s, h->ev_t0, h->ev_t1))
        return st;
    if (rows == 0 || cols == 0) return SYMTILE_OK;   // nothing launched
    SYMTILE_HIP(hipEventSynchronize(h->ev_t1));
    SYMTILE_HIP(hipEventElapsedTime(kernel_ms, h->ev_t0, h->ev_t1));
    return SYMTILE_OK;
}
