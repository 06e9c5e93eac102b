// Symmetric-heap tile copy: the pointer-based put of Section 3.3.2 applied
// to every tile of a matrix, every emulated rank r sending to rank
// (r + shift) mod w in one launch, with one release-published counter per
// tile in the destination slot.
//
// Data path: HBM-bound.  Each workgroup owns one tile; every thread moves
// 16-byte chunks, issuing a batch of loads before the matching stores so
// many requests are in flight per wave.  Consecutive lanes take consecutive
// chunks of a tile row, so each wave instruction covers whole cache lines.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <string>

#include "symtile.h"
#include "symtile_device.h"
#include "symtile_internal.h"

namespace {

using symtile::u32x4;

constexpr int kThreads = 256;
constexpr int kBatch = 8;   // chunks in flight per thread

struct CopyParams {
    const uint64_t* bases;
    int world, shift, only_rank;
    uint64_t src_off, dst_off, flag_off;
    int rows;                // matrix rows
    int row_chunks;          // 16-byte chunks per matrix row
    int ld_bytes;            // row stride in bytes
    int tile_r;              // tile rows
    int tile_chunks;         // 16-byte chunks per tile row
    int tiles_c;             // tiles per matrix row of tiles
};

template <bool NT>
__global__ __launch_bounds__(kThreads) void tile_copy_kernel(const CopyParams p) {
    const int r = p.only_rank >= 0 ? p.only_rank : (int)blockIdx.y;
    const int dst = ((r + p.shift) % p.world + p.world) % p.world;
    const int tile = blockIdx.x;
    const int tr = tile / p.tiles_c, tc = tile - tr * p.tiles_c;
    const int row0 = tr * p.tile_r;
    const int chunk0 = tc * p.tile_chunks;
    const int nrows = min(p.tile_r, p.rows - row0);
    const int nchunks = min(p.tile_chunks, p.row_chunks - chunk0);

    // The source is rank r's own buffer; the destination is the same
    // symmetric object translated into the heap of rank dst.
    const uint8_t* src = reinterpret_cast<const uint8_t*>(p.bases[r] + p.src_off);
    uint8_t* dst_local = reinterpret_cast<uint8_t*>(p.bases[r] + p.dst_off);
    uint8_t* dstp = symtile::translate(dst_local, r, dst, p.bases);

    const int total = nrows * p.tile_chunks;
    for (int base = threadIdx.x; base < total; base += kThreads * kBatch) {
        u32x4 v[kBatch];
        size_t off[kBatch];
        bool ok[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int q = base + u * kThreads;
            const int row = q / p.tile_chunks;
            const int c = q - row * p.tile_chunks;
            ok[u] = q < total && c < nchunks;
            off[u] = (size_t)(row0 + row) * p.ld_bytes + (size_t)(chunk0 + c) * 16;
            if (ok[u]) v[u] = symtile::ld16(src + off[u]);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            if (ok[u]) symtile::st16(dstp + off[u], v[u], NT);
    }

    // Publish: the tile is in rank dst's heap before its counter moves.
    symtile::wg_release_begin();
    if (threadIdx.x == 0) {
        uint32_t* flag_local = reinterpret_cast<uint32_t*>(p.bases[r] + p.flag_off) + tile;
        symtile::flag_add_release(symtile::translate(flag_local, r, dst, p.bases));
    }
}

}  // namespace

extern "C" symtile_status symtile_tile_copy(symtile_heap* h, size_t src_off, size_t dst_off,
                                            int rows, int cols, int ld, int dtype, int tile_r,
                                            int tile_c, int shift, int only_rank,
                                            size_t flag_off, symtile_stream s) {
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
    if (rows == 0 || cols == 0) return SYMTILE_OK;
    const size_t ld_bytes = (size_t)ld * esize;
    const size_t span = (size_t)(rows - 1) * ld_bytes + (size_t)cols * esize;
    const int tiles_r = (rows + tile_r - 1) / tile_r;
    const int tiles_c = (cols + tile_c - 1) / tile_c;
    const size_t ntiles = (size_t)tiles_r * tiles_c;
    if (ld_bytes > INT32_MAX || ntiles > INT32_MAX)
        return fail(SYMTILE_EINVAL, "matrix too large");
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
    p.src_off = src_off;
    p.dst_off = dst_off;
    p.flag_off = flag_off;
    p.rows = rows;
    p.row_chunks = (int)((size_t)cols * esize / 16);
    p.ld_bytes = (int)ld_bytes;
    p.tile_r = tile_r;
    p.tile_chunks = (int)((size_t)tile_c * esize / 16);
    p.tiles_c = tiles_c;

    int prev = -1;
    if (symtile_status st = symtile_host::set_device(h, &prev)) return st;
    const dim3 grid((unsigned)ntiles, only_rank >= 0 ? 1u : (unsigned)h->world);
    hipLaunchKernelGGL(tile_copy_kernel<true>, grid, dim3(kThreads), 0,
                       static_cast<hipStream_t>(s), p);
    hipError_t e = hipGetLastError();
    (void)hipSetDevice(prev);
    if (e != hipSuccess) return symtile_host::hip_fail(e, "tile_copy_kernel launch");
    return SYMTILE_OK;
}
