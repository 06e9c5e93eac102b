/*
 * symtile — one GPU's share of the fused GEMM + All-Scatter of
 * "Iris: First-Class Multi-GPU Programming Experience in Triton"
 * (arXiv 2511.12500), for AMD Instinct MI355X (gfx950).
 *
 * C ABI.  Every entry point returns a symtile_status (0 = success).  All
 * device work is enqueued on the caller's stream and is asynchronous; no
 * C++ exception crosses this boundary.  On failure the library keeps a
 * thread-local message, returned by symtile_last_error().
 *
 * Emulation of the symmetric heap on one GPU: the heap is one device
 * allocation of world_size equally sized slots; slot s plays the heap of
 * rank s.  Every symmetric allocation has the same offset in every slot, so
 * "the same object on rank s" is base[s] + offset, exactly the symmetric
 * layout of Section 3.2 (constructor, steps 3 and 6).
 */
#ifndef SYMTILE_H
#define SYMTILE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct symtile_heap symtile_heap;   /* opaque */
typedef void* symtile_stream;               /* a hipStream_t; NULL = null stream */

typedef enum {
    SYMTILE_OK = 0,
    SYMTILE_EINVAL = -1,        /* bad argument, shape, pointer or rank */
    SYMTILE_ENOMEM = -2,        /* device allocation or heap exhausted */
    SYMTILE_EHIP = -3,          /* a HIP runtime call failed */
    SYMTILE_ETIMEOUT = -4,      /* a bounded device-side wait expired */
    SYMTILE_EUNSUPPORTED = -5   /* valid request this build does not run */
} symtile_status;

typedef enum { SYMTILE_F16 = 1, SYMTILE_BF16 = 2, SYMTILE_F32 = 3 } symtile_dtype;

/* The schedules of Section 4 built here. */
typedef enum {
    SYMTILE_BULK_SYNC = 0,   /* Section 4.1.1: GEMM kernel, then scatter kernel, one stream */
    SYMTILE_FUSED_SEQ = 1,   /* Section 4.2.1: each tile stored to every rank after its K loop */
    SYMTILE_WG_SPEC = 2,     /* Section 4.2.2: producer WGs compute, consumer WGs scatter */
    SYMTILE_UNFUSED_PC = 3,  /* Section 4.1.2: a GEMM kernel and a copy kernel on two streams,
                                CUs partitioned by their grid sizes, per-tile ready counters */
    SYMTILE_WAVE_SPEC = 4    /* Section 4.2.3: each workgroup's compute waves store tiles
                                locally and one extra wave copies the previous tile to the
                                other slots during the next K loop (256x128 tiles) */
} symtile_variant;

/* Atomic verbs of the device API (Section 3.3.3, device API table). */
typedef enum {
    SYMTILE_ATOMIC_ADD = 0, SYMTILE_ATOMIC_XCHG = 1, SYMTILE_ATOMIC_CAS = 2,
    SYMTILE_ATOMIC_AND = 3, SYMTILE_ATOMIC_OR = 4, SYMTILE_ATOMIC_XOR = 5,
    SYMTILE_ATOMIC_MIN = 6, SYMTILE_ATOMIC_MAX = 7
} symtile_atomic_op;
typedef enum { SYMTILE_RELAXED = 0, SYMTILE_ACQUIRE = 1, SYMTILE_RELEASE = 2,
               SYMTILE_ACQ_REL = 3 } symtile_sem;
typedef enum { SYMTILE_SCOPE_BLOCK = 0, SYMTILE_SCOPE_GPU = 1,
               SYMTILE_SCOPE_SYS = 2 } symtile_scope;

/* Launch configuration of symtile_gemm_all_scatter.  Zero fields take the
 * documented defaults. */
typedef struct {
    int variant;          /* symtile_variant */
    int tile_m, tile_n;   /* output tile; (64,64) (128,128) (256,128) (256,256)
                             (256,224); 0,0 = 256x256 */
    int gemm_wgs;         /* producer workgroups; 0 = min(work units, CU count) for
                             BULK_SYNC/FUSED_SEQ (a unit is a tile, or one K slice
                             of a tile with split_k > 1), CU count - copy_wgs for
                             WG_SPEC and UNFUSED_PC */
    int copy_wgs;         /* WG_SPEC and UNFUSED_PC consumers (0 = CU count / 8) and
                             BULK_SYNC scatter-kernel workgroups (0 = CU count) */
    uint32_t epoch;       /* WG_SPEC, UNFUSED_PC: consumers wait until
                             ready[tile] >= epoch, so ready must hold epoch - 1
                             on entry and holds epoch after the call; 0 is taken
                             as 1 */
    uint32_t spin_limit;  /* polls of one consumer wait before it gives up and
                             raises SYMTILE_ETIMEOUT; 0 = 1<<22 */
    int nontemporal;      /* store policy of the output: 0 default, 1 streaming
                             (non-temporal), 2 write-through (leaves no dirty L2
                             line for the release to write back) */
    int group_m;          /* tile rows per L2 swizzle group; 0 = 4 */
    int waves_per_wg;     /* 4 or 8 wavefronts per workgroup; 0 = the tile's default
                             (4 for 64x64, and for 256x256 in FUSED_SEQ and
                             BULK_SYNC calls without split-K; 8 for the others).
                             Built: 64x64 with 4; 128x128, 256x128 and 256x256
                             with 4 or 8; 256x224 with 8 (others EUNSUPPORTED).
                             256x256 with 4 stages 64 k at a time through
                             registers; same results bit for bit */
    symtile_stream copy_stream; /* UNFUSED_PC: stream of the copy kernel; NULL = a
                             stream the heap creates on first use.  It must not
                             be the call's stream. */
    uint64_t* trace;      /* optional per-tile timeline (Section 3.4, instrumentation):
                             device uint64 [tiles_m*tiles_n][SYMTILE_TRACE_WORDS],
                             tile (m, n) at row m*tiles_n + n; NULL = off.  See
                             symtile_trace_word for the layout.  With split_k > 1
                             the start, location and main-loop words are those of
                             the tile's first K slice, the stored and released
                             words those of the slice that reduces the tile. */
    int split_k;          /* BULK_SYNC and FUSED_SEQ: each output tile is computed
                             as split_k slices of K (0 or 1 = no split; at most
                             64 and at most ceil(K/32)), so a problem with fewer
                             tiles than CUs still fills the chip.  The slices of
                             a tile add their fp32 partial products in slice
                             order, whichever finishes last, so the result is
                             the same on every call (it differs from split_k = 1
                             only by fp32 rounding). */
    void* workspace;      /* split_k > 1: device memory of workspace_bytes >=
                             symtile_gas_workspace_bytes(...) bytes, 16-byte
                             aligned, outside the output and counters.  Its first
                             round_up(8 * tiles, 256) bytes are counters that must
                             be zero before the first call that uses it; every
                             call that completes leaves them zero again.  A call
                             whose wait timed out (ETIMEOUT) leaves them as they
                             are, since slices of that call may still count
                             themselves after the timeout: zero the workspace
                             after the barrier that reports it.  A later call
                             that finds them non-zero skips the affected tiles
                             and reports EINVAL at the next barrier rather than
                             summing stale partials.  Calls that share a
                             workspace must not overlap in time (same stream, or
                             synchronised). */
    size_t workspace_bytes;
    int split_reduce;     /* split_k > 1: who sums a tile's K slices (symtile_split_reduce).
                             SYMTILE_SPLIT_REDUCE_LAST: the slice that arrives last
                             sums all partials and stores the whole tile (any grid).
                             SYMTILE_SPLIT_REDUCE_BANDED: the tile's rows form
                             split_k bands and slice s sums and stores band s, so
                             the reduction and the stores are spread over all
                             slices; needs one co-resident workgroup per slice
                             (tiles * split_k <= symtile_device_info's
                             max_coresident_wgs, gemm_wgs 0 or tiles * split_k) and
                             tile_m / split_k a multiple of 32 (16 for 256x224),
                             else EUNSUPPORTED.
                             SYMTILE_SPLIT_REDUCE_KERNEL: every slice writes its
                             partial and a second kernel on the same stream sums
                             each tile's rows in bands spread over the CUs and
                             stores them (any grid); gemm_wgs sizes the first
                             kernel only.
                             0 = for split_k = 2 BANDED where it applies, else
                             LAST; for split_k > 2 KERNEL.  All give the same
                             bits. */
} symtile_gas_config;

/* Reduction of split-K slices (symtile_gas_config.split_reduce). */
typedef enum {
    SYMTILE_SPLIT_REDUCE_AUTO = 0,
    SYMTILE_SPLIT_REDUCE_LAST = 1,
    SYMTILE_SPLIT_REDUCE_BANDED = 2,
    SYMTILE_SPLIT_REDUCE_KERNEL = 3
} symtile_split_reduce;

/* Per-tile trace record.  Times are ticks of the device's constant-rate
 * realtime counter (symtile_clock_rate_khz), comparable across workgroups.
 * Words a schedule has no event for are not written. */
#define SYMTILE_TRACE_WORDS 8
typedef enum {
    SYMTILE_TRACE_START = 0,     /* producer picked the tile up */
    SYMTILE_TRACE_MAINLOOP = 1,  /* accumulators final (K loop done, all waves) */
    SYMTILE_TRACE_STORED = 2,    /* producer's stores acknowledged (all waves) */
    SYMTILE_TRACE_RELEASED = 3,  /* producer's release fence and counter updates issued */
    SYMTILE_TRACE_WHERE = 4,     /* producer location: HW_ID << 32 | XCC_ID << 16 | workgroup id */
    SYMTILE_TRACE_COPY_WAIT = 5, /* WG_SPEC consumer starts waiting; BULK_SYNC copy start */
    SYMTILE_TRACE_COPY_GO = 6,   /* WG_SPEC consumer acquired the ready counter; BULK_SYNC = word 5 */
    SYMTILE_TRACE_COPY_DONE = 7  /* copy to the other slots stored and released */
} symtile_trace_word;

/* ---- heap (Section 3.2: constructor steps 3 and 6, host API table) -------- */

/* Create a heap of world_size slots of at least slot_bytes each on HIP
 * device `device`.  The slot stride is slot_bytes rounded up to 2 MiB.  The
 * library allocates (hipMalloc) and owns the memory, zeroes it, and builds
 * the device array of per-slot base addresses.  world_size in [1, 8].
 * Errors: EINVAL (bad device, world_size, slot_bytes == 0), ENOMEM, EHIP. */
symtile_status symtile_heap_create(int device, int world_size, size_t slot_bytes,
                                   symtile_heap** out);

/* Same, over caller-owned device memory [base, base + total_bytes) on
 * `device` (e.g. a framework tensor).  base must be 256-byte aligned and
 * total_bytes >= world_size * slot stride.  The memory is not zeroed and is
 * never freed by the library; it must outlive the heap. */
symtile_status symtile_heap_create_on(int device, int world_size, size_t slot_bytes,
                                      void* base, size_t total_bytes, symtile_heap** out);

/* Release the heap (and its memory if the library allocated it).  Waits for
 * the device.  NULL is accepted. */
symtile_status symtile_heap_destroy(symtile_heap* h);

/* Symmetric bump allocation: reserve `bytes` at the same offset in every
 * slot, aligned to `align` (a power of two; 0 = 256).  *offset_out receives
 * the offset from the slot base.  No per-allocation free.  ENOMEM when the
 * slot is full. */
symtile_status symtile_heap_alloc(symtile_heap* h, size_t bytes, size_t align,
                                  size_t* offset_out);

/* Device address of `offset` in slot `rank`: the symmetric object at that
 * offset as rank `rank` holds it (Section 3.2.3, tensors in the symmetric
 * heap).  EINVAL for a bad rank or an offset past the slot. */
symtile_status symtile_heap_ptr(const symtile_heap* h, int rank, size_t offset, void** out);

/* Heap geometry (Section 3.2.1, get_num_ranks): world size, slot stride,
 * bytes allocated per slot, device.  Any output may be NULL. */
symtile_status symtile_heap_info(const symtile_heap* h, int* world_size, size_t* slot_stride,
                                 size_t* used, int* device);

/* Per-rank heap bases (Section 3.2, get_heap_bases).  *dev_bases receives
 * the device array of world_size uint64 addresses (owned by the heap);
 * host_bases, if non-NULL, receives a copy (world_size entries). */
symtile_status symtile_heap_bases(const symtile_heap* h, const uint64_t** dev_bases,
                                  uint64_t* host_bases);

/* Host twin of the device translation (Section 3.3.1): for p inside slot
 * from_rank, *out = base[to_rank] + (p - base[from_rank]).  EINVAL when p is
 * not inside slot from_rank or a rank is out of range. */
symtile_status symtile_translate(const symtile_heap* h, const void* p, int from_rank,
                                 int to_rank, void** out);

/* Device translation (Section 3.3.1) applied to n addresses: out[i] =
 * translate(in[i], from_rank, to_rank) computed by a kernel with the same
 * device routine the hot path uses.  in and out are device arrays of n uint64.  Addresses are
 * not range-checked on the device (the caller checks with the host twin). */
symtile_status symtile_translate_device(const symtile_heap* h, const uint64_t* in, int n,
                                        int from_rank, int to_rank, uint64_t* out,
                                        symtile_stream s);

/* Host barrier (Section 3.2, barrier): wait for the stream (device when
 * NULL), then read and clear the heap's device error word.  Returns
 * ETIMEOUT if a device-side wait expired since the last barrier; EINVAL if a
 * split-K call found its workspace counters non-zero at entry (that call
 * skipped the affected tiles); EHIP for any other device error. */
symtile_status symtile_barrier(symtile_heap* h, symtile_stream s);

/* Fill `bytes` at `offset` of slot `rank` (every slot when rank < 0) with
 * the byte `value` (Section 3.2.3, tensor creation: zeros / full in the
 * symmetric heap), with a fill kernel on stream s (no memset node, so it may
 * be captured into a graph).  EINVAL for a bad rank or a range past the slot. */
symtile_status symtile_heap_fill(symtile_heap* h, int rank, size_t offset, size_t bytes,
                                 int value, symtile_stream s);

/* ---- device API exercise (Section 3.3.3) --------------------------------- */

/* n_threads device threads each apply atomic `op` with ordering `sem` and
 * scope `scope` to the uint32 at `offset` of slot to_rank, reached by
 * translating the address of `offset` in slot from_rank.  Thread t uses
 * operand + t (ADD/AND/OR/XOR/MIN/MAX/XCHG) or compares with `compare`
 * and swaps in operand + t (CAS).  If old_out (device, n_threads uint32) is
 * non-NULL, thread t writes the value it observed there.  Orderings that
 * do not apply to a read-modify-write are rejected with EINVAL. */
symtile_status symtile_atomic_exercise(symtile_heap* h, int op, int sem, int scope,
                                       size_t offset, int from_rank, int to_rank,
                                       int n_threads, uint32_t operand, uint32_t compare,
                                       uint32_t* old_out, symtile_stream s);

/* Value-based verbs of the device API (Section 3.3.2, load and store). */
typedef enum { SYMTILE_LOAD = 0, SYMTILE_STORE = 1 } symtile_value_op;

/* Moves `bytes` between slot cur_rank and slot remote_rank, one 16-byte
 * vector per device thread. The remote address is always found by
 * translating the address of the same offset in slot cur_rank.
 * - LOAD: each vector is read with the device `load` verb from
 *   remote_rank's slot at src_off and written to cur_rank's own slot at
 *   dst_off.
 * - STORE: each vector is read from cur_rank's own slot at src_off and
 *   written with the device `store` verb to remote_rank's slot at dst_off.
 * Either way, the destination ends up holding a bitwise copy of the source.
 * With nontemporal = 1 the destination writes are nontemporal.
 * Arguments:
 * - offsets must be 16-byte aligned, and bytes a multiple of 16;
 * - both regions must lie inside the slot, and they must not overlap when
 *   cur_rank == remote_rank;
 * - otherwise, or for a bad op or rank, the call returns EINVAL.
 * bytes = 0 launches nothing.
 * The call is asynchronous on stream s, and memory ordering is relaxed. */
symtile_status symtile_value_exercise(symtile_heap* h, int op, size_t src_off, size_t dst_off,
                                      size_t bytes, int cur_rank, int remote_rank,
                                      int nontemporal, symtile_stream s);

/* Forms of the message-passing litmus test: how the counters publish and wait. */
typedef enum {
    SYMTILE_MP_RELAXED = 0,  /* relaxed +1, relaxed polls, no fences (no guarantee) */
    SYMTILE_MP_FENCES = 1,   /* release fence + relaxed +1; relaxed polls + acquire fence */
    SYMTILE_MP_RMW = 2,      /* fetch_add(+1, release); polls by fetch_add(0, acquire) */
    SYMTILE_MP_CAS = 3,      /* cas(i-1 -> i, release); polls by cas(i -> i, acquire), the lock
                                handshake of the workgroup-specialised listing (Section 4.2.2) */
    SYMTILE_MP_WT = 4,       /* data stored write-through (the stores' cache-policy bits
                                sc0 sc1), released by waiting for their acknowledgement
                                only (no L2 write-back), relaxed +1; relaxed polls +
                                acquire fence (the kernels' write-through publication) */
    SYMTILE_MP_ACK = 5,      /* the same release with ordinary write-back data stores:
                                the control, which the write-back fence exists for */
    SYMTILE_MP_WT_COHERENT = 6, /* SYMTILE_MP_WT's writer; the reader polls, then reads
                                the data with coherent loads (sc0 sc1) and no acquire
                                fence (no L2 invalidate) */
    SYMTILE_MP_WT_PLAIN = 7  /* SYMTILE_MP_WT's writer; the reader polls and reads with
                                ordinary loads, no acquire fence: the control */
} symtile_mp_form;

/* Message-passing litmus test of the flag protocol (Section 3.3.3, memory
 * model: atomics with an ordering and a scope).  pairs writer/reader
 * workgroup pairs (pair p: writer rank p % w, reader rank (p + 1) % w, placed
 * on different XCDs) run `rounds` rounds: the writer writes `words` uint32 of
 * a round-specific pattern into the reader's slot at data_off + 4 * words *
 * p, then publishes a counter in the reader's slot (flag_off + 8p) in the
 * given form at the given scope (symtile_scope); the reader waits for it,
 * checks every word, and acknowledges through a counter in the writer's slot
 * (flag_off + 8p + 4) the same way.  In the RELAXED and FENCES forms the
 * counters are updated and polled at agent scope or wider (only the data's
 * ordering depends on `scope`); in RMW and CAS the counters take `scope`.
 * result (device, 2 uint32, zeroed by the caller) accumulates [0] words that
 * did not hold the round's value when read and [1] rounds checked.  The
 * counters must be zero on entry.  Every wait is bounded by spin_limit polls
 * (0 = 1<<22); a timeout records ETIMEOUT for the next symtile_barrier and
 * ends the pair (its partner then times out as well).  EINVAL for bad sizes,
 * regions, form or scope; EUNSUPPORTED when 2*pairs exceeds the CU count
 * (all must be resident). */
symtile_status symtile_litmus_mp(symtile_heap* h, size_t data_off, size_t flag_off, int pairs,
                                 int rounds, int words, int form, int scope, uint32_t spin_limit,
                                 uint32_t* result, symtile_stream s);

/* Forms of the store-buffering litmus test. */
typedef enum {
    SYMTILE_SB_RELAXED = 0,  /* relaxed atomic store, relaxed atomic load */
    SYMTILE_SB_ACQ_REL = 1,  /* exchange and fetch_add(0), both acq_rel */
    SYMTILE_SB_SEQ_CST = 2   /* seq_cst atomic store, seq_cst atomic load */
} symtile_sb_form;

/* Store-buffering litmus test (Section 3.3.3, memory model).  pairs pairs of
 * single threads (pair p: side 0 on rank p % w, side 1 on rank (p + 1) % w,
 * on different XCDs) run `rounds` rounds; round i of pair p uses the 16
 * bytes at flag_off + 16 * (p * rounds + i) of the two slots, which must be
 * zero on entry: x (word 0, side 1's slot), y (word 1, side 0's slot) and an
 * arrival counter (word 2, side 0's slot).  Both sides arrive and wait for
 * each other (bounded by spin_limit, 0 = 1<<22), then side 0 writes x = 1 and
 * reads y while side 1 writes y = 1 and reads x, in the given form at the
 * given scope.  out (device uint32 [pairs][rounds][2]) receives what each
 * side read, or 2 for a round not run after a timeout (ETIMEOUT at the next
 * symtile_barrier).  Both sides reading 0 is forbidden in the ACQ_REL and
 * SEQ_CST forms.  EINVAL for bad sizes, regions, form or scope;
 * EUNSUPPORTED when 2*pairs exceeds the CU count. */
symtile_status symtile_litmus_sb(symtile_heap* h, size_t flag_off, int pairs, int rounds,
                                 int form, int scope, uint32_t spin_limit, uint32_t* out,
                                 symtile_stream s);

/* ---- heap tile copy (Section 3.3.2, pointer-based put and get) ------------ */

/* Direction of symtile_tile_copy for executing rank r (Section 3.3.2 device
 * API table): PUT copies r's own buffer into rank (r + shift) mod w's (the
 * write is remote); GET copies rank (r - shift) mod w's buffer into r's own
 * (the read is remote).  Both leave the same post-state. */
typedef enum { SYMTILE_PUT = 0, SYMTILE_GET = 1 } symtile_copy_mode;

/* For every executing rank r (all ranks when only_rank < 0, else only_rank),
 * copy the rows x cols matrix at offset src_off of the source slot, tile by
 * tile (tile_r x tile_c, ragged edge tiles included), to offset dst_off of
 * the destination slot (PUT: source r, destination (r + shift) mod w; GET:
 * source (r - shift) mod w, destination r; addresses reached by translating
 * rank r's), then release-publish (agent scope) one uint32 counter per tile
 * at flag_off + 4 * tile of the destination slot (tile = tr * tiles_c + tc).
 * Row stride `ld` elements; element size from dtype (2 or 4 bytes).  All
 * ranks run in one launch.  Each workgroup copies tiles_per_wg consecutive
 * (rank, tile) items and publishes their counters after one release
 * (0 = about one workgroup per CU).  Requirements: cols*esize, tile_c*esize
 * and ld*esize multiples of 16; offsets 16-byte aligned; regions inside the
 * slot; the source and destination regions must not overlap; (tile_r + the
 * rows of kBatch passes) * ld*esize below 2 GiB.  EINVAL otherwise. */
symtile_status symtile_tile_copy(symtile_heap* h, size_t src_off, size_t dst_off, int rows,
                                 int cols, int ld, int dtype, int tile_r, int tile_c,
                                 int shift, int only_rank, size_t flag_off, int tiles_per_wg,
                                 int mode, symtile_stream s);

/* symtile_tile_copy launched with hipExtLaunchKernel, which records two
 * events as part of the kernel's own dispatch instead of as separate marker
 * packets around it, for measurement: the call waits for the kernel and
 * *kernel_ms receives the elapsed time between the events in milliseconds
 * (0 when nothing is launched): the kernel's duration plus less dispatch
 * overhead than a pair of stream events around the launch holds.  The
 * result in the heap is the same as symtile_tile_copy's.  The events belong
 * to the heap (created on first use).  Errors: those of symtile_tile_copy;
 * EINVAL for a NULL kernel_ms; EHIP when the events cannot be created or read. */
symtile_status symtile_tile_copy_timed(symtile_heap* h, size_t src_off, size_t dst_off, int rows,
                                       int cols, int ld, int dtype, int tile_r, int tile_c,
                                       int shift, int only_rank, size_t flag_off,
                                       int tiles_per_wg, int mode, symtile_stream s,
                                       float* kernel_ms);

/* ---- GEMM + All-Scatter (Section 4, case study) --------------------------- */

/* Bytes of the split-K workspace (symtile_gas_config.workspace) of a call
 * with this output shape, tile and split_k.  Splitting the K loop of the GEMM
 * main-loop listing (Section 4) is this library's addition for shapes with
 * fewer output tiles than CUs; the slices meet through this workspace: two
 * uint32 counters per tile
 * (rounded up to 256 bytes), then split_k fp32 partial tiles of
 * tile_m * tile_n values per tile.  *bytes = 0 when split_k <= 1.  EINVAL for
 * negative sizes, a tile shape that is not built (see tile_m, tile_n above)
 * or split_k outside 0..64. */
symtile_status symtile_gas_workspace_bytes(int M, int N_local, int tile_m, int tile_n,
                                           int split_k, size_t* bytes);

/* Rank `rank`'s share: C_r = A * B_shard with an fp32 accumulator (Section 4
 * GEMM main loop), rounded to the input dtype (nearest even), stored into the
 * rank's column block [rank*N_local, (rank+1)*N_local) of the gathered output
 * in EVERY slot, own slot included (Section 4.2.1), with one arrival counter
 * per tile per slot incremented with release semantics at agent scope after
 * that tile's data is in that slot.
 *
 *  A              device [M, K] row-major, row stride lda (>= K) elements;
 *                 any device memory (need not be in the heap).
 *  B_shard        device [K, N_local] row-major, row stride ldb (>= N_local).
 *  C_gathered_local  address inside slot `rank` of the gathered output
 *                 [M, world_size*N_local] row-major (row stride
 *                 world_size*N_local); the same offset is written in every
 *                 slot.
 *  arrived_local  address inside slot `rank` of the counters
 *                 uint32 [world_size][tiles_m][tiles_n] (rank-major), tiles
 *                 of cfg tile size; slot s receives arrived[rank][m][n] += 1.
 *  ready          WG_SPEC only: device uint32 [tiles_m*tiles_n] of
 *                 producer->consumer counters (any device memory), each
 *                 equal to cfg->epoch - 1 on entry; ignored (may be NULL)
 *                 for the other variants.
 *  dtype          SYMTILE_F16 or SYMTILE_BF16, for A, B and C.
 *
 * Requirements: K, N_local, lda, ldb multiples of 8; A and B 16-byte
 * aligned; M, N_local, K >= 0 (zero sizes are no-ops except K == 0, which
 * stores zeros).  WG_SPEC requires gemm_wgs + copy_wgs workgroups to be
 * co-resident (checked; EUNSUPPORTED otherwise).  A consumer wait that
 * exceeds cfg->spin_limit polls records ETIMEOUT for the next
 * symtile_barrier, and that consumer abandons its remaining tiles.  With
 * split_k > 1 the slice that finishes a tile last waits (bounded by
 * cfg->spin_limit) only for slices that have already started; a timeout
 * records ETIMEOUT and leaves that tile unwritten and unpublished.  split_k > 1
 * with another variant is EUNSUPPORTED; without a large enough workspace, or
 * with split_k above ceil(K/32), EINVAL. */
symtile_status symtile_gemm_all_scatter(symtile_heap* h, const void* A, const void* B_shard,
                                        void* C_gathered_local, uint32_t* arrived_local,
                                        uint32_t* ready, int M, int N_local, int K, int lda,
                                        int ldb, int dtype, int rank, int world_size,
                                        const symtile_gas_config* cfg, symtile_stream s);

/* Bytes of the scratch behind symtile_gemm_all_scatter_noalloc: 64 MiB of
 * fp32 partial tiles plus 64 KiB of tile counters (the split-K workspace of
 * the fp16 8192x8192 x 8192x1024 problem with 256x256 tiles in 2 K slices
 * fits). */
#define SYMTILE_NOALLOC_SCRATCH_BYTES ((64u << 20) + (64u << 10))

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): the same call as
 * symtile_gemm_all_scatter, with the same arguments, results and errors, but
 * the split-K workspace comes from a scratch array the library keeps in
 * static device memory, SYMTILE_NOALLOC_SCRATCH_BYTES per GPU, held from the
 * library's first use on that GPU until the process ends.  The call makes no
 * hipMalloc or hipFree and calls no allocating library routine.
 *  - cfg->workspace must be NULL and cfg->workspace_bytes 0 (EINVAL otherwise);
 *  - a split_k > 1 call whose workspace (symtile_gas_workspace_bytes) exceeds
 *    the scratch returns EINVAL and launches nothing;
 *  - the scratch's counters are zeroed by a kernel at the start of every
 *    split_k > 1 call (no memset node), so a timed-out earlier call leaves
 *    nothing behind for the next one;
 *  - UNFUSED_PC is EUNSUPPORTED (it creates a stream and events on first use);
 *  - every call on one GPU shares that GPU's scratch: split_k > 1 calls that
 *    overlap in time on one GPU (other streams, other threads) race and give
 *    wrong results.  Calls on one stream are ordered and safe.
 * The scratch's device address is looked up (hipGetSymbolAddress) on the
 * first split_k > 1 call on each device. */
symtile_status symtile_gemm_all_scatter_noalloc(symtile_heap* h, const void* A,
                                                const void* B_shard, void* C_gathered_local,
                                                uint32_t* arrived_local, uint32_t* ready, int M,
                                                int N_local, int K, int lda, int ldb, int dtype,
                                                int rank, int world_size,
                                                const symtile_gas_config* cfg, symtile_stream s);

/* Rate of the realtime counter behind trace timestamps (the per-tile
 * timeline of Section 3.4, instrumentation), in kHz.  EINVAL for a bad device
 * or NULL khz. */
symtile_status symtile_clock_rate_khz(int device, int* khz);

/* Number of compute units of `device` and the largest WG_SPEC grid
 * (gemm_wgs + copy_wgs) that is co-resident for the given tile shape: the
 * budget the workgroup-specialised schedule splits between producers and
 * consumers (Section 4.2.2).  EUNSUPPORTED for a tile shape not built. */
symtile_status symtile_device_info(int device, int tile_m, int tile_n, int* cu_count,
                                   int* max_coresident_wgs);

/* Thread-local message of the last failure in this thread ("" if none); the
 * error channel of this C ABI, which the paper's Python API does not need. */
const char* symtile_last_error(void);

/* Library version string (names the GPU target). */
const char* symtile_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SYMTILE_H */
