"""Host-side conveniences over the C ABI: a heap whose memory is a torch
tensor (so slots are zero-copy torch views, as the host API of Section 3.2
returns tensors living in the heap), and the symmetric buffers of one
GEMM + All-Scatter problem.  Argument marshalling only."""
from __future__ import annotations

import ctypes

import torch

from . import _binding as B

_SLOT_ALIGN = 2 << 20


# The raw handle of the current stream, without building a torch Stream object
# (which costs microseconds on every call's launch path); the public accessor
# when this torch has no raw one.
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def current_stream(device: int | None = None) -> int:
    """The current torch stream of ``device`` (default: the current device)
    as a raw stream handle."""
    if _raw_stream is not None:
        return _raw_stream(torch.cuda.current_device() if device is None else device)
    return torch.cuda.current_stream(device).cuda_stream


class Heap:
    """A symmetric heap of ``world`` slots on one GPU.

    Memory is a torch uint8 tensor (torch's allocator; the library never frees
    it) zeroed at creation; ``view`` returns a tensor aliasing one slot."""

    def __init__(self, world: int, slot_bytes: int, device: int = 0):
        self.world = world
        self.device = device
        self.stride = (slot_bytes + _SLOT_ALIGN - 1) // _SLOT_ALIGN * _SLOT_ALIGN
        self.mem = torch.zeros(world * self.stride, dtype=torch.uint8, device=f"cuda:{device}")
        self.handle = B.symtile_heap_create_on(device, world, slot_bytes, self.mem.data_ptr(),
                                               self.mem.numel())
        w, stride, _, _ = B.symtile_heap_info(self.handle)
        assert w == world and stride == self.stride
        self.failed_barriers = 0     # barriers that reported ETIMEOUT or a stale workspace

    def close(self) -> None:
        if self.handle:
            B.symtile_heap_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def alloc(self, nbytes: int, align: int = 256) -> int:
        return B.symtile_heap_alloc(self.handle, nbytes, align)

    def ptr(self, rank: int, offset: int) -> int:
        return B.symtile_heap_ptr(self.handle, rank, offset)

    def bases(self):
        return B.symtile_heap_bases(self.handle)

    def view(self, rank: int, offset: int, shape, dtype: torch.dtype) -> torch.Tensor:
        """Tensor of ``shape``/``dtype`` aliasing ``offset`` of slot ``rank``."""
        n = 1
        for d in shape:
            n *= d
        esize = torch.empty((), dtype=dtype).element_size()
        start = rank * self.stride + offset
        if offset % esize or offset + n * esize > self.stride:
            raise ValueError("view outside the slot or misaligned")
        return self.mem[start:start + n * esize].view(dtype).view(*shape)

    def slots_view(self, offset: int, shape, dtype: torch.dtype) -> torch.Tensor:
        """[world, *shape] strided view of the same object in every slot."""
        esize = torch.empty((), dtype=dtype).element_size()
        if self.stride % esize:
            raise ValueError("slot stride not a multiple of the element size")
        flat = self.mem.view(dtype)
        n = 1
        for d in shape:
            n *= d
        base = offset // esize
        strides = [self.stride // esize]
        acc = 1
        tail = []
        for d in reversed(shape):
            tail.append(acc)
            acc *= d
        strides += list(reversed(tail))
        return flat.as_strided([self.world, *shape], strides, base)

    def barrier(self, stream: int | None = None) -> None:
        """symtile_barrier.  A reported timeout or stale split-K workspace
        bumps ``failed_barriers``, so the GatheredOutput objects of this heap
        zero their split-K workspaces before their next split-K call (the
        barrier has drained the stream, so no slice of the failed call is
        still running)."""
        try:
            B.symtile_barrier(self.handle, current_stream() if stream is None else stream)
        except B.SymtileError as e:
            if e.name in ("ETIMEOUT", "EINVAL"):
                self.failed_barriers += 1
            raise

    def fill(self, rank: int, offset: int, nbytes: int, value: int,
             stream: int | None = None) -> None:
        B.symtile_heap_fill(self.handle, rank, offset, nbytes, value,
                            current_stream() if stream is None else stream)


def _tiles(n: int, t: int) -> int:
    return (n + t - 1) // t


class GatheredOutput:
    """The symmetric objects of one GEMM + All-Scatter problem in ``heap``:
    the gathered output [M, w*N_local] and the arrival counters
    [w, tiles_m, tiles_n], plus a (non-symmetric) ready counter array."""

    def __init__(self, heap: Heap, M: int, N_local: int, dtype: torch.dtype,
                 tile_m: int, tile_n: int):
        self.heap = heap
        self.M, self.N_local, self.dtype = M, N_local, dtype
        self.tile_m, self.tile_n = tile_m, tile_n
        self.tiles_m, self.tiles_n = _tiles(M, tile_m), _tiles(N_local, tile_n)
        w = heap.world
        self.c_bytes = M * w * N_local * 2
        self.c_off = heap.alloc(max(self.c_bytes, 16), 256)
        self.flag_count = w * self.tiles_m * self.tiles_n
        self.flag_off = heap.alloc(max(self.flag_count * 4, 4), 256)
        self.ready = torch.zeros(max(self.tiles_m * self.tiles_n, 1), dtype=torch.int32,
                                 device=heap.mem.device)
        self.ready_epoch = 0     # value of every ready counter after the last WG_SPEC call
        self.ws = None           # split-K workspace (uint8 device tensor), grown on demand
        self.ws_seen = heap.failed_barriers   # failed barriers already answered by a reset
        # per-call constants, computed once (run() is on the host's launch path):
        # the output's and counters' addresses per rank, the workspace size per
        # slice count, and one config struct filled in by every call
        self._ptrs = {}
        self._ws_need = {}
        self._cfg = B.GasConfig()
        self._cfg_ref = ctypes.byref(self._cfg)
        self._dt = B.BF16 if dtype == torch.bfloat16 else B.F16

    def C(self, rank: int) -> torch.Tensor:
        return self.heap.view(rank, self.c_off, (self.M, self.heap.world * self.N_local),
                              self.dtype)

    def C_all(self) -> torch.Tensor:
        return self.heap.slots_view(self.c_off, (self.M, self.heap.world * self.N_local),
                                    self.dtype)

    def arrived(self, rank: int) -> torch.Tensor:
        return self.heap.view(rank, self.flag_off,
                              (self.heap.world, self.tiles_m, self.tiles_n), torch.int32)

    def arrived_all(self) -> torch.Tensor:
        return self.heap.slots_view(self.flag_off, (self.heap.world, self.tiles_m, self.tiles_n),
                                    torch.int32)

    def workspace(self, split_k: int) -> torch.Tensor | None:
        """The split-K workspace for ``split_k`` slices (None when split_k <= 1):
        a zeroed uint8 device tensor, kept and reused by later calls (each call
        leaves its counters at zero), replaced by a larger one when needed."""
        need = self._ws_need.get(split_k)
        if need is None:
            need = self._ws_need[split_k] = B.symtile_gas_workspace_bytes(
                self.M, self.N_local, self.tile_m, self.tile_n, split_k)
        if need == 0:
            return None
        if self.ws is None or self.ws.numel() < need:
            self.ws = None
            self.ws = torch.zeros(need, dtype=torch.uint8, device=self.heap.mem.device)
        elif self.ws_seen != self.heap.failed_barriers:
            self.ws.zero_()      # a timed-out call may have left its counters non-zero
        self.ws_seen = self.heap.failed_barriers
        return self.ws

    def reset_workspace(self) -> None:
        """Zero the split-K workspace (its counters are left non-zero only by a
        call whose wait timed out, reported as ETIMEOUT by the heap barrier)."""
        if self.ws is not None:
            self.ws.zero_()

    def new_trace(self) -> torch.Tensor:
        """Zeroed per-tile trace buffer [tiles_m * tiles_n, 8] (int64, on the
        heap's device); tile (m, n) is row m * tiles_n + n."""
        return torch.zeros((self.tiles_m * self.tiles_n, B.TRACE_WORDS), dtype=torch.int64,
                           device=f"cuda:{self.heap.device}")

    def run(self, A: torch.Tensor, B_shard: torch.Tensor, rank: int, variant: int,
            gemm_wgs: int = 0, copy_wgs: int = 0, nontemporal: int = 0, group_m: int = 0,
            spin_limit: int = 0, epoch: int | None = None, stream: int | None = None,
            waves_per_wg: int = 0, trace: torch.Tensor | None = None,
            copy_stream: int | None = None, split_k: int = 0, split_reduce: int = 0) -> None:
        """One call of rank ``rank`` (enqueued on the stream, asynchronous).
        For WG_SPEC, ``epoch`` (the value consumers wait for) defaults to one
        more than after the previous WG_SPEC call on these buffers.
        ``trace``: optional int64 device tensor from new_trace(), filled with
        the per-tile timeline of this call.  ``copy_stream``: UNFUSED_PC's
        copy-kernel stream (default: one the heap creates).  ``split_k`` > 1
        (BULK_SYNC, FUSED_SEQ): each tile is computed as that many K slices,
        with this object's workspace; calls on one object that use split-K
        must not overlap in time.  ``split_reduce``: SPLIT_REDUCE_AUTO (0),
        SPLIT_REDUCE_LAST, SPLIT_REDUCE_BANDED or SPLIT_REDUCE_KERNEL (who sums
        the slices).  The call only launches kernels on the stream, so it can
        be captured in a graph (torch.cuda.graph) and replayed, except WG_SPEC
        and UNFUSED_PC, whose epoch is fixed at capture; make one eager split-K
        call first so that the workspace exists before the capture."""
        if A.dtype != self.dtype or B_shard.dtype != self.dtype:
            raise TypeError("A and B_shard must have the output dtype")
        if not (A.is_cuda and B_shard.is_cuda and A.is_contiguous() and B_shard.is_contiguous()):
            raise ValueError("A and B_shard must be contiguous device tensors")
        M, K = A.shape
        K2, N = B_shard.shape
        if M != self.M or N != self.N_local or K2 != K:
            raise ValueError("shape mismatch")
        if variant in (B.WG_SPEC, B.UNFUSED_PC):
            self.ready_epoch = self.ready_epoch + 1 if epoch is None else epoch
        if trace is not None and (not trace.is_cuda or trace.dtype != torch.int64 or
                                  not trace.is_contiguous() or
                                  trace.numel() < self.tiles_m * self.tiles_n * B.TRACE_WORDS):
            raise ValueError("trace must be a contiguous int64 device tensor from new_trace()")
        ptrs = self._ptrs.get(rank)
        if ptrs is None:
            ptrs = self._ptrs[rank] = (self.heap.ptr(rank, self.c_off),
                                       self.heap.ptr(rank, self.flag_off))
        cfg = self._cfg
        cfg.variant, cfg.tile_m, cfg.tile_n = variant, self.tile_m, self.tile_n
        cfg.gemm_wgs, cfg.copy_wgs, cfg.epoch = gemm_wgs, copy_wgs, max(self.ready_epoch, 1)
        cfg.spin_limit, cfg.nontemporal, cfg.group_m = spin_limit, nontemporal, group_m
        cfg.waves_per_wg, cfg.copy_stream = waves_per_wg, copy_stream
        cfg.trace = trace.data_ptr() if trace is not None else None
        cfg.split_k, cfg.split_reduce = split_k, split_reduce
        cfg.workspace, cfg.workspace_bytes = None, 0
        ws = self.workspace(split_k) if split_k > 1 else None
        if ws is not None:               # None: no tiles, nothing to keep
            cfg.workspace, cfg.workspace_bytes = ws.data_ptr(), ws.numel()
        st = B.lib.symtile_gemm_all_scatter(
            self.heap.handle, A.data_ptr(), B_shard.data_ptr(), ptrs[0], ptrs[1],
            self.ready.data_ptr(), M, N, K, K, N, self._dt, rank, self.heap.world,
            self._cfg_ref, current_stream(self.heap.device) if stream is None else stream)
        if st:
            B._check(st, "symtile_gemm_all_scatter")
