"""Caller-side runtime around libmori: the device-resident tier state of one KV
pool, the CPU tier's pinned arena, and one rebalance step.

torch provides device memory and streams only; every step of the placement
and of the byte movement runs in libmori's kernels.  Host extents of the CPU
tier are the caller's business (the library takes one address per program):
here they are first-fit extents inside one pinned, device-mapped arena.
"""
from __future__ import annotations

import bisect
import ctypes as C
import os
from dataclasses import dataclass

import numpy as np
import torch

from . import mori as M


class MoriError(RuntimeError):
    def __init__(self, what: str, code: int, detail: int = 0):
        super().__init__(f"{what}: {M.mori_strerror(code)} ({code}), device bits {detail:#x}")
        self.code = code
        self.detail = detail


def check(rc: int, what: str) -> None:
    if rc != M.MORI_OK:
        raise MoriError(what, rc)


class FirstFit:
    """First-fit allocator of byte extents inside one arena (offsets aligned)."""

    def __init__(self, capacity: int, align: int = 4096):
        self.capacity = capacity
        self.align = align
        self.free = [(0, capacity)]
        self.used = {}

    def alloc(self, size: int):
        size = max(self.align, -(-size // self.align) * self.align)
        for j, (s, n) in enumerate(self.free):
            if n >= size:
                self.free[j:j + 1] = [] if n == size else [(s + size, n - size)]
                self.used[s] = size
                return s
        return None

    def release(self, off: int) -> None:
        """Returns an extent, merged with free neighbours (free list kept sorted
        by offset: a binary search and at most two merges)."""
        size = self.used.pop(off)
        i = bisect.bisect_left(self.free, (off, 0))
        if i > 0 and self.free[i - 1][0] + self.free[i - 1][1] == off:
            i -= 1
            off, size = self.free[i][0], self.free[i][1] + size
            del self.free[i]
        if i < len(self.free) and off + size == self.free[i][0]:
            size += self.free[i][1]
            del self.free[i]
        self.free.insert(i, (off, size))

    @property
    def bytes_used(self) -> int:
        return sum(self.used.values())


class HostArena:
    """Pinned, device-mapped host memory holding the CPU tier."""

    def __init__(self, nbytes: int, align: int = 4096):
        rc, ptr = M.mori_host_alloc(nbytes)
        check(rc, f"mori_host_alloc({nbytes})")
        self.ptr = ptr
        self.nbytes = nbytes
        self.fit = FirstFit(nbytes, align)

    def view(self, addr: int, n: int) -> np.ndarray:
        """uint8 numpy view of n bytes at an absolute address inside the arena."""
        assert self.ptr <= addr and addr + n <= self.ptr + self.nbytes
        if n == 0:
            return np.zeros(0, np.uint8)
        return np.ctypeslib.as_array((C.c_uint8 * n).from_address(addr))

    def close(self) -> None:
        if self.ptr:
            M.mori_host_free(self.ptr)
            self.ptr = 0


@dataclass
class PoolGeometry:
    layers: int
    planes: int
    block_tokens: int
    row_bytes: int
    num_blocks: int

    @property
    def run_bytes(self) -> int:
        return self.block_tokens * self.row_bytes

    @property
    def block_bytes(self) -> int:
        return self.layers * self.planes * self.run_bytes

    @property
    def pool_bytes(self) -> int:
        return self.layers * self.planes * self.num_blocks * self.run_bytes


def hw_queues() -> int:
    """Hardware queues per process HIP creates (GPU_MAX_HW_QUEUES when it
    starts; its default is 4)."""
    try:
        n = int(os.environ.get("GPU_MAX_HW_QUEUES", "4"))
    except ValueError:
        return 4
    return n if n > 0 else 4


def _u32_dev(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, np.uint32).view(np.int32).copy()).to(device)


class TierPool:
    """One KV pool in HBM, its block tables / tiers / free map in HBM, a pinned
    host arena for the CPU tier, and a libmori context."""

    def __init__(self, geom, tbl_off, tbl, tier, free_map, arena_bytes: int, max_programs: int | None = None,
                 staging_bytes: int = 0, device: str = "cuda", pool: torch.Tensor | None = None,
                 copy_streams: bool | None = None):
        """copy_streams: let the context own a copy stream per direction
        (MORI_CREATE_COPY_STREAMS), which needs 8 hardware queues in the
        process; None: decided from GPU_MAX_HW_QUEUES as this process set it
        before HIP started."""
        self.geom = PoolGeometry(geom.layers, geom.planes, geom.block_tokens, geom.row_bytes, geom.num_blocks)
        self.device = torch.device(device)
        self.P = int(tier.size)
        self.nblk = np.diff(np.asarray(tbl_off, np.int64)).astype(np.int64)
        if pool is None:
            pool = torch.empty(self.geom.pool_bytes, dtype=torch.uint8, device=self.device)
        assert pool.dtype == torch.uint8 and pool.numel() == self.geom.pool_bytes and pool.is_contiguous()
        self.pool = pool
        self.tbl_off = _u32_dev(tbl_off, self.device)
        self.tbl = _u32_dev(tbl if len(tbl) else np.zeros(1, np.uint32), self.device)
        self.tbl_len = int(len(tbl))
        self.tier = torch.from_numpy(np.ascontiguousarray(tier, np.uint8).copy()).to(self.device)
        self.free_map = torch.from_numpy(np.ascontiguousarray(free_map, np.uint8).copy()).to(self.device)
        self.arena = HostArena(arena_bytes)
        self.host_off = {}  # program -> arena offset of its CPU-tier buffer
        self.host_addr = np.zeros(max(self.P, 1), np.uint64)
        self._pool_desc = M.mori_pool(self.geom.layers, self.geom.planes, self.geom.block_tokens,
                                      self.geom.row_bytes, self.geom.num_blocks, self.pool.data_ptr())
        if copy_streams is None:
            copy_streams = hw_queues() >= 8
        rc, self.ctx = M.mori_create(self._pool_desc, max_programs or max(self.P, 1), staging_bytes,
                                     M.MORI_CREATE_COPY_STREAMS if copy_streams else 0)
        check(rc, "mori_create")
        check(M.mori_register(self.ctx, self.arena.ptr, self.arena.nbytes), "mori_register(arena)")
        self._keep = []
        self.plan = None

    # ---- host extents -------------------------------------------------------
    def program_bytes(self, p: int) -> int:
        return int(self.nblk[p]) * self.geom.block_bytes

    def host_view(self, p: int) -> np.ndarray:
        return self.arena.view(int(self.host_addr[p]), self.program_bytes(p))

    def give_host_buffer(self, p: int) -> None:
        off = self.arena.fit.alloc(self.program_bytes(p))
        if off is None:
            raise MoriError(f"CPU-tier arena full (program {p}, {self.program_bytes(p)} B)", M.MORI_ENOSPC)
        self.host_off[p] = off
        self.host_addr[p] = self.arena.ptr + off

    def drop_host_buffer(self, p: int) -> None:
        off = self.host_off.pop(p, None)
        if off is not None:
            self.arena.fit.release(off)
        self.host_addr[p] = 0

    # ---- the three calls -----------------------------------------------------
    def rank_partition(self, *, gpu_bytes: int, cpu_bytes: int, window: torch.Tensor | None = None,
                       idleness: torch.Tensor | None = None, status: torch.Tensor | None = None, flags: int = 0,
                       stream: torch.cuda.Stream | None = None, ssd_bytes: int = 0) -> int:
        k = int(window.shape[1]) if window is not None else 0
        prog = M.mori_programs(self.P, k, window.data_ptr() if window is not None else None,
                               idleness.data_ptr() if idleness is not None else None,
                               status.data_ptr() if status is not None else None, self.tbl_off.data_ptr(),
                               self.tbl_len, self.tbl.data_ptr(), self.tier.data_ptr(), self.free_map.data_ptr())
        self._keep = [window, idleness, status]
        budget = M.mori_budget(int(gpu_bytes), int(cpu_bytes), int(flags), int(ssd_bytes))
        return M.mori_rank_partition(self.ctx, prog, budget, _stream(stream))

    def plan_wait(self):
        rc, p = M.mori_plan_wait(self.ctx)
        self.plan = p
        return rc, p

    def plan_arrays(self, p=None) -> dict:
        p = p or self.plan
        P = self.P
        arr = lambda ptr, n, dt: np.ctypeslib.as_array(ptr, shape=(n,)).astype(dt) if n else np.zeros(0, dt)
        return dict(order=arr(p.order, P, np.uint32), prefix=arr(p.prefix, P, np.uint64),
                    tier_old=arr(p.tier_old, P, np.uint8), tier_new=arr(p.tier_new, P, np.uint8),
                    category=arr(p.category, P, np.uint8), out_programs=arr(p.out_programs, p.n_out, np.uint32),
                    in_programs=arr(p.in_programs, p.n_in, np.uint32))

    def place_host_buffers(self) -> None:
        """Caller's host-extent bookkeeping for the current plan: drop the
        buffers of CPU (or SSD) programs sent to Waiting, give buffers to
        programs that leave the GPU and to those admitted from Waiting to the
        CPU (or SSD) tier.  An SSD program's KV is kept in its host buffer here:
        the storage I/O of the SSD tier is outside this module."""
        cat = self.plan_arrays()["category"]
        for p in np.flatnonzero((cat == M.MORI_CAT_DROP_CPU) | (cat == M.MORI_CAT_DROP_SSD)):
            self.drop_host_buffer(int(p))
        for c in (M.MORI_CAT_OUT, M.MORI_CAT_ADMIT_CPU, M.MORI_CAT_ADMIT_SSD):
            for p in np.flatnonzero(cat == c):
                self.give_host_buffer(int(p))

    def swap_out(self, mode: int = M.MORI_COPY_AUTO, stream=None) -> int:
        return M.mori_kv_swap_out(self.ctx, self.host_addr.ctypes.data, mode, _stream(stream))

    def swap_in(self, mode: int = M.MORI_COPY_AUTO, stream=None) -> int:
        return M.mori_kv_swap_in(self.ctx, self.host_addr.ctypes.data, mode, _stream(stream))

    def release_swapped_in(self) -> None:
        """After the swap-in completed: the promoted programs' host buffers are free."""
        cat = self.plan_arrays()["category"]
        for p in np.flatnonzero(cat == M.MORI_CAT_IN):
            self.drop_host_buffer(int(p))

    def step(self, *, gpu_bytes: int, cpu_bytes: int, window=None, idleness=None, status=None, flags: int = 0,
             mode: int = M.MORI_COPY_AUTO, s_out=None, s_in=None, sync: bool = True, ssd_bytes: int = 0):
        """rank -> plan on the host -> host extents -> swap-out || swap-in."""
        check(self.rank_partition(gpu_bytes=gpu_bytes, cpu_bytes=cpu_bytes, window=window, idleness=idleness,
                                  status=status, flags=flags, stream=s_out, ssd_bytes=ssd_bytes),
              "mori_rank_partition")
        rc, p = self.plan_wait()
        if rc != M.MORI_OK:
            raise MoriError("mori_plan_wait", rc, p.device_error)
        self.place_host_buffers()
        check(self.swap_out(mode, s_out), "mori_kv_swap_out")
        check(self.swap_in(mode, s_in if s_in is not None else s_out), "mori_kv_swap_in")
        if sync:
            self.synchronize()
        return p

    def synchronize(self) -> None:
        torch.cuda.synchronize(self.device)
        rc, err = M.mori_query(self.ctx, M.MORI_Q_DEVICE_ERROR)
        check(rc, "mori_query")
        if err:
            raise MoriError("device validation", M.MORI_EDEVICE, err)
        if self.plan is not None:
            self.release_swapped_in()

    # ---- state readback ---------------------------------------------------------
    def state(self):
        tbl = self.tbl.cpu().numpy().view(np.uint32)[: self.tbl_len].copy()
        return tbl, self.tier.cpu().numpy().copy(), self.free_map.cpu().numpy().copy()

    def close(self) -> None:
        if getattr(self, "ctx", None) is not None:
            M.mori_destroy(self.ctx)
            self.ctx = None
        self.arena.close()


def evict_order(block_type: torch.Tensor, last_access: torch.Tensor, size: torch.Tensor | None = None,
                unit_bytes: int = 1, tier: int = M.MORI_TIER_GPU, need_bytes: int = 0, stream=None,
                workspace: torch.Tensor | None = None):
    """Typed eviction order of one tier (Sec. 4.3.2) for device tensors of block
    metadata: type uint8 [N] (MORI_TYPE_*), last access int64 [N] (< 2^62), size
    int32 [N] in units of unit_bytes or None.  Returns device tensors (order
    int32 [N]: block evicted j-th; prefix int64 [N]: bytes freed by the first
    j+1; result int32 [2]: fewest evictions freeing need_bytes, error bits),
    enqueued on `stream`.  The workspace is allocated here unless given."""
    N = int(block_type.numel())
    dev = block_type.device
    assert last_access.numel() == N and (size is None or size.numel() == N)
    rc, wbytes = M.mori_evict_workspace(N)
    check(rc, "mori_evict_workspace")
    if workspace is None:
        workspace = torch.empty(max(wbytes, 256), dtype=torch.uint8, device=dev)
    order = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    prefix = torch.empty(max(N, 1), dtype=torch.int64, device=dev)
    result = torch.zeros(2, dtype=torch.int32, device=dev)
    blk = M.mori_blocks(N, block_type.data_ptr() if N else None, last_access.data_ptr() if N else None,
                        size.data_ptr() if size is not None else None, int(unit_bytes))
    check(M.mori_evict_order(blk, int(tier), int(need_bytes), workspace.data_ptr(), workspace.numel(),
                             order.data_ptr(), prefix.data_ptr(), result.data_ptr(), _stream(stream)),
          "mori_evict_order")
    return order[:N], prefix[:N], result


def _stream(s) -> int:
    if s is None:
        return torch.cuda.current_stream().cuda_stream
    return s.cuda_stream
