"""ctypes binding of libmori (``include/mori.h``): the same calls, argument
marshalling only.  Every step of the path runs in the library's HIP kernels;
this module fails loudly when the library is missing.

Each function returns the C return code (``MORI_OK`` = 0), or a tuple
``(code, value)`` when the C call has an output.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmori.so")

MORI_OK, MORI_EINVAL, MORI_ENOSPC, MORI_ESTATE, MORI_EHIP, MORI_EDEVICE = 0, -1, -2, -3, -4, -5
MORI_DEV_BAD_WINDOW, MORI_DEV_BAD_IDLENESS, MORI_DEV_BAD_TIER, MORI_DEV_BAD_TBL_OFF = 0x1, 0x2, 0x4, 0x8
MORI_DEV_PAGE_RANGE, MORI_DEV_PAGE_DUP, MORI_DEV_PAGE_LEAK, MORI_DEV_NONRES_PAGE = 0x10, 0x20, 0x40, 0x80
MORI_DEV_NOSPC, MORI_DEV_HOST_ADDR, MORI_DEV_BAD_BLOCK, MORI_DEV_BAD_STATUS = 0x100, 0x200, 0x400, 0x800
MORI_DEV_STALL = 0x1000
MORI_TYPE_BUSY, MORI_TYPE_IDLE, MORI_TYPE_INACTIVE = 0, 1, 2
MORI_TIER_GPU, MORI_TIER_CPU, MORI_TIER_WAIT, MORI_TIER_SSD = 0, 1, 2, 3
MORI_NO_PAGE = 0xFFFFFFFF
MORI_F_STATUS_KEY, MORI_F_SKIP_FIT, MORI_F_IDLENESS_GIVEN, MORI_F_INCREMENTAL, MORI_F_SSD_TIER = 1, 2, 4, 8, 16
MORI_ST_REASONING, MORI_ST_ACTING, MORI_ST_NEW = 0, 1, 2
MORI_COPY_AUTO, MORI_COPY_KERNEL, MORI_COPY_CE = 0, 1, 2
MORI_CREATE_COPY_STREAMS = 1
(MORI_CAT_KEPT, MORI_CAT_OUT, MORI_CAT_IN, MORI_CAT_DROP_GPU, MORI_CAT_DROP_CPU, MORI_CAT_ADMIT_GPU,
 MORI_CAT_ADMIT_CPU, MORI_CAT_CPU_SSD, MORI_CAT_SSD_CPU, MORI_CAT_DROP_SSD, MORI_CAT_ADMIT_SSD) = range(11)
MORI_MAX_PROGRAMS, MORI_MAX_WINDOW, MORI_MAX_RANGES, MORI_MAX_REPLICAS = 4096, 64, 64, 1024
MORI_ADMIT_BEST_FIT = 1
MORI_EVICT_NOALLOC_MAX_BLOCKS = 1 << 19
MORI_Q_LAST_HIP_ERROR, MORI_Q_DEVICE_ERROR, MORI_Q_LAST_MODE = 1, 2, 3
MORI_Q_PLAN_EVENT, MORI_Q_OUT_EVENT, MORI_Q_IN_EVENT = 4, 5, 6

EXPORTS = ("mori_create", "mori_destroy", "mori_register", "mori_host_alloc", "mori_host_free",
           "mori_rank_partition", "mori_plan_wait", "mori_kv_swap_out", "mori_kv_swap_in", "mori_query",
           "mori_strerror", "mori_profile", "mori_profile_read", "mori_evict_workspace", "mori_evict_order",
           "mori_replica_admit", "mori_evict_order_noalloc")


class mori_pool(C.Structure):
    _fields_ = [("layers", C.c_uint32), ("planes", C.c_uint32), ("block_tokens", C.c_uint32),
                ("row_bytes", C.c_uint32), ("num_blocks", C.c_uint32), ("base", C.c_void_p)]


class mori_programs(C.Structure):
    _fields_ = [("num_programs", C.c_uint32), ("window_k", C.c_uint32), ("window", C.c_void_p),
                ("idleness", C.c_void_p), ("status", C.c_void_p), ("tbl_off", C.c_void_p),
                ("tbl_len", C.c_uint32), ("tbl", C.c_void_p), ("tier", C.c_void_p), ("free_map", C.c_void_p)]


class mori_budget(C.Structure):
    _fields_ = [("gpu_bytes", C.c_uint64), ("cpu_bytes", C.c_uint64), ("flags", C.c_uint32),
                ("ssd_bytes", C.c_uint64)]


class mori_blocks(C.Structure):
    _fields_ = [("num_blocks", C.c_uint32), ("type", C.c_void_p), ("last_access", C.c_void_p),
                ("size", C.c_void_p), ("unit_bytes", C.c_uint64)]


class mori_plan(C.Structure):
    _fields_ = [(n, C.c_uint32) for n in (
        "num_programs", "m_gpu", "m_cpu", "n_out", "n_in", "n_drop_gpu", "n_drop_cpu", "n_admit_gpu",
        "n_admit_cpu", "device_error", "m_ssd")] + [(n, C.c_uint64) for n in (
            "pages_out", "pages_in", "pages_admit", "pages_free_before", "pages_released", "pages_recycled",
            "pages_free_after", "bytes_out", "bytes_in", "gpu_bytes_after", "cpu_bytes_after", "ssd_bytes_after",
            "pages_dropped")] + [
        ("order", C.POINTER(C.c_uint32)), ("prefix", C.POINTER(C.c_uint64)), ("tier_old", C.POINTER(C.c_uint8)),
        ("tier_new", C.POINTER(C.c_uint8)), ("category", C.POINTER(C.c_uint8)),
        ("out_programs", C.POINTER(C.c_uint32)), ("in_programs", C.POINTER(C.c_uint32))]


_lib = None


def lib():
    """Loads the in-tree libmori.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        V, U32, U64, I = C.c_void_p, C.c_uint32, C.c_uint64, C.c_int
        L.mori_create.argtypes = [C.POINTER(mori_pool), U32, U64, U32, C.POINTER(V)]
        L.mori_destroy.argtypes = [V]
        L.mori_register.argtypes = [V, V, U64]
        L.mori_host_alloc.argtypes = [U64, C.POINTER(V)]
        L.mori_host_free.argtypes = [V]
        L.mori_rank_partition.argtypes = [V, C.POINTER(mori_programs), C.POINTER(mori_budget), V]
        L.mori_plan_wait.argtypes = [V, C.POINTER(mori_plan)]
        L.mori_kv_swap_out.argtypes = [V, V, U32, V]
        L.mori_kv_swap_in.argtypes = [V, V, U32, V]
        L.mori_query.argtypes = [V, I, C.POINTER(U64)]
        L.mori_strerror.argtypes = [I]
        L.mori_profile.argtypes = [V, I]
        L.mori_profile_read.argtypes = [V, I, C.POINTER(U64), C.POINTER(U64), C.POINTER(C.c_double)]
        L.mori_evict_workspace.argtypes = [U32, C.POINTER(U64)]
        L.mori_evict_order.argtypes = [C.POINTER(mori_blocks), U32, U64, V, U64, V, V, V, V]
        L.mori_replica_admit.argtypes = [U32, V, V, V, U32, V, U32, V, V]
        L.mori_evict_order_noalloc.argtypes = [C.POINTER(mori_blocks), U32, U64, V, V, V, V]
        L.mori_strerror.restype = C.c_char_p
        for name in EXPORTS:
            if name != "mori_strerror":
                getattr(L, name).restype = I
        _lib = L
    return _lib


def mori_create(pool: mori_pool, max_programs: int, staging_bytes: int = 0, flags: int = 0):
    ctx = C.c_void_p()
    rc = lib().mori_create(C.byref(pool), max_programs, staging_bytes, flags, C.byref(ctx))
    return rc, ctx


def mori_destroy(ctx) -> int:
    return lib().mori_destroy(ctx)


def mori_register(ctx, ptr: int, nbytes: int) -> int:
    return lib().mori_register(ctx, ptr, nbytes)


def mori_host_alloc(nbytes: int):
    p = C.c_void_p()
    rc = lib().mori_host_alloc(nbytes, C.byref(p))
    return rc, (p.value or 0)


def mori_host_free(ptr: int) -> int:
    return lib().mori_host_free(ptr)


def mori_rank_partition(ctx, programs: mori_programs, budget: mori_budget, stream: int = 0) -> int:
    return lib().mori_rank_partition(ctx, C.byref(programs), C.byref(budget), stream)


def mori_plan_wait(ctx):
    p = mori_plan()
    rc = lib().mori_plan_wait(ctx, C.byref(p))
    return rc, p


def mori_kv_swap_out(ctx, host_dst_addr: int, mode: int = MORI_COPY_AUTO, stream: int = 0) -> int:
    """host_dst_addr: address of a host array of num_programs uint64 buffer addresses."""
    return lib().mori_kv_swap_out(ctx, host_dst_addr, mode, stream)


def mori_kv_swap_in(ctx, host_src_addr: int, mode: int = MORI_COPY_AUTO, stream: int = 0) -> int:
    return lib().mori_kv_swap_in(ctx, host_src_addr, mode, stream)


def mori_query(ctx, what: int):
    v = C.c_uint64()
    rc = lib().mori_query(ctx, what, C.byref(v))
    return rc, v.value


def mori_strerror(code: int) -> str:
    return lib().mori_strerror(code).decode()


def mori_profile(ctx, enable: bool) -> int:
    return lib().mori_profile(ctx, 1 if enable else 0)


def mori_profile_read(ctx, direction: int):
    """-> (code, launches, payload_bytes, kernel_ms)"""
    n, by, ms = C.c_uint64(), C.c_uint64(), C.c_double()
    rc = lib().mori_profile_read(ctx, direction, C.byref(n), C.byref(by), C.byref(ms))
    return rc, n.value, by.value, ms.value


def mori_evict_workspace(num_blocks: int):
    b = C.c_uint64()
    rc = lib().mori_evict_workspace(num_blocks, C.byref(b))
    return rc, b.value


def mori_evict_order(blocks: mori_blocks, tier: int, need_bytes: int, workspace: int, workspace_bytes: int,
                     order: int, prefix: int, result: int, stream: int = 0) -> int:
    """order / prefix / result / workspace: device addresses (prefix may be 0)."""
    return lib().mori_evict_order(C.byref(blocks), tier, need_bytes, workspace, workspace_bytes, order,
                                  prefix or None, result, stream)


def mori_evict_order_noalloc(blocks: mori_blocks, tier: int, need_bytes: int, order: int, prefix: int,
                             result: int, stream: int = 0) -> int:
    """mori_evict_order without a workspace (the library's device array is used)."""
    return lib().mori_evict_order_noalloc(C.byref(blocks), tier, need_bytes, order, prefix or None, result, stream)


def mori_replica_admit(bytes_, idleness, status, room, flags: int = 0):
    """Host arrays (numpy) -> (code, replica int32 [P], room_after uint64 [R])."""
    import numpy as np

    b = np.ascontiguousarray(bytes_, np.uint64)
    it = np.ascontiguousarray(idleness, np.float32)
    st = np.ascontiguousarray(status, np.uint8)
    rm = np.ascontiguousarray(room, np.uint64)
    assert it.size == b.size and st.size == b.size
    rep = np.zeros(max(b.size, 1), np.int32)
    after = np.zeros(max(rm.size, 1), np.uint64)
    ptr = lambda a: a.ctypes.data if a.size else None
    rc = lib().mori_replica_admit(b.size, ptr(b), ptr(it), ptr(st), rm.size, ptr(rm), flags, rep.ctypes.data,
                                  after.ctypes.data)
    return rc, rep[:b.size], after[:rm.size]
