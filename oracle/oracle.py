"""ctypes binding of the CPU oracle (``mori_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``.  The product path never imports it.

The oracle follows the paper (arXiv 2606.00866) step by step: Eq. 1 idleness
(Sec. 4.2), relative ranking, capacity-matched boundary (Sec. 4.1, 4.3, 7.2),
sticky diff, lowest-id page allocation, byte movement.  Every array passed in
is a numpy array; state arrays are updated in place only on success.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mori_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

GPU, CPU, WAIT, SSD = 0, 1, 2, 3
TYPE_BUSY, TYPE_IDLE, TYPE_INACTIVE = 0, 1, 2
NONE = 0xFFFFFFFF
F_STATUS_KEY, F_SKIP_FIT, F_IDLENESS_GIVEN, F_INCREMENTAL, F_SSD_TIER = 1, 2, 4, 8, 16
ST_REASONING, ST_ACTING, ST_NEW = 0, 1, 2
OK, E_INPUT, E_POOL, E_NOSPC = 0, 1, 2, 3
ADMIT_BEST_FIT = 1
KEPT, OUT, IN, DROP_GPU, DROP_CPU, ADMIT_GPU, ADMIT_CPU, CPU_SSD, SSD_CPU, DROP_SSD, ADMIT_SSD = range(11)


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (strict IEEE binary32, no contraction)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < max(
        os.path.getmtime(SRC), os.path.getmtime(os.path.join(HERE, "mori_oracle.h"))
    ):
        tmp = LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
             "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"]
        )
        os.replace(tmp, LIB)
    return LIB


class _Geometry(C.Structure):
    _fields_ = [(n, C.c_uint32) for n in ("layers", "planes", "block_tokens", "row_bytes", "num_blocks")]


class _Summary(C.Structure):
    _fields_ = [(n, C.c_uint32) for n in (
        "m_gpu", "m_cpu", "m_ssd", "n_out", "n_in", "n_drop_gpu", "n_drop_cpu", "n_admit_gpu", "n_admit_cpu")] + [
        (n, C.c_uint64) for n in (
            "pages_out", "pages_in", "pages_admit", "pages_free_before", "pages_released",
            "pages_recycled", "pages_free_after", "bytes_out", "bytes_in", "gpu_bytes_after",
            "cpu_bytes_after", "ssd_bytes_after", "pages_dropped")]


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = C.CDLL(build())
        P = C.c_void_p
        _lib.orc_idleness.argtypes = [C.c_uint32, C.c_uint32, P, P]
        _lib.orc_keys.argtypes = [C.c_uint32, P, P, C.c_uint32, P]
        _lib.orc_order.argtypes = [C.c_uint32, P, P, P]
        _lib.orc_order.restype = None
        _lib.orc_boundary.argtypes = [C.c_uint32, P, P, C.c_uint64, C.c_uint64, C.c_uint64, C.c_uint64,
                                      C.c_uint32, P, P, P, P, P]
        _lib.orc_boundary.restype = None
        _lib.orc_rebalance.argtypes = [P, P, C.c_uint32, C.c_uint32, P, P, P, P, C.c_uint32, P, P, P,
                                       C.c_uint64, C.c_uint64, C.c_uint64, C.c_uint32, P, P, P, P, P, P, P]
        _lib.orc_incremental.argtypes = [C.c_uint32, P, P, P, P, C.c_uint64, C.c_uint64, C.c_uint64, C.c_uint32,
                                         P, P, P, P, P, P]
        _lib.orc_replica_admit.argtypes = [C.c_uint32, P, P, P, C.c_uint32, P, C.c_uint32, P, P]
        _lib.orc_evict_order.argtypes = [C.c_uint32, P, P, P, C.c_uint64, C.c_uint32, C.c_uint64, P, P, P]
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _need(a, dtype, n=None):
    a = np.ascontiguousarray(a, dtype=dtype)
    if n is not None:
        assert a.size == n, (a.size, n)
    return a


def idleness(window: np.ndarray):
    """Eq. 1 per program.  window: float32 [P][k][2].  Returns (rc, iota)."""
    w = _need(window, np.float32)
    P, k = w.shape[0], w.shape[1]
    out = np.zeros(P, np.float32)
    rc = lib().orc_idleness(P, k, _ptr(w), _ptr(out))
    return rc, out


def keys(iota, status=None, flags=0):
    it = _need(iota, np.float32)
    st = None if status is None else _need(status, np.uint8)
    out = np.zeros(it.size, np.uint32)
    rc = lib().orc_keys(it.size, _ptr(it), _ptr(st), flags, _ptr(out))
    return rc, out


def order(key):
    k = _need(key, np.uint32)
    o = np.zeros(k.size, np.uint32)
    r = np.zeros(k.size, np.uint32)
    lib().orc_order(k.size, _ptr(k), _ptr(o), _ptr(r))
    return o, r


def boundary(order_, nblk, block_bytes, gpu_budget, cpu_budget, flags=0, ssd_budget=0, with_ssd=False):
    """-> (prefix, tier_new, m_gpu, m_cpu), plus m_ssd when with_ssd."""
    o = _need(order_, np.uint32)
    nb = _need(nblk, np.uint32)
    P = o.size
    prefix = np.zeros(P, np.uint64)
    tier_new = np.zeros(P, np.uint8)
    mg, mc, ms = C.c_uint32(0), C.c_uint32(0), C.c_uint32(0)
    lib().orc_boundary(P, _ptr(o), _ptr(nb), block_bytes, gpu_budget, cpu_budget, ssd_budget, flags, _ptr(prefix),
                       _ptr(tier_new), C.byref(mg), C.byref(mc), C.byref(ms))
    if with_ssd:
        return prefix, tier_new, mg.value, mc.value, ms.value
    return prefix, tier_new, mg.value, mc.value


def incremental(iota, status, tier_old, nblk, block_bytes, gpu_budget, cpu_budget, flags=0):
    """Incremental sticky placement (Sec. 4.3.1) -> (rc, order, prefix, tier_new, m_gpu, m_cpu)."""
    it = _need(iota, np.float32)
    P = it.size
    st = _need(status, np.uint8, P)
    to = _need(tier_old, np.uint8, P)
    nb = _need(nblk, np.uint32, P)
    order_ = np.zeros(P, np.uint32)
    prefix = np.zeros(P, np.uint64)
    tier_new = np.zeros(P, np.uint8)
    mg, mc = C.c_uint32(0), C.c_uint32(0)
    rc = lib().orc_incremental(P, _ptr(it), _ptr(st), _ptr(to), _ptr(nb), int(block_bytes), int(gpu_budget),
                               int(cpu_budget), flags, _ptr(order_), None, _ptr(prefix), _ptr(tier_new),
                               C.byref(mg), C.byref(mc))
    return rc, order_, prefix, tier_new, mg.value, mc.value


@dataclass
class Result:
    rc: int
    order: np.ndarray
    rank: np.ndarray
    tier_old: np.ndarray
    category: np.ndarray
    prefix: np.ndarray
    summary: dict


def rebalance(geom, *, window=None, iota=None, status=None, tbl_off, tbl, tier, free_map,
              gpu_budget, cpu_budget, flags=0, pool=None, host_bufs=None, k=None, ssd_budget=0) -> Result:
    """One whole rebalance.  ``geom`` has layers, planes, block_tokens, row_bytes, num_blocks.

    ``tbl`` (uint32), ``tier`` (uint8), ``free_map`` (uint8), ``pool`` (uint8) and the
    per-program ``host_bufs`` (list of uint8 arrays or None) are updated in place.
    """
    for name, a, dt in (("tbl", tbl, np.uint32), ("tier", tier, np.uint8), ("free_map", free_map, np.uint8)):
        assert a.dtype == dt and a.flags.c_contiguous, name
    P = tier.size
    g = _Geometry(geom.layers, geom.planes, geom.block_tokens, geom.row_bytes, geom.num_blocks)
    off = _need(tbl_off, np.uint32, P + 1)
    w = None
    kk = 0
    if window is not None:
        w = _need(window, np.float32)
        kk = w.shape[1] if w.ndim == 3 else (k or 0)
    it = None if iota is None else _need(iota, np.float32, P)
    st = None if status is None else _need(status, np.uint8, P)
    if pool is not None:
        assert pool.dtype == np.uint8 and pool.flags.c_contiguous
    bufs = None
    if host_bufs is not None:
        bufs = (C.c_void_p * max(P, 1))()
        for p in range(P):
            b = host_bufs[p]
            if b is not None:
                assert b.dtype == np.uint8 and b.flags.c_contiguous
                bufs[p] = b.ctypes.data
    order_ = np.zeros(P, np.uint32)
    rank = np.zeros(P, np.uint32)
    tier_old = np.zeros(P, np.uint8)
    cat = np.zeros(P, np.uint8)
    prefix = np.zeros(P, np.uint64)
    s = _Summary()
    rc = lib().orc_rebalance(C.byref(g), _ptr(pool), P, kk, _ptr(w), _ptr(it), _ptr(st), _ptr(off),
                             tbl.size, _ptr(tbl), _ptr(tier), _ptr(free_map), int(gpu_budget),
                             int(cpu_budget), int(ssd_budget), flags, None if bufs is None else C.cast(bufs, C.c_void_p),
                             _ptr(order_), _ptr(rank), _ptr(tier_old), _ptr(cat), _ptr(prefix), C.byref(s))
    summary = {name: getattr(s, name) for name, _ in _Summary._fields_} if rc == OK else {}
    return Result(rc, order_, rank, tier_old, cat, prefix, summary)


def evict_order(type_, last_access, tier, need_bytes, size=None, unit_bytes=1):
    """Typed eviction order of one tier (Sec. 4.3.2) -> (rc, order, prefix, count)."""
    t = _need(type_, np.uint8)
    la = _need(last_access, np.uint64, t.size)
    sz = None if size is None else _need(size, np.uint32, t.size)
    N = t.size
    order_ = np.zeros(N, np.uint32)
    prefix = np.zeros(N, np.uint64)
    cnt = C.c_uint32(0)
    rc = lib().orc_evict_order(N, _ptr(t), _ptr(la), _ptr(sz), int(unit_bytes), int(tier), int(need_bytes),
                               _ptr(order_), _ptr(prefix), C.byref(cnt))
    return rc, order_, prefix, cnt.value


def replica_admit(bytes_, iota, status, room, flags=0):
    """Multi-replica admission of Waiting programs -> (rc, replica [P] int32, room_after [R])."""
    b = _need(bytes_, np.uint64)
    P = b.size
    it = _need(iota, np.float32, P)
    st = _need(status, np.uint8, P)
    rm = _need(room, np.uint64)
    rep = np.zeros(P, np.int32)
    after = np.zeros(rm.size, np.uint64)
    rc = lib().orc_replica_admit(P, _ptr(b), _ptr(it), _ptr(st), rm.size, _ptr(rm), flags, _ptr(rep), _ptr(after))
    return rc, rep, after
