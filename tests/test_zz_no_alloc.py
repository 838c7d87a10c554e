"""The allocation-free eviction order (mori_evict_order_noalloc, through the
C ABI) against mori_evict_order with a caller workspace: identical order,
byte prefix and result on two calls in a row, the second smaller (the
library's array keeps the first call's contents), then at the maximum size
and empty; above the maximum it is refused on the host."""
import numpy as np
import pytest
import torch

from paper_2606_00866_amd import mori as M
from workload import eviction_blocks

pytestmark = pytest.mark.gpu


def _inputs(N, seed):
    rng = np.random.default_rng(seed)
    typ, la, size = eviction_blocks(rng, N, programs=max(1, min(1024, N)), tie_frac=0.5, var_size=bool(seed % 2))
    t = torch.from_numpy(typ).cuda()
    la_d = torch.from_numpy(la.view(np.int64)).cuda()
    sz = None if size is None else torch.from_numpy(size.view(np.int32)).cuda()
    total = int(size.astype(np.int64).sum()) if size is not None else N
    return t, la_d, sz, total


def _run_both(N, seed, tier):
    t, la_d, sz, total = _inputs(N, seed)
    blk = M.mori_blocks(N, t.data_ptr() if N else None, la_d.data_ptr() if N else None,
                        sz.data_ptr() if sz is not None else None, 4096)
    need = total * 4096 // 3
    s = torch.cuda.current_stream().cuda_stream
    rc, wb = M.mori_evict_workspace(N)
    assert rc == M.MORI_OK
    ws = torch.empty(max(wb, 256), dtype=torch.uint8, device="cuda")
    outs = []
    for noalloc in (False, True):
        order = torch.full((max(N, 1),), -1, dtype=torch.int32, device="cuda")
        prefix = torch.full((max(N, 1),), -1, dtype=torch.int64, device="cuda")
        result = torch.full((2,), -1, dtype=torch.int32, device="cuda")
        if noalloc:
            rc = M.mori_evict_order_noalloc(blk, tier, need, order.data_ptr(), prefix.data_ptr(), result.data_ptr(), s)
        else:
            rc = M.mori_evict_order(blk, tier, need, ws.data_ptr(), wb, order.data_ptr(), prefix.data_ptr(),
                                    result.data_ptr(), s)
        assert rc == M.MORI_OK, (noalloc, rc)
        outs.append((order, prefix, result))
    torch.cuda.synchronize()
    (o1, p1, r1), (o2, p2, r2) = outs
    assert int(r1[1]) == 0 and torch.equal(r1, r2), (r1.tolist(), r2.tolist())
    assert torch.equal(o1[:N], o2[:N]) and torch.equal(p1[:N], p2[:N])
    if N:
        assert sorted(o2[:N].cpu().tolist()) == list(range(N))
    return int(r2[0])


def test_noalloc_matches_workspace_entry_point():
    assert torch.cuda.is_available()
    M.lib()
    # two calls in a row, the second smaller: what the first left in the array must not leak into it
    for N, seed, tier in ((300_000, 1, M.MORI_TIER_GPU), (20_000, 2, M.MORI_TIER_CPU),
                          (M.MORI_EVICT_NOALLOC_MAX_BLOCKS, 3, M.MORI_TIER_GPU), (5, 4, M.MORI_TIER_CPU),
                          (0, 5, M.MORI_TIER_GPU)):
        k = _run_both(N, seed, tier)
        print(f"noalloc N={N} tier={tier}: identical, {k} evictions", flush=True)


def test_noalloc_refuses_beyond_its_array():
    M.lib()
    N = M.MORI_EVICT_NOALLOC_MAX_BLOCKS + 1
    result = torch.zeros(2, dtype=torch.int32, device="cuda")
    blk = M.mori_blocks(N, 16, 16, None, 1)  # refused before any pointer is used
    assert M.mori_evict_order_noalloc(blk, M.MORI_TIER_GPU, 0, 16, 0, result.data_ptr(), 0) == M.MORI_ENOSPC
    assert M.lib().mori_evict_order_noalloc(None, M.MORI_TIER_GPU, 0, 16, None, result.data_ptr(), None) == \
        M.MORI_EINVAL
    blk = M.mori_blocks(0, None, None, None, 1)
    assert M.mori_evict_order_noalloc(blk, 7, 0, 0, 0, result.data_ptr(), 0) == M.MORI_EINVAL
