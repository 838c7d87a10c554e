"""GPU parity of the typed eviction order (Sec. 4.3.2): libmori's device radix
sort and reclaim prefix against the oracle, element by element."""
import numpy as np
import pytest
import torch

from gpu_helpers import log
from oracle import oracle
from paper_2606_00866_amd import mori as M
from workload import eviction_blocks

pytestmark = pytest.mark.gpu


def run_gpu(typ, la, size, unit, tier, need):
    N = typ.size
    dev = "cuda"
    t = torch.from_numpy(np.ascontiguousarray(typ, np.uint8)).to(dev)
    l = torch.from_numpy(np.ascontiguousarray(la, np.uint64).view(np.int64)).to(dev)
    sz = None if size is None else torch.from_numpy(np.ascontiguousarray(size, np.uint32).view(np.int32)).to(dev)
    rc, wbytes = M.mori_evict_workspace(N)
    assert rc == 0
    ws = torch.empty(max(wbytes, 256), dtype=torch.uint8, device=dev)
    order = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    prefix = torch.empty(max(N, 1), dtype=torch.int64, device=dev)
    result = torch.zeros(2, dtype=torch.int32, device=dev)
    blk = M.mori_blocks(N, t.data_ptr() if N else None, l.data_ptr() if N else None,
                        sz.data_ptr() if sz is not None else None, unit)
    rc = M.mori_evict_order(blk, tier, need, ws.data_ptr(), ws.numel(), order.data_ptr(), prefix.data_ptr(),
                            result.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert rc == 0
    torch.cuda.synchronize()
    return (order.cpu().numpy().view(np.uint32)[:N], prefix.cpu().numpy().view(np.uint64)[:N],
            result.cpu().numpy().view(np.uint32))


def check(typ, la, size, unit, tier, need):
    rc, o_order, o_prefix, o_count = oracle.evict_order(typ, la, tier, need, size=size, unit_bytes=unit)
    assert rc == oracle.OK
    g_order, g_prefix, res = run_gpu(typ, la, size, unit, tier, need)
    assert res[1] == 0
    assert np.array_equal(g_order, o_order), "order"
    assert np.array_equal(g_prefix, o_prefix), "prefix"
    assert res[0] == o_count, ("count", res[0], o_count)


@pytest.mark.parametrize("seed", range(24))
def test_random_small(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.choice([0, 1, 2, 17, 255, 256, 4095, 4096, 4097, 9000, 20000]))
    typ, la, size = eviction_blocks(rng, N, programs=int(rng.integers(1, 64)), tie_frac=float(rng.random()),
                                    horizon=int(rng.choice([8, 1 << 20, 1 << 44])), var_size=bool(seed % 2))
    tier = seed % 2
    total = int(N if size is None else size.astype(np.int64).sum())
    need = int(rng.integers(0, 2 * total + 2)) * 3
    log(f"evict seed={seed} N={N} tier={tier} need={need}")
    check(typ, la, size, 3, tier, need)


def test_degenerate_keys():
    """All keys equal (every radix pass is skipped) and a single varying digit."""
    N = 10000
    check(np.zeros(N, np.uint8), np.full(N, 7, np.uint64), None, 1, 0, 5000)
    la = np.zeros(N, np.uint64)
    la[::3] = 255
    check(np.ones(N, np.uint8), la, None, 2, 1, 1)
    check(np.full(N, 2, np.uint8), np.full(N, (1 << 62) - 1, np.uint64), None, 1, 0, N + 5)


@pytest.mark.parametrize("N", [69938, 131072, 300000, 1 << 20])  # look-back passes up to 131072, three kernels above
def test_large(N):
    rng = np.random.default_rng(N)
    typ, la, size = eviction_blocks(rng, N, programs=1024, tie_frac=0.5)
    log(f"evict large N={N}")
    for tier in (0, 1):
        check(typ, la, size, 2 << 20, tier, (N // 3) * (2 << 20))


def test_bad_blocks_reported():
    typ = np.zeros(100, np.uint8)
    typ[40] = 3
    _, _, res = run_gpu(typ, np.zeros(100, np.uint64), None, 1, 0, 10)
    assert res[1] & M.MORI_DEV_BAD_BLOCK and res[0] == 0
    la = np.zeros(100, np.uint64)
    la[7] = 1 << 62
    _, _, res = run_gpu(np.zeros(100, np.uint8), la, None, 1, 1, 10)
    assert res[1] & M.MORI_DEV_BAD_BLOCK


def test_host_side_argument_errors():
    rc, w = M.mori_evict_workspace(1000)
    assert rc == 0 and w >= 32 * 1000
    ws = torch.empty(w, dtype=torch.uint8, device="cuda")
    res = torch.zeros(2, dtype=torch.int32, device="cuda")
    t = torch.zeros(1000, dtype=torch.uint8, device="cuda")
    l = torch.zeros(1000, dtype=torch.int64, device="cuda")
    o = torch.zeros(1000, dtype=torch.int32, device="cuda")
    blk = M.mori_blocks(1000, t.data_ptr(), l.data_ptr(), None, 1)
    assert M.mori_evict_order(blk, 2, 0, ws.data_ptr(), w, o.data_ptr(), 0, res.data_ptr()) == M.MORI_EINVAL
    assert M.mori_evict_order(blk, 0, 0, ws.data_ptr(), w - 8, o.data_ptr(), 0, res.data_ptr()) == M.MORI_EINVAL
    assert M.mori_evict_order(blk, 0, 0, ws.data_ptr() + 8, w, o.data_ptr(), 0, res.data_ptr()) == M.MORI_EINVAL
    assert M.mori_evict_order(blk, 0, 0, ws.data_ptr(), w, 0, 0, res.data_ptr()) == M.MORI_EINVAL


@pytest.mark.parametrize("N", [69938, 1 << 20])
def test_bench_inputs(N):
    """The eviction-order leg of bench.py times these exact inputs."""
    import bench

    typ, la, size, need = bench.evict_inputs(np, N)
    log(f"evict bench inputs N={N}")
    check(typ, la, size, 4096, 0, need)


@pytest.mark.parametrize("N", [1000, 69938, 300000])
def test_no_writes_past_outputs_or_workspace(N):
    """Sentinels past order[N], prefix[N], result[2] and the workspace's stated
    size are untouched (both radix pass forms)."""
    rng = np.random.default_rng(N + 5)
    typ, la, size = eviction_blocks(rng, N, programs=300, tie_frac=0.4, var_size=True)
    dev = "cuda"
    t = torch.from_numpy(typ).to(dev)
    l = torch.from_numpy(la.view(np.int64)).to(dev)
    sz = torch.from_numpy(size.view(np.int32)).to(dev)
    rc, wbytes = M.mori_evict_workspace(N)
    assert rc == 0
    pad = 4096
    ws = torch.full((wbytes + pad,), 0x3C, dtype=torch.uint8, device=dev)
    order = torch.full((N + 64,), -7, dtype=torch.int32, device=dev)
    prefix = torch.full((N + 64,), -9, dtype=torch.int64, device=dev)
    result = torch.full((2 + 14,), -11, dtype=torch.int32, device=dev)
    blk = M.mori_blocks(N, t.data_ptr(), l.data_ptr(), sz.data_ptr(), 1)
    assert M.mori_evict_order(blk, 0, N // 3, ws.data_ptr(), wbytes, order.data_ptr(), prefix.data_ptr(),
                              result.data_ptr(), torch.cuda.current_stream().cuda_stream) == M.MORI_OK
    torch.cuda.synchronize()
    assert (order[N:] == -7).all().item() and (prefix[N:] == -9).all().item() and (result[2:] == -11).all().item()
    assert (ws[wbytes:] == 0x3C).all().item()
    assert result[1].item() == 0


def test_python_wrapper():
    """tiering.evict_order (device tensors in, device tensors out) equals the oracle."""
    from paper_2606_00866_amd.tiering import evict_order

    rng = np.random.default_rng(321)
    N = 5000
    typ, la, size = eviction_blocks(rng, N, programs=50, tie_frac=0.5, var_size=True)
    need = int(size.astype(np.int64).sum()) * 4096 // 3
    order, prefix, result = evict_order(torch.from_numpy(typ).cuda(), torch.from_numpy(la.view(np.int64)).cuda(),
                                        torch.from_numpy(size.view(np.int32)).cuda(), unit_bytes=4096,
                                        tier=M.MORI_TIER_CPU, need_bytes=need)
    torch.cuda.synchronize()
    rc, o_order, o_prefix, o_count = oracle.evict_order(typ, la, M.MORI_TIER_CPU, need, size=size, unit_bytes=4096)
    assert rc == oracle.OK
    assert np.array_equal(order.cpu().numpy().view(np.uint32), o_order)
    assert np.array_equal(prefix.cpu().numpy().view(np.uint64), o_prefix)
    assert result.cpu().tolist() == [o_count, 0]


def test_need_at_prefix_edges():
    """The eviction count when need is 0, equals a prefix value exactly (at the
    first block, at tile edges, at the last block), lies just above one, or
    exceeds every block's bytes: each equals the oracle's."""
    rng = np.random.default_rng(5)
    N = 5000  # five tiles of 1024 keys
    typ, la, size = eviction_blocks(rng, N, programs=40, tie_frac=0.5, var_size=True)
    rc, _, prefix, _ = oracle.evict_order(typ, la, 0, 0, size=size, unit_bytes=1)
    assert rc == oracle.OK
    p = [int(x) for x in prefix]
    for need in (0, 1, p[0], p[0] + 1, p[1022], p[1023], p[1023] + 1, p[1024], p[2047], p[4095], p[-2], p[-1],
                 p[-1] + 1, 10 * p[-1]):
        log(f"evict need={need}")
        check(typ, la, size, 1, 0, need)


def test_more_tiles_than_the_single_kernel_tail():
    """2^21 + 5000 blocks: 1027 tiles of 2048 keys, so the prefix is finished by
    the tile-total scan, the fix-up and the result kernel."""
    N = (1 << 21) + 5000
    rng = np.random.default_rng(N)
    typ, la, size = eviction_blocks(rng, N, programs=4096, tie_frac=0.5, var_size=True)
    total = int(size.astype(np.int64).sum())
    log(f"evict N={N}")
    check(typ, la, size, 4096, 1, total * 4096 // 2)
