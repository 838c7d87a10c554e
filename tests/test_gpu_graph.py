"""The typed eviction order (Sec. 4.3.2) captured in a HIP graph and replayed.

mori_evict_order enqueues kernels only (no memsets, events or host
synchronisation), so a serving loop can capture it once and replay it.  Each
replay here runs on new block metadata written in place, with the program's
own eager work and synchronisation in between, and must equal the oracle; the
same call made eagerly is checked as well."""
import numpy as np
import pytest
import torch

from gpu_helpers import log
from oracle import oracle
from paper_2606_00866_amd import mori as M
from workload import eviction_blocks

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("N", [69938, 1 << 20])  # one look-back kernel per pass / three kernels per pass
def test_eviction_order_replayed_from_a_graph(N):
    rng = np.random.default_rng(N + 11)
    draws = [eviction_blocks(rng, N, programs=1024, tie_frac=0.5, var_size=True) for _ in range(4)]
    t = torch.empty(N, dtype=torch.uint8, device="cuda")
    la = torch.empty(N, dtype=torch.int64, device="cuda")
    sz = torch.empty(N, dtype=torch.int32, device="cuda")
    rc, wbytes = M.mori_evict_workspace(N)
    assert rc == 0
    ws = torch.empty(wbytes, dtype=torch.uint8, device="cuda")
    order = torch.empty(N, dtype=torch.int32, device="cuda")
    prefix = torch.empty(N, dtype=torch.int64, device="cuda")
    result = torch.zeros(2, dtype=torch.int32, device="cuda")
    blk = M.mori_blocks(N, t.data_ptr(), la.data_ptr(), sz.data_ptr(), 4096)
    need = int(draws[0][2].astype(np.int64).sum()) * 4096 // 3  # fixed when captured
    tier = M.MORI_TIER_GPU

    def load(d):
        typ, last, size = d
        t.copy_(torch.from_numpy(typ))
        la.copy_(torch.from_numpy(last.view(np.int64)))
        sz.copy_(torch.from_numpy(size.view(np.int32)))

    def check(d, what):
        typ, last, size = d
        rc, o_order, o_prefix, o_count = oracle.evict_order(typ, last, tier, need, size=size, unit_bytes=4096)
        assert rc == oracle.OK
        assert np.array_equal(order.cpu().numpy().view(np.uint32), o_order), (what, "order")
        assert np.array_equal(prefix.cpu().numpy().view(np.uint64), o_prefix), (what, "prefix")
        res = result.cpu().numpy().view(np.uint32)
        assert res[1] == 0 and res[0] == o_count, (what, res, o_count)

    s = torch.cuda.Stream()
    load(draws[0])
    torch.cuda.synchronize()
    with torch.cuda.stream(s):  # eager first, on the stream that is captured
        assert M.mori_evict_order(blk, tier, need, ws.data_ptr(), wbytes, order.data_ptr(), prefix.data_ptr(),
                                  result.data_ptr(), s.cuda_stream) == 0
    s.synchronize()
    check(draws[0], "eager")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        assert M.mori_evict_order(blk, tier, need, ws.data_ptr(), wbytes, order.data_ptr(), prefix.data_ptr(),
                                  result.data_ptr(), s.cuda_stream) == 0
    for rep, d in enumerate(draws):
        log(f"graph replay {rep} N={N}")
        load(d)  # eager work of the program between replays
        order.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        check(d, f"replay {rep}")
    g.reset()
