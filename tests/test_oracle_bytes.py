"""Pins of the oracle's byte movement: content addressing (every run's bytes are
regenerable from (program, block, plane)), an independent numpy gather,
round-trip identity and recycled pages."""
import numpy as np
import pytest

from workload import (TINY, Geometry, budget_bytes, fill_pool_np, make_bank, make_instance,
                      program_host_content, random_instance)


def _host_bufs(inst, bank, with_content=True):
    bufs = []
    for p in range(inst.P):
        n = int(inst.nblk[p]) * inst.geom.block_bytes
        if inst.tier[p] == 1 and with_content:
            bufs.append(program_host_content(inst, bank, p).copy())
        else:
            bufs.append(np.zeros(n, np.uint8))
    return bufs


def _assert_content(inst, bank, pool, bufs, tbl, tier):
    g = inst.geom
    planes = pool.reshape(g.nplanes, g.num_blocks, g.run_bytes)
    for p in range(inst.P):
        n = int(inst.nblk[p])
        if n == 0:
            continue
        expect = program_host_content(inst, bank, p).reshape(g.nplanes, n, g.run_bytes)
        if tier[p] == 0:
            pages = tbl[inst.tbl_off[p]:inst.tbl_off[p + 1]].astype(np.int64)
            assert np.array_equal(planes[:, pages], expect), p
        elif tier[p] == 1:
            assert np.array_equal(bufs[p].reshape(g.nplanes, n, g.run_bytes), expect), p


def test_tiny_rebalance_and_round_trip(orc):
    inst = make_instance(TINY)
    bank = make_bank(TINY.seed, TINY.dtype, inst.geom.run_bytes)
    pool = fill_pool_np(inst, bank)
    tbl, tier, free = inst.copy_state()
    bufs = _host_bufs(inst, bank)
    bg = budget_bytes(inst.total_bytes, TINY.gpu_pct)
    tbl_old = tbl.copy()
    res = orc.rebalance(inst.geom, window=inst.window, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free,
                        gpu_budget=bg, cpu_budget=inst.total_bytes, pool=pool, host_bufs=bufs)
    assert res.rc == 0 and res.summary["n_out"] > 0
    _assert_content(inst, bank, pool, bufs, tbl, tier)
    # independent realisation of the swap-out: numpy fancy-index gather of the old pages
    g = inst.geom
    planes0 = fill_pool_np(inst, bank).reshape(g.nplanes, g.num_blocks, g.run_bytes)
    for p in np.flatnonzero(res.category == orc.OUT):
        pages = tbl_old[inst.tbl_off[p]:inst.tbl_off[p + 1]].astype(np.int64)
        assert np.array_equal(bufs[p], planes0[:, pages].reshape(-1))
    # reversed ranking (swap reasoning and acting time): programs come back in
    inst2 = make_instance(TINY)
    w_rev = inst.window[:, :, ::-1].copy()
    res2 = orc.rebalance(inst2.geom, window=w_rev, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free,
                         gpu_budget=bg, cpu_budget=inst.total_bytes, pool=pool, host_bufs=bufs)
    assert res2.rc == 0 and res2.summary["n_in"] > 0 and res2.summary["n_out"] > 0
    _assert_content(inst, bank, pool, bufs, tbl, tier)


@pytest.mark.parametrize("seed", range(40))
def test_random_states_content_follows_programs(orc, seed):
    rng = np.random.default_rng(100 + seed)
    inst = random_instance(rng, P=int(rng.integers(1, 14)), max_blocks=6)
    bank = make_bank(seed, "fp16", inst.geom.run_bytes)
    pool = fill_pool_np(inst, bank)
    bufs = _host_bufs(inst, bank)
    tbl, tier, free = inst.copy_state()
    bb = inst.geom.block_bytes
    bg = int(rng.integers(0, inst.geom.num_blocks + 1)) * bb
    res = orc.rebalance(inst.geom, window=inst.window, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free,
                        gpu_budget=bg, cpu_budget=inst.total_bytes, pool=pool, host_bufs=bufs)
    assert res.rc == 0
    # programs admitted from Waiting have no bytes yet (prefill recomputes them); skip them
    admitted = (res.category == orc.ADMIT_GPU) | (res.category == orc.ADMIT_CPU)
    tier_chk = np.where(admitted, 2, tier)
    _assert_content(inst, bank, pool, bufs, tbl, tier_chk)


def test_recycled_page_is_read_before_written(orc):
    """Example B of the worked plan fixture: page 1 leaves with program 0 and is
    reused by program 2's swap-in; the host copy of program 0 keeps the old bytes."""
    geom = Geometry(layers=2, planes=2, block_tokens=1, row_bytes=16, num_blocks=6)
    off = np.array([0, 2, 4, 7], np.uint32)
    tbl = np.array([3, 1, 0, 4, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF], np.uint32)
    tier = np.array([0, 0, 1], np.uint8)
    free = np.array([0, 0, 1, 0, 0, 1], np.uint8)
    rng = np.random.default_rng(0)
    pool = rng.integers(0, 256, geom.pool_bytes, dtype=np.uint8)
    planes = pool.reshape(4, 6, 16).copy()
    bufs = [np.zeros(2 * 64, np.uint8), np.zeros(2 * 64, np.uint8), rng.integers(0, 256, 3 * 64, dtype=np.uint8)]
    in_bytes = bufs[2].copy()
    res = orc.rebalance(geom, iota=np.array([0.875, 0.125, 0.25], np.float32), tbl_off=off, tbl=tbl, tier=tier,
                        free_map=free, gpu_budget=5 * 64, cpu_budget=2 * 64, flags=orc.F_IDLENESS_GIVEN,
                        pool=pool, host_bufs=bufs)
    assert res.rc == 0 and res.summary["pages_recycled"] == 1
    assert tbl[4:7].tolist() == [2, 5, 1]
    assert np.array_equal(bufs[0].reshape(4, 2, 16), planes[:, [3, 1]])
    assert np.array_equal(pool.reshape(4, 6, 16)[:, [2, 5, 1]], in_bytes.reshape(4, 3, 16))
