"""GPU parity: libmori (through the C ABI) against the CPU oracle, element by
element -- rank order, prefix, categories, summary, block tables, tiers, free
map and every resident byte -- on seeded inputs, in both copy modes."""
import numpy as np
import pytest
import torch

from gpu_helpers import Pair, log
from oracle import oracle
from paper_2606_00866_amd import mori as M
from paper_2606_00866_amd.tiering import MoriError, TierPool
from workload import TINY, Geometry, budget_bytes, make_instance, random_instance

pytestmark = pytest.mark.gpu

MODES = [M.MORI_COPY_KERNEL, M.MORI_COPY_CE]


@pytest.fixture(scope="module", autouse=True)
def _lib():
    assert torch.cuda.is_available(), "GPU tests need the MI355X"
    M.lib()


@pytest.mark.parametrize("mode", MODES)
def test_tiny_rebalance_round_trip_reversal(mode):
    inst = make_instance(TINY)
    log(f"tiny mode={mode} P={inst.P} NB={inst.geom.num_blocks}")
    pair = Pair(inst, seed=TINY.seed)
    try:
        bg = budget_bytes(inst.total_bytes, TINY.gpu_pct)
        res, plan = pair.step(gpu_bytes=bg, cpu_bytes=inst.total_bytes, window=inst.window, mode=mode)
        assert plan.n_out > 0 and plan.bytes_out > 0
        rev = inst.window[:, :, ::-1].copy()
        res, plan = pair.step(gpu_bytes=bg, cpu_bytes=inst.total_bytes, window=rev, mode=mode)
        assert plan.n_in > 0 and plan.n_out > 0
        res, plan = pair.step(gpu_bytes=bg, cpu_bytes=inst.total_bytes, window=inst.window, mode=mode)
        assert plan.n_in > 0
    finally:
        pair.close()


@pytest.mark.parametrize("seed", range(48))
def test_random_instances(seed):
    rng = np.random.default_rng(1000 + seed)
    inst = random_instance(rng, P=int(rng.integers(0, 40)), max_blocks=int(rng.choice([3, 12, 40])),
                           ties=bool(seed % 2))
    mode = MODES[seed % 2]
    flags = [0, M.MORI_F_SKIP_FIT, M.MORI_F_STATUS_KEY, 0][seed % 4]
    log(f"random seed={seed} P={inst.P} NB={inst.geom.num_blocks} geom={inst.geom} mode={mode} flags={flags}")
    pair = Pair(inst, seed=seed)
    try:
        bb = inst.geom.block_bytes
        for step in range(3):
            bg = int(rng.integers(0, inst.geom.num_blocks + 1)) * bb
            bc = int(rng.integers(0, inst.total_bytes // max(bb, 1) + 2)) * bb
            w = inst.window if step != 1 else inst.window[:, :, ::-1].copy()
            pair.step(gpu_bytes=bg, cpu_bytes=bc, window=w, status=inst.status, flags=flags, mode=mode)
    finally:
        pair.close()


@pytest.mark.parametrize("mode", MODES)
def test_recycled_pages_worked_example_b(mode):
    """Example B of the plan fixture (one recycled page): the swap-in must not
    overwrite page 1 before the swap-out has read it."""
    geom = Geometry(layers=3, planes=2, block_tokens=4, row_bytes=256, num_blocks=6)
    inst = random_instance(np.random.default_rng(0), P=3, geom=geom, extra_free=0)
    inst.nblk[:] = [2, 2, 3]
    inst.tbl_off[:] = [0, 2, 4, 7]
    inst.tbl = np.array([3, 1, 0, 4, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF], np.uint32)
    inst.tier = np.array([0, 0, 1], np.uint8)
    inst.free_map = np.array([0, 0, 1, 0, 0, 1], np.uint8)
    inst.geom = geom
    pair = Pair(inst, seed=5)
    try:
        res, plan = pair.step(gpu_bytes=5 * geom.block_bytes, cpu_bytes=2 * geom.block_bytes,
                              iota=np.array([0.875, 0.125, 0.25], np.float32), flags=M.MORI_F_IDLENESS_GIVEN,
                              mode=mode)
        assert res.rc == oracle.OK and plan.pages_recycled == 1
    finally:
        pair.close()


def test_edge_cases_empty_and_degenerate():
    geom = Geometry(layers=1, planes=2, block_tokens=2, row_bytes=32, num_blocks=16)
    rng = np.random.default_rng(7)
    cases = [
        random_instance(rng, P=0, geom=geom, extra_free=4),                    # no programs
        random_instance(rng, P=1, geom=geom, extra_free=0),                    # one program
        random_instance(rng, P=9, max_blocks=0, geom=geom, extra_free=3),      # all zero-block programs
        random_instance(rng, P=12, geom=geom, extra_free=0, tier_p=(1.0, 0, 0)),  # pool exactly full
    ]
    for inst in cases:
        log(f"edge P={inst.P} NB={inst.geom.num_blocks}")
        if inst.geom.num_blocks == 0:
            continue
        pair = Pair(inst, seed=3)
        try:
            bb = inst.geom.block_bytes
            for bg in (0, inst.geom.num_blocks * bb):  # empty GPU budget, then the whole pool
                for bc in (0, inst.total_bytes):
                    pair.step(gpu_bytes=bg, cpu_bytes=bc, window=inst.window, mode=M.MORI_COPY_CE)
        finally:
            pair.close()


@pytest.mark.parametrize("k", [1, 5, 64])
def test_window_lengths_and_max_programs(k):
    """P = 4096 (the maximum) with ties, and windows of 1, 5 and 64 cycles."""
    rng = np.random.default_rng(k)
    P = 4096
    geom = Geometry(layers=1, planes=1, block_tokens=1, row_bytes=16, num_blocks=0)
    inst = random_instance(rng, P=P, max_blocks=2, geom=geom, ties=True)
    vals = np.array([0.0, 0.5, 1.0, 2.0], np.float32)
    inst.window = vals[rng.integers(0, 4, size=(P, k, 2))]
    log(f"max programs k={k} NB={inst.geom.num_blocks}")
    pair = Pair(inst, seed=k)
    try:
        bb = inst.geom.block_bytes
        pair.step(gpu_bytes=inst.geom.num_blocks * bb // 2, cpu_bytes=inst.total_bytes // 3, window=inst.window,
                  mode=M.MORI_COPY_KERNEL)
    finally:
        pair.close()


def test_device_validation_rejects_and_leaves_state():
    rng = np.random.default_rng(21)
    inst = random_instance(rng, P=10, extra_free=4, tier_p=(0.6, 0.3, 0.1))
    pair = Pair(inst, seed=1)
    try:
        bb = inst.geom.block_bytes
        before = pair.tp.state()
        bad = inst.window.copy()
        bad[3, 2, 1] = np.nan
        w = torch.from_numpy(bad).cuda()
        rc = pair.tp.rank_partition(gpu_bytes=bb, cpu_bytes=bb, window=w)
        assert rc == M.MORI_OK
        rc, plan = pair.tp.plan_wait()
        assert rc == M.MORI_EDEVICE and plan.device_error & M.MORI_DEV_BAD_WINDOW
        after = pair.tp.state()
        assert all((a == b).all() for a, b in zip(before, after))
        # an inconsistent pool: a free page that a GPU program also owns
        gpu_progs = [p for p in range(inst.P) if inst.tier[p] == 0 and inst.nblk[p] > 0]
        pg = int(inst.tbl[inst.tbl_off[gpu_progs[0]]])
        pair.tp.free_map[pg] = 1
        rc = pair.tp.rank_partition(gpu_bytes=bb, cpu_bytes=bb, window=torch.from_numpy(inst.window).cuda())
        rc, plan = pair.tp.plan_wait()
        assert rc == M.MORI_EDEVICE and plan.device_error & M.MORI_DEV_PAGE_DUP
        pair.tp.free_map[pg] = 0
        # swap without a fresh plan after a rejected one: swaps do nothing and report the error
        assert pair.tp.swap_out(M.MORI_COPY_KERNEL) == M.MORI_OK
        torch.cuda.synchronize()
        rc, err = M.mori_query(pair.tp.ctx, M.MORI_Q_DEVICE_ERROR)
        assert rc == 0 and err & M.MORI_DEV_PAGE_DUP
    finally:
        pair.close()


def test_host_side_state_errors():
    inst = make_instance(TINY)
    pair = Pair(inst, seed=1)
    try:
        tp = pair.tp
        assert tp.swap_out() == M.MORI_ESTATE  # no plan yet
        assert tp.rank_partition(gpu_bytes=inst.geom.num_blocks * inst.geom.block_bytes + 1, cpu_bytes=0,
                                 window=torch.from_numpy(inst.window).cuda()) == M.MORI_EINVAL
        w = torch.from_numpy(inst.window).cuda()
        assert tp.rank_partition(gpu_bytes=0, cpu_bytes=inst.total_bytes, window=w, flags=64) == M.MORI_EINVAL
        # more programs than the context was created for: refused before any device access
        too_many = M.mori_programs(tp.P + 1, w.shape[1], w.data_ptr(), None, None, tp.tbl_off.data_ptr(), tp.tbl_len,
                                   tp.tbl.data_ptr(), tp.tier.data_ptr(), tp.free_map.data_ptr())
        assert M.mori_rank_partition(tp.ctx, too_many, M.mori_budget(0, 0, 0, 0), None) == M.MORI_ENOSPC
        assert tp.rank_partition(gpu_bytes=0, cpu_bytes=inst.total_bytes, window=w) == M.MORI_OK
        rc, plan = tp.plan_wait()
        assert rc == 0
        tp.place_host_buffers()
        assert tp.swap_in() == M.MORI_ESTATE       # swap-out must be enqueued first
        assert tp.swap_out(mode=7) == M.MORI_EINVAL
        # a destination outside every registered range is refused before anything is enqueued
        saved = tp.host_addr.copy()
        tp.host_addr[plan.out_programs[0]] = 0x1000
        assert tp.swap_out(M.MORI_COPY_CE) == M.MORI_EINVAL
        tp.host_addr[:] = saved
        assert tp.swap_out(M.MORI_COPY_CE) == M.MORI_OK
        assert tp.swap_out(M.MORI_COPY_CE) == M.MORI_ESTATE  # once per plan
        assert tp.swap_in(M.MORI_COPY_CE) == M.MORI_OK
        tp.synchronize()
    finally:
        pair.close()


def test_kernel_mode_bad_address_is_caught_on_device():
    inst = make_instance(TINY)
    pair = Pair(inst, seed=1)
    try:
        tp = pair.tp
        w = torch.from_numpy(inst.window).cuda()
        assert tp.rank_partition(gpu_bytes=0, cpu_bytes=inst.total_bytes, window=w) == M.MORI_OK
        rc, plan = tp.plan_wait()
        tp.place_host_buffers()
        tp.host_addr[plan.out_programs[0]] += 8  # misaligned
        assert tp.swap_out(M.MORI_COPY_KERNEL) == M.MORI_OK
        torch.cuda.synchronize()
        rc, err = M.mori_query(tp.ctx, M.MORI_Q_DEVICE_ERROR)
        assert err & M.MORI_DEV_HOST_ADDR
    finally:
        pair.close()


def test_default_queue_count_in_order_copies():
    """With HIP's default of four hardware queues libmori creates no copy streams
    and runs the copy-engine copies on the caller's streams; the smoke check
    (tiny rebalance and reversal against the oracle) runs in a child process
    started with that setting."""
    import os
    import subprocess
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    env = dict(os.environ, GPU_MAX_HW_QUEUES="4")
    r = subprocess.run([sys.executable, "-c", "import __graft_entry__ as g; g.smoke()"], cwd=root, env=env,
                       capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "smoke ok" in r.stdout


@pytest.mark.parametrize("runs_per_half", [1, 2, 3, 7])
def test_copy_engine_small_staging_many_chunks(runs_per_half):
    """Copy-engine swaps through a staging buffer of a few runs per half: many
    chunks per step, programs spanning chunks, both halves reused, and the
    swap-in's wait for the swap-out falling inside the chunk sequence (a pool
    with few free pages, so slots land on released pages)."""
    rng = np.random.default_rng(300 + runs_per_half)
    geom = Geometry(layers=2, planes=2, block_tokens=2, row_bytes=48, num_blocks=0)
    run = geom.block_tokens * geom.row_bytes
    for trial in range(4):
        inst = random_instance(rng, P=int(rng.integers(4, 24)), max_blocks=9, geom=geom, ties=bool(trial % 2),
                               tier_p=(0.5, 0.35, 0.15), extra_free=int(rng.integers(0, 4)))
        if inst.geom.num_blocks == 0:
            continue
        log(f"small staging runs/half={runs_per_half} trial={trial} P={inst.P} NB={inst.geom.num_blocks}")
        pair = Pair(inst, seed=trial, staging_bytes=2 * runs_per_half * run)
        try:
            bb = inst.geom.block_bytes
            recycled = 0
            for step in range(4):
                bg = int(rng.integers(inst.geom.num_blocks // 2, inst.geom.num_blocks + 1)) * bb
                bc = int(rng.integers(0, inst.total_bytes // bb + 2)) * bb
                w = inst.window if step % 2 == 0 else inst.window[:, :, ::-1].copy()
                res, plan = pair.step(gpu_bytes=bg, cpu_bytes=bc, window=w, mode=M.MORI_COPY_CE)
                if plan is not None:
                    recycled += plan.pages_recycled
        finally:
            pair.close()


def test_idleness_extreme_windows():
    """Eq. 1 in binary32 at the edges: denormal times, times near the largest
    finite value (whose totals stay finite), zeros, exact ties and values whose
    rounding decides the order -- the device's ranking, prefix and categories
    equal the oracle's bit for bit (the keys are the idleness bits)."""
    rng = np.random.default_rng(77)
    P = 64
    geom = Geometry(layers=1, planes=1, block_tokens=1, row_bytes=16, num_blocks=0)
    inst = random_instance(rng, P=P, max_blocks=3, geom=geom, extra_free=8)
    tiny = np.float32(1.4e-45)          # smallest denormal
    sub = np.float32(3.0e-39)           # a denormal
    big = np.float32(3.0e37)            # five of them still sum below the largest finite value
    vals = np.array([0.0, tiny, sub, 1.0e-30, 0.1, 1.0, 3.0, 1.0e10, big], np.float32)
    w = vals[rng.integers(0, vals.size, size=(P, 5, 2))].astype(np.float32)
    w[0] = 0.0                                   # no history: idleness 0
    w[1, :, 0], w[1, :, 1] = tiny, tiny          # denormal totals: exactly 1/2
    w[2, :, 0], w[2, :, 1] = 1.0e10, 1.0e-30     # idleness 1e-40: a denormal result
    w[3, :, 0], w[3, :, 1] = 0.0, sub            # only tool time: 1
    w[4] = w[5]                                  # an exact tie, broken by id
    pair = Pair(inst, seed=4)
    try:
        bb = inst.geom.block_bytes
        for bg in (0, inst.geom.num_blocks * bb // 2, inst.geom.num_blocks * bb):
            res, plan = pair.step(gpu_bytes=bg, cpu_bytes=inst.total_bytes // 2, window=w, mode=M.MORI_COPY_KERNEL)
            assert res.rc == oracle.OK and plan is not None
        rc, iota = oracle.idleness(w)
        assert rc == oracle.OK and iota[1] == np.float32(0.5) and iota[3] == np.float32(1.0) and iota[0] == 0.0
        assert 0.0 < iota[2] < np.float32(1.2e-38)  # below the smallest normal
    finally:
        pair.close()


@pytest.mark.parametrize("mode", MODES)
def test_profile_counters(mode):
    """mori_profile / mori_profile_read: launches, payload bytes (each plan's own
    bytes, also when several plans run between reads) and time per direction;
    a read clears the record; nothing is recorded while profiling is off."""
    rng = np.random.default_rng(55)
    geom = Geometry(layers=2, planes=2, block_tokens=2, row_bytes=48, num_blocks=0)
    inst = random_instance(rng, P=16, max_blocks=8, geom=geom, tier_p=(0.5, 0.4, 0.1), extra_free=6)
    run = geom.block_tokens * geom.row_bytes
    pair = Pair(inst, seed=5, staging_bytes=2 * 3 * run)  # three runs per half: several chunks per step
    try:
        ctx, bb = pair.tp.ctx, inst.geom.block_bytes
        assert M.mori_profile(ctx, True) == M.MORI_OK
        moved = [0, 0]
        for step in range(3):
            w = inst.window if step % 2 == 0 else inst.window[:, :, ::-1].copy()
            bg = int(rng.integers(inst.geom.num_blocks // 3, inst.geom.num_blocks + 1)) * bb
            res, plan = pair.step(gpu_bytes=bg, cpu_bytes=inst.total_bytes, window=w, mode=mode)
            moved[0] += plan.bytes_out
            moved[1] += plan.bytes_in
        assert moved[0] > 0 and moved[1] > 0
        for d in (0, 1):
            rc, n, by, ms = M.mori_profile_read(ctx, d)
            assert rc == M.MORI_OK and by == moved[d] and n > 0 and ms > 0.0
            assert M.mori_profile_read(ctx, d)[1:] == (0, 0, 0.0)  # cleared
        assert M.mori_profile(ctx, False) == M.MORI_OK
        pair.step(gpu_bytes=0, cpu_bytes=inst.total_bytes, window=inst.window, mode=mode)
        assert M.mori_profile_read(ctx, 0)[1] == 0
        assert M.mori_profile_read(ctx, 2)[0] == M.MORI_EINVAL
    finally:
        pair.close()


@pytest.mark.parametrize("where,mode,row_bytes,tokens",
                         [("device", M.MORI_COPY_AUTO, 64, 4), ("device", M.MORI_COPY_AUTO, 1152, 64),
                          ("device", M.MORI_COPY_AUTO, 1024, 16), ("two_ranges", M.MORI_COPY_KERNEL, 64, 4),
                          ("two_ranges", M.MORI_COPY_CE, 64, 4)],
                         ids=["device-256B", "device-72KiB", "device-16KiB", "two_ranges-kernel", "two_ranges-ce"])
def test_buffers_in_other_registered_ranges(where, mode, row_bytes, tokens):
    """CPU-tier buffers in a registered device-memory range (AUTO then resolves
    to the kernels at the device grid and its copy shapes: 256 B runs sixteen
    to a workgroup, 72 KiB runs in rounds of four vectors per thread, 16 KiB
    runs one vector per thread) or alternating between two pinned host ranges
    registered beside the pool's arena: tables, tiers, free map, resident pages
    and every buffer byte equal the oracle's over three steps; then the range
    limit (ENOSPC) and unknown memory (EINVAL)."""
    import ctypes

    from workload import fill_pool_np, make_bank, program_host_content

    rng = np.random.default_rng(77)
    geom = Geometry(layers=2, planes=2, block_tokens=tokens, row_bytes=row_bytes, num_blocks=0)
    inst = random_instance(rng, P=24, max_blocks=10, geom=geom, tier_p=(0.55, 0.45), extra_free=8)
    g, bb = inst.geom, inst.geom.block_bytes
    bank = make_bank(3, inst.dtype, g.run_bytes)
    pool = fill_pool_np(inst, bank)
    bufs = [program_host_content(inst, bank, p).copy() if inst.tier[p] == 1
            else np.zeros(int(inst.nblk[p]) * bb, np.uint8) for p in range(inst.P)]
    extent = [(-(-int(n) * bb // 256)) * 256 for n in inst.nblk]
    off = np.concatenate([[0], np.cumsum(extent)]).astype(np.int64)
    tbl, tier, free = inst.copy_state()
    tp = TierPool(g, inst.tbl_off, inst.tbl, inst.tier, inst.free_map, arena_bytes=4096)
    hosts = []
    try:
        tp.pool.copy_(torch.from_numpy(pool).cuda())
        if where == "device":
            dbuf = torch.zeros(int(off[-1]) + 256, dtype=torch.uint8, device="cuda")
            assert M.mori_register(tp.ctx, dbuf.data_ptr(), dbuf.numel()) == M.MORI_OK
            addr = np.array([dbuf.data_ptr() + o for o in off[:-1]], np.uint64)
            read = lambda p: dbuf[off[p]:off[p] + bufs[p].size].cpu().numpy()
            for p in range(inst.P):
                if bufs[p].size:
                    dbuf[off[p]:off[p] + bufs[p].size] = torch.from_numpy(bufs[p]).cuda()
        else:
            for _ in range(2):
                rc, h = M.mori_host_alloc(int(off[-1]) + 256)
                assert rc == M.MORI_OK
                hosts.append(h)
                assert M.mori_register(tp.ctx, h, int(off[-1]) + 256) == M.MORI_OK
            addr = np.array([hosts[p % 2] + o for p, o in enumerate(off[:-1])], np.uint64)
            view = lambda p: np.ctypeslib.as_array((ctypes.c_uint8 * bufs[p].size).from_address(int(addr[p])))
            read = lambda p: view(p).copy()
            for p in range(inst.P):
                if bufs[p].size:
                    view(p)[:] = bufs[p]
        s_out, s_in = torch.cuda.Stream(), torch.cuda.Stream()
        for t in range(3):
            w = inst.window if t != 1 else inst.window[:, :, ::-1].copy()
            bg = int(rng.integers(g.num_blocks // 4, g.num_blocks + 1)) * bb
            res = oracle.rebalance(g, window=w, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free,
                                   gpu_budget=bg, cpu_budget=inst.total_bytes, pool=pool, host_bufs=bufs)
            assert res.rc == oracle.OK
            assert tp.rank_partition(gpu_bytes=bg, cpu_bytes=inst.total_bytes,
                                     window=torch.from_numpy(np.ascontiguousarray(w)).cuda(), stream=s_out) == 0
            rc, plan = tp.plan_wait()
            assert rc == M.MORI_OK
            assert M.mori_kv_swap_out(tp.ctx, addr.ctypes.data, mode, s_out.cuda_stream) == M.MORI_OK
            assert M.mori_kv_swap_in(tp.ctx, addr.ctypes.data, mode, s_in.cuda_stream) == M.MORI_OK
            torch.cuda.synchronize()
            assert M.mori_query(tp.ctx, M.MORI_Q_DEVICE_ERROR) == (M.MORI_OK, 0)
            used = M.mori_query(tp.ctx, M.MORI_Q_LAST_MODE)[1]
            assert used == (M.MORI_COPY_KERNEL if where == "device" else mode)
            log(f"  {where} step {t}: out {plan.n_out} in {plan.n_in} mode {used}")
            t_, r_, f_ = tp.state()
            assert (t_ == tbl).all() and (r_ == tier).all() and (f_ == free).all()
            dpool = tp.pool.cpu().numpy().reshape(g.nplanes, g.num_blocks, g.run_bytes)
            owned = tbl[tbl != 0xFFFFFFFF].astype(np.int64)
            assert np.array_equal(dpool[:, owned], pool.reshape(g.nplanes, g.num_blocks, g.run_bytes)[:, owned])
            for p in np.flatnonzero(tier == 1):
                assert np.array_equal(read(p), bufs[p]), p
        # the context holds MORI_MAX_RANGES ranges (the pool's arena is one)
        extra = []
        while True:
            rc, h = M.mori_host_alloc(4096)
            assert rc == M.MORI_OK
            extra.append(h)
            rc = M.mori_register(tp.ctx, h, 4096)
            if rc != M.MORI_OK:
                break
        assert rc == M.MORI_ENOSPC and 1 + len(hosts) + (where == "device") + len(extra) - 1 == M.MORI_MAX_RANGES
        hosts += extra
        junk = np.zeros(4096, np.uint8)
        tp2 = TierPool(g, inst.tbl_off, inst.tbl, inst.tier, inst.free_map, arena_bytes=4096)
        try:
            assert M.mori_register(tp2.ctx, junk.ctypes.data, junk.size) == M.MORI_EINVAL  # pageable memory
            assert M.mori_register(tp2.ctx, hosts[0], 0) == M.MORI_EINVAL
        finally:
            tp2.close()
    finally:
        torch.cuda.synchronize()
        tp.close()
        for h in hosts:
            M.mori_host_free(h)


def test_two_contexts_interleaved():
    """Two pools, each with its own context and streams, rebalanced in turn:
    contexts share nothing, so each matches its own oracle run."""
    rng = np.random.default_rng(31)
    geom = Geometry(layers=2, planes=2, block_tokens=2, row_bytes=64, num_blocks=0)
    insts = [random_instance(rng, P=int(rng.integers(20, 60)), max_blocks=10, geom=geom, tier_p=(0.5, 0.35, 0.15),
                             extra_free=int(rng.integers(2, 20))) for _ in range(2)]
    pairs = [Pair(inst, seed=40 + i) for i, inst in enumerate(insts)]
    try:
        for step in range(4):
            for i, (inst, pair) in enumerate(zip(insts, pairs)):
                bb = inst.geom.block_bytes
                bg = int(rng.integers(inst.geom.num_blocks // 3, inst.geom.num_blocks + 1)) * bb
                w = inst.window if (step + i) % 2 == 0 else inst.window[:, :, ::-1].copy()
                log(f"context {i} step {step} P={inst.P} NB={inst.geom.num_blocks}")
                pair.step(gpu_bytes=bg, cpu_bytes=inst.total_bytes, window=w, mode=MODES[(step + i) % 2])
    finally:
        for pair in pairs:
            pair.close()


@pytest.mark.parametrize("mode", MODES)
def test_no_writes_outside_the_pool_and_buffers(mode):
    """Guard bytes around the pool (inside one larger allocation) and past the
    end of the host arena's used extents keep their pattern through several
    rebalances in both directions: no kernel writes outside the pages and
    buffers the plan names."""
    from workload import fill_pool_np, make_bank, program_host_content

    rng = np.random.default_rng(91)
    geom = Geometry(layers=2, planes=2, block_tokens=2, row_bytes=64, num_blocks=0)
    inst = random_instance(rng, P=40, max_blocks=12, geom=geom, tier_p=(0.55, 0.45), extra_free=10)
    g, bb = inst.geom, inst.geom.block_bytes
    guard = 1 << 16
    big = torch.full((guard + g.pool_bytes + guard,), 0xA5, dtype=torch.uint8, device="cuda")
    pool_view = big[guard:guard + g.pool_bytes]
    bank = make_bank(4, inst.dtype, g.run_bytes)
    pool = fill_pool_np(inst, bank)
    pool_view.copy_(torch.from_numpy(pool).cuda())
    bufs = [program_host_content(inst, bank, p).copy() if inst.tier[p] == 1
            else np.zeros(int(inst.nblk[p]) * bb, np.uint8) for p in range(inst.P)]
    tbl, tier, free = inst.copy_state()
    need = sum(max(4096, -(-int(n) * bb // 4096) * 4096) for n in inst.nblk)  # the arena's first-fit extents
    tail = 1 << 16
    tp = TierPool(g, inst.tbl_off, inst.tbl, inst.tier, inst.free_map, arena_bytes=need + tail, pool=pool_view)
    try:
        for p in range(inst.P):  # every program keeps one extent for the whole test
            tp.give_host_buffer(p)
            if bufs[p].size:
                tp.host_view(p)[:] = bufs[p]
        tail_view = tp.arena.view(tp.arena.ptr + need, tail)
        tail_view[:] = 0x5A
        s_out, s_in = torch.cuda.Stream(), torch.cuda.Stream()
        for step in range(4):
            w = inst.window if step % 2 == 0 else inst.window[:, :, ::-1].copy()
            bg = int(rng.integers(g.num_blocks // 4, g.num_blocks + 1)) * bb
            res = oracle.rebalance(g, window=w, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free,
                                   gpu_budget=bg, cpu_budget=inst.total_bytes, pool=pool, host_bufs=bufs)
            assert res.rc == oracle.OK
            assert tp.rank_partition(gpu_bytes=bg, cpu_bytes=inst.total_bytes,
                                     window=torch.from_numpy(np.ascontiguousarray(w)).cuda(), stream=s_out) == 0
            rc, plan = tp.plan_wait()
            assert rc == M.MORI_OK
            assert tp.swap_out(mode, s_out) == M.MORI_OK
            assert tp.swap_in(mode, s_in) == M.MORI_OK
            torch.cuda.synchronize()
            log(f"  guards step {step}: out {plan.n_out} in {plan.n_in}")
            assert (big[:guard] == 0xA5).all().item() and (big[guard + g.pool_bytes:] == 0xA5).all().item()
            assert (tail_view == 0x5A).all()
            t_, r_, f_ = tp.state()
            assert (t_ == tbl).all() and (r_ == tier).all() and (f_ == free).all()
            for p in np.flatnonzero(tier == 1):
                assert np.array_equal(tp.host_view(int(p)), bufs[p]), p
    finally:
        torch.cuda.synchronize()
        tp.close()


def test_two_contexts_on_two_host_threads():
    """Two host threads, each driving its own context (own pool, streams and
    arena) through three rebalances at the same time; each matches its own
    oracle run (distinct contexts share no state)."""
    import threading

    insts = [random_instance(np.random.default_rng(500 + i), P=30, max_blocks=10,
                             geom=Geometry(layers=2, planes=2, block_tokens=2, row_bytes=64, num_blocks=0),
                             tier_p=(0.5, 0.35, 0.15), extra_free=8) for i in range(2)]
    pairs = [Pair(inst, seed=60 + i) for i, inst in enumerate(insts)]
    errors = []

    def work(i):
        try:
            inst, pair = insts[i], pairs[i]
            rng = np.random.default_rng(900 + i)
            bb = inst.geom.block_bytes
            for step in range(3):
                bg = int(rng.integers(inst.geom.num_blocks // 3, inst.geom.num_blocks + 1)) * bb
                w = inst.window if step % 2 == 0 else inst.window[:, :, ::-1].copy()
                pair.step(gpu_bytes=bg, cpu_bytes=inst.total_bytes, window=w, mode=MODES[(i + step) % 2])
        except BaseException as e:  # reported below
            errors.append(repr(e))

    try:
        threads = [threading.Thread(target=work, args=(i,)) for i in range(2)]
        for th in threads:
            th.start()
        for th in threads:
            th.join(timeout=120)
        assert not any(th.is_alive() for th in threads)
        assert not errors, errors
    finally:
        for pair in pairs:
            pair.close()


@pytest.mark.parametrize("target", [1 << 19, (1 << 19) + 1, 1_500_000])
def test_pools_around_the_tile_scan_switch(target):
    """Pools of 2^19 pages (1024 tiles of 512 pages: each page-assignment
    workgroup scans the tile counts itself), one page more (1025 tiles: the
    tile scan is a kernel of its own) and 1.5 M pages, about 85% of them owned,
    so free pages, released pages and incoming slots span many tiles and
    swap-ins land on pages the same step releases: plan, tables, free map and
    bytes equal the oracle's, two steps each."""
    geom = Geometry(layers=1, planes=1, block_tokens=1, row_bytes=16, num_blocks=0)
    P, tier_p = 300, (0.45, 0.35, 0.2)
    max_blocks = int(2 * 0.85 * target / (P * tier_p[0]))
    gpu_blocks = random_instance(np.random.default_rng(target), P=P, max_blocks=max_blocks, geom=geom, tier_p=tier_p,
                                 extra_free=0).geom.num_blocks
    assert gpu_blocks < target
    inst = random_instance(np.random.default_rng(target), P=P, max_blocks=max_blocks, geom=geom, tier_p=tier_p,
                           extra_free=target - gpu_blocks)
    assert inst.geom.num_blocks == target
    log(f"tile scan switch: NB={target} P={inst.P} owned={gpu_blocks} blocks={int(inst.nblk.sum())}")
    pair = Pair(inst, seed=target % 1000)
    try:
        bb = inst.geom.block_bytes
        recycled = 0
        for step in range(2):
            w = inst.window if step == 0 else inst.window[:, :, ::-1].copy()
            res, plan = pair.step(gpu_bytes=min(inst.total_bytes // 2 // bb, target) * bb,
                                  cpu_bytes=int(inst.total_bytes * 0.3) // bb * bb, window=w,
                                  mode=(M.MORI_COPY_KERNEL, M.MORI_COPY_CE)[step])
            assert res.rc == oracle.OK and plan.n_in + plan.n_out > 0
            recycled += plan.pages_recycled
        assert recycled > 0
    finally:
        pair.close()


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("row_bytes,tokens", [(2048, 16), (1536, 16), (1024, 16), (512, 16), (256, 16), (128, 16),
                                               (16, 4)],
                         ids=["32KiB", "24KiB", "16KiB", "8KiB", "4KiB", "2KiB", "64B"])
def test_runs_per_pass(row_bytes, tokens, mode):
    """Runs of 32 KiB (between HBM buffers one round of four vectors per
    thread, half of them past the run's end), 24 KiB and 16 KiB (one vector
    per thread per round: two rounds, the second half past the end, and one;
    over the host link two runs per workgroup), and runs a workgroup copies
    several at a time, one vector per thread: 8, 4 and 2 KiB (two, four and
    eight per pass) and 64 B (sixteen, most threads past the end): every byte
    lands where the oracle puts it, three steps with swaps both ways, in both
    copy modes."""
    rng = np.random.default_rng(row_bytes * 100 + tokens)
    geom = Geometry(layers=2, planes=2, block_tokens=tokens, row_bytes=row_bytes, num_blocks=0)
    inst = random_instance(rng, P=40, max_blocks=12, geom=geom, tier_p=(0.5, 0.3, 0.2), extra_free=20)
    log(f"runs per pass: run={row_bytes * tokens} B mode={mode} NB={inst.geom.num_blocks}")
    pair = Pair(inst, seed=row_bytes + tokens, staging_bytes=int(rng.choice([0, 5 * inst.geom.run_bytes])))
    try:
        bb = inst.geom.block_bytes
        for step in range(3):
            w = inst.window if step % 2 == 0 else inst.window[:, :, ::-1].copy()
            res, plan = pair.step(gpu_bytes=inst.geom.num_blocks * bb * 2 // 3 // bb * bb,
                                  cpu_bytes=inst.total_bytes // 3 // bb * bb, window=w, mode=mode)
            assert res.rc == oracle.OK and plan is not None
    finally:
        pair.close()


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("row_bytes,tokens,staging_runs", [(1152, 64, 0), (1152, 64, 3), (768, 64, 5), (2560, 16, 2),
                                                           (1152, 32, 0), (1024, 64, 0), (1536, 64, 2), (1792, 64, 0),
                                                           (2048, 64, 3), (2176, 64, 0), (4096, 64, 2)],
                         ids=["72KiB", "72KiB-small-staging", "48KiB", "40KiB", "36KiB", "64KiB", "96KiB", "112KiB",
                              "128KiB", "136KiB", "256KiB"])
def test_runs_ending_inside_a_pass(row_bytes, tokens, staging_runs, mode):
    """Long runs, which between HBM buffers a workgroup copies one at a time
    in rounds of four vectors per thread (64 KiB): 36, 40 and 48 KiB (one
    round, the rest of it past the run's end), 64 KiB (exactly one), 72 KiB as
    in the compressed-latent workload (a full round and one of 8 KiB), 96 and
    112 KiB, 128 KiB (exactly two), 136 KiB (three, the last mostly past the
    end) and 256 KiB (four); over the host link two at a time in rounds of
    8 KiB: every byte lands where the oracle puts it, three steps both ways, in
    both copy modes and with staging halves of a few runs."""
    rng = np.random.default_rng(row_bytes * 7 + tokens + staging_runs)
    geom = Geometry(layers=3, planes=1, block_tokens=tokens, row_bytes=row_bytes, num_blocks=0)
    inst = random_instance(rng, P=30, max_blocks=9, geom=geom, tier_p=(0.5, 0.3, 0.2), extra_free=12)
    log(f"runs inside a pass: run={row_bytes * tokens} B mode={mode} staging runs={staging_runs}")
    pair = Pair(inst, seed=row_bytes + tokens, staging_bytes=2 * staging_runs * inst.geom.run_bytes)
    try:
        bb = inst.geom.block_bytes
        # drawn, reversed, then another program's windows for each program
        wins = [inst.window, inst.window[:, :, ::-1].copy(), np.ascontiguousarray(inst.window[rng.permutation(inst.P)])]
        moved = 0
        for w in wins:
            res, plan = pair.step(gpu_bytes=inst.geom.num_blocks * bb * 2 // 3 // bb * bb,
                                  cpu_bytes=inst.total_bytes // 3 // bb * bb, window=w, mode=mode)
            assert res.rc == oracle.OK and plan is not None
            moved += (plan.n_in > 0) + (plan.n_out > 0)
        assert moved >= 4  # swaps in both directions in at least two of the steps
    finally:
        pair.close()


SUMMARY = ("m_gpu", "m_cpu", "n_out", "n_in", "n_drop_gpu", "n_drop_cpu", "n_admit_gpu", "n_admit_cpu", "pages_out",
           "pages_in", "pages_admit", "pages_free_before", "pages_released", "pages_recycled", "pages_free_after",
           "bytes_out", "bytes_in", "gpu_bytes_after", "cpu_bytes_after")


def test_plans_supersede_without_swaps():
    """Placement-only use: four plans in a row with no swap in between (each
    new plan supersedes the last; tables, tiers and the free map stand as the
    last plan wrote them), each equal to the oracle's placement from the state
    the previous one left -- summary, tables, tiers, free map.  Then the last
    plan's swaps: its swap-ins read host buffers that the skipped swap-outs
    never filled or placed, so the device refuses them (MORI_DEV_HOST_ADDR)
    and reports it, rather than copying from an unregistered address."""
    rng = np.random.default_rng(606)
    geom = Geometry(layers=2, planes=2, block_tokens=2, row_bytes=64, num_blocks=0)
    inst = random_instance(rng, P=120, max_blocks=10, geom=geom, tier_p=(0.5, 0.3, 0.2), extra_free=40)
    tp = TierPool(inst.geom, inst.tbl_off, inst.tbl, inst.tier, inst.free_map, arena_bytes=1 << 20)
    try:
        tbl, tier, free = inst.copy_state()
        bb = inst.geom.block_bytes
        for step in range(4):
            w = rng.choice(np.array([0.0, 0.5, 1.0, 2.0, 8.0], np.float32), size=inst.window.shape)
            bg = int(rng.integers(0, inst.geom.num_blocks + 1)) * bb
            bc = int(rng.integers(0, inst.total_bytes // bb + 1)) * bb
            res = oracle.rebalance(inst.geom, window=w, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free,
                                   gpu_budget=bg, cpu_budget=bc)
            assert res.rc == oracle.OK
            assert tp.rank_partition(gpu_bytes=bg, cpu_bytes=bc, window=torch.from_numpy(w).cuda()) == M.MORI_OK
            rc, plan = tp.plan_wait()
            assert rc == M.MORI_OK
            for k in SUMMARY:
                assert getattr(plan, k) == res.summary[k], (step, k)
            g_tbl, g_tier, g_free = tp.state()
            assert (g_tbl == tbl).all() and (g_tier == tier).all() and (g_free == free).all(), step
            log(f"placement-only plan {step}: out {plan.n_out} in {plan.n_in} admitted {plan.n_admit_gpu}")
        assert plan.n_in > 0
        tp.place_host_buffers()
        assert tp.swap_out(M.MORI_COPY_KERNEL) == M.MORI_OK
        assert tp.swap_in(M.MORI_COPY_KERNEL) == M.MORI_OK
        with pytest.raises(MoriError) as e:
            tp.synchronize()
        assert e.value.code == M.MORI_EDEVICE and e.value.detail & M.MORI_DEV_HOST_ADDR
    finally:
        tp.close()


@pytest.mark.parametrize("P", [63, 64, 65, 255, 256, 257, 1023, 1024, 1025, 4095, 4096])
def test_program_counts_at_the_shape_switches(P):
    """Program counts on both sides of each switch between the rank kernel's
    shapes (one wave up to 64 and 256 threads up to 256, both counting ranks
    directly; one item per thread up to 1024, four above): boundary,
    incremental and skip-fit plans with exact ties, equal to the oracle."""
    rng = np.random.default_rng(P)
    geom = Geometry(layers=1, planes=2, block_tokens=1, row_bytes=16, num_blocks=0)
    inst = random_instance(rng, P=P, max_blocks=4, geom=geom, extra_free=int(rng.integers(1, 100)), ties=True)
    pair = Pair(inst, seed=P)
    try:
        bb = inst.geom.block_bytes
        status = rng.integers(0, 3, P).astype(np.uint8)
        for step, flags in enumerate((0, M.MORI_F_INCREMENTAL, M.MORI_F_SKIP_FIT | M.MORI_F_STATUS_KEY)):
            kw = dict(gpu_bytes=int(rng.integers(0, inst.geom.num_blocks + 1)) * bb,
                      cpu_bytes=int(rng.integers(0, inst.total_bytes // bb + 1)) * bb, flags=flags,
                      window=inst.window if step % 2 == 0 else inst.window[:, :, ::-1].copy(),
                      mode=(M.MORI_COPY_KERNEL, M.MORI_COPY_CE)[step % 2])
            if flags & (M.MORI_F_INCREMENTAL | M.MORI_F_STATUS_KEY):
                kw["status"] = status
            log(f"shape switch P={P} step={step} flags={flags}")
            res, plan = pair.step(**kw)
            assert res.rc == oracle.OK and plan is not None
            status = np.where((status == 2) & (pair.tier != 2), 0, status).astype(np.uint8)
    finally:
        pair.close()
