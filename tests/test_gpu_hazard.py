"""The ordering that overlapping the two swaps relies on, tested under
pressure: the swap-out stream is held back by a bounded spin before the
swap-out is enqueued, while the swap-in stream is free to run at once.

- Recycled pages (Sec. 4.3: both directions move in one tick): most swap-in
  slots are pages the delayed swap-out still has to read.  If the swap-in
  wrote any of them early, the swapped-out programs' host buffers would hold
  the promoted programs' bytes; every byte is compared with the oracle.  The
  copy-engine case includes a staging size where the wait falls in the
  middle of the chunk sequence.
- A program dropped to Waiting while it runs (Sec. 4.3.1 lazy demotion):
  its inference step is ordered on the swap-out stream after the spin (here
  it reads the victim's pages).  It must see the victim's own KV, although a
  promoted program takes some of those pages in the same step.

Each case also checks that the pressure was real (the swap-out began at
least a few milliseconds after the swap-in was free to start) and that the
swap-in ended after the swap-out.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import NONE, Pair, log
from oracle import oracle
from paper_2606_00866_amd import mori as M
from workload import Geometry, random_instance

pytestmark = pytest.mark.gpu

SPIN_CYCLES = 50_000_000   # a bounded spin kernel: tens of milliseconds at the shader clock
MIN_HOLD_MS = 2.0


def _instance(blocks, tier, status, free_pages, geom, seed=0):
    """A consistent pool: GPU programs own a random permutation of the pages
    less `free_pages`, which are free."""
    rng = np.random.default_rng(seed)
    P = len(blocks)
    nblk = np.array(blocks, np.uint32)
    tier = np.array(tier, np.uint8)
    NB = int(nblk[tier == 0].sum()) + free_pages
    inst = random_instance(rng, P=P, geom=Geometry(geom.layers, geom.planes, geom.block_tokens, geom.row_bytes, 0),
                           extra_free=0)
    off = np.zeros(P + 1, np.uint32)
    off[1:] = np.cumsum(nblk)
    tbl = np.full(int(off[-1]), NONE, np.uint32)
    perm = rng.permutation(NB).astype(np.uint32)
    used = 0
    for p in range(P):
        if tier[p] == 0:
            tbl[off[p]:off[p + 1]] = perm[used:used + nblk[p]]
            used += int(nblk[p])
    free = np.zeros(NB, np.uint8)
    free[perm[used:]] = 1
    inst.geom = Geometry(geom.layers, geom.planes, geom.block_tokens, geom.row_bytes, NB)
    inst.nblk, inst.tbl_off, inst.tbl, inst.tier, inst.free_map = nblk, off, tbl, tier, free
    inst.ctx = nblk.astype(np.int64) * geom.block_tokens
    inst.status = np.array(status, np.uint8)
    return inst


def _delayed_step(pair, *, gpu_bytes, cpu_bytes, iota, flags, mode, status=None, readers=()):
    """One rebalance with the swap-out stream held back; `readers` are
    programs whose inference step (a read of their pages) is ordered on the
    swap-out stream after the hold.  Returns (plan, hold_ms, tail_ms, reads)."""
    inst, g, tp = pair.inst, pair.g, pair.tp
    tbl0, pool0 = pair.tbl.copy(), pair.pool.copy()
    flags |= M.MORI_F_IDLENESS_GIVEN
    res = oracle.rebalance(g, iota=iota, status=status, tbl_off=inst.tbl_off, tbl=pair.tbl, tier=pair.tier,
                           free_map=pair.free, gpu_budget=gpu_bytes, cpu_budget=cpu_bytes, flags=flags,
                           pool=pair.pool, host_bufs=pair.bufs)
    assert res.rc == oracle.OK
    dev = tp.device
    it = torch.from_numpy(np.ascontiguousarray(iota, np.float32)).to(dev)
    st = None if status is None else torch.from_numpy(np.ascontiguousarray(status, np.uint8)).to(dev)
    s_out, s_in = pair.s_out, pair.s_in
    assert tp.rank_partition(gpu_bytes=gpu_bytes, cpu_bytes=cpu_bytes, idleness=it, status=st, flags=flags,
                             stream=s_out) == M.MORI_OK
    rc, plan = tp.plan_wait()
    assert rc == M.MORI_OK, plan.device_error
    tp.place_host_buffers()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    dpool = tp.pool.view(g.nplanes, g.num_blocks, g.run_bytes)
    reads = {}
    ev[0].record(s_in)  # the swap-in stream is free from here
    with torch.cuda.stream(s_out):
        torch.cuda._sleep(SPIN_CYCLES)
        for p in readers:
            pages = torch.from_numpy(tbl0[inst.tbl_off[p]:inst.tbl_off[p + 1]].astype(np.int64)).to(dev)
            reads[p] = (dpool.index_select(1, pages), pages.cpu().numpy())
    ev[1].record(s_out)  # the swap-out may start only from here
    assert tp.swap_out(mode, s_out) == M.MORI_OK
    ev[2].record(s_out)
    assert tp.swap_in(mode, s_in) == M.MORI_OK
    ev[3].record(s_in)
    tp.synchronize()
    hold = ev[0].elapsed_time(ev[1])
    tail = ev[2].elapsed_time(ev[3])
    pair.compare(res, plan)
    pair.prefill(res)
    got = {p: (t.cpu().numpy(), pg) for p, (t, pg) in reads.items()}
    opool = pool0.reshape(g.nplanes, g.num_blocks, g.run_bytes)
    for p, (t, pg) in got.items():
        assert np.array_equal(t, opool[:, pg]), f"program {p}'s running step read another program's bytes"
    return plan, hold, tail


@pytest.mark.parametrize("mode,runs_per_half", [(M.MORI_COPY_KERNEL, 0), (M.MORI_COPY_CE, 0), (M.MORI_COPY_CE, 2),
                                                (M.MORI_COPY_CE, 7)])
def test_recycled_slots_wait_for_a_delayed_swap_out(mode, runs_per_half):
    geom = Geometry(layers=3, planes=2, block_tokens=4, row_bytes=512, num_blocks=0)
    rng = np.random.default_rng(77)
    P_gpu, P_cpu = 14, 10
    blocks = rng.integers(2, 9, size=P_gpu + P_cpu).tolist()
    tier = [0] * P_gpu + [1] * P_cpu
    inst = _instance(blocks, tier, [1] * (P_gpu + P_cpu), free_pages=6, geom=geom)
    run = geom.block_tokens * geom.row_bytes
    staging = 2 * runs_per_half * run
    pair = Pair(inst, seed=8, staging_bytes=staging)
    try:
        g = inst.geom
        # CPU programs busiest, GPU programs next by id: the whole pool stays
        # the GPU budget, so the CPU programs come in and as many GPU-resident
        # bytes go out, nearly all onto pages the swap-out still reads
        iota = np.array([0.2 + 0.03 * p for p in range(P_gpu)] + [0.1] * P_cpu, np.float32)
        plan, hold, tail = _delayed_step(pair, gpu_bytes=g.num_blocks * g.block_bytes, cpu_bytes=inst.total_bytes,
                                         iota=iota, flags=0, mode=mode)
        gated = plan.pages_in - min(plan.pages_in, plan.pages_free_before + plan.pages_dropped)
        log(f"mode={mode} staging={staging}: in {plan.pages_in} pages, {gated} on pages the swap-out reads; "
            f"swap-out held {hold:.1f} ms, swap-in ended {tail:.2f} ms after it")
        assert plan.n_out > 0 and gated >= plan.pages_in // 2
        assert hold >= MIN_HOLD_MS and tail >= 0.0
        # and back: the programs just swapped out return onto pages of the ones just swapped in
        iota2 = np.where(pair.tier == 1, 0.05, np.where(pair.tier == 0, 0.6, 0.9)).astype(np.float32)
        plan, hold, tail = _delayed_step(pair, gpu_bytes=g.num_blocks * g.block_bytes, cpu_bytes=inst.total_bytes,
                                         iota=iota2, flags=0, mode=mode)
        assert plan.n_in > 0 and hold >= MIN_HOLD_MS and tail >= 0.0
    finally:
        pair.close()


@pytest.mark.parametrize("policy", ["incremental", "status_key"])
@pytest.mark.parametrize("mode", [M.MORI_COPY_KERNEL, M.MORI_COPY_CE])
def test_running_victim_keeps_its_pages_until_its_step_ends(policy, mode):
    geom = Geometry(layers=2, planes=2, block_tokens=4, row_bytes=256, num_blocks=0)
    R, A = M.MORI_ST_REASONING, M.MORI_ST_ACTING
    if policy == "incremental":
        # GPU 4+6+2 = 12 blocks over a budget of 7: the Acting p2 goes first, then
        # the Reasoning p1 (both to Waiting: the CPU tier has no room); p3 (3
        # blocks, a CPU program waiting for inference) fills the room of 3 and
        # takes p2's two pages and one of p1's.
        blocks, tier, status = [4, 6, 2, 3, 4], [0, 0, 0, 1, 1], [R, R, A, R, R]
        iota = np.array([0.25, 0.5, 0.75, 0.125, 0.3], np.float32)
        flags, bg, bc = M.MORI_F_INCREMENTAL, 7, 7
        victim = 1
    else:
        # boundary policy with the status key: p2 (CPU, busiest) and p0 fit the
        # GPU budget of 7 blocks; the Reasoning p1 has no CPU room and waits
        blocks, tier, status = [4, 4, 3], [0, 0, 1], [R, R, R]
        iota = np.array([0.5, 0.6, 0.1], np.float32)
        flags, bg, bc = M.MORI_F_STATUS_KEY, 7, 0
        victim = 1
    inst = _instance(blocks, tier, status, free_pages=0, geom=geom, seed=3)
    pair = Pair(inst, seed=4, staging_bytes=4 * geom.block_tokens * geom.row_bytes)
    try:
        bb = inst.geom.block_bytes
        plan, hold, tail = _delayed_step(pair, gpu_bytes=bg * bb, cpu_bytes=bc * bb, iota=iota,
                                         status=np.array(status, np.uint8), flags=flags, mode=mode,
                                         readers=(victim,))
        log(f"{policy} mode={mode}: dropped {plan.n_drop_gpu}, pages at once {plan.pages_dropped}, "
            f"in {plan.pages_in}; hold {hold:.1f} ms, tail {tail:.2f} ms")
        assert pair.tier[victim] == 2 and plan.n_in == 1
        # the promoted program reaches into the running victim's pages
        assert plan.pages_in > plan.pages_free_before + plan.pages_dropped
        assert hold >= MIN_HOLD_MS and tail >= 0.0
    finally:
        pair.close()
