"""GPU parity of the incremental sticky policy (Sec. 4.3.1; MORI_F_INCREMENTAL):
libmori through the C ABI against the CPU oracle, element by element -- listing
order, prefix, categories, summary, block tables, tiers, free map and every
resident byte -- on the hand-derived examples, random pools over several
steps, the 4096-program maximum and a multi-step sequence with phase changes
and new arrivals, in both copy modes."""
import numpy as np
import pytest
import torch

from golden_io import incremental_cases
from gpu_helpers import Pair, instance_from_blocks, log
from oracle import oracle
from paper_2606_00866_amd import mori as M
from workload import Geometry, random_instance

pytestmark = pytest.mark.gpu

MODES = [M.MORI_COPY_KERNEL, M.MORI_COPY_CE]
INC = M.MORI_F_INCREMENTAL


@pytest.fixture(scope="module", autouse=True)
def _lib():
    assert torch.cuda.is_available(), "GPU tests need the MI355X"
    M.lib()


@pytest.mark.parametrize("name", sorted(incremental_cases()))
def test_worked_examples(name):
    c = incremental_cases()[name]
    inst = instance_from_blocks(c["blocks"], c["tier"], c["gpu_budget"], status=c["status"])
    flags = INC | M.MORI_F_IDLENESS_GIVEN | (M.MORI_F_SKIP_FIT if c["skip_fit"] else 0)
    log(f"incremental worked example {name}")
    pair = Pair(inst, seed=11)
    try:
        res, plan = pair.step(gpu_bytes=16 * c["gpu_budget"], cpu_bytes=16 * c["cpu_budget"],
                              iota=np.array(c["idleness"], np.float32), status=inst.status, flags=flags,
                              mode=M.MORI_COPY_KERNEL)
        assert res.rc == oracle.OK
        arr = pair.tp.plan_arrays(plan)
        assert arr["order"].tolist() == c["order"]
        assert pair.tier.tolist() == c["new_tier"]
        assert (plan.m_gpu, plan.m_cpu) == (c["m_gpu"], c["m_cpu"])
    finally:
        pair.close()


@pytest.mark.parametrize("seed", range(32))
def test_random_instances(seed):
    """Random pools, statuses (new arrivals included, also outside Waiting) and
    budgets; three steps with statuses and windows changing in between."""
    rng = np.random.default_rng(5000 + seed)
    max_blocks = int(rng.choice([3, 12, 40]))
    inst = random_instance(rng, P=int(rng.integers(1, 48)), max_blocks=max_blocks, ties=bool(seed % 2),
                           extra_free=int(rng.integers(1, 2 * max_blocks + 2)))  # a pool of at least one page
    mode = MODES[seed % 2]
    flags = INC | (M.MORI_F_SKIP_FIT if seed % 4 >= 2 else 0)
    status = rng.integers(0, 3, inst.P).astype(np.uint8)
    log(f"incremental random seed={seed} P={inst.P} NB={inst.geom.num_blocks} mode={mode} flags={flags}")
    pair = Pair(inst, seed=seed)
    try:
        bb = inst.geom.block_bytes
        for step in range(3):
            bg = int(rng.integers(0, inst.geom.num_blocks + 1)) * bb
            bc = int(rng.integers(0, inst.total_bytes // max(bb, 1) + 2)) * bb
            w = inst.window if step != 1 else inst.window[:, :, ::-1].copy()
            pair.step(gpu_bytes=bg, cpu_bytes=bc, window=w, status=status, flags=flags, mode=mode)
            flip = rng.random(inst.P) < 0.3
            status = np.where(flip, rng.integers(0, 3, inst.P), status).astype(np.uint8)
    finally:
        pair.close()


@pytest.mark.parametrize("skip_fit", [0, 1])
def test_max_programs_with_walks(skip_fit):
    """P = 4096 with tied idleness and new arrivals of many sizes; a CPU room
    smaller than the victims forces the one-by-one victim walk, skip-fit the
    one-by-one promotion walk."""
    rng = np.random.default_rng(77 + skip_fit)
    P = 4096
    geom = Geometry(layers=1, planes=1, block_tokens=1, row_bytes=16, num_blocks=0)
    inst = random_instance(rng, P=P, max_blocks=6, geom=geom, ties=True, tier_p=(0.45, 0.3, 0.25),
                           extra_free=2000)
    status = rng.choice(3, size=P, p=[0.45, 0.4, 0.15]).astype(np.uint8)
    bb = inst.geom.block_bytes
    gpu_now = int(inst.nblk[inst.tier == 0].astype(np.int64).sum()) * bb
    cpu_now = int(inst.nblk[inst.tier == 1].astype(np.int64).sum()) * bb
    log(f"incremental P=4096 skip_fit={skip_fit} NB={inst.geom.num_blocks}")
    pair = Pair(inst, seed=9, max_programs=P)
    try:
        flags = INC | (M.MORI_F_SKIP_FIT if skip_fit else 0)
        # GPU over budget by a third; the CPU tier has a little room: some victims go to Waiting
        res, plan = pair.step(gpu_bytes=gpu_now * 2 // 3, cpu_bytes=cpu_now + gpu_now // 10, window=inst.window,
                              status=status, flags=flags, mode=M.MORI_COPY_CE)
        assert plan.n_out > 0 and plan.n_drop_gpu > 0
        # then a roomy GPU: promotions from the CPU tier and from Waiting
        res, plan = pair.step(gpu_bytes=inst.geom.num_blocks * bb, cpu_bytes=cpu_now, window=inst.window,
                              status=status, flags=flags, mode=M.MORI_COPY_KERNEL)
        assert plan.n_in > 0 and plan.n_admit_gpu > 0
    finally:
        pair.close()


@pytest.mark.parametrize("P", [256, 700])  # the rank kernel's 256 x 1 and 1024 x 1 shapes
@pytest.mark.parametrize("mode", MODES)
def test_phase_changes_and_arrivals(mode, P):
    """P programs over 12 steps: a GPU budget swinging around 55% of the KV,
    20% of the programs switching between Reasoning and Acting each step, and
    new arrivals joining in Waiting; admitted arrivals become Reasoning."""
    rng = np.random.default_rng(404 + mode + P)
    geom = Geometry(layers=2, planes=2, block_tokens=4, row_bytes=64, num_blocks=0)
    inst = random_instance(rng, P=P, max_blocks=24, geom=geom, ties=False, tier_p=(0.5, 0.3, 0.2),
                           extra_free=200)
    status = rng.integers(0, 2, P).astype(np.uint8)
    status[(inst.tier == 2) & (rng.random(P) < 0.5)] = M.MORI_ST_NEW
    bb = inst.geom.block_bytes
    total = inst.total_bytes
    pair = Pair(inst, seed=12)
    try:
        moved = 0
        for t in range(12):
            pct = 55 + 10 * np.sin(2 * np.pi * t / 6)
            bg = min(int(total * pct / 100) // bb * bb, inst.geom.num_blocks * bb)
            window = inst.window if t % 2 == 0 else inst.window[:, :, ::-1].copy()
            res, plan = pair.step(gpu_bytes=bg, cpu_bytes=total // 4, window=window, status=status,
                                  flags=INC, mode=mode)
            moved += plan.bytes_out + plan.bytes_in
            log(f"  step {t}: out {plan.n_out} in {plan.n_in} admit {plan.n_admit_gpu} drop {plan.n_drop_gpu}")
            status[(res.category == oracle.ADMIT_GPU) & (status == M.MORI_ST_NEW)] = M.MORI_ST_REASONING
            flip = (rng.random(P) < 0.2) & (status != M.MORI_ST_NEW)
            status[flip] ^= 1
        assert moved > 0
    finally:
        pair.close()


def test_device_validation_and_host_checks():
    rng = np.random.default_rng(3)
    inst = random_instance(rng, P=10, extra_free=4, tier_p=(0.6, 0.3, 0.1))
    pair = Pair(inst, seed=1)
    try:
        before = pair.tp.state()
        bad = np.zeros(inst.P, np.uint8)
        bad[4] = 3
        w = torch.from_numpy(np.ascontiguousarray(inst.window)).cuda()
        rc = pair.tp.rank_partition(gpu_bytes=0, cpu_bytes=0, window=w, status=torch.from_numpy(bad).cuda(),
                                    flags=INC)
        assert rc == M.MORI_OK
        rc, plan = pair.tp.plan_wait()
        assert rc == M.MORI_EDEVICE and plan.device_error & M.MORI_DEV_BAD_STATUS
        after = pair.tp.state()
        assert all((a == b).all() for a, b in zip(before, after))
        # the incremental policy needs the status vector
        rc = pair.tp.rank_partition(gpu_bytes=0, cpu_bytes=0, window=w, status=None, flags=INC)
        assert rc == M.MORI_EINVAL
        # a status of 3 means nothing to the boundary policy: only Acting (1) counts there
        rc = pair.tp.rank_partition(gpu_bytes=0, cpu_bytes=0, window=w, status=torch.from_numpy(bad).cuda(),
                                    flags=M.MORI_F_STATUS_KEY)
        assert rc == M.MORI_OK
        rc, plan = pair.tp.plan_wait()
        assert rc == M.MORI_OK
    finally:
        pair.close()


def test_bench_plan_cases():
    """The rank/partition leg of bench.py times these exact inputs (the
    Llama-3-8B programs and pool pages, and 4096 random programs) under every
    policy it times (boundary, incremental, three tiers): two consecutive
    plans, each compared with the oracle's."""
    import bench
    from paper_2606_00866_amd.tiering import TierPool
    from workload import LLAMA3_8B, budget_bytes, make_instance

    inst = make_instance(LLAMA3_8B)
    bg = budget_bytes(inst.total_bytes, LLAMA3_8B.gpu_pct)
    for label, geom, src, gb, cb, status, wins in bench.plan_cases(np, inst, bg, 28 << 30):
        for policy, flags, sfrac in bench.POLICIES:
            sb = bench.ssd_budget(src, sfrac)
            log(f"bench plan case {label} {policy}")
            tp = TierPool(geom, src.tbl_off, src.tbl, src.tier, src.free_map, arena_bytes=64 << 20,
                          max_programs=src.P, staging_bytes=1 << 20)
            try:
                tbl, tier, free = src.copy_state()
                st_d = torch.from_numpy(status).cuda()
                for i in range(2):
                    res = oracle.rebalance(geom, window=wins[i], status=status, tbl_off=src.tbl_off, tbl=tbl,
                                           tier=tier, free_map=free, gpu_budget=gb, cpu_budget=cb, flags=flags,
                                           ssd_budget=sb)
                    assert res.rc == oracle.OK
                    assert tp.rank_partition(gpu_bytes=gb, cpu_bytes=cb, window=torch.from_numpy(wins[i]).cuda(),
                                             status=st_d, flags=flags, ssd_bytes=sb) == M.MORI_OK
                    rc, p = tp.plan_wait()
                    assert rc == M.MORI_OK
                    arr = tp.plan_arrays(p)
                    assert (arr["order"] == res.order).all() and (arr["category"] == res.category).all()
                    assert (arr["prefix"] == res.prefix).all()
                    t_, r_, f_ = tp.state()
                    assert (t_ == tbl).all() and (r_ == tier).all() and (f_ == free).all()
                    for k, v in res.summary.items():
                        assert getattr(p, k) == v, k
            finally:
                torch.cuda.synchronize()
                tp.close()
