"""Randomised sweep of the whole path against the oracle, beyond the targeted
tests: every policy form (boundary with and without skip-fit and the status
key, three tiers, the incremental policy), random geometries and pool
fragmentation, random budgets, both copy modes and small staging buffers
(many chunks), several steps per pool, all through the C ABI and compared
element by element (plan, tables, tiers, free map, every resident and host
byte).  Then eviction orders at sizes on both sides of the switch between the
one-kernel and the three-kernel radix passes, pools whose policy changes from
step to step, and pools of 700-4096 programs (the rank kernel's radix-sort
shapes) with windows of 1 to 64 cycles."""
import numpy as np
import pytest
import torch

from gpu_helpers import Pair, log
from oracle import oracle
from paper_2606_00866_amd import mori as M
from workload import Geometry, eviction_blocks, random_instance

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    assert torch.cuda.is_available(), "GPU tests need the MI355X"
    M.lib()


def _policy(rng):
    form = int(rng.integers(0, 4))
    if form == 0:
        return "boundary", int(rng.integers(0, 4)) & (M.MORI_F_SKIP_FIT | M.MORI_F_STATUS_KEY), (0.5, 0.3, 0.2)
    if form == 1:
        return "ssd", M.MORI_F_SSD_TIER | (M.MORI_F_SKIP_FIT if rng.random() < 0.5 else 0), (0.4, 0.25, 0.15, 0.2)
    if form == 2:
        return "incremental", M.MORI_F_INCREMENTAL | (M.MORI_F_SKIP_FIT if rng.random() < 0.5 else 0), (0.5, 0.3, 0.2)
    return "given", M.MORI_F_IDLENESS_GIVEN | (M.MORI_F_SKIP_FIT if rng.random() < 0.5 else 0), (0.5, 0.3, 0.2)


@pytest.mark.parametrize("block", range(12))
def test_random_rebalances(block):
    """24 pools per block, three steps each."""
    for seed in range(block * 24, block * 24 + 24):
        rng = np.random.default_rng(70000 + seed)
        name, flags, tier_p = _policy(rng)
        P = int(rng.choice([1, 5, 40, 300, 1500]))
        if P < 300:
            geom = Geometry(int(rng.integers(1, 4)), int(rng.integers(1, 3)), int(rng.choice([1, 2, 4, 16])),
                            int(rng.choice([16, 48, 64, 512, 1152])), 0)
        else:  # many programs: small blocks keep the pool and the host copies small
            geom = Geometry(int(rng.integers(1, 3)), int(rng.integers(1, 3)), int(rng.choice([1, 2])),
                            int(rng.choice([16, 48, 64])), 0)
        max_blocks = int(rng.choice([2, 8, 30]))
        inst = random_instance(rng, P=P, max_blocks=max_blocks, geom=geom, tier_p=tier_p, ties=bool(rng.random() < 0.5),
                               extra_free=int(rng.integers(1, 3 * max_blocks + 2)))
        run = inst.geom.run_bytes
        staging = int(rng.choice([0, 2 * run, 6 * run, 64 * run]))
        log(f"fuzz seed={seed} {name} flags={flags} P={inst.P} NB={inst.geom.num_blocks} geom={inst.geom} "
            f"staging={staging}")
        pair = Pair(inst, seed=seed, staging_bytes=staging)
        try:
            bb = inst.geom.block_bytes
            nb_total = inst.total_bytes // max(bb, 1)
            status = rng.integers(0, 3 if name == "incremental" else 2, inst.P).astype(np.uint8)
            for step in range(3):
                bg = int(rng.integers(0, inst.geom.num_blocks + 1)) * bb
                bc = int(rng.integers(0, nb_total + 2)) * bb
                bs = int(rng.integers(0, nb_total + 2)) * bb if name == "ssd" else 0
                mode = (M.MORI_COPY_KERNEL, M.MORI_COPY_CE)[(seed + step) % 2]
                kw = dict(gpu_bytes=bg, cpu_bytes=bc, ssd_bytes=bs, flags=flags, mode=mode)
                if name == "given":
                    kw["iota"] = rng.choice(np.array([0.0, 0.125, 0.5, 0.75, 1.0], np.float32), inst.P)
                else:
                    kw["window"] = inst.window if step != 1 else inst.window[:, :, ::-1].copy()
                if flags & (M.MORI_F_STATUS_KEY | M.MORI_F_INCREMENTAL):
                    kw["status"] = status
                res, plan = pair.step(**kw)
                assert res.rc == oracle.OK, (seed, step, res.rc)
                if name == "incremental":  # statuses move on between steps; new arrivals stay new until placed
                    status = np.where((status == 2) & (pair.tier != 2), 0, status).astype(np.uint8)
                    flip = rng.random(inst.P) < 0.3
                    status = np.where(flip & (status != 2), 1 - status, status).astype(np.uint8)
        finally:
            pair.close()


@pytest.mark.parametrize("N", [1, 1023, 1024, 1025, 131071, 131072, 131073, 200000])
def test_eviction_sizes_around_the_pass_switch(N):
    from test_gpu_evict import check

    rng = np.random.default_rng(N)
    typ, la, size = eviction_blocks(rng, N, programs=int(rng.integers(1, 400)), tie_frac=0.3,
                                    horizon=int(rng.choice([1 << 20, 1 << 40])), var_size=True)
    total = int(size.astype(np.int64).sum())
    need = int(rng.integers(0, total + 1)) * 7
    log(f"fuzz evict N={N} need={need}")
    check(typ, la, size, 7, int(N % 2), need)


@pytest.mark.parametrize("seed", range(8))
def test_policy_changes_between_steps(seed):
    """One pool whose policy changes from step to step (boundary, incremental,
    skip-fit variants, given idleness, three tiers and back once no program is
    left on the SSD tier): each step equals the oracle's from the same state."""
    rng = np.random.default_rng(81000 + seed)
    geom = Geometry(2, 2, 2, 48, 0)
    inst = random_instance(rng, P=int(rng.choice([20, 200])), max_blocks=10, geom=geom, tier_p=(0.5, 0.3, 0.2),
                           extra_free=int(rng.integers(2, 30)))
    pair = Pair(inst, seed=seed, staging_bytes=int(rng.choice([0, 4 * inst.geom.run_bytes])))
    try:
        bb = inst.geom.block_bytes
        nb_total = inst.total_bytes // bb
        status = rng.integers(0, 3, inst.P).astype(np.uint8)
        forms = [0, M.MORI_F_INCREMENTAL, M.MORI_F_SKIP_FIT, M.MORI_F_INCREMENTAL | M.MORI_F_SKIP_FIT,
                 M.MORI_F_IDLENESS_GIVEN, M.MORI_F_SSD_TIER, M.MORI_F_SSD_TIER | M.MORI_F_SKIP_FIT, 0]
        for step, flags in enumerate(forms):
            if not flags & M.MORI_F_SSD_TIER and (pair.tier == 3).any():
                flags |= M.MORI_F_SSD_TIER  # programs on the SSD tier need the three-tier policy
                flags &= ~M.MORI_F_INCREMENTAL
            kw = dict(gpu_bytes=int(rng.integers(0, inst.geom.num_blocks + 1)) * bb,
                      cpu_bytes=int(rng.integers(0, nb_total + 1)) * bb, flags=flags,
                      mode=(M.MORI_COPY_KERNEL, M.MORI_COPY_CE)[step % 2])
            if flags & M.MORI_F_SSD_TIER:
                kw["ssd_bytes"] = int(rng.integers(0, nb_total + 1)) * bb
            if flags & M.MORI_F_IDLENESS_GIVEN:
                kw["iota"] = rng.random(inst.P).astype(np.float32)
            else:
                kw["window"] = inst.window if step % 2 == 0 else inst.window[:, :, ::-1].copy()
            if flags & M.MORI_F_INCREMENTAL:
                kw["status"] = status
            log(f"policy change seed={seed} step={step} flags={flags}")
            res, plan = pair.step(**kw)
            assert res.rc == oracle.OK, (seed, step, flags, res.rc)
            status = np.where((status == 2) & (pair.tier != 2), 0, status).astype(np.uint8)
    finally:
        pair.close()


@pytest.mark.parametrize("block", range(2))
def test_random_large_program_counts(block):
    """24 pools per block of 700-4096 programs (the rank kernel's larger
    shapes) with windows of 1 to 64 cycles, every policy form, two steps each."""
    for seed in range(block * 24, block * 24 + 24):
        rng = np.random.default_rng(90000 + seed)
        name, flags, tier_p = _policy(rng)
        P = int(rng.choice([700, 1024, 1025, 3000, 4096]))
        k = int(rng.choice([1, 5, 17, 64]))
        inst = random_instance(rng, P=P, max_blocks=int(rng.choice([1, 3, 6])), geom=Geometry(1, 2, 1, 16, 0),
                               tier_p=tier_p, ties=bool(rng.random() < 0.5), extra_free=int(rng.integers(1, 200)))
        inst.window = rng.choice(np.array([0.0, 0.25, 0.5, 1.0, 3.0, 60.0], np.float32), size=(P, k, 2))
        log(f"fuzz large seed={seed} {name} flags={flags} P={P} k={k} NB={inst.geom.num_blocks}")
        pair = Pair(inst, seed=seed)
        try:
            bb = inst.geom.block_bytes
            nb_total = inst.total_bytes // bb
            status = rng.integers(0, 3 if name == "incremental" else 2, P).astype(np.uint8)
            for step in range(2):
                kw = dict(gpu_bytes=int(rng.integers(0, inst.geom.num_blocks + 1)) * bb,
                          cpu_bytes=int(rng.integers(0, nb_total + 2)) * bb, flags=flags,
                          ssd_bytes=int(rng.integers(0, nb_total + 2)) * bb if name == "ssd" else 0,
                          mode=(M.MORI_COPY_KERNEL, M.MORI_COPY_CE)[(seed + step) % 2])
                if name == "given":
                    kw["iota"] = rng.random(P).astype(np.float32)
                else:
                    kw["window"] = inst.window if step == 0 else inst.window[:, :, ::-1].copy()
                if flags & (M.MORI_F_STATUS_KEY | M.MORI_F_INCREMENTAL):
                    kw["status"] = status
                res, plan = pair.step(**kw)
                assert res.rc == oracle.OK, (seed, step, res.rc)
        finally:
            pair.close()
