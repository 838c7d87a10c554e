"""GPU parity of the three-tier boundary (Sec. 7.1; MORI_F_SSD_TIER): libmori
through the C ABI against the CPU oracle, element by element -- order, prefix,
categories, summary (m_ssd, ssd_bytes_after included), block tables, tiers,
free map and every resident byte, SSD programs' KV held in host buffers -- on
the hand-derived examples, random pools with SSD programs over several steps
and the tiny workload, in both copy modes."""
import numpy as np
import pytest
import torch

from golden_io import ssd_cases
from gpu_helpers import Pair, instance_from_blocks, log
from oracle import oracle
from paper_2606_00866_amd import mori as M
from workload import TINY, make_instance, random_instance

pytestmark = pytest.mark.gpu

MODES = [M.MORI_COPY_KERNEL, M.MORI_COPY_CE]
SSD = M.MORI_F_SSD_TIER


@pytest.fixture(scope="module", autouse=True)
def _lib():
    assert torch.cuda.is_available(), "GPU tests need the MI355X"
    M.lib()


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", sorted(ssd_cases()))
def test_worked_examples(name, mode):
    c = ssd_cases()[name]
    inst = instance_from_blocks(c["blocks"], c["tier"], c["gpu_budget"])
    flags = SSD | M.MORI_F_IDLENESS_GIVEN | (M.MORI_F_SKIP_FIT if c["skip_fit"] else 0)
    log(f"ssd worked example {name} mode={mode}")
    pair = Pair(inst, seed=21)
    try:
        res, plan = pair.step(gpu_bytes=16 * c["gpu_budget"], cpu_bytes=16 * c["cpu_budget"],
                              ssd_bytes=16 * c["ssd_budget"], iota=np.array(c["idleness"], np.float32),
                              flags=flags, mode=mode)
        assert res.rc == oracle.OK
        assert pair.tier.tolist() == c["new_tier"]
        assert pair.tp.plan_arrays(plan)["category"].tolist() == c["category"]
        assert [plan.m_gpu, plan.m_cpu, plan.m_ssd] == c["m"]
    finally:
        pair.close()


@pytest.mark.parametrize("seed", range(24))
def test_random_instances(seed):
    rng = np.random.default_rng(9000 + seed)
    max_blocks = int(rng.choice([3, 12, 40]))
    inst = random_instance(rng, P=int(rng.integers(1, 40)), max_blocks=max_blocks, ties=bool(seed % 2),
                           tier_p=(0.4, 0.25, 0.15, 0.2), extra_free=int(rng.integers(1, 2 * max_blocks + 2)))
    mode = MODES[seed % 2]
    flags = SSD | (M.MORI_F_SKIP_FIT if seed % 4 >= 2 else 0) | (M.MORI_F_STATUS_KEY if seed % 3 == 0 else 0)
    log(f"ssd random seed={seed} P={inst.P} NB={inst.geom.num_blocks} mode={mode} flags={flags}")
    pair = Pair(inst, seed=seed)
    try:
        bb = inst.geom.block_bytes
        nb_total = inst.total_bytes // max(bb, 1)
        for step in range(3):
            bg = int(rng.integers(0, inst.geom.num_blocks + 1)) * bb
            bc = int(rng.integers(0, nb_total + 2)) * bb
            bs = int(rng.integers(0, nb_total + 2)) * bb
            w = inst.window if step != 1 else inst.window[:, :, ::-1].copy()
            pair.step(gpu_bytes=bg, cpu_bytes=bc, ssd_bytes=bs, window=w, status=inst.status, flags=flags, mode=mode)
    finally:
        pair.close()


def test_mid_size_program_count():
    """600 programs (the rank kernel's 1024 x 1 shape) over three tiers, two steps."""
    rng = np.random.default_rng(600)
    inst = random_instance(rng, P=600, max_blocks=10, ties=False, tier_p=(0.4, 0.25, 0.15, 0.2), extra_free=50)
    pair = Pair(inst, seed=6)
    try:
        bb = inst.geom.block_bytes
        nb_total = inst.total_bytes // bb
        for step in range(2):
            w = inst.window if step == 0 else inst.window[:, :, ::-1].copy()
            pair.step(gpu_bytes=int(rng.integers(1, inst.geom.num_blocks + 1)) * bb,
                      cpu_bytes=int(rng.integers(0, nb_total)) * bb, ssd_bytes=int(rng.integers(0, nb_total)) * bb,
                      window=w, flags=SSD, mode=MODES[step])
    finally:
        pair.close()


@pytest.mark.parametrize("mode", MODES)
def test_tiny_three_tiers(mode):
    """The tiny workload split 40% GPU / 20% CPU / 30% SSD, then the reversed
    ranking (every tier changes hands), then back."""
    inst = make_instance(TINY)
    total = inst.total_bytes
    bb = inst.geom.block_bytes
    bg, bc, bs = (total * 40 // 100) // bb * bb, (total * 20 // 100) // bb * bb, (total * 30 // 100) // bb * bb
    pair = Pair(inst, seed=TINY.seed)
    try:
        seen = set()
        for t, w in enumerate((inst.window, inst.window[:, :, ::-1].copy(), inst.window)):
            res, plan = pair.step(gpu_bytes=bg, cpu_bytes=bc, ssd_bytes=bs, window=w, flags=SSD, mode=mode)
            seen |= set(np.unique(res.category).tolist())
            log(f"  step {t}: m {plan.m_gpu}/{plan.m_cpu}/{plan.m_ssd} out {plan.n_out} in {plan.n_in}")
            assert plan.m_ssd > 0
        assert {oracle.OUT, oracle.IN, oracle.CPU_SSD, oracle.SSD_CPU} <= seen
    finally:
        pair.close()


def test_validation():
    rng = np.random.default_rng(4)
    inst = random_instance(rng, P=8, extra_free=4, tier_p=(0.5, 0.2, 0.1, 0.2))
    assert (inst.tier == 3).any()
    pair = Pair(inst, seed=2)
    try:
        w = torch.from_numpy(np.ascontiguousarray(inst.window)).cuda()
        before = pair.tp.state()
        # an SSD program without the flag is a bad tier, found on the device; nothing changes
        assert pair.tp.rank_partition(gpu_bytes=0, cpu_bytes=0, window=w) == M.MORI_OK
        rc, plan = pair.tp.plan_wait()
        assert rc == M.MORI_EDEVICE and plan.device_error & M.MORI_DEV_BAD_TIER
        assert all((a == b).all() for a, b in zip(before, pair.tp.state()))
        # the SSD tier belongs to the boundary policy only
        st = torch.zeros(inst.P, dtype=torch.uint8, device="cuda")
        assert pair.tp.rank_partition(gpu_bytes=0, cpu_bytes=0, window=w, status=st,
                                      flags=SSD | M.MORI_F_INCREMENTAL) == M.MORI_EINVAL
    finally:
        pair.close()
