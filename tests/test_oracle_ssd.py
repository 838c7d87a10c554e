"""Pins of the oracle's three-tier boundary (Sec. 7.1, an SSD tier below the CPU
tier reached through a further threshold in the same ranking): hand-derived
examples, brute force over all prefixes and all 4^P placements, the reduction
to the two-tier boundary, and a GPU -> SSD -> GPU round trip of KV bytes."""
import itertools

import numpy as np
import pytest

from golden_io import NONE, ssd_cases
from workload import Geometry, fill_pool_np, make_bank, program_host_content, random_instance

GPU, CPU, WAIT, SSD = 0, 1, 2, 3


def _pool_state(blocks, tier, gpu_budget, rng=None):
    """Tables of a consistent pool holding the programs (one page per block)."""
    P = len(blocks)
    off = np.zeros(P + 1, np.uint32)
    off[1:] = np.cumsum(blocks)
    gpu_blocks = int(sum(b for b, t in zip(blocks, tier) if t == GPU))
    NB = max(gpu_blocks, gpu_budget) + 2
    tbl = np.full(int(off[-1]), NONE, np.uint32)
    perm = np.arange(NB, dtype=np.uint32) if rng is None else rng.permutation(NB).astype(np.uint32)
    used = 0
    for p in range(P):
        if tier[p] == GPU:
            tbl[off[p]:off[p + 1]] = perm[used:used + blocks[p]]
            used += blocks[p]
    free = np.zeros(NB, np.uint8)
    free[perm[used:]] = 1
    return NB, off, tbl, free


@pytest.mark.parametrize("name", sorted(ssd_cases()))
def test_worked_examples(orc, name):
    c = ssd_cases()[name]
    NB, off, tbl, free = _pool_state(c["blocks"], c["tier"], c["gpu_budget"])
    geom = Geometry(num_blocks=NB, layers=1, planes=1, block_tokens=1, row_bytes=16)
    tier = np.array(c["tier"], np.uint8)
    flags = orc.F_IDLENESS_GIVEN | orc.F_SSD_TIER | (orc.F_SKIP_FIT if c["skip_fit"] else 0)
    res = orc.rebalance(geom, iota=np.array(c["idleness"], np.float32), tbl_off=off, tbl=tbl, tier=tier,
                        free_map=free, gpu_budget=16 * c["gpu_budget"], cpu_budget=16 * c["cpu_budget"],
                        ssd_budget=16 * c["ssd_budget"], flags=flags)
    assert res.rc == orc.OK
    assert tier.tolist() == c["new_tier"]
    assert res.category.tolist() == c["category"]
    assert [res.summary[k] for k in ("m_gpu", "m_cpu", "m_ssd")] == c["m"]
    nb = np.array(c["blocks"])
    assert res.summary["ssd_bytes_after"] == 16 * nb[tier == SSD].sum()
    # programs off the GPU own no page; SSD programs are neither counted as CPU nor GPU
    for p in range(len(nb)):
        if tier[p] != GPU:
            assert (tbl[off[p]:off[p + 1]] == NONE).all()


def _brute_strict(sizes_ranked, budgets):
    """Longest fitting prefix for the GPU, then the longest fitting run for the
    CPU, then for the SSD, by enumerating every split point."""
    P = len(sizes_ranked)
    start, ms = 0, []
    for b in budgets:
        best = 0
        for m in range(P - start + 1):
            if sum(sizes_ranked[start:start + m]) <= b:
                best = m
        ms.append(best)
        start += best
    return ms


def _brute_skip(sizes_ranked, budgets):
    """Lexicographically greatest placement (GPU > CPU > SSD > Wait per program,
    in rank order) that respects the three budgets."""
    P = len(sizes_ranked)
    best = None
    for tiers in itertools.product((0, 1, 2, 3), repeat=P):  # 0 GPU, 1 CPU, 2 SSD, 3 Wait: ascending = greatest
        load = [0, 0, 0]
        for s, t in zip(sizes_ranked, tiers):
            if t < 3:
                load[t] += s
        if all(l <= b for l, b in zip(load, budgets)):
            best = tiers
            break
    return best


@pytest.mark.parametrize("skip_fit", [0, 1])
def test_boundary_brute_force(orc, skip_fit):
    rng = np.random.default_rng(31 + skip_fit)
    for _ in range(400):
        P = int(rng.integers(0, 7 if skip_fit else 10))
        nblk = rng.integers(0, 5, P).astype(np.uint32)
        order = rng.permutation(P).astype(np.uint32)
        total = int(nblk.sum())
        budgets = [int(rng.integers(0, total + 2)) for _ in range(3)]
        flags = orc.F_SSD_TIER | (orc.F_SKIP_FIT if skip_fit else 0)
        prefix, tier_new, mg, mc, ms = orc.boundary(order, nblk, 1, *budgets[:2], flags=flags,
                                                   ssd_budget=budgets[2], with_ssd=True)
        ranked = [int(nblk[p]) for p in order]
        assert prefix.tolist() == np.cumsum(ranked).tolist()
        if skip_fit:
            want = _brute_skip(ranked, budgets)
            code = {0: GPU, 1: CPU, 2: SSD, 3: WAIT}
            assert [int(tier_new[p]) for p in order] == [code[t] for t in want]
            assert (mg, mc, ms) == tuple(sum(1 for t in want if t == k) for k in (0, 1, 2))
        else:
            want = _brute_strict(ranked, budgets)
            assert [mg, mc, ms] == want
            tiers = [GPU] * want[0] + [CPU] * want[1] + [SSD] * want[2] + [WAIT] * (P - sum(want))
            assert [int(tier_new[p]) for p in order] == tiers


def test_reduces_to_two_tiers(orc):
    """With no SSD room and no zero-block program the SSD flag changes nothing;
    with room for everything, nothing waits."""
    rng = np.random.default_rng(5)
    for _ in range(200):
        P = int(rng.integers(1, 30))
        nblk = rng.integers(1, 9, P).astype(np.uint32)
        order = rng.permutation(P).astype(np.uint32)
        total = int(nblk.sum())
        bg, bc = int(rng.integers(0, total + 1)), int(rng.integers(0, total + 1))
        for skip in (0, orc.F_SKIP_FIT):
            a = orc.boundary(order, nblk, 1, bg, bc, flags=skip)
            b = orc.boundary(order, nblk, 1, bg, bc, flags=skip | orc.F_SSD_TIER, ssd_budget=0, with_ssd=True)
            assert (a[1] == b[1]).all() and a[2:] == b[2:4] and b[4] == 0
            c = orc.boundary(order, nblk, 1, bg, bc, flags=skip | orc.F_SSD_TIER, ssd_budget=total, with_ssd=True)
            assert not (c[1] == WAIT).any()


def test_tier_and_flag_validation(orc):
    geom = Geometry(num_blocks=2, layers=1, planes=1, block_tokens=1, row_bytes=16)
    base = dict(iota=np.array([0.5], np.float32), tbl_off=np.array([0, 1], np.uint32), gpu_budget=16,
                cpu_budget=16)

    def run(flags, tier=SSD, status=None):
        return orc.rebalance(geom, tbl=np.array([NONE], np.uint32), tier=np.array([tier], np.uint8),
                             free_map=np.ones(2, np.uint8), status=status, flags=orc.F_IDLENESS_GIVEN | flags,
                             **base).rc

    assert run(0) == orc.E_INPUT  # an SSD tier without the flag
    assert run(orc.F_SSD_TIER) == orc.OK
    assert run(orc.F_SSD_TIER, tier=4) == orc.E_INPUT
    assert run(orc.F_SSD_TIER | orc.F_INCREMENTAL, tier=WAIT, status=np.zeros(1, np.uint8)) == orc.E_INPUT


def test_ssd_round_trip_bytes(orc):
    """GPU -> SSD then SSD -> GPU: every run of every program comes back to its
    new pages unchanged (the SSD program's KV sits in its host buffer)."""
    rng = np.random.default_rng(8)
    inst = random_instance(rng, P=12, max_blocks=6, geom=Geometry(2, 2, 2, 32, 0), extra_free=4,
                           tier_p=(1.0, 0.0, 0.0))
    g = inst.geom
    bank = make_bank(3, "fp16", g.run_bytes)
    pool = fill_pool_np(inst, bank)
    bufs = [np.zeros(int(n) * g.block_bytes, np.uint8) for n in inst.nblk]
    tbl, tier, free = inst.copy_state()
    iota = rng.random(inst.P).astype(np.float32)
    total = inst.total_bytes
    common = dict(iota=iota, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free, pool=pool, host_bufs=bufs,
                  flags=orc.F_IDLENESS_GIVEN | orc.F_SSD_TIER)
    res = orc.rebalance(g, gpu_budget=total // 3, cpu_budget=0, ssd_budget=total, **common)
    assert res.rc == orc.OK and (tier == SSD).any() and not (tier == WAIT).any()
    ssd_bytes = int(inst.nblk[tier == SSD].astype(np.int64).sum()) * g.block_bytes
    assert (res.summary["ssd_bytes_after"], res.summary["cpu_bytes_after"]) == (ssd_bytes, 0)
    assert res.summary["bytes_out"] == ssd_bytes and res.summary["n_out"] == int((tier == SSD).sum())
    for p in np.flatnonzero(tier == SSD):
        assert np.array_equal(bufs[p], program_host_content(inst, bank, int(p)))
    res = orc.rebalance(g, gpu_budget=g.num_blocks * g.block_bytes, cpu_budget=0, ssd_budget=0, **common)
    assert res.rc == orc.OK and (tier == GPU).all()
    planes = pool.reshape(g.nplanes, g.num_blocks, g.run_bytes)
    for p in range(inst.P):
        n = int(inst.nblk[p])
        pages = tbl[inst.tbl_off[p]:inst.tbl_off[p + 1]].astype(np.int64)
        got = planes[:, pages].reshape(-1)
        assert np.array_equal(got, program_host_content(inst, bank, p)), p
        assert n == pages.size
