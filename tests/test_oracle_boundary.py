"""Pins of the oracle's capacity-matched boundary (Sec. 4.1 per-tier capacity,
Sec. 4.3, Sec. 7.2 fill from the busiest end) by brute force and special cases."""
import itertools

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

from golden_io import boundary_case
from workload import LLAMA3_70B, TIER_CPU, TIER_GPU, TIER_WAIT, budget_bytes, make_instance


def brute_prefix(sizes_in_rank_order, b_gpu, b_cpu):
    """Largest m with the first m programs within the GPU budget; then the largest
    following run within the CPU budget (enumerating every m)."""
    P = len(sizes_in_rank_order)
    m_g = max(m for m in range(P + 1) if sum(sizes_in_rank_order[:m]) <= b_gpu)
    m_c = max(m for m in range(P - m_g + 1) if sum(sizes_in_rank_order[m_g:m_g + m]) <= b_cpu)
    return m_g, m_c


def brute_skip_fit(sizes, b_gpu, b_cpu):
    """Lexicographically greatest feasible GPU indicator vector in rank order
    (enumerating all 2^P subsets), then the same for the CPU tier on the rest."""
    P = len(sizes)
    best = None
    for bits in itertools.product([1, 0], repeat=P):  # lexicographically descending
        if sum(s for s, b in zip(sizes, bits) if b) <= b_gpu:
            best = bits
            break
    rest = [r for r in range(P) if not best[r]]
    best_c = None
    for bits in itertools.product([1, 0], repeat=len(rest)):
        if sum(sizes[r] for r, b in zip(rest, bits) if b) <= b_cpu:
            best_c = bits
            break
    tier = [TIER_GPU if best[r] else TIER_WAIT for r in range(P)]
    for r, b in zip(rest, best_c):
        if b:
            tier[r] = TIER_CPU
    return tier


def test_worked_example(orc):
    kv = boundary_case()
    iota = np.array([float(x) for x in kv["idleness"].split()], np.float32)
    blocks = np.array([int(x) for x in kv["blocks"].split()], np.uint32)
    bb = int(kv["block_bytes"])
    _, key = orc.keys(iota)
    order, _ = orc.order(key)
    assert order.tolist() == [int(x) for x in kv["order"].split()]
    for flags, tier_key, mg_key, mc_key in ((0, "tier", "m_gpu", "m_cpu"),
                                            (orc.F_SKIP_FIT, "skipfit_tier", "skipfit_m_gpu", "skipfit_m_cpu")):
        prefix, tier, mg, mc = orc.boundary(order, blocks, bb, int(kv["gpu_budget"]), int(kv["cpu_budget"]), flags)
        assert (prefix // bb).tolist() == [int(x) for x in kv["prefix_blocks"].split()]
        assert tier.tolist() == [int(x) for x in kv[tier_key].split()]
        assert (mg, mc) == (int(kv[mg_key]), int(kv[mc_key]))


sizes_st = st.lists(st.integers(min_value=0, max_value=9), min_size=0, max_size=10)


@settings(max_examples=300, deadline=None)
@given(sizes_st, st.integers(0, 60), st.integers(0, 60), st.booleans())
def test_prefix_and_skip_fit_brute_force(orc, sizes, bg, bc, skip):
    P = len(sizes)
    order = np.arange(P, dtype=np.uint32)[::-1].copy()  # rank r holds program P-1-r
    nblk = np.array(sizes, np.uint32)
    bb = 16
    sz_rank = [sizes[o] * bb for o in order]
    prefix, tier, mg, mc = orc.boundary(order, nblk, bb, bg * bb, bc * bb, orc.F_SKIP_FIT if skip else 0)
    assert prefix.tolist() == list(itertools.accumulate(sz_rank))
    if skip:
        expect_rank = brute_skip_fit(sz_rank, bg * bb, bc * bb)
        assert [int(tier[o]) for o in order] == expect_rank
        assert mg == expect_rank.count(TIER_GPU) and mc == expect_rank.count(TIER_CPU)
    else:
        emg, emc = brute_prefix(sz_rank, bg * bb, bc * bb)
        assert (mg, mc) == (emg, emc)
        assert [int(tier[o]) for o in order] == [TIER_GPU] * emg + [TIER_CPU] * emc + [TIER_WAIT] * (P - emg - emc)
    # capacity invariants (Sec. 4.1): neither tier exceeds its budget
    assert sum(sizes[p] * bb for p in range(P) if tier[p] == TIER_GPU) <= bg * bb
    assert sum(sizes[p] * bb for p in range(P) if tier[p] == TIER_CPU) <= bc * bb


def test_special_cases(orc):
    order = np.array([0, 1, 2, 3], np.uint32)
    nblk = np.array([5, 1, 1, 1], np.uint32)
    # budget at least the total: everything on the GPU
    _, tier, mg, mc = orc.boundary(order, nblk, 1, 8, 0)
    assert mg == 4 and mc == 0 and (tier == TIER_GPU).all()
    # budget below the busiest program: nothing on the GPU even though later ones fit
    _, tier, mg, mc = orc.boundary(order, nblk, 1, 4, 0)
    assert mg == 0 and mc == 0 and (tier == TIER_WAIT).all()
    # budget equal to a prefix sum: that program is included (budget is inclusive)
    _, tier, mg, _ = orc.boundary(order, nblk, 1, 6, 0)
    assert mg == 2 and tier.tolist() == [0, 0, 2, 2]
    # zero-block programs always fit, even with a zero budget
    _, tier, mg, _ = orc.boundary(order, np.array([0, 0, 1, 0], np.uint32), 1, 0, 0)
    assert mg == 2 and tier.tolist() == [0, 0, 2, 2]


@settings(max_examples=100, deadline=None)
@given(sizes_st.filter(lambda s: len(s) > 0), st.integers(0, 90))
def test_monotone_in_budget(orc, sizes, b):
    order = np.arange(len(sizes), dtype=np.uint32)
    nblk = np.array(sizes, np.uint32)
    m1 = orc.boundary(order, nblk, 1, b, 0)[2]
    m2 = orc.boundary(order, nblk, 1, b + 1, 0)[2]
    assert m1 <= m2


@pytest.mark.parametrize("ratio", [1.0, 1.6, 2.0, 3.1])
def test_paper_capacity_ratios(orc, ratio):
    """CPU:GPU capacity ratios of the paper's setup (1x and 2x, Sec. 6.1) and of
    the 1:1.6 / 1:3.1 examples (Sec. 3.4): capacities hold and overflow waits."""
    rng = np.random.default_rng(11)
    P = 200
    nblk = rng.integers(1, 50, P).astype(np.uint32)
    order = rng.permutation(P).astype(np.uint32)
    total = int(nblk.sum())
    bg = total // 5
    bc = int(bg * ratio)
    _, tier, mg, mc = orc.boundary(order, nblk, 1, bg, bc)
    assert nblk[tier == TIER_GPU].sum() <= bg and nblk[tier == TIER_CPU].sum() <= bc
    assert (tier == TIER_WAIT).sum() == P - mg - mc > 0
    # prefix structure: ranks are GPU, then CPU, then Wait
    assert list(tier[order]) == sorted(tier[order])


def test_boundary_shifts_away_from_phase_label(orc):
    """Llama-3-70B workload: 30% busy programs vs a 60% GPU budget -> the GPU tier
    also holds idle-labeled programs, the least idle of them (Sec. 1: a binary
    label cannot match the capacity ratio)."""
    inst = make_instance(LLAMA3_70B)
    tbl, tier, free_map = inst.copy_state()
    res = orc.rebalance(inst.geom, window=inst.window, tbl_off=inst.tbl_off, tbl=tbl, tier=tier,
                        free_map=free_map, gpu_budget=budget_bytes(inst.total_bytes, 60.0),
                        cpu_budget=inst.total_bytes)
    assert res.rc == 0
    on_gpu = tier == TIER_GPU
    assert (on_gpu & ~inst.busy).any()
    busy_ranks = res.rank[inst.busy]
    idle_ranks = res.rank[~inst.busy]
    # the busy-labeled programs rank (almost all) ahead of idle-labeled ones
    assert np.median(busy_ranks) < np.median(idle_ranks)
