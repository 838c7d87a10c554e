"""Pins of the oracle's sticky diff and page allocation (Sec. 4.3; paged KV,
Sec. 2.1): worked examples, pool invariants and error handling."""
import numpy as np
import pytest

from golden_io import NONE, plan_cases
from workload import Geometry, random_instance

ONE = dict(layers=1, planes=1, block_tokens=1, row_bytes=16)


def _state_from_case(c):
    P = len(c["blocks"])
    off = np.zeros(P + 1, np.uint32)
    off[1:] = np.cumsum(c["blocks"])
    tbl = np.array([x for grp in c["tables"] for x in grp], np.uint32)
    free = np.zeros(c["num_blocks"], np.uint8)
    free[c["free"]] = 1
    return off, tbl, np.array(c["tier"], np.uint8), free


@pytest.mark.parametrize("name", sorted(plan_cases()))
def test_worked_examples(orc, name):
    c = plan_cases()[name]
    geom = Geometry(num_blocks=c["num_blocks"], **ONE)
    off, tbl, tier, free = _state_from_case(c)
    flags = orc.F_IDLENESS_GIVEN | (orc.F_INCREMENTAL if "incremental" in c["flags"] else 0)
    status = None if c["status"] is None else np.array(c["status"], np.uint8)
    res = orc.rebalance(geom, iota=np.array(c["idleness"], np.float32), status=status, tbl_off=off, tbl=tbl,
                        tier=tier, free_map=free, gpu_budget=c["gpu_budget"], cpu_budget=c["cpu_budget"],
                        flags=flags)
    assert res.rc == orc.OK
    assert tier.tolist() == c["new_tier"]
    assert tbl.tolist() == [x for grp in c["new_tables"] for x in grp]
    assert np.flatnonzero(free).tolist() == c["new_free"]
    for k, v in c["summary"].items():
        assert res.summary[k] == v, k


def _check_invariants(orc, inst, res, tbl0, tier0, free0, tbl, tier, free, budgets, running=None):
    """running[p]: program p may still be running an inference step (Sec. 4.3.1
    lazy demotion), so pages it leaves become free only after its step."""
    P, NB = inst.P, inst.geom.num_blocks
    off = inst.tbl_off
    nblk = inst.nblk.astype(np.int64)
    # exactly one tier per program; capacities respected (Sec. 4.1)
    bb = inst.geom.block_bytes
    assert nblk[tier == 0].sum() * bb <= budgets[0]
    assert nblk[tier == 1].sum() * bb <= budgets[1]
    # conservation: resident blocks + free pages = pool size; no page owned twice
    owned = np.concatenate([tbl[off[p]:off[p + 1]] for p in range(P) if tier[p] == 0] + [np.zeros(0, np.uint32)])
    assert owned.size + int(free.sum()) == NB
    assert np.unique(owned).size == owned.size
    assert not free[owned].any() if owned.size else True
    # non-resident programs own no page
    for p in range(P):
        if tier[p] != 0:
            assert (tbl[off[p]:off[p + 1]] == NONE).all()
    # sticky placement: a program that stays put keeps its pages
    for p in range(P):
        if tier[p] == tier0[p]:
            assert (tbl[off[p]:off[p + 1]] == tbl0[off[p]:off[p + 1]]).all()
    # allocation: pages handed out in the order free-before ++ dropped ++ swapped out, each ascending
    f0 = np.flatnonzero(free0)

    if running is None:
        running = np.zeros(P, bool)

    def pages_of(keep):
        return np.sort(np.concatenate([tbl0[off[p]:off[p + 1]] for p in range(P)
                                       if tier0[p] == 0 and tier[p] != 0 and keep(p)] + [np.zeros(0, np.uint32)]))

    # nothing reads these: dropped to Waiting and idle
    dropped = pages_of(lambda p: tier[p] == 2 and not running[p])
    # free only later: swapped out (after the swap-out read them) or dropped while running
    later = pages_of(lambda p: tier[p] in (1, 3) or running[p])
    avail = np.concatenate([f0, dropped, later]).astype(np.int64)
    assert res.summary["pages_dropped"] == dropped.size
    incoming = [p for p in res.order if tier0[p] == 1 and tier[p] == 0] + \
               [p for p in res.order if tier0[p] == 2 and tier[p] == 0]
    got = np.concatenate([tbl[off[p]:off[p + 1]] for p in incoming] + [np.zeros(0, np.uint32)]).astype(np.int64)
    assert got.tolist() == avail[:got.size].tolist()
    assert sorted(np.flatnonzero(free).tolist()) == sorted(avail[got.size:].tolist())
    # the ranking prefix structure
    assert list(tier[res.order]) == sorted(tier[res.order])
    s = res.summary
    assert s["pages_recycled"] == max(0, got.size - f0.size)
    assert s["n_out"] == int(((tier0 == 0) & (tier == 1)).sum())
    assert s["n_in"] == int(((tier0 == 1) & (tier == 0)).sum())
    assert s["pages_out"] == int(nblk[(tier0 == 0) & (tier == 1)].sum())
    assert s["bytes_in"] == int(nblk[(tier0 == 1) & (tier == 0)].sum()) * bb


@pytest.mark.parametrize("seed", range(60))
def test_random_instances_invariants(orc, seed):
    rng = np.random.default_rng(seed)
    inst = random_instance(rng)
    total = inst.total_bytes
    bb = inst.geom.block_bytes
    bg = int(rng.integers(0, inst.geom.num_blocks + 1)) * bb
    bc = int(rng.integers(0, total // max(bb, 1) + 2)) * bb
    tbl0, tier0, free0 = inst.copy_state()
    tbl, tier, free = inst.copy_state()
    flags = int(rng.choice([0, orc.F_SKIP_FIT, orc.F_STATUS_KEY]))
    res = orc.rebalance(inst.geom, window=inst.window, status=inst.status, tbl_off=inst.tbl_off, tbl=tbl,
                        tier=tier, free_map=free, gpu_budget=bg, cpu_budget=bc, flags=flags)
    assert res.rc == orc.OK
    if flags == orc.F_SKIP_FIT:
        return _check_invariants_skip(inst, tbl, tier, free, (bg, bc))
    running = inst.status != orc.ST_ACTING if flags == orc.F_STATUS_KEY else None
    _check_invariants(orc, inst, res, tbl0, tier0, free0, tbl, tier, free, (bg, bc), running)


def _check_invariants_skip(inst, tbl, tier, free, budgets):
    nblk = inst.nblk.astype(np.int64)
    bb = inst.geom.block_bytes
    assert nblk[tier == 0].sum() * bb <= budgets[0]
    assert nblk[tier == 1].sum() * bb <= budgets[1]
    off = inst.tbl_off
    owned = np.concatenate([tbl[off[p]:off[p + 1]] for p in range(inst.P) if tier[p] == 0] + [np.zeros(0, np.uint32)])
    assert owned.size + int(free.sum()) == inst.geom.num_blocks
    assert np.unique(owned).size == owned.size


def _inconsistent(kind, inst):
    tbl, tier, free = inst.copy_state()
    off = inst.tbl_off
    gpu = [p for p in range(inst.P) if tier[p] == 0 and inst.nblk[p] > 0]
    cpu = [p for p in range(inst.P) if tier[p] != 0 and inst.nblk[p] > 0]
    if kind == "duplicate":
        a, b = gpu[0], gpu[1]
        tbl[off[b]] = tbl[off[a]]
    elif kind == "free_owned":
        free[tbl[off[gpu[0]]]] = 1
    elif kind == "out_of_range":
        tbl[off[gpu[0]]] = inst.geom.num_blocks
    elif kind == "leaked":
        free[np.flatnonzero(free)[0]] = 0
    elif kind == "nonresident_page":
        tbl[off[cpu[0]]] = 0
    return tbl, tier, free


@pytest.mark.parametrize("kind", ["duplicate", "free_owned", "out_of_range", "leaked", "nonresident_page"])
def test_inconsistent_pool_rejected_and_untouched(orc, kind):
    rng = np.random.default_rng(5)
    while True:
        inst = random_instance(rng, P=12, extra_free=4, tier_p=(0.5, 0.4, 0.1))
        if sum((inst.tier == 0) & (inst.nblk > 0)) >= 2 and sum((inst.tier != 0) & (inst.nblk > 0)) >= 1:
            break
    tbl, tier, free = _inconsistent(kind, inst)
    before = (tbl.copy(), tier.copy(), free.copy())
    res = orc.rebalance(inst.geom, window=inst.window, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free,
                        gpu_budget=inst.geom.num_blocks * inst.geom.block_bytes, cpu_budget=inst.total_bytes)
    assert res.rc == orc.E_POOL
    assert (tbl == before[0]).all() and (tier == before[1]).all() and (free == before[2]).all()


def test_bad_program_data_rejected(orc):
    rng = np.random.default_rng(9)
    inst = random_instance(rng, P=6, extra_free=3)
    kw = dict(window=inst.window, gpu_budget=0, cpu_budget=0)
    tbl, tier, free = inst.copy_state()
    tier[2] = 3
    assert orc.rebalance(inst.geom, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free, **kw).rc == orc.E_INPUT
    tbl, tier, free = inst.copy_state()
    off = inst.tbl_off.copy()
    off[-1] = off[-2] - 1 if off[-2] > 0 else 5
    r = orc.rebalance(inst.geom, tbl_off=off, tbl=tbl, tier=tier, free_map=free, **kw)
    assert r.rc == orc.E_INPUT
    w = inst.window.copy()
    w[0, 0, 0] = np.nan
    tbl, tier, free = inst.copy_state()
    r = orc.rebalance(inst.geom, window=w, tbl_off=inst.tbl_off, tbl=tbl, tier=tier, free_map=free,
                      gpu_budget=0, cpu_budget=0)
    assert r.rc == orc.E_INPUT and (tier == inst.tier).all()


def test_empty_program_set(orc):
    geom = Geometry(num_blocks=4, **ONE)
    free = np.ones(4, np.uint8)
    res = orc.rebalance(geom, window=np.zeros((0, 5, 2), np.float32), tbl_off=np.zeros(1, np.uint32),
                        tbl=np.zeros(0, np.uint32), tier=np.zeros(0, np.uint8), free_map=free, gpu_budget=64,
                        cpu_budget=0)
    assert res.rc == 0 and free.tolist() == [1, 1, 1, 1] and res.summary["m_gpu"] == 0
