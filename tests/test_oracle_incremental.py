"""Pins of the oracle's incremental sticky policy (Sec. 4.3 sticky placement;
Sec. 4.3.1 demotion from GPU and promotion to GPU).

The oracle runs the paper's loops (pick the next victim while a tier is over
budget, promote while the next candidate fits).  It is pinned here by
hand-derived examples and by brute force on tiny inputs against independent
characterisations of each step:
  * the CPU drops and the GPU victims are the shortest prefix of the demotion
    order (Acting first, then idleness high to low) whose removal fits;
  * the victims' destinations are the lexicographically greatest feasible
    CPU/Wait assignment in demotion order (what placing each victim in the CPU
    tier when it still fits yields);
  * the promoted set is the longest prefix of the candidate order that fits,
    or with skip-fit the lexicographically greatest feasible selection.
"""
import itertools

import numpy as np
import pytest

from golden_io import NONE, incremental_cases
from workload import Geometry

GPU, CPU, WAIT = 0, 1, 2
R, A, N = 0, 1, 2


@pytest.mark.parametrize("name", sorted(incremental_cases()))
def test_worked_examples(orc, name):
    c = incremental_cases()[name]
    flags = orc.F_SKIP_FIT if c["skip_fit"] else 0
    rc, order, prefix, tier_new, mg, mc = orc.incremental(
        np.array(c["idleness"], np.float32), c["status"], c["tier"], c["blocks"], 1, c["gpu_budget"],
        c["cpu_budget"], flags)
    assert rc == orc.OK
    assert tier_new.tolist() == c["new_tier"]
    assert order.tolist() == c["order"]
    assert prefix.tolist() == np.cumsum(np.array(c["blocks"])[c["order"]]).tolist()
    assert (mg, mc) == (c["m_gpu"], c["m_cpu"])


def test_worked_example_b_pages(orc):
    """Example B through a whole rebalance: the promoted CPU program takes the
    first free pages, then the admitted Waiting programs in promotion order
    (returning before new, smallest new first)."""
    c = incremental_cases()["B"]
    P = len(c["blocks"])
    geom = Geometry(num_blocks=6, layers=1, planes=1, block_tokens=1, row_bytes=16)
    off = np.zeros(P + 1, np.uint32)
    off[1:] = np.cumsum(c["blocks"])
    tbl = np.full(off[-1], NONE, np.uint32)
    tbl[0:2] = [4, 1]  # p0 on the GPU
    free = np.array([1, 0, 1, 1, 0, 1], np.uint8)
    tier = np.array(c["tier"], np.uint8)
    res = orc.rebalance(geom, iota=np.array(c["idleness"], np.float32), status=np.array(c["status"], np.uint8),
                        tbl_off=off, tbl=tbl, tier=tier, free_map=free, gpu_budget=16 * c["gpu_budget"],
                        cpu_budget=16 * c["cpu_budget"], flags=orc.F_IDLENESS_GIVEN | orc.F_INCREMENTAL)
    assert res.rc == orc.OK
    assert tier.tolist() == c["new_tier"]
    assert res.category.tolist() == [orc.KEPT, orc.DROP_CPU, orc.IN, orc.DROP_CPU, orc.ADMIT_GPU, orc.KEPT,
                                     orc.ADMIT_GPU, orc.KEPT]
    # free before: 0 2 3 5 -> p2 (in) takes 0 2, p4 takes 3, p6 takes 5
    assert tbl[off[2]:off[3]].tolist() == [0, 2]
    assert tbl[off[4]:off[5]].tolist() == [3]
    assert tbl[off[6]:off[7]].tolist() == [5]
    assert tbl[off[0]:off[1]].tolist() == [4, 1]
    assert free.tolist() == [0] * 6
    s = res.summary
    assert (s["n_in"], s["n_admit_gpu"], s["n_drop_cpu"], s["pages_in"], s["pages_admit"]) == (1, 2, 2, 2, 2)


# ---- brute force ------------------------------------------------------------------------------------------

def _demote_key(p, status, iota):
    return (0 if status[p] == A else 1, -float(iota[p]), -p)


def _shortest_fitting_prefix(seq, size, budget):
    """Smallest k such that dropping seq[:k] leaves at most budget."""
    total = sum(size[p] for p in seq)
    for k in range(len(seq) + 1):
        if total - sum(size[p] for p in seq[:k]) <= budget:
            return k
    raise AssertionError("unreachable")


def _lex_greatest(items, size, room):
    """Lexicographically greatest 0/1 vector over items whose selected sizes fit room."""
    best = None
    for bits in itertools.product((1, 0), repeat=len(items)):  # lexicographically descending
        if sum(size[p] for p, b in zip(items, bits) if b) <= room:
            best = bits
            break
    return best


def brute(iota, status, tier, size, bg, bc, skip_fit):
    P = len(size)
    new = list(tier)
    moved = [False] * P
    used_c = sum(size[p] for p in range(P) if tier[p] == CPU)
    cpu_seq = sorted((p for p in range(P) if tier[p] == CPU), key=lambda p: _demote_key(p, status, iota))
    for p in cpu_seq[:_shortest_fitting_prefix(cpu_seq, size, bc)]:
        new[p], moved[p] = WAIT, True
        used_c -= size[p]
    gpu_seq = sorted((p for p in range(P) if tier[p] == GPU), key=lambda p: _demote_key(p, status, iota))
    victims = gpu_seq[:_shortest_fitting_prefix(gpu_seq, size, bg)]
    for p, b in zip(victims, _lex_greatest(victims, size, bc - used_c)):
        new[p], moved[p] = (CPU if b else WAIT), True
    used_g = sum(size[p] for p in range(P) if new[p] == GPU)

    def level(p):
        return 0 if tier[p] == CPU else (2 if status[p] == N else 1)

    cand = sorted((p for p in range(P) if not moved[p] and tier[p] != GPU and status[p] != A),
                  key=lambda p: (level(p), size[p] if level(p) == 2 else 0, float(iota[p]), p))
    room = bg - used_g
    if skip_fit:
        pick = _lex_greatest(cand, size, room)
    else:
        k = 0
        while k < len(cand) and sum(size[p] for p in cand[:k + 1]) <= room:
            k += 1
        pick = [1] * k + [0] * (len(cand) - k)
    for p, b in zip(cand, pick):
        if b:
            new[p] = GPU

    def group(p):
        if tier[p] in (GPU, CPU):
            return (tier[p], 0 if status[p] != A else 1, float(iota[p]), p)
        g = {R: 2, N: 3, A: 4}[status[p]]
        return (g, size[p] if g == 3 else 0, float(iota[p]), p)

    order = sorted(range(P), key=group)
    return new, order


def _random_case(rng):
    P = int(rng.integers(1, 10))
    size = rng.integers(0, 5, P).tolist()
    tier = rng.integers(0, 3, P).tolist()
    status = rng.integers(0, 3, P).tolist()
    iota = rng.choice(np.array([0, 0.25, 0.5, 0.75, 1.0], np.float32), P)
    total = sum(size)
    bg = int(rng.integers(0, total + 3))
    bc = int(rng.integers(0, total + 3))
    return iota, status, tier, size, bg, bc


@pytest.mark.parametrize("skip_fit", [0, 1])
def test_brute_force_small(orc, skip_fit):
    rng = np.random.default_rng(2606 + skip_fit)
    moved_any = 0
    for _ in range(1500):
        iota, status, tier, size, bg, bc = _random_case(rng)
        rc, order, prefix, tier_new, mg, mc = orc.incremental(iota, status, tier, size, 1, bg, bc,
                                                              orc.F_SKIP_FIT if skip_fit else 0)
        assert rc == orc.OK
        want, want_order = brute(iota, status, tier, size, bg, bc, skip_fit)
        assert tier_new.tolist() == want, (iota, status, tier, size, bg, bc)
        assert order.tolist() == want_order
        assert (mg, mc) == (want.count(GPU), want.count(CPU))
        moved_any += tier_new.tolist() != tier
    assert moved_any > 500


def test_invariants_and_stickiness(orc):
    """Capacities hold after every step; within budgets, nothing leaves a tier
    and only waiting-for-inference programs move up; Acting programs are never
    promoted; Waiting programs never land on the CPU tier."""
    rng = np.random.default_rng(7)
    for _ in range(2000):
        iota, status, tier, size, bg, bc = _random_case(rng)
        rc, _, _, new, _, _ = orc.incremental(iota, status, tier, size, 1, bg, bc)
        assert rc == orc.OK
        size_a = np.array(size)
        new = new.tolist()
        assert size_a[[t == GPU for t in new]].sum() <= bg
        assert size_a[[t == CPU for t in new]].sum() <= bc
        used_g = size_a[[t == GPU for t in tier]].sum()
        used_c = size_a[[t == CPU for t in tier]].sum()
        for p in range(len(size)):
            if tier[p] == WAIT:
                assert new[p] in (WAIT, GPU)
            if new[p] == GPU and tier[p] != GPU:
                assert status[p] != A
            if used_g <= bg and tier[p] == GPU:
                assert new[p] == GPU
            if used_c <= bc and tier[p] == CPU:
                assert new[p] in (CPU, GPU)
            # Acting before Reasoning: a Reasoning program leaves the GPU only if no Acting one stays
            if tier[p] == GPU and new[p] != GPU and status[p] != A:
                assert all(new[q] != GPU for q in range(len(size)) if tier[q] == GPU and status[q] == A)


def test_special_cases(orc):
    iota = np.array([0.5, 0.25, 0.75, 0.0], np.float32)
    status = [A, R, R, N]
    size = [2, 3, 1, 4]
    # a zero GPU budget empties the GPU tier, every victim fitting the CPU tier
    rc, _, _, new, _, _ = orc.incremental(iota, status, [GPU, GPU, GPU, WAIT], size, 1, 0, 100)
    assert rc == orc.OK and new.tolist() == [CPU, CPU, CPU, WAIT]
    # ample GPU room takes every candidate that waits for inference, never an Acting one
    rc, _, _, new, _, _ = orc.incremental(iota, status, [CPU, CPU, WAIT, WAIT], size, 1, 100, 100)
    assert rc == orc.OK and new.tolist() == [CPU, GPU, GPU, GPU]
    # no CPU room: the victim (the Acting program, which alone restores the budget) goes to Waiting
    rc, _, _, new, _, _ = orc.incremental(iota, status, [GPU, GPU, GPU, WAIT], size, 1, 4, 0)
    assert rc == orc.OK and new.tolist() == [WAIT, GPU, GPU, WAIT]
    # empty input
    rc, order, _, new, mg, mc = orc.incremental(np.zeros(0, np.float32), [], [], [], 1, 0, 0)
    assert rc == orc.OK and order.size == 0 and (mg, mc) == (0, 0)


def test_rejects_bad_input(orc):
    ok = dict(iota=np.array([0.5], np.float32), status=[R], tier_old=[WAIT], nblk=[1])

    def run(**kw):
        d = dict(ok, **kw)
        return orc.incremental(d["iota"], d["status"], d["tier_old"], d["nblk"], 1, 10, 10)[0]

    assert run() == orc.OK
    assert run(status=[3]) == orc.E_INPUT
    assert run(iota=np.array([1.5], np.float32)) == orc.E_INPUT
    assert run(iota=np.array([np.nan], np.float32)) == orc.E_INPUT
    assert run(status=[N], nblk=[1 << 31]) == orc.E_INPUT
    assert run(status=[R], nblk=[1 << 31]) == orc.OK  # the limit concerns new arrivals only
    # a whole rebalance needs the status vector
    geom = Geometry(num_blocks=1, layers=1, planes=1, block_tokens=1, row_bytes=16)
    res = orc.rebalance(geom, iota=np.array([0.5], np.float32), tbl_off=np.array([0, 1], np.uint32),
                        tbl=np.array([NONE], np.uint32), tier=np.array([WAIT], np.uint8),
                        free_map=np.ones(1, np.uint8), gpu_budget=16, cpu_budget=0,
                        flags=orc.F_IDLENESS_GIVEN | orc.F_INCREMENTAL)
    assert res.rc == orc.E_INPUT


def test_concurrent_calls_match_sequential(orc):
    """The oracle's sort context is per thread: incremental placements run on
    eight threads at once (the C call releases the GIL) give the results of the
    same calls run one after another."""
    import threading

    rng = np.random.default_rng(808)
    cases = []
    for _ in range(16):
        P = int(rng.integers(50, 400))
        iota = rng.choice(np.array([0.0, 0.25, 0.5, 0.75, 1.0], np.float32), P)  # ties exercise the comparators
        status = rng.integers(0, 3, P).astype(np.uint8)
        tier = rng.integers(0, 3, P).astype(np.uint8)
        nblk = rng.integers(0, 30, P).astype(np.uint32)
        total = int(nblk.sum())
        cases.append((iota, status, tier, nblk, int(rng.integers(0, total + 1)), int(rng.integers(0, total + 1))))
    expect = [orc.incremental(i, s, t, n, 1, g, c) for i, s, t, n, g, c in cases]
    got, errors = {}, []

    def work(k):
        try:
            for rep in range(20):
                j = (k + rep) % len(cases)
                i, s, t, n, g, c = cases[j]
                got.setdefault(j, []).append(orc.incremental(i, s, t, n, 1, g, c))
        except Exception as e:  # pragma: no cover - reported below
            errors.append(e)

    threads = [threading.Thread(target=work, args=(k,)) for k in range(8)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors
    for j, runs in got.items():
        for r in runs:
            assert r[0] == expect[j][0] and r[4:] == expect[j][4:]
            for a, b in zip(r[1:4], expect[j][1:4]):
                assert np.array_equal(a, b)
