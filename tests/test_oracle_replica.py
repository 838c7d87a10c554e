"""Pins of the oracle's multi-replica admission (Sec. 4.1 shared Waiting queue;
Sec. 4.3.1 bin packing of Waiting promotions across replicas): hand-derived
examples, the one-replica case against brute force, closed forms for equal
sizes, and invariants that hold at any size."""
import itertools

import numpy as np
import pytest

from golden_io import replica_cases

R_, A_, N_ = 0, 1, 2


@pytest.mark.parametrize("name", sorted(replica_cases()))
def test_worked_examples(orc, name):
    c = replica_cases()[name]
    rc, rep, after = orc.replica_admit(c["bytes"], c["idleness"], c["status"], c["room"],
                                       orc.ADMIT_BEST_FIT if c["best_fit"] else 0)
    assert rc == orc.OK
    assert rep.tolist() == c["replica"]
    assert after.tolist() == c["room_after"]


def _order(bytes_, iota, status):
    cand = [p for p in range(len(bytes_)) if status[p] != A_]
    return sorted(cand, key=lambda p: (status[p] == N_, -int(bytes_[p]), float(iota[p]), p))


def test_one_replica_is_greedy_in_packing_order(orc):
    """With one replica both rules place a candidate whenever it still fits: the
    admitted set is the lexicographically greatest feasible selection in
    packing order (enumerated over all subsets)."""
    rng = np.random.default_rng(12)
    for _ in range(400):
        P = int(rng.integers(0, 10))
        b = rng.integers(0, 8, P).astype(np.uint64)
        iota = rng.choice(np.array([0, 0.5, 1], np.float32), P)
        st = rng.integers(0, 3, P).astype(np.uint8)
        room = int(rng.integers(0, int(b.sum()) + 3))
        order = _order(b, iota, st)
        want = None
        for bits in itertools.product((1, 0), repeat=len(order)):
            if sum(int(b[p]) for p, x in zip(order, bits) if x) <= room:
                want = bits
                break
        for flags in (0, orc.ADMIT_BEST_FIT):
            rc, rep, after = orc.replica_admit(b, iota, st, [room], flags)
            assert rc == orc.OK
            assert [int(rep[p] == 0) for p in order] == list(want)
            assert all(rep[p] == -1 for p in range(P) if st[p] == A_)


@pytest.mark.parametrize("R,k,s,room", [(3, 10, 2, 7), (4, 9, 3, 9), (5, 3, 1, 1), (2, 7, 5, 11)])
def test_equal_sizes_closed_forms(orc, R, k, s, room):
    """k programs of s bytes onto R replicas of equal room: the default rule
    spreads them (per-replica counts differ by at most one while every replica
    has room), best fit fills replica 0 first, then 1, ...; both admit
    min(k, R * floor(room / s))."""
    per = room // s
    admitted = min(k, R * per)
    iota = np.linspace(0, 1, k).astype(np.float32)
    st = np.zeros(k, np.uint8)
    rc, rep, _ = orc.replica_admit(np.full(k, s), iota, st, np.full(R, room))
    counts = np.bincount(rep[rep >= 0], minlength=R)
    assert rc == orc.OK and counts.sum() == admitted
    assert counts.max() - counts.min() <= 1
    rc, rep, _ = orc.replica_admit(np.full(k, s), iota, st, np.full(R, room), orc.ADMIT_BEST_FIT)
    counts = np.bincount(rep[rep >= 0], minlength=R)
    want = [min(per, max(0, admitted - r * per)) for r in range(R)]
    assert rc == orc.OK and counts.tolist() == want


def test_invariants(orc):
    """Room is conserved and never negative; Acting programs stay; a candidate
    left waiting fits no replica even at the end (rooms only shrink); ids of
    replicas are in range."""
    rng = np.random.default_rng(99)
    for _ in range(500):
        P = int(rng.integers(0, 60))
        R = int(rng.integers(1, 9))
        b = rng.integers(0, 50, P).astype(np.uint64)
        iota = rng.random(P).astype(np.float32)
        st = rng.integers(0, 3, P).astype(np.uint8)
        room = rng.integers(0, 120, R).astype(np.uint64)
        for flags in (0, orc.ADMIT_BEST_FIT):
            rc, rep, after = orc.replica_admit(b, iota, st, room, flags)
            assert rc == orc.OK
            assert ((rep >= -1) & (rep < R)).all()
            used = np.zeros(R, np.int64)
            for p in range(P):
                if rep[p] >= 0:
                    used[rep[p]] += int(b[p])
            assert (after.astype(np.int64) + used == room.astype(np.int64)).all()
            assert (rep[st == A_] == -1).all()
            left = (rep == -1) & (st != A_)
            assert (b[left] > after.max()).all()


def test_rejects_bad_input(orc):
    ok = dict(bytes_=[1], iota=[0.5], status=[0], room=[4])

    def run(**kw):
        d = dict(ok, **kw)
        return orc.replica_admit(d["bytes_"], d["iota"], d["status"], d["room"])[0]

    assert run() == orc.OK
    assert run(room=np.zeros(0, np.uint64)) == orc.E_INPUT
    assert run(status=[3]) == orc.E_INPUT
    assert run(iota=[np.nan]) == orc.E_INPUT
    assert run(iota=[-0.5]) == orc.E_INPUT
