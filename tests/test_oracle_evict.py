"""Pins of the oracle's typed eviction order (Sec. 4.3.2): tier-reversed type
priority, least-recently-used within a type, minimal reclaim prefix."""
import os

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

from golden_io import GOLDEN

# the paper's type orders, written from its text: GPU evicts inactive, idle, busy;
# CPU evicts inactive, busy, idle (0 busy, 1 idle, 2 inactive)
PAPER_ORDER = {0: [2, 1, 0], 1: [2, 0, 1]}


def _fixture():
    kv = {}
    for line in open(os.path.join(GOLDEN, "evict_worked.txt")):
        if line.strip() and not line.startswith("#"):
            k, v = line.split(":")
            kv[k.strip()] = [int(x) for x in v.split()]
    return kv


@pytest.mark.parametrize("tier,name", [(0, "gpu"), (1, "cpu")])
def test_worked_example(orc, tier, name):
    kv = _fixture()
    rc, order, prefix, count = orc.evict_order(kv["type"], kv["last_access"], tier, kv["need"][0], size=kv["size"])
    assert rc == 0
    assert order.tolist() == kv[f"{name}_order"]
    assert prefix.tolist() == kv[f"{name}_prefix"]
    assert count == kv[f"{name}_count"][0]


blocks = st.lists(st.tuples(st.integers(0, 2), st.integers(0, 50), st.integers(0, 9)), min_size=0, max_size=120)


@settings(max_examples=200, deadline=None)
@given(blocks, st.integers(0, 1), st.integers(0, 400))
def test_against_python_sort_and_brute_force_count(orc, bl, tier, need):
    t = np.array([b[0] for b in bl], np.uint8)
    la = np.array([b[1] for b in bl], np.uint64)
    sz = np.array([b[2] for b in bl], np.uint32)
    rc, order, prefix, count = orc.evict_order(t, la, tier, need, size=sz, unit_bytes=3)
    assert rc == 0
    pos = {ty: PAPER_ORDER[tier].index(ty) for ty in range(3)}
    expect = sorted(range(len(bl)), key=lambda b: (pos[bl[b][0]], bl[b][1], b))
    assert order.tolist() == expect
    freed = np.cumsum([bl[b][2] * 3 for b in expect]).tolist()
    assert prefix.tolist() == freed
    # fewest evictions freeing at least `need` bytes, by trying every count
    if need == 0:
        assert count == 0
    else:
        ok = [m for m in range(1, len(bl) + 1) if freed[m - 1] >= need]
        assert count == (ok[0] if ok else len(bl))


@settings(max_examples=100, deadline=None)
@given(blocks, st.integers(0, 1))
def test_type_segments_and_lru(orc, bl, tier):
    t = np.array([b[0] for b in bl], np.uint8)
    la = np.array([b[1] for b in bl], np.uint64)
    rc, order, _, _ = orc.evict_order(t, la, tier, 0)
    pos = np.array([PAPER_ORDER[tier].index(x) for x in range(3)])
    seg = pos[t[order]] if len(bl) else np.zeros(0)
    assert (np.diff(seg) >= 0).all()  # inactive first; then idle (GPU) / busy (CPU); the tier's own type last
    for ty in range(3):
        times = la[order][t[order] == ty]
        assert (np.diff(times.astype(np.int64)) >= 0).all()  # least recently used first


def test_reversed_between_tiers(orc):
    """Same timestamps: the GPU keeps busy blocks longest, the CPU keeps idle ones longest."""
    t = np.array([0, 1, 2], np.uint8)
    la = np.zeros(3, np.uint64)
    assert orc.evict_order(t, la, 0, 0)[1].tolist() == [2, 1, 0]
    assert orc.evict_order(t, la, 1, 0)[1].tolist() == [2, 0, 1]


def test_rejects_bad_input(orc):
    assert orc.evict_order(np.array([3], np.uint8), np.zeros(1, np.uint64), 0, 0)[0] == orc.E_INPUT
    assert orc.evict_order(np.array([0], np.uint8), np.zeros(1, np.uint64), 2, 0)[0] == orc.E_INPUT
