"""Pins of the oracle's relative ranking (Sec. 1, Sec. 4.3): ascending idleness,
busiest first, ties by program id."""
import numpy as np
from hypothesis import given, settings
from hypothesis import strategies as st

keys_strategy = st.lists(st.integers(min_value=0, max_value=2 ** 32 - 1), min_size=0, max_size=300)
small_keys = st.lists(st.integers(min_value=0, max_value=7), min_size=0, max_size=60)


@settings(max_examples=200, deadline=None)
@given(st.one_of(keys_strategy, small_keys))
def test_order_equals_python_sort_of_pairs(orc, keys):
    k = np.array(keys, np.uint32)
    order, rank = orc.order(k)
    expect = [p for _, p in sorted((int(k[p]), p) for p in range(k.size))]
    assert order.tolist() == expect
    assert (rank[order] == np.arange(k.size)).all()


@settings(max_examples=100, deadline=None)
@given(small_keys)
def test_rank_by_counting(orc, keys):
    """rank[p] = number of programs strictly before p in (key, id) order (brute force)."""
    k = np.array(keys, np.int64)
    _, rank = orc.order(k.astype(np.uint32))
    for p in range(k.size):
        before = int(((k < k[p]) | ((k == k[p]) & (np.arange(k.size) < p))).sum())
        assert rank[p] == before


@settings(max_examples=100, deadline=None)
@given(st.lists(st.floats(min_value=0.0, max_value=1.0, width=32), min_size=1, max_size=80))
def test_monotone_transform_keeps_order(orc, vals):
    """Ranking depends only on the relative order of idleness (it is relative)."""
    iota = np.array(vals, np.float32)
    _, k1 = orc.keys(iota)
    o1, _ = orc.order(k1)
    squashed = (iota.astype(np.float64) ** 3 * 0.5).astype(np.float32)  # strictly monotone on [0,1] ...
    # ... but binary32 rounding may merge neighbours; only compare when it stays injective on distinct values
    if len(np.unique(squashed)) == len(np.unique(iota)):
        _, k2 = orc.keys(squashed)
        o2, _ = orc.order(k2)
        assert o1.tolist() == o2.tolist()


def test_busiest_first_from_windows(orc):
    rng = np.random.default_rng(7)
    w = rng.random((50, 5, 2)).astype(np.float32)
    w[13, :, 1] = 0.0  # never in a tool call: idleness 0, busiest
    w[31, :, 0] = 0.0  # never reasoning: idleness 1, most idle
    rc, iota = orc.idleness(w)
    assert rc == 0
    _, key = orc.keys(iota)
    order, _ = orc.order(key)
    assert order[0] == 13 and order[-1] == 31
    assert np.all(np.diff(iota[order]) >= 0)


def test_relabeling_permutes_order(orc):
    rng = np.random.default_rng(3)
    key = rng.permutation(100).astype(np.uint32)  # distinct keys
    order, _ = orc.order(key)
    perm = rng.permutation(100)
    key2 = key[perm]  # program j of the relabeled set is program perm[j]
    order2, _ = orc.order(key2)
    inv = np.argsort(perm)
    assert (perm[order2] == order).all()
    assert (inv[order] == order2).all()
