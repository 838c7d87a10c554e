"""Host-side bookkeeping of the caller runtime: the first-fit extent allocator
of the CPU tier's arena, against a byte map of the same arena."""
import numpy as np

from paper_2606_00866_amd.tiering import FirstFit


def _check(ff, cap):
    """Free extents are sorted, disjoint, maximal (no two adjacent), and with the
    used extents they tile the arena exactly."""
    owner = np.zeros(cap // ff.align, np.int8)
    for s, n in ff.free:
        assert s % ff.align == 0 and n > 0 and n % ff.align == 0
        assert (owner[s // ff.align:(s + n) // ff.align] == 0).all()
        owner[s // ff.align:(s + n) // ff.align] = 1
    for (a, m), (b, _) in zip(ff.free, ff.free[1:]):
        assert a + m < b  # sorted, and never adjacent (would have been merged)
    for s, n in ff.used.items():
        assert (owner[s // ff.align:(s + n) // ff.align] == 0).all()
        owner[s // ff.align:(s + n) // ff.align] = 2
    assert (owner != 0).all()


def test_first_fit_random_sequence():
    rng = np.random.default_rng(11)
    cap, align = 1 << 20, 64
    ff = FirstFit(cap, align)
    live = []
    for it in range(3000):
        if live and (rng.random() < 0.45 or len(live) > 200):
            ff.release(live.pop(int(rng.integers(len(live)))))
        else:
            size = int(rng.integers(1, 20000))
            need = -(-size // align) * align
            first = next((s for s, n in ff.free if n >= need), None)  # the lowest extent that holds it
            off = ff.alloc(size)
            assert off == first
            if off is not None:
                assert ff.used[off] == need
                live.append(off)
        if it % 50 == 0:
            _check(ff, cap)
    for off in live:
        ff.release(off)
    assert ff.free == [(0, cap)] and ff.bytes_used == 0


def test_first_fit_merges_both_sides():
    ff = FirstFit(4096 * 4, 4096)
    a, b, c, d = (ff.alloc(4096) for _ in range(4))
    assert (a, b, c, d) == (0, 4096, 8192, 12288) and ff.free == []
    ff.release(a)
    ff.release(c)
    assert ff.free == [(0, 4096), (8192, 4096)]
    ff.release(b)  # joins both neighbours
    assert ff.free == [(0, 12288)]
    assert ff.alloc(8192) == 0 and ff.free == [(8192, 4096)]
