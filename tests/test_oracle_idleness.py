"""Pins of the oracle's Eq. 1 (Sec. 4.2) against closed forms and exact arithmetic."""
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

from golden_io import idleness_cases, round_to_f32

U = Fraction(1, 2 ** 24)  # unit roundoff of binary32


@pytest.mark.parametrize("case", idleness_cases())
def test_hand_cases(orc, case):
    r, a, exact = case
    w = np.stack([r, a], axis=1)[None]
    rc, iota = orc.idleness(w)
    assert rc == orc.OK
    assert iota[0] == round_to_f32(exact)
    assert not np.signbit(iota[0])


def test_paper_k_is_five_and_order_of_columns(orc):
    # Reasoning time only -> 0 (busiest); acting time only -> 1 (most idle).
    w = np.zeros((2, 5, 2), np.float32)
    w[0, :, 0] = 3.0
    w[1, :, 1] = 3.0
    rc, iota = orc.idleness(w)
    assert rc == 0 and iota[0] == 0.0 and iota[1] == 1.0


def test_window_uses_every_cycle(orc):
    # Changing any single cycle changes the result: no term is dropped.
    base = np.ones((1, 5, 2), np.float32)
    _, ref = orc.idleness(base)
    for j in range(5):
        for c in range(2):
            w = base.copy()
            w[0, j, c] = 3.0
            _, it = orc.idleness(w)
            assert it[0] != ref[0], (j, c)


finite = st.floats(min_value=0.0, max_value=1e6, allow_nan=False, allow_infinity=False, width=32)


@settings(max_examples=400, deadline=None)
@given(st.lists(finite, min_size=10, max_size=10))
def test_within_rounding_bound_of_exact(orc, vals):
    """binary32 result within the error bound of 5+5 additions, one addition and
    one division of the exact rational value of Eq. 1."""
    w = np.array(vals, np.float32).reshape(1, 5, 2)
    rc, iota = orc.idleness(w)
    assert rc == orc.OK
    tr = sum(Fraction(float(x)) for x in w[0, :, 0])
    ta = sum(Fraction(float(x)) for x in w[0, :, 1])
    if tr + ta == 0:
        assert iota[0] == 0.0
        return
    exact = ta / (tr + ta)
    # each total has at most 4 rounded additions, plus the denominator's and the quotient's roundings
    bound = (2 * 4 + 2 + 1) * U * exact * Fraction(11, 10) + Fraction(1, 2 ** 149)
    assert abs(Fraction(float(iota[0])) - exact) <= bound
    assert 0.0 <= iota[0] <= 1.0


@pytest.mark.parametrize("bad", [np.nan, np.inf, -np.inf, -1.0, -1e-30])
@pytest.mark.parametrize("col", [0, 1])
def test_rejects_invalid_windows(orc, bad, col):
    w = np.ones((3, 5, 2), np.float32)
    w[1, 2, col] = bad
    rc, _ = orc.idleness(w)
    assert rc == orc.E_INPUT


def test_rejects_total_overflow(orc):
    w = np.full((1, 5, 2), 3e38, np.float32)
    rc, _ = orc.idleness(w)
    assert rc == orc.E_INPUT


def test_negative_zero_is_canonical(orc):
    w = np.ones((1, 5, 2), np.float32)
    w[0, :, 1] = -0.0
    rc, iota = orc.idleness(w)
    assert rc == 0 and iota.view(np.uint32)[0] == 0


def test_keys_order_like_values_and_status_bit(orc):
    iota = np.array([0.0, 0.25, 1.0, 0.5], np.float32)
    rc, k = orc.keys(iota)
    assert rc == 0
    assert list(np.argsort(k, kind="stable")) == list(np.argsort(iota, kind="stable"))
    status = np.array([1, 0, 0, 1], np.uint8)
    rc, k2 = orc.keys(iota, status, orc.F_STATUS_KEY)
    # every Reasoning program (status 0) ranks before every Acting one (demotion order of Sec. 4.3.1)
    assert k2[status == 0].max() < k2[status == 1].min()
    # a given idleness of -0 keys like +0 (it must not rank after every positive value)
    rc, k3 = orc.keys(np.array([-0.0, 0.5], np.float32))
    assert rc == 0 and k3[0] == 0
    rc, _ = orc.keys(np.array([1.5], np.float32))
    assert rc == orc.E_INPUT
    rc, _ = orc.keys(np.array([np.nan], np.float32))
    assert rc == orc.E_INPUT
