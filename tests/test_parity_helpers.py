"""The GPU parity bars themselves (tests/parity.py), on the CPU: a check
that passed everything would make every parity test vacuous."""
import numpy as np
import pytest

from parity import rel_check, scaled_check


def test_rel_check_bar_and_count():
    o = np.array([1.0, -2.5, 3e-20, 0.0, np.nan], dtype=np.float32)
    assert rel_check(o.copy(), o, "same") == 0
    one_ulp = o.copy()
    one_ulp[0] = np.nextafter(o[0], np.float32(2))
    assert rel_check(one_ulp, o, "1 ulp") == 1              # within 1e-6, counted
    for i, bad in ((0, o[0] * (1 + 2e-6)), (3, np.float32(1e-30)), (1, np.nan)):
        g = o.copy()
        g[i] = bad
        with pytest.raises(AssertionError):
            rel_check(g, o, "outside the bar")


def test_scaled_check_bound():
    o = np.array([1.0, 2.0])
    scaled_check(o + 31 * 2.0 ** -24, o, np.ones(2), "inside")
    with pytest.raises(AssertionError):
        scaled_check(o + 33 * 2.0 ** -24, o, np.ones(2), "outside")
    scaled_check(o + np.array([0.0, 1.0]), o, np.ones(2), "masked", mask=np.array([True, False]))
