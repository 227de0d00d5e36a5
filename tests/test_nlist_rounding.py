"""The neighbour-list kernel takes rint(d / box) of the minimum image from
d * (1 / box) when that product lies more than 1e-6 from a half-integer and
|d / box| < 2^20, and from the division otherwise.  The claim that both
give the same integer on the fast path is checked here in float64 on
differences spread over +-5 boxes and on differences at and one unit in the
last place beside half-integer quotients."""
import numpy as np
import pytest


@pytest.mark.parametrize("box", [20.0, 232.576, 14.536, 3.0000000001, 81.0, 1e-3, 7.3e4])
def test_fast_quotient_rounds_like_the_division(box):
    rng = np.random.default_rng(int(box * 1000) % 2**32)
    half = (rng.integers(-9, 9, 20000) + 0.5) * box
    d = np.concatenate([rng.uniform(-5 * box, 5 * box, 200000), half,
                        np.nextafter(half, np.inf), np.nextafter(half, -np.inf),
                        rng.uniform(-1e5, 1e5, 20000) * box])
    q = d * (1.0 / box)
    n = np.rint(q)
    fast = (np.abs(q - n) < 0.499999) & (np.abs(q) < 1048576.0)
    assert fast.mean() > 0.5
    np.testing.assert_array_equal(n[fast], np.rint(d[fast] / box))
    # and the minimum image itself, computed both ways
    np.testing.assert_array_equal(d[fast] - box * n[fast], d[fast] - box * np.rint(d[fast] / box))
