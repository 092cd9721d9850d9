"""The refresh-set rule the GPU parity tests apply (CPU only).

``tests.gpu_util.check_refresh_set`` accepts a GPU refresh set when it equals
the oracle's top-k (boundary gap above the tolerance) or, with a gap within
the tolerance, when it is valid on both sides of the k-th score.  These cases
feed it hand-made sets, so that a checker too lenient to notice a wrong
selection fails here first.
"""
import numpy as np
import pytest

from tests.gpu_util import check_refresh_set

TOL = 2e-2


def _near_uniform(n=40, seed=3):
    # attention mass as random weights give it: near-uniform, tiny gaps
    rng = np.random.default_rng(seed)
    return 1.0 + 1e-4 * rng.standard_normal(n)


def test_ambiguous_boundary_accepts_any_tolerance_valid_set():
    s = _near_uniform()
    excl = [0, 1, 2]
    k = 5
    order = sorted(set(range(40)) - set(excl), key=lambda j: -s[j])
    assert check_refresh_set(sorted(order[:k]), s, excl, k, TOL) == "ambiguous"
    # a different but valid choice inside the tolerance band
    assert check_refresh_set(sorted(order[3:3 + k]), s, excl, k, TOL) == "ambiguous"


def test_dropping_a_clear_winner_is_caught_even_at_an_ambiguous_boundary():
    s = _near_uniform()
    s[17] = 1.5                      # clearly above every other candidate
    excl = [0, 1, 2]
    k = 5
    order = sorted(set(range(40)) - set(excl), key=lambda j: -s[j])
    assert order[0] == 17
    good = sorted(order[:k])
    assert check_refresh_set(good, s, excl, k, TOL) == "ambiguous"
    bad = sorted(order[1:k + 1])     # the top-1 token left out
    with pytest.raises(AssertionError, match="clearly past"):
        check_refresh_set(bad, s, excl, k, TOL)


def test_lowest_first_mirror():
    s = _near_uniform()
    s[9] = 0.5                       # clearly the lowest candidate
    excl = [0, 1]
    k = 4
    order = sorted(set(range(40)) - set(excl), key=lambda j: s[j])
    assert check_refresh_set(sorted(order[:k]), s, excl, k, TOL, lowest=True) == "ambiguous"
    with pytest.raises(AssertionError, match="clearly past"):
        check_refresh_set(sorted(order[1:k + 1]), s, excl, k, TOL, lowest=True)


def test_gap_above_tolerance_requires_the_exact_set():
    s = np.linspace(1.0, 2.0, 30)
    s[[4, 8, 15]] = 10.0
    excl = [29]
    assert check_refresh_set([4, 8, 15], s, excl, 3, TOL) == "exact"
    with pytest.raises(AssertionError, match="differs"):
        check_refresh_set([4, 8, 28], s, excl, 3, TOL)


@pytest.mark.parametrize("bad", [[3, 3, 4], [0, 5, 6], [5, 6]])
def test_invalid_sets(bad):
    s = _near_uniform(12)
    with pytest.raises(AssertionError):
        check_refresh_set(bad, s, [0], 3, TOL)
