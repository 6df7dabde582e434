"""The mask comparator itself (CPU only): it must accept exactly the rows the
selection rule allows to differ (near-ties in the order, a top-p stopping test
on the boundary) and reject every other difference, including a wrong block
taken at the boundary and a count the floor fixed."""

import math

import numpy as np

from tests.compare import compare_row


def ln(*m):
    return np.log(np.array(m, dtype=np.float64))


def test_identical_rows_are_exact():
    s = ln(0.5, 0.3, 0.15, 0.05)
    assert compare_row([0, 1], [0, 1], s, 0.8, 0.0) == "exact"


def test_extra_boundary_block_must_be_the_next_in_order():
    # masses 0.5, 0.3, 0.15, 0.05; top_p on the cumulative 0.8 after two
    # blocks, so one more block is excusable -- but only block 2, the next in
    # the order, not the lowest-mass block 3
    s = ln(0.5, 0.3, 0.15, 0.05)
    top_p = float(np.cumsum(np.exp(s) / np.exp(s).sum())[1])
    assert compare_row([0, 1, 2], [0, 1], s, top_p, 0.0) == "excused"
    res = compare_row([0, 1, 3], [0, 1], s, top_p, 0.0)
    assert res not in ("exact", "excused"), res


def test_missing_boundary_block_must_be_the_last_in_order():
    s = ln(0.5, 0.3, 0.15, 0.05)
    top_p = float(np.cumsum(np.exp(s) / np.exp(s).sum())[1])
    # oracle keeps {0, 1, 2} when its cumulative lands just below top_p
    assert compare_row([0, 1], [0, 1, 2], s, top_p + 1e-9, 0.0) == "excused"
    res = compare_row([0, 2], [0, 1, 2], s, top_p + 1e-9, 0.0)
    assert res not in ("exact", "excused"), res


def test_count_difference_away_from_the_boundary_fails():
    s = ln(0.5, 0.3, 0.15, 0.05)
    res = compare_row([0, 1, 2], [0, 1], s, 0.7, 0.0)
    assert res not in ("exact", "excused"), res


def test_count_fixed_by_the_floor_is_never_excused():
    # floor ceil(0.75 * 4) = 3 blocks; the top-p count (1) is below it, so
    # the count is the floor's and may not differ, even if the mass after
    # two blocks sits exactly on top_p
    s = ln(0.5, 0.3, 0.15, 0.05)
    top_p = float(np.cumsum(np.exp(s) / np.exp(s).sum())[1])
    res = compare_row([0, 1], [0, 1, 2], s, top_p, 0.75)
    assert res not in ("exact", "excused"), res
    # with the floor at 2 blocks the same pair of rows is a boundary case
    assert compare_row([0, 1, 2], [0, 1], s, top_p, 0.5) == "excused"


def test_near_tie_swap_is_excused_and_a_real_swap_is_not():
    s = ln(0.4, 0.2, 0.2 * (1 + 1e-9), 0.2 * (1 - 1e-9))
    # oracle order 0, 2, 1, 3; keeping 1 instead of 2 is a near-tie
    assert compare_row([0, 1], [0, 2], s, 0.0, 0.5) == "excused"
    s2 = ln(0.4, 0.25, 0.2, 0.15)
    res = compare_row([0, 2], [0, 1], s2, 0.0, 0.5)
    assert res not in ("exact", "excused"), res


def test_custom_tie_and_boundary_tolerances():
    s = ln(0.4, 0.3, 0.3001, 1e-4)
    loose = lambda a, b: abs(math.exp(a) - math.exp(b)) <= 1e-3
    assert compare_row([0, 1], [0, 2], s, 0.0, 0.5, tie=loose) == "excused"
    assert compare_row([0, 1], [0, 2], s, 0.0, 0.5) not in ("exact", "excused")


def test_malformed_rows_fail():
    s = ln(0.5, 0.3, 0.15, 0.05)
    assert compare_row([1, 0], [0, 1], s, 0.8, 0.0) == "gpu row not strictly ascending"
    assert compare_row([0, 0], [0, 1], s, 0.8, 0.0) == "gpu row not strictly ascending"
    assert compare_row([0, 1, 2, 3], [0, 1], s, 0.8, 0.0).startswith("count")
