"""The weight-gradient group checker accepts a valid grouping and rejects
each kind of mistake a plan kernel could make (CPU only)."""
import copy

import pytest

from plan_invariants import check_weight_grad_groups

# tile rows with 0, 5, 4 and 1 kept tiles
ROW_PTR = [0, 0, 5, 9, 10]
ROW_COLS = [0, 2, 3, 5, 7, 1, 2, 3, 4, 6]
GOOD = [4, 0, 0, 0,
        1, 0, 4, 0, 0, 2, 3, 5,
        1, 4, 1, 0, 7, 7, 7, 7,
        2, 5, 4, 0, 1, 2, 3, 4,
        3, 9, 1, 0, 6, 6, 6, 6]


def test_valid_groupings_pass():
    check_weight_grad_groups(GOOD, ROW_PTR, ROW_COLS)
    check_weight_grad_groups([0, 0, 0, 0], [0, 0, 0], [])
    # other valid splits of the same rows: a short group first, single tiles
    alt = [4, 0, 0, 0,
           1, 0, 2, 0, 0, 2, 2, 2,
           1, 2, 3, 0, 3, 5, 7, 7,
           2, 5, 4, 0, 1, 2, 3, 4,
           3, 9, 1, 0, 6, 6, 6, 6]
    check_weight_grad_groups(alt, ROW_PTR, ROW_COLS)


def mutated(edit):
    r = copy.deepcopy(GOOD)
    edit(r)
    return r


@pytest.mark.parametrize("edit", [
    lambda r: r.__setitem__(1, 1),                          # header
    lambda r: r.__setitem__(0, 3),                          # count does not match the records
    lambda r: r.__setitem__(4 + 8 + 7, 6),                  # padding differs from the last column
    lambda r: r.__setitem__(4 + 9, 6),                      # a column that is not the CSR's
    lambda r: r.__setitem__(4 + 2, 5),                      # more than 4 tiles
    lambda r: r.__setitem__(4 + 8 + 2, 0),                  # empty group
    lambda r: r.__setitem__(4 + 8 + 1, 3),                  # a tile twice, another missing
    lambda r: r.__setitem__(4 + 16, 1),                     # group outside its tile row
    lambda r: r.__setitem__(4 + 3, 2),                      # reserved entry
    lambda r: r.__setitem__(slice(4, 20), r[12:20] + r[4:12]),  # out of row order
])
def test_planted_mistakes_fail(edit):
    with pytest.raises(AssertionError):
        check_weight_grad_groups(mutated(edit), ROW_PTR, ROW_COLS)


def test_missing_group_fails():
    short = GOOD[:4] + GOOD[12:]
    short[0] = 3
    with pytest.raises(AssertionError):
        check_weight_grad_groups(short, ROW_PTR, ROW_COLS)
