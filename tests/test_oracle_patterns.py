"""Pins of the oracle's row and tile patterns and their compaction (Secs. III-A, III-B)."""
import json
import os

import numpy as np
import pytest

from oracle import patterns, prng

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
EX = json.load(open(os.path.join(GOLDEN, "paper_examples.json")))


def test_kept_count_closed_form_against_brute_force():
    for n in range(0, 41):
        for period in range(1, 18):
            for offset in range(period):
                brute = sum(1 for j in range(n) if j % period == offset)
                assert patterns.row_kept_count(n, period, offset) == brute
                assert len(patterns.row_kept_list(n, period, offset)) == brute


def test_row_example_of_the_paper():
    ex = EX["row_pattern_example"]
    dp, b = ex["dp"], ex["b"]
    m = patterns.row_mask(30, dp, b - 1)
    for start in range(0, 30, ex["block"]):
        block = m[start:start + ex["block"]]
        assert int((block == 0).sum()) == ex["dropped_per_block"]
    # reading of Eq. 1: the rows it selects ((i - b) mod dp == 0, 1-based) are kept
    kept_1based = [i for i in range(1, 31) if (i - b) % dp == 0]
    assert [j + 1 for j in patterns.row_kept_list(30, dp, b - 1)] == kept_1based


def test_tile_example_of_the_paper():
    ex = EX["tile_pattern_example"]
    words = prng.tile_bitmap_tdp(4, 8, ex["dp"], ex["b"] - 1)
    bits = [(words[t // 32] >> (t % 32)) & 1 for t in range(32)]
    for start in range(0, 32, ex["block"]):
        assert ex["block"] - sum(bits[start:start + ex["block"]]) == ex["dropped_per_block"]


def test_kept_fraction_is_one_over_dp():
    for dp in EX["kept_fraction"]["dp_values"]:
        n = 16 * 9 * 5 * 7 * dp
        for off in range(dp):
            assert patterns.row_kept_count(n, dp, off) * dp == n


def test_dp_max_and_sub_model_count():
    ex = EX["dp_max_tdp"]
    assert (ex["M"] // ex["x"]) * (ex["N"] // ex["y"]) == ex["dp_max"]
    # every (dp, b) pair is a distinct sub-model: n(n+1)/2 of them for dp <= n
    for n in range(1, 20):
        pairs = {(d, o) for d in range(1, n + 1) for o in range(d)}
        masks = {tuple(patterns.row_mask(n * (n + 1), d, o)) for d, o in pairs}
        assert len(pairs) == n * (n + 1) // 2 == len(masks)


def test_edge_cases():
    assert patterns.row_kept_list(10, 1, 0) == list(range(10))
    assert patterns.row_kept_list(5, 8, 6) == []
    assert patterns.row_kept_count(5, 8, 6) == 0
    assert patterns.row_kept_list(0, 3, 1) == []
    with pytest.raises(ValueError):
        patterns.row_kept_list(10, 0, 0)
    with pytest.raises(ValueError):
        patterns.row_kept_list(10, 3, 3)


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_tile_lists_reconstruct_the_grid(seed):
    rng = np.random.default_rng(seed)
    tn, tk = int(rng.integers(1, 9)), int(rng.integers(1, 9))
    words = prng.tile_bitmap_bernoulli(tn, tk, 0.5, seed, 3, 4)
    grid = patterns.bitmap_to_grid(words, tn, tk)
    L = patterns.tile_lists(words, tn, tk)
    g1 = np.zeros_like(grid)
    for r in range(tn):
        cols = L["row_cols"][L["row_ptr"][r]:L["row_ptr"][r + 1]]
        assert cols == sorted(cols)
        g1[r, cols] = True
    g2 = np.zeros_like(grid)
    for c in range(tk):
        rows = L["col_rows"][L["col_ptr"][c]:L["col_ptr"][c + 1]]
        assert rows == sorted(rows)
        g2[rows, c] = True
    g3 = np.zeros_like(grid)
    for t in L["flat"]:
        g3[t // tk, t % tk] = True
    assert (g1 == grid).all() and (g2 == grid).all() and (g3 == grid).all()
    assert L["flat"] == sorted(L["flat"])
    assert patterns.bitmap_popcount(words, tn * tk) == int(grid.sum()) == len(L["flat"])


def test_tile_mask_expansion():
    words = prng.tile_bitmap_tdp(2, 3, 2, 1)
    M = patterns.tile_mask(words, 2, 3, 4)
    assert M.shape == (8, 12)
    for r in range(8):
        for c in range(12):
            t = (r // 4) * 3 + (c // 4)
            assert M[r, c] == (1.0 if t % 2 == 1 else 0.0)
