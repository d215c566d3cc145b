"""Row-based and tile-based dropout patterns as masks and gather lists.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Row-based dropout pattern (Sec. III-A, Eq. 1). The pattern is (dp, b) with
b in {1..dp}. Eq. 1 selects the rows with (i - b) mod dp == 0; the text then
says (dp-1)/dp of the rows are dropped and only 1/dp of the weight matrix is
fetched, so the rows Eq. 1 selects are read as the KEPT ones. In 0-based terms
with period = dp and offset = b - 1: neuron j is kept iff j mod period == offset.

Tile-based dropout pattern (Sec. III-B): the same rule over the row-major tile
index of the weight matrix W[N][K], or an arbitrary kept-tile bitmap.
"""

import numpy as np


def row_kept_list(n, period, offset):
    """Ascending kept indices in [0, n): j with j mod period == offset."""
    if period < 1 or not (0 <= offset < period):
        raise ValueError("need period >= 1 and 0 <= offset < period")
    return [j for j in range(n) if j % period == offset]


def row_kept_count(n, period, offset):
    """Number of kept rows: 0 if offset >= n, else ceil((n - offset) / period)."""
    if offset >= n:
        return 0
    return (n - offset + period - 1) // period


def row_mask(n, period, offset):
    """fp64 0/1 mask of length n, 1 at kept neurons."""
    m = np.zeros(n, dtype=np.float64)
    for j in row_kept_list(n, period, offset):
        m[j] = 1.0
    return m


def bitmap_to_grid(words, tiles_n, tiles_k):
    """Bitmap words -> bool array [tiles_n][tiles_k] (True = kept)."""
    grid = np.zeros((tiles_n, tiles_k), dtype=bool)
    for t in range(tiles_n * tiles_k):
        if (words[t // 32] >> (t % 32)) & 1:
            grid[t // tiles_k, t % tiles_k] = True
    return grid


def tile_mask(words, tiles_n, tiles_k, tile):
    """Element mask of W[N][K]: the tile grid expanded to tile x tile blocks."""
    grid = bitmap_to_grid(words, tiles_n, tiles_k).astype(np.float64)
    return np.kron(grid, np.ones((tile, tile), dtype=np.float64))


def tile_lists(words, tiles_n, tiles_k):
    """The compaction of a kept-tile bitmap into gather lists.

    Returns a dict of int lists:
      row_ptr[tiles_n + 1], row_cols[nnz]  - kept tile columns of each tile row
      col_ptr[tiles_k + 1], col_rows[nnz]  - kept tile rows of each tile column
      flat[nnz]                            - kept linear tile indices t
    Every list is ascending within its segment.
    """
    grid = bitmap_to_grid(words, tiles_n, tiles_k)
    row_ptr, row_cols = [0], []
    for tn in range(tiles_n):
        for tk in range(tiles_k):
            if grid[tn, tk]:
                row_cols.append(tk)
        row_ptr.append(len(row_cols))
    col_ptr, col_rows = [0], []
    for tk in range(tiles_k):
        for tn in range(tiles_n):
            if grid[tn, tk]:
                col_rows.append(tn)
        col_ptr.append(len(col_rows))
    flat = [t for t in range(tiles_n * tiles_k) if grid[t // tiles_k, t % tiles_k]]
    return {"row_ptr": row_ptr, "row_cols": row_cols,
            "col_ptr": col_ptr, "col_rows": col_rows, "flat": flat}


def bitmap_popcount(words, total):
    """Number of kept tiles among the first ``total`` bits."""
    return sum((words[t // 32] >> (t % 32)) & 1 for t in range(total))
