"""Checks of the tile plan's weight-gradient work records by their properties.

The plan kernel also writes work records for the tile weight-gradient kernel:
groups of up to four kept tiles of one tile row. Their layout is the kernel's
own schedule, not something the paper defines (Sec. III-B defines only the
kept tiles and their compact matrices), so the oracle has no copy of it.
Instead the device's records are checked against the oracle's CSR lists: every
kept tile appears exactly once, each group holds 1 to 4 tiles of one tile row
at consecutive CSR positions, the groups come in row order, and the padding
repeats the group's last column.

Record layout: a 4-int header [count, 0, 0, 0], then per group 8 ints:
tile row, first position in row_cols, tile count n, 0, the n tile columns and
the last of them repeated up to 4 entries.
"""

GROUP = 4
REC = 4 + GROUP


def check_weight_grad_groups(recs, row_ptr, row_cols):
    """Raises AssertionError unless recs (a flat int list, header included)
    is a valid grouping of the kept tiles given by the CSR lists."""
    assert len(recs) >= 4, "record array shorter than its header"
    count = recs[0]
    assert count >= 0 and recs[1:4] == [0, 0, 0], f"bad header {recs[:4]}"
    assert len(recs) == 4 + REC * count, f"{len(recs)} ints for {count} groups"
    tiles_n = len(row_ptr) - 1
    covered = [0] * len(row_cols)
    prev = (-1, -1)
    for g in range(count):
        r, first, n, zero, *cols = recs[4 + REC * g: 4 + REC * (g + 1)]
        assert zero == 0, f"group {g}: reserved entry {zero}"
        assert 0 <= r < tiles_n, f"group {g}: tile row {r}"
        assert 1 <= n <= GROUP, f"group {g}: {n} tiles"
        assert row_ptr[r] <= first and first + n <= row_ptr[r + 1], f"group {g}: positions outside row {r}"
        assert (r, first) > prev, f"group {g}: not in row order"
        prev = (r, first)
        for j in range(n):
            assert cols[j] == row_cols[first + j], f"group {g}: column {j} is {cols[j]}"
            covered[first + j] += 1
        for j in range(n, GROUP):
            assert cols[j] == cols[n - 1], f"group {g}: padding {j} is {cols[j]}"
    missing = [i for i, c in enumerate(covered) if c != 1]
    assert not missing, f"kept tiles covered {[covered[i] for i in missing[:4]]} times at positions {missing[:4]}"
