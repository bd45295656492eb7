"""How a rank's vector is cut into per-collective segments and blocks (oracle side).

Test infrastructure only (see the package docstring).

The paper assumes a vector of m bytes that splits into n equal blocks of m/n (Sec. 2.2, Sec. 4.1)
and, on a torus, D equal parts of m/D, one per collective (Sec. 5). It never says how to round
when the element count is not divisible. Reading used throughout (it decides which block, hence
which owner and which floating-point summation tree, each element belongs to):

  * elements are grouped into granules of 64 consecutive elements; G = ceil(E / 64);
  * segment c (c = 0..D-1) holds granules [floor(c G / D), floor((c + 1) G / D));
  * inside a segment of G_c granules, block j (j = 0..n-1) holds the segment's granules
    [floor(j G_c / n), floor((j + 1) G_c / n));
  * every bound is converted to elements by multiplying by 64 and clipping at E.

Blocks may be empty. All element ranges are half-open.
"""

from __future__ import annotations

import numpy as np

GRANULE = 64


def segment_bounds(E: int, D: int) -> list:
    """[(begin, end)] element ranges of the D segments."""
    G = -(-E // GRANULE)
    out = []
    for c in range(D):
        g0 = (c * G) // D
        g1 = ((c + 1) * G) // D
        out.append((min(g0 * GRANULE, E), min(g1 * GRANULE, E)))
    return out


def block_bounds(E: int, D: int, n: int) -> list:
    """out[c][j] = (begin, end) element range of block j in segment c."""
    G = -(-E // GRANULE)
    out = []
    for c in range(D):
        g0 = (c * G) // D
        g1 = ((c + 1) * G) // D
        Gc = g1 - g0
        row = []
        for j in range(n):
            b = g0 + (j * Gc) // n
            e = g0 + ((j + 1) * Gc) // n
            row.append((min(b * GRANULE, E), min(e * GRANULE, E)))
        out.append(row)
    return out


def column_labels(E: int, D: int, n: int, cols=None) -> tuple:
    """Segment and block label of each listed column (all columns by default).

    Returns (seg, blk) int64 arrays aligned with `cols`. Used both for whole vectors and for
    column samples of large runs: every step of either variant acts column-wise inside a block,
    so a column's result depends only on its own values and its labels."""
    cols = np.arange(E, dtype=np.int64) if cols is None else np.asarray(cols, dtype=np.int64)
    if cols.size and (cols.min() < 0 or cols.max() >= E):
        raise ValueError("column index outside [0, E)")
    bounds = block_bounds(E, D, n)
    begins = np.array([b for row in bounds for (b, _) in row], dtype=np.int64)
    ends = np.array([e for row in bounds for (_, e) in row], dtype=np.int64)
    # last (segment, block) whose range starts at or before the column; empty blocks share their
    # start with the next block and are skipped by taking the right-most match
    flat = np.searchsorted(begins, cols, side="right") - 1
    if cols.size and not ((begins[flat] <= cols) & (cols < ends[flat])).all():
        raise AssertionError("partition does not cover the columns")
    return flat // n, flat % n
