"""Message-contiguous block placement: an option next to the default partition (oracle side).

Test infrastructure only (see the package docstring).

The default partition puts block j of a segment at the j-th of the segment's n granule ranges
(`partition`). The paper fixes which rank owns block j (Sec. 4.1) but not where in the vector block
j lies. This option places block j at position pos_c(j) instead: write block j's coordinates in
base 3 and take their digits in the order in which collective c's steps fix them (step t works on
dimension d at distance 3^k and so fixes digit k of coordinate j_d), most significant first.

Why: after reduce-scatter step t a rank keeps the blocks that agree with it in the digits fixed by
steps 0..t (the closed form of Sec. 4.3: j congruent to the rank modulo 3^(t+1), per dimension on
a torus). Under this placement those blocks, and therefore every message, occupy one contiguous
run of positions. The floating-point summation tree of an element depends on which block it lies
in, so results differ in fp32 bits from the default partition (not in int32).

Only power-of-three sides use it (equal or not; the option is rejected elsewhere).
"""

from __future__ import annotations

import numpy as np

from . import partition, schedule


def positions(dims) -> list:
    """pos[c][j] = position of block j in segment c (a permutation of range(n) per collective)."""
    torus = schedule.Torus(tuple(dims))
    S = torus.steps
    out = []
    for c in range(torus.D):
        steps = []
        for t in range(S):
            d, dist = schedule.step_dim_and_distance(torus, c, t)
            steps.append((d, schedule.log3_exact(dist)))
        pos = np.zeros(torus.n, dtype=np.int64)
        for j in range(torus.n):
            xs = torus.coords(j)
            p = 0
            for d, k in steps:
                p = 3 * p + (xs[d] // 3 ** k) % 3
            pos[j] = p
        out.append(pos)
    return out


def column_labels(E: int, dims, cols=None) -> tuple:
    """(seg, blk) of each listed column under this placement: the column's position in the
    default granule partition, mapped to the block placed there."""
    torus = schedule.Torus(tuple(dims))
    seg, place = partition.column_labels(E, torus.D, torus.n, cols)
    block_at = np.stack([np.argsort(p) for p in positions(dims)])  # [c][position] -> block
    return seg, block_at[seg, place] if seg.size else place
