"""Latency-optimal Trivance on rings and tori whose sides are not all powers of three (oracle side,
Sec. 4.2 with Sec. 4.4).

Test infrastructure only (see the package docstring).

What the paper fixes: the steps (Sec. 4.4: distances 3^0 .. 3^(f-1), then d = ceil((n - 3^f) / 2)
on a side of n with 3^f < n < 3^(f+1)); in the latency-optimal variant every rank sends what it
has accumulated to both peers and reduces both messages with its own partial (Sec. 4.2, 4.3); in
the final step a rank obtains only the contributions it is still missing (Sec. 4.4). The paper
does not say how a rank forwards "only the missing ones" once its partial has merged them with
others; this module is the reading used here.

Reading. A rank holds partial sums, each over a set of sources given by offsets relative to the
rank (the same sets at every rank, by symmetry):
  * the window: after the k-th full step along a dimension it covers the offsets |o| <= R_k =
    (3^(k+1) - 1) / 2 along it, as in Lemma 2;
  * in the final step along a dimension a rank combines its window (|o| <= R, R = R_(f-1)) with
    the sources beyond it: those at offsets R+1 .. R+d come from the peer at +d (they are the top d
    of that peer's window) and those at -R-b .. -R-1, b = n - 3^f - d, from the peer at -d (offsets
    taken in (-n/2, n/2], so an odd remainder gives the + side the extra source, as in the
    bandwidth-optimal trees);
  * every other partial a rank needs is the one its peers must send it later, worked out backwards
    from the final result: a partial over a set S, formed in a full step at distance 3^k, takes
    the part of S inside the left peer's previous window from the left peer, the part inside its
    own previous window from itself and the part inside the right peer's from the right peer
    (three disjoint windows that tile the new one, Appendix A); parts that are whole windows are
    the windows themselves, the others are partials the peers keep for that purpose.
  * Every partial is formed as (own + from_left) + from_right with absent parts skipped (the joint
    reduction of Sec. 4.3). Steps along other dimensions extend each partial along those
    dimensions in the same way, so each partial is a box of offsets.
On sides that are powers of three the window is the only partial and this is the ordinary
latency-optimal schedule. A rank sends in each step the window plus the partials its peers need,
so some messages carry more than one vector (the cost model counts them).
"""

from __future__ import annotations

import numpy as np

from . import nonpow3


def _ring_offsets(side: int) -> list:
    lo = -((side - 1) // 2)
    return list(range(lo, lo + side))


def _canon(side: int, o: int) -> int:
    lo = -((side - 1) // 2)
    return (o - lo) % side + lo


class _Dim:
    """The step structure of one side (Sec. 4.4): distances, and the window of offsets after each
    number of steps taken along it."""

    def __init__(self, side: int):
        self.side = side
        self.dist = nonpow3.distances(side) if side > 1 else []
        self.f = nonpow3.levels(side)[0] if side > 1 else 0  # full steps; a final one follows
                                                              # when the side is not 3^f

    def window(self, taken: int) -> frozenset:
        """Offsets (canonical) covered after `taken` steps along this dimension."""
        if self.side == 1:
            return frozenset([0])
        if taken > self.f:  # after the final step: the whole ring
            return frozenset(_ring_offsets(self.side))
        R = (3 ** taken - 1) // 2
        return frozenset(_canon(self.side, o) for o in range(-R, R + 1))


def _box_window(dims_info, taken):
    return tuple(dims_info[d].window(taken[d]) for d in range(len(dims_info)))


def _shift(side, offs, delta):
    return frozenset(_canon(side, o + delta) for o in offs)


def program(dims, c: int = 0) -> list:
    """The partials of collective c, pass by pass.

    Returns a list `states` of length S + 1: states[t] is the list of boxes (tuples of frozensets of
    offsets, one per dimension) a rank holds before pass t (states[0] = [the rank's own value]),
    and `recipes[t][i]` (in the second returned list) gives, for box i of states[t + 1], the
    indices (own, left, right) into states[t] of its parts (None when absent)."""
    dims = tuple(int(x) for x in dims)
    D = len(dims)
    info = [_Dim(s) for s in dims]
    rot = nonpow3.torus_rotation(dims, c)
    S = len(rot)
    taken = [[0] * D]
    for (dim, _) in rot:
        nxt = list(taken[-1])
        nxt[dim] += 1
        taken.append(nxt)
    full = _box_window(info, taken[S])
    needed = [None] * (S + 1)
    needed[S] = [full]
    recipes = [None] * S
    for t in reversed(range(S)):
        dim, k = rot[t]
        side = dims[dim]
        dist = info[dim].dist[k]
        prev_win = info[dim].window(taken[t][dim])
        cur_win = info[dim].window(taken[t + 1][dim])
        final = k == info[dim].f  # the Sec. 4.4 final step of this dimension
        parts_all = []
        order = []
        for box in needed[t + 1]:
            I = box[dim]
            assert I <= cur_win, "a partial outside the window"
            if final:
                assert I == cur_win, "after the final step only whole rings are needed"
                R = max(prev_win)
                own = prev_win
                right = frozenset(o for o in cur_win if o > R)        # from the peer at +d
                left = frozenset(o for o in cur_win if o < -R)        # from the peer at -d
            else:
                # three disjoint windows tile the new one (Appendix A)
                lw = _shift(side, prev_win, -dist)
                rw = _shift(side, prev_win, +dist)
                assert not (lw & prev_win) and not (rw & prev_win) and not (lw & rw)
                assert lw | prev_win | rw == cur_win
                own, left, right = I & prev_win, I & lw, I & rw
            assert own | left | right == I and not (own & left) and not (own & right) \
                and not (left & right)
            pieces = []
            for part, delta in ((own, 0), (left, +dist), (right, -dist)):
                if not part:
                    pieces.append(None)
                    continue
                # in the sender's frame: offset o from x is o + dist from x - dist
                pbox = tuple(_shift(side, part, delta) if d == dim else box[d] for d in range(D))
                pwin = info[dim].window(taken[t][dim])
                assert pbox[dim] <= pwin, "a part the sender cannot hold"
                pieces.append(pbox)
            order.append(pieces)
            for pb in pieces:
                if pb is not None and pb not in parts_all:
                    parts_all.append(pb)
        # keep the window first
        win_t = _box_window(info, taken[t])
        parts_all.sort(key=lambda b: (b != win_t,))
        needed[t] = parts_all
        recipes[t] = [tuple(None if pb is None else parts_all.index(pb) for pb in pieces)
                      for pieces in order]
    start = tuple(frozenset([0]) for _ in range(D))
    assert needed[0] == [start], "the first pass must start from the rank's own value"
    return needed, recipes


def latency_optimal(V: np.ndarray, dims, col_seg=None, trace=None) -> np.ndarray:
    """Run the latency-optimal schedule on (n, E) inputs V; every rank ends with the reduction of
    all ranks' values over its segment's columns.

    col_seg   segment (collective) of every column (default: the partition rule).
    trace     optional list; receives, per pass, {box: (n, cols) array} of every collective."""
    from . import partition

    dims = tuple(int(x) for x in dims)
    D = len(dims)
    n, E = V.shape
    if col_seg is None:
        col_seg, _ = partition.column_labels(E, D, n)
    col_seg = np.asarray(col_seg)
    coords = np.array([nonpow3._coords(dims, r) for r in range(n)], dtype=np.int64)
    strides = np.cumprod((1,) + dims[:-1])

    def peer(dim, delta):
        Y = coords.copy()
        Y[:, dim] = (Y[:, dim] + delta) % dims[dim]
        return (Y * strides).sum(axis=1)

    out = V.copy()
    for c in range(D):
        cols = np.nonzero(col_seg == c)[0]
        needed, recipes = program(dims, c)
        rot = nonpow3.torus_rotation(dims, c)
        state = [V[:, cols].copy()]
        for t, (dim, k) in enumerate(rot):
            dist = nonpow3.distances(dims[dim])[k]
            L, R = peer(dim, -dist), peer(dim, +dist)
            new = []
            for own_i, left_i, right_i in recipes[t]:
                # joint reduction (Sec. 4.3): (own + from_left) + from_right, absent parts skipped
                acc = None
                for idx, rows in ((own_i, None), (left_i, L), (right_i, R)):
                    if idx is None:
                        continue
                    val = state[idx] if rows is None else state[idx][rows]
                    acc = val.copy() if acc is None else np.add(acc, val, dtype=val.dtype)
                new.append(acc)
            state = new
            if trace is not None:
                trace.append((c, t, dict(zip(needed[t + 1], state))))
        assert len(state) == 1
        out[:, cols] = state[0]
    return out


def message_slots(dims, c: int = 0) -> list:
    """Per pass of collective c: (partials sent towards +, partials sent towards -) by every rank:
    the distinct parts its +d peer takes from its left and its -d peer takes from its right."""
    _, recipes = program(dims, c)
    out = []
    for rec in recipes:
        lefts = {r[1] for r in rec if r[1] is not None}
        rights = {r[2] for r in rec if r[2] is not None}
        out.append((len(lefts), len(rights)))
    return out
