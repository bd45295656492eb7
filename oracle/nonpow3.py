"""Trivance on rings and tori whose sides are not all powers of three (oracle side, Sec. 4.4).

Test infrastructure only (see the package docstring).

What the paper fixes (Sec. 4.4, figure fig:trivanceNonPowerThree):
  * for 3^f < n < 3^(f+1) the first f steps are the usual ones (distances 3^0 .. 3^(f-1)) and one
    final step at distance d = ceil((n - 3^f) / 2) follows: ceil(log3 n) steps in total;
  * the final step is uniform, its congestion equals d;
  * every block is forwarded at most once per phase, so a rank sends at most m per phase;
  * n = 7: two blocks per direction in the first step, one in the final step.
The paper describes this for the bandwidth-optimal variant (blocks forwarded by Algorithm 1); it
does not say how the latency-optimal variant, which forwards whole pre-reduced vectors, would avoid
counting the final step's overlap twice, so only the bandwidth-optimal variant is modelled.

Reading (the paper gives no construction). For a block j, offsets are taken in (-n/2, n/2].
  * Three reduction trees of the ordinary Trivance pattern are used: rooted at j (window
    |offset| <= R, R = (3^f - 1) / 2), at j + d and at j - d; a rank's path inside a tree moves by
    the balanced-ternary digits of its offset from the root, lowest digit first, and the roots
    j + d and j - d deliver to j in the final step.
  * Ranks outside j's window start in the tree on their side (+ for offsets > R, - for < -R;
    with n - 3^f odd the + side gets the extra rank).
  * Closure, repeated until nothing changes: every rank on the path of a member of the + (or -)
    tree joins that tree; a member of j's tree whose path passes a rank of another tree joins
    that tree instead (it must lie in that tree's window).
  This makes every block a single tree: each rank forwards each block exactly once.
  * A rank combines what arrives for a block as (own + from_left) + from_right, absent terms
    skipped; the all-gather retraces each tree edge backwards (reverse step order).
On a torus every side gets its own tree of this kind (the ordinary one for a power of three); see
the section on tori below.
"""

from __future__ import annotations

from functools import lru_cache
from itertools import product

import numpy as np


def levels(n: int) -> tuple:
    """(f, d): number of full steps and the final distance; d = 0 when n is a power of three."""
    if n < 2:
        raise ValueError("need at least two ranks")
    f, p = 0, 1
    while p * 3 <= n:
        p *= 3
        f += 1
    if p == n:
        return f, 0
    return f, -(-(n - p) // 2)


def is_tree(dims) -> bool:
    """True if some side is not a power of three (the schedules of this module apply)."""
    return any(int(s) >= 2 and levels(int(s))[1] != 0 for s in dims)


def distances(n: int) -> list:
    """Peer distance of every step (Sec. 4.4)."""
    f, d = levels(n)
    return [3 ** k for k in range(f)] + ([d] if d else [])


def offsets(n: int) -> list:
    """Ring offsets in (-n/2, n/2]."""
    lo = -((n - 1) // 2)
    return list(range(lo, lo + n))


def canon(n: int, o: int) -> int:
    lo = -((n - 1) // 2)
    return (o - lo) % n + lo


@lru_cache(maxsize=None)
def _digits_to(f: int, value: int):
    """Digits (e_0..e_{f-1}) in {-1,0,1} with sum e_i 3^i == value, by exhaustive search."""
    hits = [e for e in product((-1, 0, 1), repeat=f) if sum(x * 3 ** i for i, x in enumerate(e)) == value]
    return hits[0] if len(hits) == 1 else None


def _tree_path(n: int, o: int, side: int):
    """Positions (offsets) visited in the first f steps by a rank at offset o inside the tree
    rooted at side * d, or None if o is outside that tree's window (any representative)."""
    f, d = levels(n)
    root = side * d
    for rep in (o, o + n, o - n):
        e = _digits_to(f, rep - root)
        if e is not None:
            pos = [rep]
            for i, x in enumerate(e):
                pos.append(pos[-1] - x * 3 ** i)
            return [canon(n, p) for p in pos], e
    return None


@lru_cache(maxsize=None)
def families(n: int) -> dict:
    """Offset -> tree (0: rooted at j, +1: at j + d, -1: at j - d), by the closure above."""
    f, d = levels(n)
    R = (3 ** f - 1) // 2
    fam = {o: (0 if abs(o) <= R else (1 if o > R else -1)) for o in offsets(n)}
    while True:
        changed = False
        for o in offsets(n):
            tp = _tree_path(n, o, fam[o])
            if tp is None:
                raise AssertionError(f"offset {o} is outside its tree on a ring of {n}")
            path, _ = tp
            for q in path[1:]:
                if fam[o] != 0 and fam[q] != fam[o]:
                    if fam[q] != 0 or q == 0:
                        raise AssertionError("trees collide")
                    fam[q] = fam[o]
                    changed = True
                if fam[o] == 0 and fam[q] != 0:
                    fam[o] = fam[q]
                    changed = True
                    break
        if not changed:
            return fam


@lru_cache(maxsize=None)
def path_digits(n: int, u: int, j: int) -> tuple:
    """Digits (e_0, ..., e_{S-1}) of the path of u's contribution to block j: the digits of its
    tree, then the final-step digit (+1: delivered from j + d, -1: from j - d, 0: already at j).
    For n a power of three this is the balanced-ternary path of the ordinary schedule."""
    f, d = levels(n)
    o = canon(n, u - j)
    if d == 0:
        return tuple(_tree_path(n, o, 0)[1])
    side = families(n)[o]
    return tuple(_tree_path(n, o, side)[1]) + (side,)


def position(n: int, u: int, j: int, k: int) -> int:
    """Rank holding u's contribution to block j at the start of step k."""
    e = path_digits(n, u, j)
    dist = distances(n)
    return (u - sum(e[i] * dist[i] for i in range(k))) % n


def _joint(parts: dict) -> np.ndarray:
    """Joint reduction of what a rank holds for one block after a step: (own + from_left) +
    from_right, absent terms skipped (Sec. 4.3 reduces both messages with the local partial)."""
    acc = None
    for side in ("own", "left", "right"):
        if side in parts:
            acc = parts[side].copy() if acc is None else np.add(acc, parts[side],
                                                                 dtype=parts[side].dtype)
    return acc


def bandwidth_optimal_ring(V: np.ndarray, col_blk=None, stats=None) -> np.ndarray:
    """Reduce-scatter + all-gather on a ring of any size n >= 2 (mailbox emulation).

    V        (n, E) inputs; col_blk: block of every column (default: the partition rule).
    stats    optional dict; receives per-step message block counts per rank and direction.
    """
    from . import partition

    n, E = V.shape
    dist = distances(n)
    S = len(dist)
    if col_blk is None:
        _, col_blk = partition.column_labels(E, 1, n)
    col_blk = np.asarray(col_blk)
    cols = {j: np.nonzero(col_blk == j)[0] for j in range(n)}

    # held[x] maps (block, remaining digits) -> partial values of that block's columns
    held = [dict() for _ in range(n)]
    for u in range(n):
        for j in range(n):
            held[u][(j, path_digits(n, u, j))] = V[u, cols[j]].copy()
    sent = np.zeros((S, n, 2), dtype=np.int64)  # blocks per message, [step][rank][+/-]
    for k in range(S):
        inbox = [dict() for _ in range(n)]
        for x in range(n):
            going = {+1: set(), -1: set()}
            for (j, rest), val in held[x].items():
                e = rest[0]
                to = (x - e * dist[k]) % n
                # e = +1: the partial moves towards -, so the receiver gets it from its right
                side = "own" if e == 0 else ("right" if e == +1 else "left")
                slot = inbox[to].setdefault((j, rest[1:]), {})
                if side in slot:
                    raise AssertionError("two partials of one block arrive from one side")
                slot[side] = val
                if e != 0:
                    if j in going[-e]:
                        raise AssertionError("a block is forwarded twice in one message")
                    going[-e].add(j)
            sent[k, x, 0] = len(going[+1])
            sent[k, x, 1] = len(going[-1])
        # barrier: every rank combines what it received, own first, then left, then right
        for x in range(n):
            new = {}
            for key, parts in inbox[x].items():
                acc = _joint(parts)
                if (key[0], key[1]) in new:
                    raise AssertionError("duplicate partial")
                new[key] = acc
            held[x] = new
    for x in range(n):
        if set(held[x]) != {(x, ())}:
            raise AssertionError(f"after reduce-scatter rank {x} holds {sorted(held[x])}")

    # all-gather: retrace every tree edge backwards, latest step first
    out = np.empty_like(V)
    final = {j: held[j][(j, ())] for j in range(n)}
    have = {j: {j} for j in range(n)}
    for k in reversed(range(S)):
        for j in range(n):
            edges = {(position(n, u, j, k + 1), position(n, u, j, k)) for u in range(n)}
            for a, b in edges:
                if a != b:
                    if a not in have[j] or b in have[j]:
                        raise AssertionError("all-gather edge out of order")
                    have[j].add(b)
    for j in range(n):
        if have[j] != set(range(n)):
            raise AssertionError("all-gather left ranks without a block")
        out[:, cols[j]] = final[j][None, :]
    if stats is not None:
        stats["blocks_sent"] = sent
    return out


def link_loads_ring(n: int) -> np.ndarray:
    """Messages per directed link per pass of the bandwidth-optimal schedule, walking every
    non-empty message hop by hop. [pass][rank][port], port 0 = towards +, 1 = towards -;
    reduce-scatter passes, then the all-gather passes in reverse step order (each retraces the
    messages of its step in the opposite direction)."""
    dist = distances(n)
    S = len(dist)
    stats = {}
    bandwidth_optimal_ring(np.zeros((n, 0), np.int32), stats=stats)
    sent = stats["blocks_sent"]
    rs = np.zeros((S, n, 2), dtype=np.int64)
    ag = np.zeros((S, n, 2), dtype=np.int64)
    for k in range(S):
        for x in range(n):
            for port, sign in ((0, +1), (1, -1)):
                if sent[k, x, port] == 0:
                    continue
                node = x
                for _ in range(dist[k]):
                    rs[k, node, port] += 1
                    node = (node + sign) % n
                node = (x + sign * dist[k]) % n
                for _ in range(dist[k]):
                    ag[k, node, 1 - port] += 1
                    node = (node - sign) % n
    return np.concatenate([rs, ag[::-1]])


# ---- tori with sides that are not all powers of three (Sec. 4.4 applied per dimension) ----
#
# Reading: one collective per dimension on its own segment (Sec. 5); collective c takes
# ceil(log3 side_d) steps in every dimension d, choosing at global step t the first dimension in
# cyclic order from (c + t) mod D in which it still has steps left (the rule used for unequal
# sides); a step in dimension d moves contributions along d exactly as the ring of that side
# does (its tree above; the ordinary balanced-ternary tree for a power of three). A
# contribution's position in dimension d depends only on its own offset there, so a rank holds a
# partial of block j while, in every dimension, its offset from j has not yet been forwarded.


def dim_steps(side: int) -> int:
    return 0 if side == 1 else len(distances(side))


def torus_rotation(dims, c: int) -> list:
    """[(dimension, per-dimension step k)] of collective c for every global step."""
    D = len(dims)
    left = [dim_steps(s) for s in dims]
    taken = [0] * D
    out = []
    for t in range(sum(left)):
        order = [(c + t + i) % D for i in range(D)]
        dim = next(d for d in order if taken[d] < left[d])
        out.append((dim, taken[dim]))
        taken[dim] += 1
    return out


def _coords(dims, r):
    out = []
    for s in dims:
        out.append(r % s)
        r //= s
    return out


def _rank(dims, xs):
    r, stride = 0, 1
    for x, s in zip(xs, dims):
        r += (x % s) * stride
        stride *= s
    return r


def torus_paths(dims, j: int, c: int) -> list:
    """pos[t][u]: rank holding u's contribution to block j of collective c at the start of
    global step t, for t = 0..S."""
    dims = tuple(int(x) for x in dims)
    n = int(np.prod(dims))
    js = _coords(dims, j)
    xs = [_coords(dims, u) for u in range(n)]
    digs = [[path_digits(dims[d], xs[u][d], js[d]) if dims[d] > 1 else () for d in range(len(dims))]
            for u in range(n)]
    pos = [[_rank(dims, x) for x in xs]]
    for (dim, k) in torus_rotation(dims, c):
        step = distances(dims[dim])[k]
        for u in range(n):
            xs[u][dim] = (xs[u][dim] - digs[u][dim][k] * step) % dims[dim]
        pos.append([_rank(dims, x) for x in xs])
    return pos


def torus_position(dims, u: int, j: int, c: int, t: int) -> int:
    """Rank holding u's contribution to block j of collective c at the start of global step t."""
    return torus_paths(dims, j, c)[t][u]


def bandwidth_optimal_torus(V: np.ndarray, dims, col_seg=None, col_blk=None,
                            stats=None) -> np.ndarray:
    """Reduce-scatter + all-gather on a torus with any sides (mailbox emulation, see above).

    stats  optional dict; receives "sent" [S][D collectives][n][2]: blocks per message of every
           reduce-scatter step, port 0 towards + and 1 towards - along the active dimension.
    """
    from . import partition

    dims = tuple(int(x) for x in dims)
    D = len(dims)
    n, E = V.shape
    if col_seg is None or col_blk is None:
        col_seg, col_blk = partition.column_labels(E, D, n)
    col_seg = np.asarray(col_seg)
    col_blk = np.asarray(col_blk)
    S = sum(dim_steps(s) for s in dims)
    sent = np.zeros((S, D, n, 2), dtype=np.int64)
    out = np.empty_like(V)
    for c in range(D):
        rot = torus_rotation(dims, c)
        cols = {j: np.nonzero((col_seg == c) & (col_blk == j))[0] for j in range(n)}

        def digits(u, j):
            cu, cj = _coords(dims, u), _coords(dims, j)
            return tuple(path_digits(dims[d], cu[d], cj[d]) if dims[d] > 1 else ()
                         for d in range(D))

        # held[x] maps (block, remaining digits per dimension) -> partial of that block
        held = [dict() for _ in range(n)]
        for u in range(n):
            for j in range(n):
                held[u][(j, digits(u, j))] = V[u, cols[j]].copy()
        for t, (dim, k) in enumerate(rot):
            step = distances(dims[dim])[k]
            inbox = [dict() for _ in range(n)]
            for x in range(n):
                going = {+1: set(), -1: set()}
                for (j, rest), val in held[x].items():
                    e = rest[dim][0]
                    xs = _coords(dims, x)
                    xs[dim] -= e * step
                    to = _rank(dims, xs)
                    # e = +1: the partial moves towards -, so the receiver gets it from its right
                    side = "own" if e == 0 else ("right" if e == +1 else "left")
                    nrest = tuple(r[1:] if d == dim else r for d, r in enumerate(rest))
                    slot = inbox[to].setdefault((j, nrest), {})
                    if side in slot:
                        raise AssertionError("two partials of one block arrive from one side")
                    slot[side] = val
                    if e != 0:
                        if j in going[-e]:
                            raise AssertionError("a block is forwarded twice in one message")
                        going[-e].add(j)
                sent[t, c, x, 0] = len(going[+1])
                sent[t, c, x, 1] = len(going[-1])
            # barrier: every rank combines what it received, own first, then left, then right
            for x in range(n):
                new = {}
                for key, parts in inbox[x].items():
                    new[key] = _joint(parts)
                held[x] = new
        done = tuple(() for _ in range(D))
        for x in range(n):
            if set(held[x]) != {(x, done)}:
                raise AssertionError("reduce-scatter did not finish every block at its owner")
        # all-gather: reverse step order, every tree edge retraced from parent to child (a copy);
        # the parent must already hold the block and the child must not
        for j in range(n):
            have = {j}
            pos = torus_paths(dims, j, c)
            for t in reversed(range(len(rot))):
                edges = {(pos[t + 1][u], pos[t][u]) for u in range(n)}
                for src, dst in edges:
                    if src != dst:
                        if src not in have or dst in have:
                            raise AssertionError("all-gather edge out of order")
                        have.add(dst)
            if have != set(range(n)):
                raise AssertionError("all-gather left ranks without a block")
            out[:, cols[j]] = held[j][(j, done)][None, :]
    if stats is not None:
        stats["sent"] = sent
    return out


def link_loads_torus(dims, form: str = "columns") -> np.ndarray:
    """Messages per directed link per pass of the bandwidth-optimal schedule on a torus with any
    sides, walking every non-empty message hop by hop; layout [pass][rank][port], port 2d towards
    +d, 2d+1 towards -d; reduce-scatter passes, then the all-gather passes in reverse step order
    (each retraces the messages of its step in the opposite direction). Which messages are
    non-empty comes from the gather form on one column per block ("columns") or from the
    mailbox form ("mailbox"); both agree (pinned on small tori)."""
    dims = tuple(int(x) for x in dims)
    D = len(dims)
    n = int(np.prod(dims))
    stats = {}
    if form == "mailbox":
        bandwidth_optimal_torus(np.zeros((n, 0), np.int32), dims, stats=stats)
    else:
        seg = np.repeat(np.arange(D), n)
        blk = np.tile(np.arange(n), D)
        bandwidth_optimal_torus_columns(np.zeros((n, D * n), np.int32), dims, seg, blk,
                                        stats=stats)
    sent = stats["sent"]
    S = sent.shape[0]
    rs = np.zeros((S, n, 2 * D), dtype=np.int64)
    ag = np.zeros((S, n, 2 * D), dtype=np.int64)
    for c in range(D):
        for t, (dim, k) in enumerate(torus_rotation(dims, c)):
            step = distances(dims[dim])[k]
            for x in range(n):
                for port, sign in ((0, +1), (1, -1)):
                    if sent[t, c, x, port] == 0:
                        continue
                    xs = _coords(dims, x)
                    for _ in range(step):
                        rs[t, _rank(dims, xs), 2 * dim + port] += 1
                        xs[dim] += sign
                    # xs is now the receiver: the all-gather message walks back to x
                    for _ in range(step):
                        ag[t, _rank(dims, xs), 2 * dim + 1 - port] += 1
                        xs[dim] -= sign
    return np.concatenate([rs, ag[::-1]])


def _tree_tables(side: int):
    """(send_step[o], digit[o][k]) of a side's tree for every offset residue o = 0..side-1: the
    step at which offset o forwards (S for the root, offset 0) and its path digits."""
    S = dim_steps(side)
    digit = np.zeros((side, max(S, 1)), dtype=np.int64)
    send = np.full(side, S, dtype=np.int64)
    for o in range(1, side):
        e = path_digits(side, o, 0)
        digit[o, :S] = e
        send[o] = next(k for k, x in enumerate(e) if x != 0)
    return send, digit


def _gather_joint(own, left, right, from_left, from_right):
    """(own + from_left) + from_right, where a child sends (the gather form of _joint)."""
    acc = np.where(from_left, np.add(own, left, dtype=own.dtype), own)
    return np.where(from_right, np.add(acc, right, dtype=own.dtype), acc)


def bandwidth_optimal_torus_columns(V: np.ndarray, dims, col_seg, col_blk,
                                    stats=None) -> np.ndarray:
    """The schedule of bandwidth_optimal_torus, executed column by column in gather form: at
    every step each rank combines its own partial with those of the children that forward to it
    in that step, (own + from_left) + from_right; the all-gather copies each forwarded block back
    from the parent. For tori with thousands of ranks, where the mailbox form is too slow; it
    equals the mailbox form bit for bit (pinned on small tori).

    stats  optional dict; "sent" [S][D][n][2] counts, per reduce-scatter step, collective, rank
           and direction (0 towards +, 1 towards -), the columns whose partial the rank forwards
           (with one column per block: the blocks of the message, as the mailbox form counts)."""
    dims = tuple(int(x) for x in dims)
    D = len(dims)
    n, E = V.shape
    col_seg = np.asarray(col_seg)
    col_blk = np.asarray(col_blk)
    tables = [_tree_tables(s) for s in dims]
    X = np.array([_coords(dims, r) for r in range(n)], dtype=np.int64)  # (n, D)

    def neighbour(dim, delta):
        Y = X.copy()
        Y[:, dim] = (Y[:, dim] + delta) % dims[dim]
        strides = np.cumprod((1,) + dims[:-1])
        return (Y * strides).sum(axis=1)

    out = V.copy()
    S = sum(dim_steps(x) for x in dims)
    sent = np.zeros((S, D, n, 2), dtype=np.int64)
    for c in range(D):
        cols = np.nonzero(col_seg == c)[0]
        if cols.size == 0:
            continue
        J = np.array([_coords(dims, int(j)) for j in col_blk[cols]], dtype=np.int64).reshape(-1, D)
        off = [(X[:, d][:, None] - J[:, d][None, :]) % dims[d] for d in range(D)]  # (n, m) each
        rot = torus_rotation(dims, c)
        Q = out[:, cols].copy()

        def state(t):
            taken = [sum(1 for (dd, _) in rot[:t] if dd == d) for d in range(D)]
            dim, k = rot[t]
            alive = np.ones(Q.shape, dtype=bool)
            for d in range(D):
                alive &= tables[d][0][off[d]] >= taken[d]
            e = np.where(alive, tables[dim][1][off[dim], k], 0)
            return dim, distances(dims[dim])[k], alive, e

        for t in range(len(rot)):
            dim, dist, alive, e = state(t)
            sent[t, c, :, 0] = (e == -1).sum(axis=1)
            sent[t, c, :, 1] = (e == +1).sum(axis=1)
            L, R = neighbour(dim, -dist), neighbour(dim, +dist)
            from_left = e[L] == -1   # the rank at y - dist moves by +dist onto y
            from_right = e[R] == +1  # the rank at y + dist moves by -dist onto y
            recv = from_left | from_right
            if not (alive[recv].all() and (e[recv] == 0).all()):
                raise AssertionError("a receiver is not holding its own partial")
            Q = _gather_joint(Q, Q[L], Q[R], from_left, from_right)
        for t in reversed(range(len(rot))):
            dim, dist, alive, e = state(t)
            L, R = neighbour(dim, -dist), neighbour(dim, +dist)
            # a sender (e = +1 moved to y - dist, e = -1 to y + dist) receives its parent's copy
            Q = np.where(e == +1, Q[L], np.where(e == -1, Q[R], Q))
        out[:, cols] = Q
    if stats is not None:
        stats["sent"] = sent
    return out
