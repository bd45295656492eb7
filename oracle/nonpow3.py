"""Trivance on rings whose size is not a power of three (oracle side, Sec. 4.4).

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
                acc = None
                for side in ("own", "left", "right"):
                    if side in parts:
                        acc = parts[side].copy() if acc is None else \
                            np.add(acc, parts[side], dtype=V.dtype)
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
