"""Step-by-step message-passing emulation of Trivance AllReduce (oracle side).

Test infrastructure only (see the package docstring).

Every rank is an explicit mailbox participant. In each step every rank first posts its messages
(copies of its current data), then -- after all messages of the step exist, the per-step barrier
of Sec. 4.3 -- every rank combines the two messages it received with its own partial result.

Arithmetic is done in the element type of the input (numpy float32 / int32; int32 adds wrap
modulo 2^32 like two's-complement hardware). Floating-point association of the joint reduction
(a reading; Sec. 4.3 and Appendix D only say that both received messages are combined with the
local partial result): (own + from_left) + from_right, where `left` is the peer at -distance.

Variants
--------
'L'  latency-optimal (Sec. 4.2): every step, every rank sends its whole segment to both peers.
'B'  bandwidth-optimal (Sec. 4.1): reduce-scatter with the block sets of Algorithm 1, then an
     all-gather in reverse step order in which every rank forwards every finished block it holds
     to both peers (no reduction; Appendix D).
On a torus one collective per dimension runs on its own segment (Sec. 5).
"""

from __future__ import annotations

import numpy as np

from . import nonpow3, partition, schedule


def _check_input(V: np.ndarray, torus: schedule.Torus) -> None:
    if V.ndim != 2 or V.shape[0] != torus.n:
        raise ValueError(f"expected an (n={torus.n}, E) array, got shape {V.shape}")
    if V.dtype not in (np.float32, np.int32, np.float64):
        raise ValueError(f"unsupported dtype {V.dtype}")


def _reduce3(own: np.ndarray, from_left: np.ndarray, from_right: np.ndarray) -> np.ndarray:
    """Joint reduction of one rank: (own + from_left) + from_right in the element type."""
    with np.errstate(over="ignore"):
        tmp = np.add(own, from_left, dtype=own.dtype)
        return np.add(tmp, from_right, dtype=own.dtype)


def latency_optimal(V: np.ndarray, dims, col_seg=None, passes=None, trace=None) -> np.ndarray:
    """Latency-optimal Trivance on a ring or torus; returns every rank's final vector.

    V        (n, E) inputs, row r = rank r's vector (not modified).
    col_seg  segment (collective) of each column; defaults to the partition rule for all E
             columns. Pass it explicitly when V holds a column sample of a larger vector.
    passes   optional number of passes to run (default: all S); used for per-step checks.
    trace    optional list; receives (t, c, sender, receiver, payload copy) of every message.
    """
    torus = schedule.Torus(tuple(dims))
    _check_input(V, torus)
    n, E = V.shape
    if col_seg is None:
        col_seg, _ = partition.column_labels(E, torus.D, n)
    col_seg = np.asarray(col_seg)
    state = V.copy()
    S = torus.steps if passes is None else passes
    for t in range(S):
        for c in range(torus.D):
            cols = np.nonzero(col_seg == c)[0]
            # post: every rank copies its whole segment into both outgoing messages
            inbox = {}
            for r in range(n):
                left, right = schedule.peers(torus, c, r, t)
                payload = state[r, cols].copy()
                inbox[(r, left)] = payload
                inbox[(r, right)] = payload
                if trace is not None:
                    trace.append((t, c, r, left, payload))
                    trace.append((t, c, r, right, payload))
            # barrier passed: combine both received messages with the local partial
            for r in range(n):
                left, right = schedule.peers(torus, c, r, t)
                state[r, cols] = _reduce3(state[r, cols], inbox[(left, r)], inbox[(right, r)])
    return state


def bandwidth_optimal(V: np.ndarray, dims, col_seg=None, col_blk=None, rs_passes=None,
                      ag_passes=None, stats=None) -> np.ndarray:
    """Bandwidth-optimal Trivance (reduce-scatter + all-gather); returns every rank's vector.

    col_seg, col_blk  segment and block label of every column (default: the partition rule).
    rs_passes         optional number of reduce-scatter steps to run (default all S).
    ag_passes         optional number of all-gather steps to run after a full reduce-scatter.
    stats             optional dict; filled with per-rank message/block counts for the pins.

    Bookkeeping: `live[c][r]` is the set of blocks for which rank r still holds a partial result
    it is responsible for; `final[c][r]` is the set of finished blocks it holds during the
    all-gather. Both are checked at every step, so a wrong block set aborts instead of silently
    producing a plausible number.
    """
    torus = schedule.Torus(tuple(dims))
    _check_input(V, torus)
    n, E = V.shape
    D, S = torus.D, torus.steps
    if col_seg is None or col_blk is None:
        col_seg, col_blk = partition.column_labels(E, D, n)
    col_seg = np.asarray(col_seg)
    col_blk = np.asarray(col_blk)
    cols_of = [{j: np.nonzero((col_seg == c) & (col_blk == j))[0] for j in range(n)}
               for c in range(D)]

    def columns(c, blocks):
        if not blocks:
            return np.zeros(0, dtype=np.int64)
        return np.concatenate([cols_of[c][j] for j in blocks])

    state = V.copy()
    live = [[set(range(n)) for _ in range(n)] for _ in range(D)]
    sent_blocks = np.zeros((D, n), dtype=np.int64)
    reduced_blocks = np.zeros((D, n), dtype=np.int64)

    # ---- reduce-scatter, t = 0..S-1 ----
    n_rs = S if rs_passes is None else rs_passes
    for t in range(n_rs):
        for c in range(D):
            inbox = {}
            for r in range(n):
                going = set()
                for p in schedule.peers(torus, c, r, t):
                    blocks = schedule.message_blocks(torus, c, p, t)
                    if not set(blocks) <= live[c][r]:
                        raise AssertionError(f"rank {r} would send blocks it no longer holds")
                    inbox[(r, p)] = (blocks, state[r, columns(c, blocks)].copy())
                    going |= set(blocks)
                    sent_blocks[c, r] += len(blocks)
                reduced_blocks[c, r] += len(live[c][r])  # partial data touched this step
                live[c][r] -= going
            for r in range(n):
                left, right = schedule.peers(torus, c, r, t)
                lb, lv = inbox[(left, r)]
                rb, rv = inbox[(right, r)]
                if lb != rb or set(lb) != live[c][r]:
                    raise AssertionError("the two incoming messages do not match the kept blocks")
                cols = columns(c, lb)
                state[r, cols] = _reduce3(state[r, cols], lv, rv)
    if n_rs == S:
        for c in range(D):
            for r in range(n):
                if live[c][r] != {r}:
                    raise AssertionError(f"after reduce-scatter rank {r} holds {live[c][r]}")

    # ---- all-gather, t = S-1..0 ----
    final = [[set(live[c][r]) for r in range(n)] for c in range(D)]
    n_ag = (S if ag_passes is None else ag_passes) if n_rs == S else 0
    for t in list(reversed(range(S)))[:n_ag]:
        for c in range(D):
            inbox = {}
            for r in range(n):
                blocks = sorted(final[c][r])
                payload = state[r, columns(c, blocks)].copy()
                for p in schedule.peers(torus, c, r, t):
                    inbox[(r, p)] = (blocks, payload)
            for r in range(n):
                left, right = schedule.peers(torus, c, r, t)
                lb, lv = inbox[(left, r)]
                rb, rv = inbox[(right, r)]
                if set(lb) & set(rb) or (set(lb) | set(rb)) & final[c][r]:
                    raise AssertionError("all-gather messages overlap")
                state[r, columns(c, lb)] = lv
                state[r, columns(c, rb)] = rv
                final[c][r] |= set(lb) | set(rb)
    if n_ag == S:
        for c in range(D):
            for r in range(n):
                if final[c][r] != set(range(n)):
                    raise AssertionError("all-gather left blocks missing")
    if stats is not None:
        stats["sent_blocks_rs"] = sent_blocks
        stats["reduced_blocks_rs"] = reduced_blocks
    return state


def allreduce(V: np.ndarray, dims, variant: str, **kw) -> np.ndarray:
    if nonpow3.is_tree(dims):
        if variant == "L":
            from . import latency_nonpow3

            return latency_nonpow3.latency_optimal(V, dims, col_seg=kw.get("col_seg"))
        if variant != "B":
            raise ValueError(f"unknown variant {variant!r}")
        if len(dims) == 1:
            return nonpow3.bandwidth_optimal_ring(V, col_blk=kw.get("col_blk"))
        seg, blk = kw.get("col_seg"), kw.get("col_blk")
        if seg is None or blk is None:
            seg, blk = partition.column_labels(V.shape[1], len(dims), V.shape[0])
        # the gather form: equal bit for bit to the mailbox form (pinned), fast for large tori
        return nonpow3.bandwidth_optimal_torus_columns(V, dims, seg, blk)
    if variant == "L":
        return latency_optimal(V, dims, **kw)
    if variant == "B":
        return bandwidth_optimal(V, dims, **kw)
    raise ValueError(f"unknown variant {variant!r}")


# ---- reference sums (the plain definition of AllReduce, Sec. 2.2) ----

def exact_int_sum(V: np.ndarray) -> np.ndarray:
    """sum_u v_u per column in exact integers, wrapped to int32 (two's complement)."""
    s = V.astype(np.int64).sum(axis=0)
    return ((s + 2 ** 31) % 2 ** 32 - 2 ** 31).astype(np.int32)


def fp64_sum(V: np.ndarray) -> np.ndarray:
    return V.astype(np.float64).sum(axis=0)


def abs_sum(V: np.ndarray) -> np.ndarray:
    return np.abs(V.astype(np.float64)).sum(axis=0)


def ceil_log3(n: int) -> int:
    """Smallest s with 3^s >= n: the step count of Theorem 1 and Sec. 4.4 on a ring of n."""
    s, p = 0, 1
    while p < n:
        p *= 3
        s += 1
    return s


def fp32_error_bound(V: np.ndarray) -> np.ndarray:
    """Per-column bound 4 * ceil(log3 n) * 2^-23 * sum_u |v_u| on |fp32 result - exact sum|, n the
    number of ranks (rows of V).

    Each input passes through at most two float additions per step (a ternary joint reduction),
    so the classical summation bound is about 2 S * 2^-24 * sum |v| = S * 2^-23 * sum |v| for S
    steps. S is ceil(log3 n) on rings and on tori whose sides are powers of three; a torus with
    other sides can take a few more steps than that (32x32: 8 against 7), which the factor 4
    covers."""
    return 4.0 * max(ceil_log3(V.shape[0]), 1) * 2.0 ** -23 * abs_sum(V)
