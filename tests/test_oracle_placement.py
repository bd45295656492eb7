"""The optional message-contiguous block placement of the oracle (CPU only).

Pins: it is a permutation; on a ring it is base-3 digit reversal (written out here with Python's
own base conversion); every set of blocks a rank keeps after a reduce-scatter step, as Algorithm 1
(reachability) yields it, is one aligned run of positions, and so is every message; the AllReduce
under it gives exact int32 sums, and in fp32 every element equals the latency-optimal result at
its block's owner (the same association, Sec. 4.2 vs 4.1).
"""

import numpy as np
import pytest

from oracle import allreduce, partition, placement, schedule

SHAPES = [(3,), (9,), (27,), (81,), (243,), (3, 3), (9, 9), (27, 27), (3, 3, 3), (9, 9, 9),
          (3, 3, 3, 3), (3, 9), (27, 3), (3, 3, 9), (9, 27)]


def _digits_reversed(j: int, s: int) -> int:
    text = np.base_repr(j, 3).rjust(s, "0") if s else ""
    return int(text[::-1], 3) if s else 0


@pytest.mark.parametrize("dims", SHAPES, ids=lambda d: "x".join(map(str, d)))
def test_positions_are_a_permutation(dims):
    n = int(np.prod(dims))
    for pos in placement.positions(dims):
        assert sorted(pos.tolist()) == list(range(n))


@pytest.mark.parametrize("n", [3, 9, 27, 81, 243, 729])
def test_ring_placement_is_digit_reversal(n):
    s = schedule.log3_exact(n)
    (pos,) = placement.positions((n,))
    assert pos.tolist() == [_digits_reversed(j, s) for j in range(n)]


def _kept_after(torus, c, r, t):
    """Blocks rank r still reduces after reduce-scatter step t: all blocks minus those it sent,
    the messages being Algorithm 1's (schedule.message_blocks)."""
    kept = set(range(torus.n))
    for t2 in range(t + 1):
        for p in schedule.peers(torus, c, r, t2):
            kept -= set(schedule.message_blocks(torus, c, p, t2))
    return kept


@pytest.mark.parametrize("dims", [(9,), (27,), (81,), (3, 3), (9, 9), (3, 3, 3), (3, 3, 3, 3),
                                  (3, 9), (9, 3), (3, 27), (3, 3, 9)],
                         ids=lambda d: "x".join(map(str, d)))
def test_kept_sets_and_messages_are_contiguous(dims):
    torus = schedule.Torus(dims)
    pos = placement.positions(dims)
    for c in range(torus.D):
        for t in range(torus.steps):
            size = torus.n // 3 ** (t + 1)
            for r in range(torus.n):
                kept = _kept_after(torus, c, r, t)
                assert len(kept) == size
                p = sorted(pos[c][j] for j in kept)
                assert p == list(range(p[0], p[0] + size)) and p[0] % size == 0
                for q in schedule.peers(torus, c, r, t):
                    m = sorted(pos[c][j] for j in schedule.message_blocks(torus, c, q, t))
                    assert m == list(range(m[0], m[0] + len(m)))


def test_natural_order_is_not_contiguous():
    """The default partition keeps every third block after the first step of a 9-ring."""
    torus = schedule.Torus((9,))
    kept = sorted(_kept_after(torus, 0, 0, 0))
    assert kept == [0, 3, 6]


@pytest.mark.parametrize("dims,E", [((9,), 64 * 9 * 3 + 20), ((27,), 64 * 27 * 2 + 4),
                                    ((3, 3), 64 * 9 * 4 + 12), ((9, 9), 64 * 81 * 2 + 4),
                                    ((3, 3, 3), 64 * 27 * 3 + 16), ((3, 9), 64 * 27 * 2 + 8),
                                    ((9, 3, 3), 777)],
                         ids=lambda x: "x".join(map(str, x)) if isinstance(x, tuple) else str(x))
def test_allreduce_under_placement(dims, E):
    n = int(np.prod(dims))
    rng = np.random.default_rng(n + E)
    seg, blk = placement.column_labels(E, dims)
    Vi = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    out = allreduce.bandwidth_optimal(Vi, dims, col_seg=seg, col_blk=blk)
    assert (out == allreduce.exact_int_sum(Vi)[None]).all()
    Vf = rng.standard_normal((n, E), dtype=np.float32)
    out = allreduce.bandwidth_optimal(Vf, dims, col_seg=seg, col_blk=blk)
    lat = allreduce.latency_optimal(Vf, dims)
    assert np.array_equal(out, np.broadcast_to(lat[blk, np.arange(E)], out.shape))
    # and it differs from the default partition somewhere (other blocks, other trees)
    assert not np.array_equal(out, allreduce.bandwidth_optimal(Vf, dims))


def test_placed_labels_of_a_sample_match_the_whole_vector():
    dims, E = (9, 9), 64 * 81 * 2 + 36
    seg, blk = placement.column_labels(E, dims)
    cols = np.array([0, 5, 64 * 81, E - 1, 1000])
    s2, b2 = placement.column_labels(E, dims, cols)
    assert (s2 == seg[cols]).all() and (b2 == blk[cols]).all()
    _, nat = partition.column_labels(E, 2, 81)
    assert not (nat == blk).all()


def _contiguous(dims, pos) -> bool:
    torus = schedule.Torus(dims)
    for c in range(torus.D):
        for t in range(torus.steps):
            size = torus.n // 3 ** (t + 1)
            for r in range(torus.n):
                p = sorted(pos[c][j] for j in _kept_after(torus, c, r, t))
                if p != list(range(p[0], p[0] + size)):
                    return False
    return True


@pytest.mark.parametrize("dims", [(27,), (3, 3), (9, 9), (3, 3, 3)], ids=lambda d: "x".join(map(str, d)))
def test_planted_placement_mistakes_are_caught(dims):
    torus = schedule.Torus(dims)
    good = placement.positions(dims)
    assert _contiguous(dims, good)
    # digits least significant first (the natural order on a ring)
    low_first = []
    for c in range(torus.D):
        steps = [schedule.step_dim_and_distance(torus, c, t) for t in range(torus.steps)]
        pos = []
        for j in range(torus.n):
            xs, p = torus.coords(j), 0
            for d, dist in reversed(steps):
                p = 3 * p + (xs[d] // dist) % 3
            pos.append(p)
        low_first.append(np.array(pos))
    assert not _contiguous(dims, low_first)
    # on a torus, digits taken dimension by dimension instead of in the schedule's order
    if torus.D > 1:
        by_dim = []
        for c in range(torus.D):
            pos = []
            for j in range(torus.n):
                xs, p = torus.coords(j), 0
                for d in range(torus.D):
                    for k in range(schedule.log3_exact(dims[d])):
                        p = 3 * p + (xs[d] // 3 ** k) % 3
                pos.append(p)
            by_dim.append(np.array(pos))
        assert not _contiguous(dims, by_dim)
