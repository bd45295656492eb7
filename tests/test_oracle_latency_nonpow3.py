"""Pins of the latency-optimal oracle for sides that are not powers of three
(oracle/latency_nonpow3.py; Sec. 4.2 with Sec. 4.4), CPU only."""

import json
import os

import numpy as np
import pytest

from oracle import allreduce, latency_nonpow3 as LN, nonpow3, partition

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

RINGS = [2, 4, 5, 6, 7, 8, 10, 11, 13, 14, 16, 20, 22, 26, 28, 32, 40, 50, 64, 80, 82, 100]
TORI = [(4, 4), (2, 3), (3, 8), (8, 3), (5, 7), (1, 8), (2, 3, 4), (4, 4, 4), (2, 2, 2, 2),
        (8, 8), (10, 3, 3), (16, 16), (32, 32), (8, 64)]


@pytest.mark.parametrize("dims", [(n,) for n in RINGS] + TORI,
                         ids=lambda d: "x".join(map(str, d)))
def test_int32_exact_sums_on_every_rank(dims):
    """Integer results equal the exact column sums on every rank (Sec. 2.2), with wrapping."""
    n = int(np.prod(dims))
    E = 3 * len(dims) + 1 if n > 300 else 64 * len(dims) + 13
    V = np.random.default_rng(n).integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    out = LN.latency_optimal(V, dims)
    np.testing.assert_array_equal(out, np.broadcast_to(allreduce.exact_int_sum(V), out.shape))


@pytest.mark.parametrize("dims", [(n,) for n in RINGS if n <= 64] + [(4, 4), (5, 7), (2, 3, 4)],
                         ids=lambda d: "x".join(map(str, d)))
def test_one_hot_every_source_exactly_once(dims):
    """With one-hot inputs (column u holds 1 at rank u only) every rank ends with all ones: each
    source reaches each rank exactly once after ceil(log3) steps per side, as Lemma 2 and
    Theorem 1 require of the full schedule."""
    n = int(np.prod(dims))
    D = len(dims)
    V = np.zeros((n, D * n), dtype=np.int32)
    for c in range(D):
        V[np.arange(n), c * n + np.arange(n)] = 1
    seg = np.repeat(np.arange(D), n)
    out = LN.latency_optimal(V, dims, col_seg=seg)
    assert (out == 1).all()


@pytest.mark.parametrize("n", [4, 5, 7, 8, 10, 16, 32, 64])
def test_window_after_the_full_steps_is_lemma2(n):
    """Before the final step a rank's first partial is its Lemma 2 window: the sources within
    R = (3^f - 1) / 2, each once (one-hot inputs)."""
    f, d = nonpow3.levels(n)
    V = np.eye(n, dtype=np.int32)
    trace = []
    LN.latency_optimal(V, (n,), col_seg=np.zeros(n, dtype=np.int64), trace=trace)
    c, t, parts = trace[f - 1]
    R = (3 ** f - 1) // 2
    win = next(iter(parts.values()))  # the window comes first
    for x in range(n):
        want = np.zeros(n, dtype=np.int32)
        want[[(x + o) % n for o in range(-R, R + 1)]] = 1
        np.testing.assert_array_equal(win[x], want)


def test_n7_figure_steps_and_final_distance():
    with open(os.path.join(GOLDEN, "n7_nonpower3.json")) as f:
        g = json.load(f)
    needed, recipes = LN.program((7,))
    assert len(recipes) == g["n7_steps"]["value"]
    assert nonpow3.distances(7)[-1] == g["n7_final_distance"]["value"]
    # a rank sends one vector each way in both steps
    assert LN.message_slots((7,)) == [(1, 1), (1, 1)]


@pytest.mark.parametrize("dims", [(3,), (9,), (27,), (81,), (3, 3), (9, 9), (3, 9), (1, 9), (3, 3, 3)],
                         ids=lambda d: "x".join(map(str, d)))
def test_powers_of_three_are_the_ordinary_schedule(dims):
    """On sides that are powers of three the window is the only partial: bit for bit the ordinary
    latency-optimal oracle."""
    n = int(np.prod(dims))
    E = 64 * len(dims) * 2 + 7
    V = (np.random.default_rng(n).standard_normal((n, E)) * np.logspace(-5, 5, E)).astype(np.float32)
    assert all(len(s) == 1 for s in LN.program(dims)[0])
    np.testing.assert_array_equal(LN.latency_optimal(V, dims), allreduce.latency_optimal(V, dims))


def test_rank0_trees_written_out():
    """fp32 association at rank 0, derived by hand from the reading.

    n = 4 (f = 1, window of 3, final distance 1, one missing source, on the + side): the rank at +1
    keeps its right neighbour's value and sends it: ((v0 + v3) + v1) + v2.
    n = 7 (final distance 2): the rank at -2 sends its own plus its left neighbour's value, the rank
    at +2 its own plus its right neighbour's: (((v0 + v6) + v1) + (v5 + v4)) + (v2 + v3).
    n = 8 (final distance 3, the + side supplies three sources): the rank at +3 sends its whole
    window, the rank at -3 its own plus its right neighbour's value:
    (((v0 + v7) + v1) + (v5 + v6)) + ((v3 + v2) + v4)."""
    trees = {4: lambda v: ((v[0] + v[3]) + v[1]) + v[2],
             7: lambda v: (((v[0] + v[6]) + v[1]) + (v[5] + v[4])) + (v[2] + v[3]),
             8: lambda v: (((v[0] + v[7]) + v[1]) + (v[5] + v[6])) + ((v[3] + v[2]) + v[4])}
    for n, tree in trees.items():
        E = 512
        V = (np.random.default_rng(40 + n).standard_normal((n, E)) *
             np.logspace(-6, 6, E)).astype(np.float32)
        out = LN.latency_optimal(V, (n,), col_seg=np.zeros(E, dtype=np.int64))
        np.testing.assert_array_equal(out[0], tree(V))
        naive = V[0].copy()
        for u in range(1, n):
            naive = naive + V[u]
        assert not np.array_equal(naive, out[0])


@pytest.mark.parametrize("n", RINGS[:12])
def test_shift_equivariance(n):
    """Every rank runs the same program relative to itself: rolling the inputs by one rank rolls
    the results, bit for bit."""
    E = 200
    V = (np.random.default_rng(3 * n).standard_normal((n, E)) * np.logspace(-4, 4, E)).astype(np.float32)
    seg = np.zeros(E, dtype=np.int64)
    a = LN.latency_optimal(np.roll(V, 1, axis=0), (n,), col_seg=seg)
    b = np.roll(LN.latency_optimal(V, (n,), col_seg=seg), 1, axis=0)
    np.testing.assert_array_equal(a, b)


BLOCK_EQUALS_OWNER = [2, 6, 7, 8, 18, 19, 20, 21, 24, 25, 26]


@pytest.mark.parametrize("n", [n for n in range(2, 28) if nonpow3.levels(n)[1] != 0])
def test_bandwidth_block_equals_latency_owner_where_windows_match(n):
    """On powers of three block j of the bandwidth-optimal result equals rank j's latency-optimal
    result. With the Sec. 4.4 trees the same holds exactly where the owner's tree holds its whole
    window before the final step (tests/test_nonpow3_trees.py), and the two associations differ
    elsewhere."""
    E = 64 * n * 2
    V = (np.random.default_rng(n).standard_normal((n, E)) * np.logspace(-4, 4, E)).astype(np.float32)
    Lr = LN.latency_optimal(V, (n,))
    B = nonpow3.bandwidth_optimal_ring(V)
    _, blk = partition.column_labels(E, 1, n)
    same = all(np.array_equal(B[0, blk == j], Lr[j, blk == j]) for j in range(n))
    assert same == (n in BLOCK_EQUALS_OWNER)


@pytest.mark.parametrize("dims", [(7,), (32,), (4, 4), (5, 7), (32, 32)], ids=lambda d: "x".join(map(str, d)))
def test_fp32_within_the_summation_bound(dims):
    n = int(np.prod(dims))
    E = 64 * len(dims) * 3 + 5
    V = np.random.default_rng(9 + n).standard_normal((n, E)).astype(np.float32)
    out = LN.latency_optimal(V, dims)
    err = np.abs(out.astype(np.float64) - allreduce.fp64_sum(V)[None, :])
    assert (err <= allreduce.fp32_error_bound(V)[None, :]).all()
