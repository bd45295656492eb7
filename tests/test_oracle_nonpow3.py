"""Pins of the oracle for rings and tori whose sides are not all powers of three (Sec. 4.4), CPU
only."""

import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import allreduce, congestion, nonpow3

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SIZES = [2, 4, 5, 6, 7, 8, 10, 11, 14, 15, 16, 20, 26, 28, 31, 32, 40, 50, 64, 80, 82, 100]


def _golden():
    with open(os.path.join(GOLDEN, "n7_nonpower3.json")) as f:
        return json.load(f)


def test_n7_figure():
    g = _golden()
    assert len(nonpow3.distances(7)) == g["n7_steps"]["value"]
    assert nonpow3.distances(7)[-1] == g["n7_final_distance"]["value"]
    stats = {}
    nonpow3.bandwidth_optimal_ring(np.zeros((7, 0), np.int32), stats=stats)
    for k, want in enumerate(g["n7_blocks_per_direction"]["value"]):
        assert (stats["blocks_sent"][k] == want).all()


def test_n32_reading_departs_from_the_27_of_32_count():
    """Reading 13 on the 32-ring: the final distance is ceil((32 - 27) / 2) = 3 (Sec. 4.4), the
    owner of a block holds 15 of the 32 contributions before the final step and receives 17 in
    it, and every rank forwards every block exactly once (31 forwards per block and phase).

    Sec. 4.4 counts 27 held before the final step and 5 arriving in it. That count is the reading
    NOT taken: the ranks at +/-3 that send in the final step lie inside the owner's 27-window, so
    holding the whole window before the final step would need them to forward the block twice,
    against the paper's at-most-once bound (tests/test_nonpow3_trees.py proves this and shows by
    enumeration that the reading holds as many contributions before the final step as any
    single-forwarding tree can)."""
    g = _golden()
    f, d = nonpow3.levels(32)
    assert d == math.ceil((32 - g["n32_blocks_before_final"]["value"]) / 2) == 3
    # which contributions reach block 0's owner without the final step
    S = len(nonpow3.distances(32))
    held = {u for u in range(32) if nonpow3.position(32, u, 0, S - 1) == 0}
    assert len(held) == 15 and len(held) != g["n32_blocks_before_final"]["value"]
    arriving = {u for u in range(32) if nonpow3.position(32, u, 0, S - 1) in (3, 29)}
    assert len(arriving) == 17 and held | arriving == set(range(32))
    # one forward per block and rank: 31 forwards of each block over the phase
    stats = {}
    nonpow3.bandwidth_optimal_ring(np.zeros((32, 0), np.int32), stats=stats)
    assert stats["blocks_sent"].sum() == 32 * 31
    assert (stats["blocks_sent"].sum(axis=(0, 2)) == 31).all()


def test_n7_and_n8_block0_trees_written_out():
    """fp32 association of block 0 on the 7- and 8-rings, derived by hand from reading 13.

    n = 7 (f = 1, window |o| <= 1, final distance 2): ranks 2 and 3 form the + tree (3 sends to 2
    in step 0), ranks 5 and 4 the - tree (4 sends to 5); the owner first combines its neighbours,
    then in the final step the partial from 5 (its left peer at distance 2) and the one from 2:
        ((((v0 + v6) + v1) + (v5 + v4)) + (v2 + v3)).
    n = 8 (final distance 3; the odd remainder puts the extra rank on the + side): ranks 2, 3, 4
    form the + tree rooted at 3 (2 from its left, 4 from its right), ranks 6, 5 the - tree rooted
    at 5 (6 sends from its right):
        (((v0 + v7) + v1) + (v5 + v6)) + ((v3 + v2) + v4).
    Each is a (own + left) + right joint reduction at every receiver (Sec. 4.3), absent terms
    skipped. Inputs spanning twelve decades make other associations round differently."""
    from oracle import partition

    for n, tree in ((7, lambda v: (((v[0] + v[6]) + v[1]) + (v[5] + v[4])) + (v[2] + v[3])),
                    (8, lambda v: (((v[0] + v[7]) + v[1]) + (v[5] + v[6])) + ((v[3] + v[2]) + v[4]))):
        rng = np.random.default_rng(70 + n)
        E = 64 * n * 4
        V = (rng.standard_normal((n, E)) * np.logspace(-6, 6, E)).astype(np.float32)
        want = tree(V)
        out = nonpow3.bandwidth_optimal_ring(V)
        _, blk = partition.column_labels(E, 1, n)
        np.testing.assert_array_equal(out[0, blk == 0], want[blk == 0])
        # the written-out order is observable: summing left to right gives other bits
        naive = V[0].copy()
        for u in range(1, n):
            naive = naive + V[u]
        assert not np.array_equal(naive[blk == 0], want[blk == 0])


@pytest.mark.parametrize("n", range(2, 244))
def test_step_count_and_distance_rule(n):
    """ceil(log3 n) steps; the final distance grows by one for every two ranks beyond 3^f."""
    dist = nonpow3.distances(n)
    S = 0
    while 3 ** S < n:
        S += 1
    assert len(dist) == S
    f, d = nonpow3.levels(n)
    assert dist[:f] == [3 ** k for k in range(f)]
    if 3 ** f != n:
        assert d == -(-(n - 3 ** f) // 2)
        assert nonpow3.levels(n + 1)[1] in (d, d + 1) or 3 ** (f + 1) == n + 1


@pytest.mark.parametrize("n", SIZES)
def test_int32_bruteforce_and_forwarded_once(n):
    """Exact integer sums, and every rank forwards every block exactly once per phase (Sec. 4.4:
    each block at most once per phase, at most m per rank)."""
    rng = np.random.default_rng(n)
    V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, 64 * n + 13), dtype=np.int32)
    stats = {}
    out = nonpow3.bandwidth_optimal_ring(V, stats=stats)
    np.testing.assert_array_equal(out, np.broadcast_to(allreduce.exact_int_sum(V), out.shape))
    assert (stats["blocks_sent"].sum(axis=(0, 2)) == n - 1).all()
    np.testing.assert_array_equal(allreduce.allreduce(V, (n,), "B"), out)


@pytest.mark.parametrize("n", [7, 8, 10, 20, 32, 50, 100])
def test_fp32_bound_and_identical_ranks(n):
    rng = np.random.default_rng(100 + n)
    V = rng.standard_normal((n, 64 * n + 7), dtype=np.float32)
    out = nonpow3.bandwidth_optimal_ring(V)
    assert (out == out[0:1]).all()
    err = np.abs(out[0].astype(np.float64) - allreduce.fp64_sum(V))
    assert (err <= allreduce.fp32_error_bound(V)).all()


@pytest.mark.parametrize("n", [3, 9, 27, 81])
def test_powers_of_three_reduce_to_the_ordinary_schedule(n):
    rng = np.random.default_rng(7 * n)
    V = rng.standard_normal((n, 64 * n + 3), dtype=np.float32)
    np.testing.assert_array_equal(nonpow3.bandwidth_optimal_ring(V),
                                  allreduce.bandwidth_optimal(V, (n,)))


@pytest.mark.parametrize("n", [4, 7, 8, 10, 20, 32, 64])
def test_congestion_uniform_and_final_equals_distance(n):
    """Sec. 4.4: the final step is uniform and its congestion equals its distance; every step
    loads each used link with exactly its distance (one message per rank and direction)."""
    loads = congestion.link_loads((n,), "B")
    dist = nonpow3.distances(n)
    S = len(dist)
    assert loads.shape == (2 * S, n, 2)
    for k in range(S):
        for p in (k, 2 * S - 1 - k):
            for port in (0, 1):
                col = loads[p, :, port]
                assert (col == 0).all() or (col == dist[k]).all()
            assert loads[p].max() == dist[k]
    f, d = nonpow3.levels(n)
    if n - 3 ** f >= 2:
        assert (loads[S - 1] == d).all()


def test_latency_variant_dispatches_to_its_oracle():
    from oracle import latency_nonpow3

    V = np.random.default_rng(8).integers(-99, 99, size=(8, 77), dtype=np.int32)
    np.testing.assert_array_equal(allreduce.allreduce(V, (8,), "L"),
                                  latency_nonpow3.latency_optimal(V, (8,)))
    with pytest.raises(ValueError):
        allreduce.allreduce(V, (8,), "X")


# ---- tori with a side that is not a power of three ----

TORI = [(4, 4), (2, 3), (8, 8), (5, 7), (3, 8), (8, 3), (4, 4, 4), (2, 3, 4), (2, 2, 2, 2)]


@pytest.mark.parametrize("dims", TORI)
def test_torus_int32_bruteforce_and_forwarded_once(dims):
    """Exact integer sums on every rank, and per collective every rank forwards n - 1 blocks over
    the reduce-scatter (each block's contributions meet along one tree of n - 1 edges, Sec. 4.4:
    each block forwarded once per phase)."""
    n = int(np.prod(dims))
    rng = np.random.default_rng(n + len(dims))
    V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, 64 * len(dims) * n + 13), dtype=np.int32)
    stats = {}
    out = nonpow3.bandwidth_optimal_torus(V, dims, stats=stats)
    np.testing.assert_array_equal(out, np.broadcast_to(allreduce.exact_int_sum(V), out.shape))
    assert (stats["sent"].sum(axis=(0, 3)) == n - 1).all()
    assert stats["sent"].shape[0] == sum(math.ceil(math.log(s, 3) - 1e-12) for s in dims)
    np.testing.assert_array_equal(allreduce.allreduce(V, dims, "B"), out)


@pytest.mark.parametrize("dims", [(4, 4), (5, 7), (8, 3), (2, 3, 4)])
def test_torus_fp32_bound_and_identical_ranks(dims):
    n = int(np.prod(dims))
    V = np.random.default_rng(200 + n).standard_normal((n, 64 * len(dims) * n + 7),
                                                       dtype=np.float32)
    out = nonpow3.bandwidth_optimal_torus(V, dims)
    assert (out == out[0:1]).all()
    err = np.abs(out[0].astype(np.float64) - allreduce.fp64_sum(V))
    assert (err <= allreduce.fp32_error_bound(V)).all()


@pytest.mark.parametrize("dims", [(3, 3), (9, 3), (3, 9), (3, 3, 3), (1, 9)])
def test_torus_powers_of_three_reduce_to_the_ordinary_schedule(dims):
    """Bits and link loads equal the ordinary torus schedule (Sec. 5) when every side is 3^s."""
    n = int(np.prod(dims))
    V = np.random.default_rng(11 * n).standard_normal((n, 64 * len(dims) * n + 3),
                                                      dtype=np.float32)
    np.testing.assert_array_equal(nonpow3.bandwidth_optimal_torus(V, dims),
                                  allreduce.bandwidth_optimal(V, dims))
    np.testing.assert_array_equal(nonpow3.link_loads_torus(dims), congestion.link_loads(dims, "B"))


@pytest.mark.parametrize("n", [4, 7, 8, 16])
def test_torus_with_unit_side_is_the_ring(n):
    """A side of 1 takes no steps: both collectives of a 1 x n torus run the ring of n on their
    own segment, bit for bit, and a 1-dimensional torus is the ring itself."""
    from oracle import partition

    V = np.random.default_rng(n).standard_normal((n, 128 * n + 9), dtype=np.float32)
    seg, blk = partition.column_labels(V.shape[1], 2, n)
    np.testing.assert_array_equal(nonpow3.bandwidth_optimal_torus(V, (1, n)),
                                  nonpow3.bandwidth_optimal_ring(V, col_blk=blk))
    np.testing.assert_array_equal(nonpow3.bandwidth_optimal_torus(V, (n,)),
                                  nonpow3.bandwidth_optimal_ring(V))
    np.testing.assert_array_equal(nonpow3.link_loads_torus((n,)), nonpow3.link_loads_ring(n))


@pytest.mark.parametrize("dims", [(4, 4), (8, 8), (5, 7), (8, 3), (4, 4, 4)])
def test_torus_congestion_per_dimension(dims):
    """Every pass loads only the links of the collectives' active dimensions, each used link by
    its distance times the number of collectives working on that dimension at that step (one
    message per rank, direction and collective), and the all-gather mirrors the reduce-scatter."""
    D = len(dims)
    loads = congestion.link_loads(dims, "B")
    S = sum(nonpow3.dim_steps(s) for s in dims)
    assert loads.shape == (2 * S, int(np.prod(dims)), 2 * D)
    rot = [nonpow3.torus_rotation(dims, c) for c in range(D)]
    for t in range(S):
        for dim in range(D):
            users = [nonpow3.distances(dims[dim])[rot[c][t][1]] for c in range(D)
                     if rot[c][t][0] == dim]
            for p in (t, 2 * S - 1 - t):
                for port in (2 * dim, 2 * dim + 1):
                    col = loads[p, :, port]
                    sums = {sum(x for x, b in zip(users, bits) if b)
                            for bits in itertools.product((0, 1), repeat=len(users))}
                    assert (col == col[0]).all() and int(col[0]) in sums
        np.testing.assert_array_equal(loads[t].sum(axis=0)[0::2] + loads[t].sum(axis=0)[1::2],
                                      loads[2 * S - 1 - t].sum(axis=0)[0::2]
                                      + loads[2 * S - 1 - t].sum(axis=0)[1::2])


@pytest.mark.parametrize("dims", [(4, 4), (2, 3), (5, 7), (8, 3), (1, 8), (4, 4, 4), (2, 3, 4),
                                  (2, 2, 2, 2), (3, 3), (9, 3), (3, 3, 3), (7,), (8,)])
@pytest.mark.parametrize("dtype", ["f32", "i32"])
def test_torus_gather_form_equals_mailbox_form(dims, dtype):
    """The gather form used for thousands of ranks is the mailbox form, bit for bit (fp32 sums
    in the same association), with the same message statistics and link loads."""
    from oracle import partition

    n = int(np.prod(dims))
    E = 64 * len(dims) * n + 37
    rng = np.random.default_rng(3 * n + len(dims))
    if dtype == "f32":
        V = rng.standard_normal((n, E), dtype=np.float32)
    else:
        V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    seg, blk = partition.column_labels(E, len(dims), n)
    a = nonpow3.bandwidth_optimal_torus_columns(V, dims, seg, blk)
    b = nonpow3.bandwidth_optimal_torus(V, dims)
    np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))
    np.testing.assert_array_equal(nonpow3.link_loads_torus(dims, "columns"),
                                  nonpow3.link_loads_torus(dims, "mailbox"))


@pytest.mark.parametrize("dims", [(8, 8), (10, 10), (16, 16), (8, 16), (5, 5, 5), (6, 6, 6),
                                  (350,)], ids=lambda d: "x".join(map(str, d)))
def test_gather_form_equals_mailbox_form_on_larger_shapes(dims):
    """The same pin on the shapes between the small ones above and the 1024- and 4096-rank
    workloads the gather form checks alone (and on a ring above the 300 ranks where the GPU tests
    switch to it): one column per block, so every partial of every block is compared."""
    n = int(np.prod(dims))
    D = len(dims)
    seg = np.repeat(np.arange(D), n)
    blk = np.tile(np.arange(n), D)
    V = (np.random.default_rng(n + D).standard_normal((n, D * n)) *
         np.logspace(-4, 4, D * n)).astype(np.float32)
    a = nonpow3.bandwidth_optimal_torus_columns(V, dims, seg, blk)
    if D == 1:
        b = nonpow3.bandwidth_optimal_ring(V, col_blk=blk)
    else:
        b = nonpow3.bandwidth_optimal_torus(V, dims, seg, blk)
    np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))


def test_rectangular_tree_torus_final_steps_share_the_long_dimension():
    """8 x 64 under the rotation rule for unequal step counts: the side of 8 is done after two
    steps of each collective, so both collectives take the last two steps of the side of 64
    together (distances 9 and then 19 = ceil((64 - 27) / 2)), doubling those links' loads."""
    loads = congestion.link_loads((8, 64), "B")
    assert [int(loads[p].max()) for p in range(6)] == [1, 1, 3, 3, 18, 38]
    assert (loads[5][:, 2:] == 38).all() and (loads[5][:, :2] == 0).all()
