"""Pins of the oracle for rings whose size is not a power of three (Sec. 4.4), CPU only."""

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


def test_n32_final_distance():
    """Sec. 4.4: 27 of 32 blocks before the final step; the 5 missing ones come from both sides,
    so the final distance is ceil(5 / 2) = 3."""
    f, d = nonpow3.levels(32)
    assert 3 ** f == _golden()["n32_blocks_before_final"]["value"]
    assert d == math.ceil((32 - 27) / 2) == 3


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
    S = len(nonpow3.distances(n))
    err = np.abs(out[0].astype(np.float64) - allreduce.fp64_sum(V))
    assert (err <= allreduce.fp32_error_bound(V, S)).all()


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


def test_latency_variant_rejected():
    with pytest.raises(ValueError):
        allreduce.allreduce(np.zeros((8, 4), np.float32), (8,), "L")
