"""Pins of the oracle's AllReduce results (CPU only).

Integers: the method reaches the plain definition exactly (Sec. 2.2 + Theorem 1), so the oracle
is compared with a brute-force column sum. Floating point: the paper fixes no summation order;
the oracle's order (own + left) + right is a reading, pinned here by
  (a) the classical summation error bound against an fp64 sum,
  (b) n = 3, where one joint reduction is the whole AllReduce,
  (c) the explicit n = 9 tree that follows from the worked example of Sec. 4.3,
  (d) values for which a different association gives a different float,
  (e) cross-variant identities (the bandwidth-optimal block j is reduced by the same tree as the
      latency-optimal result of rank j, and the all-gather copies bits unchanged),
  (f) ring shift-equivariance,
  (g) exactly representable float inputs, where every association gives the exact sum.
"""

import numpy as np
import pytest

from oracle import allreduce, partition, schedule

TOPOS = [(1,), (3,), (9,), (27,), (81,), (3, 3), (9, 9), (3, 3, 3), (3, 9), (27, 3), (3, 9, 3)]
ELEMS = [0, 1, 3, 63, 64, 65, 200, 1023]


@pytest.mark.parametrize("dims", TOPOS)
@pytest.mark.parametrize("variant", ["L", "B"])
def test_int32_equals_bruteforce_sum(dims, variant):
    rng = np.random.default_rng(31 * sum(dims) + len(dims) + (0 if variant == "L" else 1000))
    n = schedule.Torus(dims).n
    for E in ELEMS:
        V = rng.integers(-1000, 1000, size=(n, E), dtype=np.int32)
        out = allreduce.allreduce(V, dims, variant)
        np.testing.assert_array_equal(out, np.broadcast_to(allreduce.exact_int_sum(V), out.shape))


@pytest.mark.parametrize("variant", ["L", "B"])
def test_int32_wraps_like_twos_complement(variant):
    rng = np.random.default_rng(7)
    V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(27, 300), dtype=np.int32)
    out = allreduce.allreduce(V, (27,), variant)
    want = (V.astype(np.int64).sum(axis=0) % 2 ** 32).astype(np.uint32).view(np.int32)
    np.testing.assert_array_equal(out, np.broadcast_to(want, out.shape))


def test_9x9x9_int32_small():
    rng = np.random.default_rng(3)
    V = rng.integers(-(2 ** 20), 2 ** 20, size=(729, 3 * 64 + 5), dtype=np.int32)
    out = allreduce.allreduce(V, (9, 9, 9), "B")
    np.testing.assert_array_equal(out, np.broadcast_to(allreduce.exact_int_sum(V), out.shape))


@pytest.mark.parametrize("dims", [(9,), (27,), (81,), (3, 3), (9, 9), (3, 3, 3)])
@pytest.mark.parametrize("variant", ["L", "B"])
def test_fp32_within_summation_bound(dims, variant):
    """(a): |fp32 - exact| <= 4 ceil(log3 n) 2^-23 sum|v| per column."""
    rng = np.random.default_rng(11)
    t = schedule.Torus(dims)
    V = rng.standard_normal((t.n, 64 * t.n + 17), dtype=np.float32)
    out = allreduce.allreduce(V, dims, variant).astype(np.float64)
    err = np.abs(out - allreduce.fp64_sum(V)[None, :])
    assert (err <= allreduce.fp32_error_bound(V)[None, :]).all()


def test_n3_is_one_joint_reduction():
    """(b): with n = 3 there is one step; rank r reduces (v_r + v_{r-1}) + v_{r+1} (L), and
    block j is finished at its owner j by the same expression (B)."""
    rng = np.random.default_rng(5)
    E = 3 * 64
    V = rng.standard_normal((3, E), dtype=np.float32)
    L = allreduce.allreduce(V, (3,), "L")
    for r in range(3):
        want = (V[r] + V[(r - 1) % 3]) + V[(r + 1) % 3]
        np.testing.assert_array_equal(L[r], want)
    B = allreduce.allreduce(V, (3,), "B")
    _, blk = partition.column_labels(E, 1, 3)
    for j in range(3):
        m = blk == j
        want = (V[j, m] + V[(j - 1) % 3, m]) + V[(j + 1) % 3, m]
        for r in range(3):
            np.testing.assert_array_equal(B[r, m], want)


def test_n9_tree_of_rank0():
    """(c): Sec. 4.3 example: after step 0 node 0 holds (v0 + v8) + v1, node 3 holds
    (v3 + v2) + v4 and node 6 holds (v6 + v5) + v7; in step 1 node 0 combines its partial with
    the one from node 6 (its left peer at distance 3) and then the one from node 3."""
    rng = np.random.default_rng(9)
    V = (rng.standard_normal((9, 256)) * np.logspace(-6, 6, 256)).astype(np.float32)
    v = V
    want = (((v[0] + v[8]) + v[1]) + ((v[6] + v[5]) + v[7])) + ((v[3] + v[2]) + v[4])
    L = allreduce.allreduce(V, (9,), "L")
    np.testing.assert_array_equal(L[0], want)
    # B: block 0 is finished at rank 0 by the same tree
    B = allreduce.allreduce(V, (9,), "B")
    _, blk = partition.column_labels(256, 1, 9)
    np.testing.assert_array_equal(B[0, blk == 0], want[blk == 0])


def test_association_is_observable():
    """(d): 1 + 2^-24 rounds to 1 (ties to even), so (1 + e) + e = 1 while 1 + (e + e) = 1 + 2^-23.
    With v_r = 1 and both neighbours e, the oracle's order yields exactly 1."""
    e = np.float32(2.0 ** -24)
    V = np.array([[1.0], [e], [e]], dtype=np.float32)  # rank 0 own = 1, left = rank 2, right = rank 1
    L = allreduce.allreduce(V, (3,), "L")
    assert L[0, 0] == np.float32(1.0)
    assert np.float32(1.0) + (e + e) != np.float32(1.0)


@pytest.mark.parametrize("dims", [(9,), (27,), (81,), (9, 9), (3, 3, 3), (3, 27), (9, 3, 3)])
def test_bandwidth_variant_block_equals_latency_variant_owner(dims):
    """(e): block j of the B result equals, bit for bit, rank j's L result; and B leaves every rank
    with identical bits."""
    rng = np.random.default_rng(13)
    t = schedule.Torus(dims)
    E = 2 * 64 * t.n + 29
    V = rng.standard_normal((t.n, E), dtype=np.float32)
    L = allreduce.allreduce(V, dims, "L")
    B = allreduce.allreduce(V, dims, "B")
    assert (B == B[0:1]).all()
    seg, blk = partition.column_labels(E, t.D, t.n)
    for j in range(t.n):
        m = blk == j
        np.testing.assert_array_equal(B[0, m], L[j, m])


@pytest.mark.parametrize("n", [9, 27, 81])
def test_latency_variant_shift_equivariant(n):
    """(f): relabelling ranks by a cyclic shift relabels the results the same way."""
    rng = np.random.default_rng(17)
    V = rng.standard_normal((n, 100), dtype=np.float32)
    L = allreduce.allreduce(V, (n,), "L")
    for s in (1, 2, n // 3):
        Ls = allreduce.allreduce(np.roll(V, s, axis=0), (n,), "L")
        np.testing.assert_array_equal(Ls, np.roll(L, s, axis=0))


@pytest.mark.parametrize("dims", [(27,), (9, 9), (3, 3, 3)])
@pytest.mark.parametrize("variant", ["L", "B"])
def test_exact_small_integers_in_float(dims, variant):
    """(g): small integers in fp32 add exactly, so any correct schedule gives the exact sum."""
    rng = np.random.default_rng(19)
    t = schedule.Torus(dims)
    V = rng.integers(-1000, 1000, size=(t.n, 500)).astype(np.float32)
    out = allreduce.allreduce(V, dims, variant)
    np.testing.assert_array_equal(out, np.broadcast_to(V.astype(np.float64).sum(0), out.shape))


def test_column_sample_matches_full_run():
    """Verification of huge runs uses column samples with their original labels; the sampled
    emulation must reproduce the full emulation on those columns."""
    rng = np.random.default_rng(23)
    dims, E = (9, 9), 3000
    t = schedule.Torus(dims)
    V = rng.standard_normal((t.n, E), dtype=np.float32)
    full = allreduce.allreduce(V, dims, "B")
    cols = np.sort(rng.choice(E, 50, replace=False))
    seg, blk = partition.column_labels(E, t.D, t.n, cols)
    part = allreduce.bandwidth_optimal(V[:, cols], dims, col_seg=seg, col_blk=blk)
    np.testing.assert_array_equal(part, full[:, cols])
    fullL = allreduce.allreduce(V, dims, "L")
    partL = allreduce.latency_optimal(V[:, cols], dims, col_seg=seg)
    np.testing.assert_array_equal(partL, fullL[:, cols])


def test_partition_rule_examples():
    """The block partition reading on the workload shapes: 27x27 torus, 4 MiB per rank."""
    bb = partition.block_bounds(1_048_576, 2, 729)
    sizes = {e - b for row in bb for (b, e) in row}
    assert sizes == {704, 768}
    assert partition.segment_bounds(1_048_576, 2) == [(0, 524288), (524288, 1048576)]
    bb5 = partition.block_bounds(33_554_432, 3, 729)
    assert {e - b for row in bb5 for (b, e) in row} == {15296, 15360}
    bb3 = partition.block_bounds(8_388_608, 1, 243)
    assert {e - b for row in bb3 for (b, e) in row} == {34496, 34560}
    # ragged: every element is covered once, blocks are contiguous and ordered
    for E, D, n in [(1, 1, 3), (65, 2, 9), (1000, 3, 27), (0, 1, 9)]:
        flat = [be for row in partition.block_bounds(E, D, n) for be in row]
        pos = 0
        for b, e in flat:
            assert b == pos and e >= b
            pos = e
        assert pos == E
