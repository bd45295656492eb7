"""Pins of the oracle's schedule against what the paper fixes (CPU only)."""

import json
import os

import numpy as np
import pytest

from oracle import allreduce, partition, schedule

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RINGS = [3, 9, 27, 81, 243]


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


@pytest.mark.parametrize("dims,S", [((1,), 0), ((3,), 1), ((9,), 2), ((81,), 4), ((243,), 5),
                                    ((27, 27), 6), ((9, 9, 9), 6), ((3, 3), 2)])
def test_step_count_is_log3_n(dims, S):
    """Theorem 1: n = 3^s needs s steps; the torus runs log3(n) steps in total (Sec. 5)."""
    t = schedule.Torus(dims)
    assert t.steps == S
    assert 3 ** t.steps == t.n
    assert len(schedule.pass_list(t, "L")) == S
    assert len(schedule.pass_list(t, "B")) == 2 * S  # Sec. 3.2: 2 log3 n steps for RS + AG


def test_non_power_of_three_rejected():
    for bad in (2, 4, 8, 10, 32):
        with pytest.raises(ValueError):
            schedule.Torus((bad,))


def test_ring_peers_are_pm_3k():
    """Sec. 4.1: pi(r, k, n) = (r - 3^k, r + 3^k) mod n."""
    for n in RINGS:
        t = schedule.Torus((n,))
        for k in range(t.steps):
            for r in range(n):
                assert schedule.peers(t, 0, r, k) == ((r - 3 ** k) % n, (r + 3 ** k) % n)


@pytest.mark.parametrize("n", RINGS)
def test_algorithm1_matches_closed_form(n):
    """Sec. 4.3: the message blocks (the step-by-step reachability), Algorithm 1's recursive
    BlockPropagation (plus the receiver it never marks) and the closed form Pi(n, r, p, k) are
    the same sets, and a message at step k carries 3^(s-1-k) blocks."""
    t = schedule.Torus((n,))
    s = t.steps
    for k in range(s):
        for r in range(n):
            for p in schedule.peers(t, 0, r, k):
                blocks = schedule.message_blocks(t, 0, p, k)
                assert blocks == schedule.pi_closed_form_ring(n, p, k)
                assert blocks == sorted({p} | set(schedule.reach(t, 0, p, k + 1)))
                assert len(blocks) == 3 ** (s - 1 - k)


@pytest.mark.parametrize("dims", [(3, 3), (9, 9), (3, 3, 3), (3, 9), (9, 3, 3), (27, 3)])
def test_algorithm1_matches_reachability_on_tori(dims):
    """On tori (Sec. 5) the step-by-step reachability and Algorithm 1 over the collective's step
    list give the same block sets for every collective, receiver and step."""
    t = schedule.Torus(dims)
    for c in range(t.D):
        for k in range(t.steps):
            for p in range(t.n):
                assert schedule.message_blocks(t, c, p, k) == \
                    sorted({p} | set(schedule.reach(t, c, p, k + 1)))


def test_n9_golden_message_sizes():
    g = _golden("n9_example.json")
    t = schedule.Torus((9,))
    assert t.steps == g["steps"]["value"]
    sizes = [len(schedule.message_blocks(t, 0, 1, k)) for k in range(t.steps)]
    assert sizes == g["blocks_per_message"]["value"]


def test_n9_golden_worked_example():
    """Sec. 4.3 example, replayed with one-hot integer inputs so that a value of 1 at column u
    means 'holds data of node u exactly once'."""
    g = _golden("n9_example.json")
    V = np.eye(9, dtype=np.int32)
    trace = []
    after0 = allreduce.latency_optimal(V, (9,), passes=1)
    assert sorted(np.nonzero(after0[0])[0].tolist()) == g["node0_after_step0"]["value"]
    assert set(np.unique(after0)) <= {0, 1}
    final = allreduce.latency_optimal(V, (9,), trace=trace)
    step1_to0 = {src: np.nonzero(p)[0].tolist() for (t, c, src, dst, p) in trace
                 if t == 1 and dst == 0}
    assert sorted(step1_to0[3]) == g["node0_step1_via_node3"]["value"]
    assert sorted(step1_to0[6]) == g["node0_step1_via_node6"]["value"]
    assert g["all_covered_after_step"]["value"] == 1
    assert (final == 1).all()


@pytest.mark.parametrize("n", [9, 27, 81])
def test_lemma2_coverage_window(n):
    """Lemma 2: after step k, node r holds data of exactly the nodes within ring distance
    R_k = (3^(k+1) - 1) / 2, each once."""
    V = np.eye(n, dtype=np.int32)
    s = schedule.log3_exact(n)
    for k in range(s):
        out = allreduce.latency_optimal(V, (n,), passes=k + 1)
        Rk = (3 ** (k + 1) - 1) // 2
        for r in range(n):
            want = np.array([1 if schedule.ring_distance(u, r, n) <= Rk else 0
                             for u in range(n)], dtype=np.int32)
            np.testing.assert_array_equal(out[r], want)


@pytest.mark.parametrize("dims", [(3, 3), (9, 9), (3, 3, 3), (3, 9), (9, 3), (3, 3, 9)])
def test_torus_coverage_is_product_of_ring_windows(dims):
    """Sec. 5: each collective applies the ring pattern per dimension, so after some steps the
    covered sources are the product of per-dimension Lemma-2 windows (R = (3^k - 1) / 2 after k
    steps in a dimension), each source counted once."""
    t = schedule.Torus(dims)
    n, D = t.n, t.D
    # segment c spans granules [c n, (c+1) n) of 64 columns; its first n columns get a one-hot
    # marker per source rank
    Eh = n * D * 64
    seg_cols = [np.arange(c * n * 64, c * n * 64 + n) for c in range(D)]
    seg, _ = partition.column_labels(Eh, D, n)
    V = np.zeros((n, Eh), dtype=np.int32)
    for c in range(D):
        assert (seg[seg_cols[c]] == c).all()
        V[np.arange(n), seg_cols[c]] = 1
    for steps_done in range(t.steps + 1):
        out = allreduce.latency_optimal(V, dims, passes=steps_done)
        for c in range(D):
            kd = [0] * D
            for tt in range(steps_done):
                kd[schedule.step_dim_and_distance(t, c, tt)[0]] += 1
            for r in range(n):
                rc = t.coords(r)
                want = []
                for u in range(n):
                    uc = t.coords(u)
                    ok = all(schedule.ring_distance(uc[d], rc[d], dims[d]) <= (3 ** kd[d] - 1) // 2
                             for d in range(D))
                    want.append(1 if ok else 0)
                np.testing.assert_array_equal(out[r, seg_cols[c]], np.array(want, np.int32))


@pytest.mark.parametrize("dims", [(9,), (27,), (243,), (3, 3), (9, 9), (27, 27), (9, 9, 9),
                                  (3, 27), (9, 3, 3)])
def test_lemma1_bandwidth_and_reduction_volume(dims):
    """Lemma 1: a rank sends n - 1 blocks per reduce-scatter phase (m (1 - 1/n) bytes).
    Sec. 7 (reduction volume): the partial data reduced per rank sums to 1.5 m (1 - 1/n),
    i.e. 1.5 (n - 1) blocks."""
    t = schedule.Torus(dims)
    n = t.n
    stats = {}
    allreduce.bandwidth_optimal(np.zeros((n, 0), np.int32), dims, stats=stats)
    assert (stats["sent_blocks_rs"] == n - 1).all()
    assert (2 * stats["reduced_blocks_rs"] == 3 * (n - 1)).all()


def test_torus_message_sizes_shrink_by_three():
    """Sec. 5 + Appendix B: on a torus the data fraction of global step t is 3^-(t+1)."""
    for dims in [(3, 3), (9, 9), (27, 27), (9, 9, 9)]:
        t = schedule.Torus(dims)
        for c in range(t.D):
            for step in range(t.steps):
                assert len(schedule.message_blocks(t, c, 0, step)) * 3 ** (step + 1) == t.n


def test_dimension_rotation():
    """Sec. 5 (fig:trivanceexamplemultid): on a 9x9 torus the two collectives start on different
    dimensions, switch at step 1 and return at step 2; distance stays 1 for the first D steps."""
    t = schedule.Torus((9, 9))
    assert [schedule.step_dim_and_distance(t, 0, s) for s in range(4)] == [(0, 1), (1, 1), (0, 3), (1, 3)]
    assert [schedule.step_dim_and_distance(t, 1, s) for s in range(4)] == [(1, 1), (0, 1), (1, 3), (0, 3)]


@pytest.mark.parametrize("dims", [(3, 9), (9, 27), (27, 3), (3, 3, 9), (9, 3, 27)])
def test_rectangular_rotation_reading(dims):
    """Unequal sides (not covered by Sec. 5): every collective takes exactly log3(side) steps in
    each dimension, the k-th step in a dimension has distance 3^k, and while no dimension is
    exhausted the collectives use pairwise distinct dimensions (as in Sec. 5)."""
    t = schedule.Torus(dims)
    for c in range(t.D):
        seq = [schedule.step_dim_and_distance(t, c, s) for s in range(t.steps)]
        for d in range(t.D):
            dists = [dist for (dd, dist) in seq if dd == d]
            assert dists == [3 ** k for k in range(schedule.log3_exact(dims[d]))]
    short = min(schedule.log3_exact(d) for d in dims)
    for s in range(short * t.D):
        used = [schedule.step_dim_and_distance(t, c, s)[0] for c in range(t.D)]
        assert len(set(used)) == t.D
