"""Race freedom of the in-place bandwidth-optimal passes, checked on the host (CPU only).

Every reduce-scatter and all-gather pass updates the rank buffers in place, one work unit per
(collective, rank, block) pair, all units of a pass concurrently. That is safe only if, within a
pass, no location is written by two units and no location written by one unit is read by another
(Sec. 4.3's barrier is the kernel boundary; inside a pass there is no ordering). This file
enumerates the units of every pass as the kernels form them and checks both properties, plus that
every location a unit reads still holds a live partial (one that has not been forwarded yet).

* Power-of-three sides: the units of pass t are the pairs (centre r, block j) with j_d = r_d
  (mod 3^(steps collective c has taken along d up to and including t)) for every d, the closed
  form of Sec. 4.3 the block step decodes. The moduli are re-derived here from the plan's own
  introspection (trivance_plan_step: dimension and distance per pass and collective). A
  reduce-scatter unit reads (r, j), (r - d, j), (r + d, j) and writes (r, j); an all-gather unit
  reads (r, j) and writes (r - d, j) and (r + d, j).
* Sides that are not powers of three: the units come from the plan's reduction trees (printed by
  tests/c/tree_tables.cpp): at step k a receiver at offset o from the block's owner reads its own
  partial and those of the children at o - d / o + d that send, and writes o; the all-gather
  copies o back to those children.
Blocks are disjoint element ranges (checked from trivance_block_range), so disjoint (rank, block)
pairs are disjoint memory.

The latency-optimal step reads and writes every location of a pass: it is in place because each
thread owns whole (cycle, column) strips and loads every row of its strip before storing it (and
waves of one cycle exchange their boundary rows through LDS before any store); the slot steps of
sides that are not powers of three read one workspace state and write the other. Neither is a set
property of units, so neither is checked here; both are covered by the GPU parity tests.
"""

import os
import shutil
import sys

import pytest

T = pytest.importorskip("paper_2602_17254_amd")

POW3 = [(9,), (27,), (81,), (3, 3), (9, 9), (3, 3, 3), (3, 9), (9, 3), (3, 27), (3, 3, 9), (27, 27)]


def _coords(dims, r):
    out = []
    for s in dims:
        out.append(r % s)
        r //= s
    return tuple(out)


def _rank(dims, xs):
    r, stride = 0, 1
    for x, s in zip(xs, dims):
        r += (x % s) * stride
        stride *= s
    return r


def _check_pass(units_reads_writes, live):
    """units_reads_writes: list of (reads, writes) per unit, each a list of (rank, block)."""
    written = {}
    for u, (_, writes) in enumerate(units_reads_writes):
        for loc in writes:
            assert loc not in written, f"location {loc} written by two units"
            written[loc] = u
    for u, (reads, _) in enumerate(units_reads_writes):
        for loc in reads:
            assert written.get(loc, u) == u, f"location {loc} read by one unit, written by another"
            assert loc in live, f"location {loc} read after its partial was forwarded"


@pytest.mark.parametrize("dims", POW3, ids=lambda d: "x".join(map(str, d)))
def test_power_of_three_passes_are_race_free(dims):
    plan = T.trivance_plan(dims, "B")
    n, D = plan.n, plan.D
    S = plan.num_steps
    # blocks are disjoint element ranges that tile each segment
    E = 64 * D * n + 37
    for c in range(D):
        b0, e0 = T.trivance_block_range(plan, E, c, -1)
        spans = sorted(T.trivance_block_range(plan, E, c, j) for j in range(n))
        assert spans[0][0] == b0 and spans[-1][1] == e0
        assert all(a[1] == b[0] for a, b in zip(spans, spans[1:]))
    for c in range(D):
        taken = [0] * D
        moduli = []
        dist = []
        for t in range(S):
            _, dim, d = T.trivance_plan_step(plan, t, c)
            assert d == 3 ** taken[dim]
            taken[dim] += 1
            moduli.append([3 ** x for x in taken])
            dist.append((dim, d))
        # live before reduce-scatter step t: (r, j) with j = r mod the moduli before the step
        live = {(r, j) for r in range(n) for j in range(n)}
        for t in range(S):
            dim, d = dist[t]
            K = moduli[t]
            units = []
            keep = set()
            for r in range(n):
                xr = _coords(dims, r)
                for j in range(n):
                    xj = _coords(dims, j)
                    if all(xj[q] % K[q] == xr[q] % K[q] for q in range(D)):
                        rl = _rank(dims, [x - d if q == dim else x for q, x in enumerate(xr)])
                        rr = _rank(dims, [x + d if q == dim else x for q, x in enumerate(xr)])
                        units.append(([(r, j), (rl, j), (rr, j)], [(r, j)]))
                        keep.add((r, j))
            assert len(units) == n * n // 3 ** (t + 1)
            _check_pass(units, live)
            live = keep
        # after the reduce-scatter every rank keeps only its own block
        assert live == {(r, r) for r in range(n)}
        # all-gather steps t = S-1 .. 0: the same pairs send to both peers
        for t in reversed(range(S)):
            dim, d = dist[t]
            K = moduli[t]
            units = []
            for r in range(n):
                xr = _coords(dims, r)
                for j in range(n):
                    xj = _coords(dims, j)
                    if all(xj[q] % K[q] == xr[q] % K[q] for q in range(D)):
                        rl = _rank(dims, [x - d if q == dim else x for q, x in enumerate(xr)])
                        rr = _rank(dims, [x + d if q == dim else x for q, x in enumerate(xr)])
                        units.append(([(r, j)], [(rl, j), (rr, j)]))
            _check_pass(units, live)
            live = live | {w for _, ws in units for w in ws}
        assert live == {(r, j) for r in range(n) for j in range(n)}


@pytest.fixture(scope="module")
def trees(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ not found")
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import test_nonpow3_trees as tt

    return tt.plan_trees(list(range(2, 41)) + [64, 100, 728],
                         str(tmp_path_factory.mktemp("race")))


@pytest.mark.parametrize("n", [2, 4, 5, 7, 8, 10, 13, 20, 32, 40, 64, 100, 728])
def test_tree_passes_are_race_free(n, trees):
    """Rings whose size is not a power of three, from the plan's own trees (units of every block j
    at every step, with offsets taken relative to j)."""
    p = trees[n]
    tree, dist = p["tree"], p["dist"]
    S = len(dist)
    # blocks j at every offset: a unit is (block j, receiver offset o)
    recv = [{} for _ in range(S)]
    for child, (k, par) in tree.items():
        recv[k].setdefault(par, []).append(child)
    live = {(x, j) for x in range(n) for j in range(n)}
    for k in range(S):
        # the live partials agree with the plan's own table of offsets not yet forwarded
        if k in p["alive"]:
            assert live == {((j + o) % n, j) for o in p["alive"][k] for j in range(n)}
        units = []
        for j in range(n):
            for o, kids in recv[k].items():
                reads = [((j + o) % n, j)] + [((j + ch) % n, j) for ch in kids]
                units.append((reads, [((j + o) % n, j)]))
        _check_pass(units, live)
        # forwarded offsets are dead after the step
        sent = {ch for kids in recv[k].values() for ch in kids}
        live = {(x, j) for (x, j) in live if (x - j) % n not in sent}
    assert live == {(j, j) for j in range(n)}
    for k in reversed(range(S)):
        units = []
        for j in range(n):
            for o, kids in recv[k].items():
                units.append(([((j + o) % n, j)], [((j + ch) % n, j) for ch in kids]))
        _check_pass(units, live)
        live = live | {w for _, ws in units for w in ws}
    assert live == {(x, j) for x in range(n) for j in range(n)}


def test_checker_catches_a_planted_overlap():
    """A pass in which one unit writes a location another unit reads, and one in which a unit reads
    a forwarded partial, are both rejected."""
    live = {(0, 0), (1, 0), (2, 0)}
    with pytest.raises(AssertionError):
        _check_pass([([(0, 0), (1, 0)], [(0, 0)]), ([(1, 0)], [(1, 0)])], live)
    with pytest.raises(AssertionError):
        _check_pass([([(0, 0)], [(0, 0)]), ([(2, 0)], [(0, 0)])], live)
    with pytest.raises(AssertionError):
        _check_pass([([(0, 0), (3, 0)], [(0, 0)])], live)
