"""The Sec. 4.4 reduction trees (rings whose size is not a power of three) checked by brute force,
CPU only.

Sec. 4.4 fixes the steps (distances 3^0 .. 3^(f-1), then a final one at d = ceil((n - 3^f) / 2))
and states that every block is forwarded at most once per phase. Which partials travel where is
left open; the oracle (oracle/nonpow3.py) and the plan (csrc/plan.cpp) build one tree per block
from a reading. This file checks that reading against everything the paper's constraints allow,
with code that shares nothing with either side: it enumerates, for small n, every reduction tree
a schedule with those steps can have, directly from the definition.

A tree of block 0 gives every other offset o one forward: at some step k, to o - e d_k (e = +/-1,
d_k the step's distance). Following the forwards from o must reach 0, each at a later step than
the one before (a rank forwards after it has received from all its children, Sec. 4.3), and must
not pass through 0 on the way (the owner never forwards its own block in the reduce-scatter).
So a tree is one digit vector e in {-1, 0, 1}^S per offset with sum_k e_k d_k = o (mod n), such
that zeroing the lowest non-zero digit of any offset's vector gives its parent's vector. Each
rank then forwards each block exactly once, which is the paper's at-most-once bound.

The offsets o whose path to 0 does not use the final step are the contributions the owner holds
before the final step. Sec. 4.4 counts 27 of 32 for n = 32, i.e. the whole window |o| <= R,
R = (3^f - 1) / 2. The tests show that with single forwarding that count is impossible whenever
d <= R (as for 32, where d = 3 <= R = 13), and that the reading's tree holds as many contributions
before the final step as any valid tree does.
"""

import itertools
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import nonpow3

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2602_17254_amd")


# ---- the definition, written out independently ----

def _steps(n):
    """(f, d, distances) of Sec. 4.4: f full steps at 3^k, then d = ceil((n - 3^f) / 2) (none
    when n is a power of three)."""
    f, p = 0, 1
    while p * 3 <= n:
        p *= 3
        f += 1
    d = 0 if p == n else (n - p + 1) // 2
    return f, d, [3 ** k for k in range(f)] + ([d] if d else [])


def _paths(n):
    """offset -> every digit vector that can carry it to 0 (see the module docstring)."""
    _, _, dist = _steps(n)
    out = {o: [] for o in range(1, n)}
    for e in itertools.product((-1, 0, 1), repeat=len(dist)):
        o = sum(x * w for x, w in zip(e, dist)) % n
        if o == 0:
            continue
        cur, pos, ok = list(e), o, True
        while any(cur):
            k = next(i for i, x in enumerate(cur) if x)
            pos = (pos - cur[k] * dist[k]) % n
            cur[k] = 0
            if pos == 0 and any(cur):
                ok = False
                break
        if ok:
            out[o].append(tuple(e))
    return out


def _edge(n, o, e):
    """(step, parent) of offset o with digit vector e."""
    _, _, dist = _steps(n)
    k = next(i for i, x in enumerate(e) if x)
    return k, (o - e[k] * dist[k]) % n


def valid_trees(n):
    """Every reduction tree of block 0 on a ring of n, as {offset: (step, parent)}."""
    cand = _paths(n)
    offs = sorted(cand)
    trees = []
    for choice in itertools.product(*(cand[o] for o in offs)):
        vec = dict(zip(offs, choice))
        ok = True
        for o, e in vec.items():
            k, par = _edge(n, o, e)
            if par != 0:
                want = tuple(0 if i == k else x for i, x in enumerate(e))
                if vec[par] != want:
                    ok = False
                    break
        if ok:
            trees.append({o: _edge(n, o, e) for o, e in vec.items()})
    return trees


def held_before_final(n, tree):
    """Offsets (0 included) whose contribution reaches the owner without the final step."""
    f, d, _ = _steps(n)
    if d == 0:
        return set(range(n))
    out = {0}
    for o in tree:
        x, last = o, None
        while x != 0:
            last, x = tree[x]
        if last < f:
            out.add(o)
    return out


def window(n):
    f, _, _ = _steps(n)
    R = (3 ** f - 1) // 2
    return {o % n for o in range(-R, R + 1)}


# ---- the two implementations under test ----

def oracle_tree(n):
    """The oracle's tree of block 0: where each contribution first moves."""
    S = len(nonpow3.distances(n))
    tree = {}
    for u in range(1, n):
        for k in range(S):
            a, b = nonpow3.position(n, u, 0, k), nonpow3.position(n, u, 0, k + 1)
            if a != b:
                tree[u] = (k, b)
                break
    return tree


def plan_trees(sides, tmp):
    """The plan's trees, read from tests/c/tree_tables.cpp (plan.cpp built with g++)."""
    exe = os.path.join(tmp, "tree_tables")
    if not os.path.exists(exe):
        csrc = os.path.join(PKG, "csrc")
        subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Wextra", "-Werror", "-I", csrc,
                        "-I", os.path.join(ROOT, "include"),
                        os.path.join(ROOT, "tests", "c", "tree_tables.cpp"),
                        os.path.join(csrc, "plan.cpp"), "-o", exe], check=True)
    res = subprocess.run([exe] + [str(s) for s in sides], capture_output=True, text=True,
                         timeout=120, check=True)
    out, side, dist = {}, None, None
    for line in res.stdout.splitlines():
        w = line.split()
        if w[0] == "tree":
            side, dist = int(w[1]), [int(x) for x in w[3:]]
            out[side] = {"dist": dist, "tree": {}, "alive": {}, "recv": {}}
        elif w[0] == "recv":
            k = int(w[1])
            out[side]["recv"][k] = {}
            for item in w[2:]:
                o, fl = item.split(":")
                o = int(o)
                out[side]["recv"][k][o] = fl
                if "L" in fl:  # the child at o - d moves towards + onto o
                    out[side]["tree"][(o - dist[k]) % side] = (k, o)
                if "R" in fl:
                    out[side]["tree"][(o + dist[k]) % side] = (k, o)
        elif w[0] == "alive":
            out[side]["alive"][int(w[1])] = sorted(int(x) for x in w[2:])
    return out


@pytest.fixture(scope="module")
def plans(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ not found")
    tmp = str(tmp_path_factory.mktemp("trees"))
    return plan_trees(list(range(2, 201)) + [728, 2200], tmp)


def tree_sum(V0, recv, dist):
    """Block 0's value at its owner, evaluated directly from a tree: a rank starts from its own
    contribution and, at every step at which it receives, adds the partial of the child on its
    left (the rank at -distance) and then that of the child on its right, absent ones skipped
    (Sec. 4.3's joint reduction); a child's partial is what it holds after its own earlier steps.
    fp32, IEEE round to nearest. V0: the (n, m) inputs of the block's columns."""
    n = V0.shape[0]

    def value(o, upto):
        v = V0[o].copy()
        for k in range(upto):
            fl = recv[k].get(o)
            if fl is None:
                continue
            if "L" in fl:
                v = v + value((o - dist[k]) % n, k)
            if "R" in fl:
                v = v + value((o + dist[k]) % n, k)
        return v

    return value(0, len(dist))


SMALL = [n for n in range(2, 28) if _steps(n)[1] != 0]


# ---- the enumeration itself against what the paper fixes ----

@pytest.mark.parametrize("n", [3, 9, 27])
def test_power_of_three_has_exactly_the_ordinary_tree(n):
    """With n = 3^s the definition admits one tree only: each offset forwards at the step of its
    lowest non-zero balanced-ternary digit (the closed form of Sec. 4.3), and the owner holds
    everything after the last step (Theorem 1)."""
    trees = valid_trees(n)
    assert len(trees) == 1
    s = _steps(n)[0]
    for o, (k, par) in trees[0].items():
        v, digits = (o + (n - 1) // 2) % n - (n - 1) // 2, []
        for _ in range(s):
            r = ((v % 3) + 3) % 3
            digits.append(-1 if r == 2 else r)
            v = (v - digits[-1]) // 3
        k0 = next(i for i, x in enumerate(digits) if x)
        assert (k, par) == (k0, (o - digits[k0] * 3 ** k0) % n)


@pytest.mark.parametrize("n", SMALL)
def test_every_enumerated_tree_is_a_reduction_tree(n):
    """n - 1 forwards, every path reaches the owner with increasing steps and the listed
    distances, and no rank receives two partials of the block from one side in one step."""
    _, _, dist = _steps(n)
    trees = valid_trees(n)
    assert trees
    for tree in trees:
        assert sorted(tree) == list(range(1, n))
        seen = set()
        for o, (k, par) in tree.items():
            assert (o - par) % n in (dist[k] % n, (-dist[k]) % n)
            side = +1 if (par - o) % n == dist[k] % n else -1
            assert (k, par, side) not in seen
            seen.add((k, par, side))
            if par != 0:
                assert tree[par][0] > k


# ---- the oracle's and the plan's trees are among them ----

@pytest.mark.parametrize("n", SMALL)
def test_oracle_and_plan_trees_are_valid_schedules(n, plans):
    trees = valid_trees(n)
    mine = oracle_tree(n)
    assert mine in trees
    assert plans[n]["tree"] == mine
    assert plans[n]["dist"] == _steps(n)[2]


@pytest.mark.parametrize("n", list(range(28, 201)) + [728, 2200])
def test_plan_trees_are_reduction_trees_beyond_enumeration(n, plans):
    """Larger rings: the plan's tree has the Sec. 4.4 distances, one forward per offset, steps
    increasing towards the owner, every path reaching it, and its not-yet-forwarded lists are
    the offsets whose forward comes at that step or later."""
    _, _, dist = _steps(n)
    p = plans[n]
    assert p["dist"] == dist
    tree = p["tree"]
    assert sorted(tree) == list(range(1, n))
    for o, (k, par) in tree.items():
        assert (o - par) % n in (dist[k] % n, (-dist[k]) % n)
        if par != 0:
            assert tree[par][0] > k
        x, hops = o, 0
        while x != 0:
            x = tree[x][1]
            hops += 1
            assert hops <= len(dist)
    S = len(dist)
    for m in range(S + 1):
        want = sorted([0] + [o for o, (k, _) in tree.items() if k >= m])
        assert p["alive"][m] == want


# ---- the paper's 27-of-32 count ----

# n: the whole 3^f window can be held before the final step by some tree (from the enumeration)
WINDOW_REACHABLE = {2, 6, 7, 8, 18, 19, 20, 21, 24, 25, 26}


@pytest.mark.parametrize("n", SMALL)
def test_reading_holds_the_most_before_the_final_step(n):
    """Sec. 4.4 counts the owner's whole 3^f window as held before the final step. Among all
    trees single forwarding allows, the reading's tree holds as many contributions before the
    final step as any (the maximum of the enumeration), and the whole window whenever some tree
    can. The window cannot be held when d <= R (the argument of the 32-ring below), nor for
    n = 22, 23, where reaching +/-7 within two steps passes through the window."""
    f, d, _ = _steps(n)
    R = (3 ** f - 1) // 2
    W = window(n)
    trees = valid_trees(n)
    best = max(len(held_before_final(n, t)) for t in trees)
    mine = held_before_final(n, oracle_tree(n))
    assert len(mine) == best
    reachable = any(held_before_final(n, t) == W for t in trees)
    assert reachable == (n in WINDOW_REACHABLE)
    if d <= R:
        assert not reachable
    assert (mine == W) == reachable


def test_n32_owner_holds_15_of_32_before_the_final_step():
    """Reading 13 on the 32-ring: the owner of a block holds 15 of the 32 contributions before the
    final step, 17 arrive in it (through the ranks at +/-3), and each rank forwards each block
    exactly once (31 forwards per block).

    Sec. 4.4 counts 27 held and 5 arriving. That count is not taken, because with single
    forwarding it cannot happen when d <= R (here d = 3, R = 13):
      (a) within the first f = 3 steps a contribution moves by at most sum 3^k = 13, so the
          contributions that reach the owner before the final step lie in the window |o| <= 13;
      (b) in the final step only the ranks at +3 and -3 can send to the owner, and both lie in
          that window;
      (c) if the owner held the whole window before the final step, +3 and -3 would have
          forwarded their partials of the block already and send nothing in the final step, so
          the owner would end with 27 of 32 contributions.
    Keeping the 27 would need the ranks at +/-3 to forward the block twice (once inside the
    window, once with the 5 outer contributions): 35 forwards per block instead of 31."""
    n = 32
    f, d, dist = _steps(n)
    R = (3 ** f - 1) // 2
    assert (f, d, R) == (3, 3, 13)
    # (a) every offset reachable with the first f steps lies in the window, and all of it is
    reach = {sum(e * 3 ** k for k, e in enumerate(v)) % n
             for v in itertools.product((-1, 0, 1), repeat=f)}
    assert reach == window(n) and len(reach) == 27
    # (b) the final step's senders into 0 are +/-d, inside the window
    assert {d % n, (-d) % n} <= window(n)
    # the reading's tree
    mine = oracle_tree(n)
    assert sorted(mine) == list(range(1, n))  # one forward per offset: 31 per block
    held = held_before_final(n, mine)
    assert len(held) == 15 and held < window(n)
    final_senders = {o for o, (k, _) in mine.items() if k == f}
    assert final_senders == {d, n - d}


# sizes where no distance equals n / 2 (there a child's side is a matter of naming only)
TREE_SUM_SIZES = [4, 5, 7, 8, 10, 11, 13, 14, 16, 20, 22, 23, 28, 32, 40, 50, 64, 80, 100, 128, 200]


@pytest.mark.parametrize("n", TREE_SUM_SIZES)
def test_oracle_arithmetic_is_the_plan_trees_sum(n, plans):
    """The oracle's fp32 results on rings whose size is not a power of three equal, bit for bit,
    block 0's sum evaluated directly from the plan's own tree tables (tree_sum above, code that
    shares nothing with the oracle's mailbox emulation). With every column labelled block 0 the
    bandwidth-optimal result on every rank is that sum. Inputs span twelve orders of magnitude so
    that any other association or side order would change bits."""
    _, _, dist = _steps(n)
    assert all((2 * d) % n for d in dist)
    p = plans[n]
    E = 96
    V = (np.random.default_rng(1000 + n).standard_normal((n, E)) *
         np.logspace(-6, 6, E)[None, :] * np.logspace(-3, 3, n)[:, None]).astype(np.float32)
    want = tree_sum(V, p["recv"], p["dist"])
    got = nonpow3.bandwidth_optimal_ring(V, col_blk=np.zeros(E, dtype=np.int64))
    for r in range(n):
        assert np.array_equal(got[r].view(np.uint32), want.view(np.uint32)), r
    naive = V[0].copy()
    for u in range(1, n):
        naive = naive + V[u]
    assert not np.array_equal(naive.view(np.uint32), want.view(np.uint32))


TORUS_SUM = [(4, 4), (5, 7), (3, 8), (8, 3), (2, 3, 4), (8, 8), (10, 3, 3), (4, 4, 4), (2, 2, 2, 2)]


def torus_sum(V0, dims, steps, recv, dist):
    """Block 0's value at its owner on a torus, evaluated directly: steps[t] = (dimension, level)
    of collective c's step t (the plan's rotation); recv[side] / dist[side] the plan's tree of a
    side. A rank holding the block's partial receives, at a step along dimension a, from the
    children its offset along a has at that level in a's tree (left before right); dimension 0
    is the fastest-varying coordinate."""
    n = V0.shape[0]
    D = len(dims)
    stride = [1] * D
    for d in range(1, D):
        stride[d] = stride[d - 1] * dims[d - 1]

    def move(x, a, delta):
        xa = (x // stride[a]) % dims[a]
        return x + (((xa + delta) % dims[a]) - xa) * stride[a]

    def value(x, upto):
        v = V0[x].copy()
        for t in range(upto):
            a, k = steps[t]
            side = dims[a]
            fl = recv[side][k].get((x // stride[a]) % side)
            if fl is None:
                continue
            if "L" in fl:
                v = v + value(move(x, a, -dist[side][k]), t)
            if "R" in fl:
                v = v + value(move(x, a, +dist[side][k]), t)
        return v

    return value(0, len(steps))


@pytest.mark.parametrize("dims", TORUS_SUM, ids=lambda d: "x".join(map(str, d)))
def test_torus_oracle_arithmetic_is_the_plan_trees_sum(dims, tmp_path):
    """The torus form: for every collective, the oracle's fp32 result (mailbox emulation, and the
    gather form used for large tori) equals, bit for bit, block 0's sum evaluated from the plan's
    per-side trees in the order of the plan's rotation (trivance_plan_step)."""
    T = pytest.importorskip("paper_2602_17254_amd")
    if shutil.which("g++") is None:
        pytest.skip("g++ not found")
    sides = sorted(set(dims) - {1})
    trees = plan_trees(sides, str(tmp_path))
    plan = T.trivance_plan(dims, "B")
    D, n = len(dims), int(np.prod(dims))
    E = 96
    V = (np.random.default_rng(7 * n + D).standard_normal((n, E)) *
         np.logspace(-6, 6, E)[None, :] * np.logspace(-3, 3, n)[:, None]).astype(np.float32)
    recv = {s: trees[s]["recv"] for s in sides}
    dist = {s: trees[s]["dist"] for s in sides}
    for c in range(D):
        level = [0] * D
        steps = []
        for t in range(plan.num_steps):
            _, a, d = T.trivance_plan_step(plan, t, c)
            assert d == dist[dims[a]][level[a]]
            steps.append((a, level[a]))
            level[a] += 1
        want = torus_sum(V, dims, steps, recv, dist)
        seg = np.full(E, c, dtype=np.int64)
        blk = np.zeros(E, dtype=np.int64)
        for got in (nonpow3.bandwidth_optimal_torus(V, dims, col_seg=seg, col_blk=blk),
                    nonpow3.bandwidth_optimal_torus_columns(V, dims, seg, blk)):
            for r in range(n):
                assert np.array_equal(got[r].view(np.uint32), want.view(np.uint32)), (c, r)
