"""The C ABI without a GPU: the library loads, exports what include/trivance.h declares, and its
host-side schedule logic agrees with the oracle (CPU only; no kernel is launched)."""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2602_17254_amd as T
from oracle import partition, schedule

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def _built():
    if not os.path.exists(T.binding.LIB_PATH):
        import __graft_entry__

        __graft_entry__.build()
    yield


def test_exports_every_declared_symbol():
    with open(os.path.join(ROOT, "include", "trivance.h")) as f:
        header = f.read()
    declared = set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(trivance_\w+)\s*\(", header, re.M))
    assert len(declared) >= 14
    lib = ctypes.CDLL(T.binding.LIB_PATH)
    missing = [s for s in sorted(declared) if not hasattr(lib, s)]
    assert not missing, missing
    assert set(T.binding.exported_symbols()) == declared


@pytest.mark.parametrize("dims,variant", [((1,), "L"), ((3,), "B"), ((9,), "L"), ((81,), "L"),
                                          ((243,), "B"), ((27, 27), "B"), ((9, 9, 9), "B"),
                                          ((27, 27), "L"), ((9, 9, 9), "L"), ((81,), "BRUCK"),
                                          ((9, 27), "B"), ((27, 3), "L"), ((3, 9, 27), "B")])
def test_plan_matches_oracle_schedule(dims, variant):
    p = T.trivance_plan(dims, variant)
    t = schedule.Torus(dims)
    assert p.num_steps == t.steps
    plist = schedule.pass_list(t, "L" if variant == "BRUCK" else variant)
    assert p.num_passes == len(plist)
    phase_code = {"L": T.binding.PHASE_LATENCY, "RS": T.binding.PHASE_REDUCE_SCATTER,
                  "AG": T.binding.PHASE_ALLGATHER}
    for i, (ph, step) in enumerate(plist):
        for c in range(t.D):
            got = T.trivance_plan_step(p, i, c)
            dim, dist = schedule.step_dim_and_distance(t, c, step)
            assert got == (phase_code[ph], dim, dist)
        assert T.trivance_plan_step_index(p, i) == step


@pytest.mark.parametrize("E,dims", [(0, (9,)), (1, (9,)), (1000, (27,)), (64 * 243 * 3 + 17, (243,)),
                                    (1_048_576, (27, 27)), (33_554_432, (9, 9, 9)), (12345, (3, 3, 3))])
def test_block_range_matches_oracle_partition(E, dims):
    p = T.trivance_plan(dims, "B")
    n, D = p.n, p.D
    bb = partition.block_bounds(E, D, n)
    js = range(n) if n <= 81 else list(range(0, n, 7)) + [n - 1]
    for c in range(D):
        assert T.trivance_block_range(p, E, c, -1) == partition.segment_bounds(E, D)[c]
        for j in js:
            assert T.trivance_block_range(p, E, c, j) == bb[c][j]


@pytest.mark.parametrize("dims", [(9,), (81,), (243,), (27, 27), (9, 9, 9)])
def test_algorithmic_bytes(dims):
    """L: 2 S n E w per AllReduce; B: reduce-scatter step t reads n E w / 3^t and writes a third of
    it, all-gather step t reads n E w / 3^(t+1) and writes twice that: 3.5 w E (n - 1) in total
    (Sec. 7's reduction volume 1.5 m (1 - 1/n) per rank is the reduce-scatter read volume)."""
    n = int(np.prod(dims))
    S = schedule.Torus(dims).steps
    for E in (0, 1, 4096, 33_554_432):
        pl = T.trivance_plan(dims, "L")
        assert T.trivance_algorithmic_bytes(pl, E) == 2 * S * n * E * 4
        pb = T.trivance_plan(dims, "B")
        assert 2 * T.trivance_algorithmic_bytes(pb, E) == 7 * 4 * E * (n - 1)
        rs_reads = sum(3 * T.trivance_pass_bytes(pb, E, t) // 4 for t in range(S))
        assert 2 * rs_reads == 3 * 4 * E * (n - 1)  # 1.5 m (1 - 1/n) per rank, times n ranks


def test_plan_errors():
    with pytest.raises(T.TrivanceError) as e:
        T.trivance_plan((8,), "BRUCK")
    assert e.value.status == -2
    with pytest.raises(T.TrivanceError) as e:
        T.trivance_plan((9, 9), "BRUCK")
    assert e.value.status == -2
    lib = T.binding._lib()
    h = ctypes.c_void_p()
    dims = (ctypes.c_int * 2)(9, 9)
    assert lib.trivance_plan(80, dims, 2, 0, ctypes.byref(h)) == -1
    assert lib.trivance_plan(0, None, 0, 0, ctypes.byref(h)) == -1
    assert lib.trivance_plan(9, None, 0, 7, ctypes.byref(h)) == -1
    assert lib.trivance_plan(9, None, 0, 0, None) == -1
    p = T.trivance_plan((9,), "L")
    with pytest.raises(T.TrivanceError):
        T.trivance_plan_step(p, 2, 0)
    with pytest.raises(T.TrivanceError):
        T.trivance_block_range(p, 100, 1, 0)
    assert lib.trivance_strerror(-5) == b"output buffer too small"


@pytest.mark.parametrize("dims,E", [((9,), 64 * 9 * 3 + 20), ((243,), 8 * 2 ** 20), ((27, 27), 1_048_576),
                                    ((9, 9, 9), 12345), ((3, 3, 3, 3), 5000), ((1,), 100),
                                    ((3, 9), 5000), ((27, 3), 64 * 81 * 2 + 4), ((3, 3, 9), 7777),
                                    ((9, 27), 64 * 243 * 2), ((1, 9), 999)])
def test_placed_block_range_matches_oracle_placement(dims, E):
    from oracle import placement

    p = T.trivance_plan(dims, "B", placement="schedule")
    nat = partition.block_bounds(E, p.D, p.n)
    pos = placement.positions(dims)
    for c in range(p.D):
        for j in range(p.n):
            assert T.trivance_block_range(p, E, c, j) == nat[c][pos[c][j]]
        assert T.trivance_block_range(p, E, c, -1) == partition.segment_bounds(E, p.D)[c]


def test_placement_is_rejected_where_it_does_not_apply():
    lib = T.binding._lib()
    for dims, variant in [((8,), "B"), ((9,), "L"), ((9,), "BRUCK"), ((4, 4), "B"), ((3, 8), "B")]:
        with pytest.raises(T.TrivanceError) as e:
            T.trivance_plan(dims, variant, placement="schedule")
        assert e.value.status == -2
    h = ctypes.c_void_p()
    arr = (ctypes.c_int * 1)(9)
    assert lib.trivance_plan_ex(9, arr, 1, 1, 2, ctypes.byref(h)) == -1
    assert lib.trivance_plan_ex(9, arr, 1, 1, 0, ctypes.byref(h)) == 0
    lib.trivance_plan_destroy(h)


def test_dispatch_limit_is_a_derived_plan():
    """The dispatch limit lives in a plan: a derived plan carries the lower limit and the same
    schedule, the original is unchanged, and limits outside [1024, 2^31] are rejected."""
    p = T.trivance_plan((27, 27), "B")
    q = T.trivance_plan_with_dispatch_limit(p, 4096)
    assert q.num_passes == p.num_passes and q.num_steps == p.num_steps
    for i in range(p.num_passes):
        for c in range(2):
            assert T.trivance_plan_step(q, i, c) == T.trivance_plan_step(p, i, c)
    for bad in (0, -1, 1023, 2 ** 31 + 1):
        with pytest.raises(T.TrivanceError):
            T.trivance_plan_with_dispatch_limit(p, bad)
    assert T.trivance_plan_with_dispatch_limit(p, 2 ** 31).num_passes == p.num_passes
    del p  # the derived plan stays usable
    assert T.trivance_algorithmic_bytes(q, 1000) > 0


def test_congestion_length_query_and_size_check():
    """loads == NULL returns the required length; a short array is rejected before any GPU work."""
    lib = T.binding._lib()
    p = T.trivance_plan((27, 27), "B")
    need = lib.trivance_congestion(p.handle, None, None, 0)
    assert need == 12 * 729 * 4
    buf = np.zeros(need - 1, dtype=np.int64)
    rc = lib.trivance_congestion(p.handle, None, buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                 need - 1)
    assert rc == -5


def test_executor_argument_checks_without_gpu():
    """Argument validation happens before any HIP call: these return errors on a CPU-only host."""
    lib = T.binding._lib()
    p = T.trivance_plan((9,), "L")
    assert lib.trivance_allreduce_emulated(None, 9, 100, 0, p.handle, None) == -1  # NULL buffers
    assert lib.trivance_allreduce_emulated(None, 8, 100, 0, p.handle, None) == -1  # n mismatch
    assert lib.trivance_allreduce_emulated(None, 9, -1, 0, p.handle, None) == -1
    assert lib.trivance_allreduce_emulated(None, 9, 100, 5, p.handle, None) == -1  # dtype
    assert lib.trivance_allreduce_emulated(None, 9, 0, 0, p.handle, None) == 0     # no-op
    assert lib.trivance_allreduce_emulated_steps(None, 9, 10, 0, p.handle, None, 1, 3) == -1
    b = T.trivance_plan((9,), "BRUCK")
    assert lib.trivance_allreduce_emulated(None, 9, 10, 0, b.handle, None) == -2


@pytest.mark.parametrize("n", [2, 4, 5, 7, 8, 10, 20, 32, 100, 728])
def test_nonpower3_ring_plan_matches_oracle_tree(n):
    """Sec. 4.4 rings: the plan's passes (distances, order) and, through the per-pass byte
    accounting, its per-step receivers and sending children equal the oracle's tree."""
    from oracle import nonpow3

    p = T.trivance_plan((n,), "B")
    dist = nonpow3.distances(n)
    S = len(dist)
    assert p.num_steps == S and p.num_passes == 2 * S
    E = 1000
    for i in range(2 * S):
        phase, dim, d = T.trivance_plan_step(p, i)
        step = T.trivance_plan_step_index(p, i)
        assert (phase, step, dim, d) == ((1 if i < S else 2), i if i < S else 2 * S - 1 - i, 0,
                                          dist[i if i < S else 2 * S - 1 - i])
    # oracle tree: receivers (parent offsets) and children per step, from the contribution paths
    recv = [dict() for _ in range(S)]
    for u in range(n):
        for k in range(S):
            a, b = nonpow3.position(n, u, 0, k), nonpow3.position(n, u, 0, k + 1)
            if a != b:
                recv[k].setdefault(b, set()).add(a)
    for k in range(S):
        kids = sum(len(v) for v in recv[k].values())
        rs = T.trivance_pass_bytes(p, E, k)
        ag = T.trivance_pass_bytes(p, E, 2 * S - 1 - k)
        assert rs == (2 * len(recv[k]) + kids) * E * 4
        assert ag == (len(recv[k]) + kids) * E * 4
    # each rank forwards each block once: n - 1 child reads per block over the reduce-scatter
    assert sum(T.trivance_pass_bytes(p, E, k) for k in range(S)) == \
        (2 * sum(len(r) for r in recv) + (n - 1)) * E * 4


@pytest.mark.parametrize("dims", [(4, 4), (2, 3), (8, 8), (5, 7), (3, 8), (8, 3), (1, 8),
                                  (4, 4, 4), (2, 3, 4), (9, 2, 3), (2, 2, 2, 2)])
def test_nonpower3_torus_plan_matches_oracle(dims):
    """Tori with a side that is not a power of three: every pass's dimension and distance per
    collective equal the oracle's rotation, and the per-pass bytes, which count the receivers
    and sending children of every block's step, equal the edges of the oracle's contribution
    paths (so the plan's receiver and not-yet-forwarded offset lists are the oracle's)."""
    from oracle import nonpow3, partition

    dims = tuple(dims)
    D = len(dims)
    n = int(np.prod(dims))
    p = T.trivance_plan(dims, "B")
    S = sum(nonpow3.dim_steps(s) for s in dims)
    assert p.num_steps == S and p.num_passes == 2 * S
    rot = [nonpow3.torus_rotation(dims, c) for c in range(D)]
    for i in range(2 * S):
        t = i if i < S else 2 * S - 1 - i
        for c in range(D):
            phase, dim, d = T.trivance_plan_step(p, i, c)
            step = T.trivance_plan_step_index(p, i)
            want_dim, k = rot[c][t]
            assert (phase, step, dim, d) == ((1 if i < S else 2), t, want_dim,
                                              nonpow3.distances(dims[want_dim])[k])
    E = 64 * D * n + 37 * 64 + 5  # blocks of unequal sizes and a ragged tail
    bounds = partition.block_bounds(E, D, n)
    for t in range(S):
        rs = ag = 0
        for c in range(D):
            for j in range(n):
                pos = nonpow3.torus_paths(dims, j, c)
                edges = {(pos[t][u], pos[t + 1][u]) for u in range(n)}
                moves = {(a, b) for a, b in edges if a != b}
                recv = {b for _, b in moves}
                size = bounds[c][j][1] - bounds[c][j][0]
                rs += (2 * len(recv) + len(moves)) * size
                ag += (len(recv) + len(moves)) * size
        assert T.trivance_pass_bytes(p, E, t) == rs * 4
        assert T.trivance_pass_bytes(p, E, 2 * S - 1 - t) == ag * 4


def test_nonpower3_limits():
    for dims, variant in [((8,), "BRUCK"), ((2201,), "B"), ((2201,), "L"), ((5, 5, 5, 5), "L"),
                          ((2, 2, 2, 2, 2), "B"), ((2, 2, 2, 2, 2), "L"), ((2201, 2), "B"),
                          ((1000, 1000, 1000), "B")]:
        with pytest.raises(T.TrivanceError) as e:
            T.trivance_plan(dims, variant)
        assert e.value.status == -2


def _random_shapes(seed, count, max_n):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        D = int(rng.integers(1, 4))
        dims = tuple(int(x) for x in rng.integers(1, 14 if D > 1 else 200, size=D))
        n = int(np.prod(dims))
        if 2 <= n <= max_n and dims not in out:
            out.append(dims)
    return out


@pytest.mark.parametrize("dims", _random_shapes(11, 30, 300))
def test_plan_matches_oracle_on_seeded_random_shapes(dims):
    """Seeded random rings and tori, with sides that are and are not powers of three: passes,
    distances and per-pass bytes of the bandwidth-optimal plan against the oracle's contribution
    paths (tree plans) or its schedule and the 3.5 w E (n - 1) total (powers of three)."""
    from oracle import nonpow3, partition

    D = len(dims)
    n = int(np.prod(dims))
    p = T.trivance_plan(dims, "B")
    E = 64 * D * n + 23 * 64 + 7
    if not nonpow3.is_tree(dims):
        assert T.trivance_algorithmic_bytes(p, E) * 2 == 7 * 4 * E * (n - 1)
        return
    S = sum(nonpow3.dim_steps(s) for s in dims)
    assert p.num_passes == 2 * S
    rot = [nonpow3.torus_rotation(dims, c) for c in range(D)]
    for t in range(S):
        for c in range(D):
            _, dim, d = T.trivance_plan_step(p, t, c)
            step = T.trivance_plan_step_index(p, t)
            assert (step, dim, d) == (t, rot[c][t][0], nonpow3.distances(dims[rot[c][t][0]])[rot[c][t][1]])
    bounds = partition.block_bounds(E, D, n)
    rs = [0] * S
    ag = [0] * S
    for c in range(D):
        for j in range(n):
            pos = nonpow3.torus_paths(dims, j, c)
            size = bounds[c][j][1] - bounds[c][j][0]
            for t in range(S):
                moves = {(a, b) for a, b in zip(pos[t], pos[t + 1]) if a != b}
                recv = {b for _, b in moves}
                rs[t] += (2 * len(recv) + len(moves)) * size
                ag[t] += (len(recv) + len(moves)) * size
    for t in range(S):
        assert T.trivance_pass_bytes(p, E, t) == rs[t] * 4
        assert T.trivance_pass_bytes(p, E, 2 * S - 1 - t) == ag[t] * 4


def test_copy_helper_rejects_bad_arguments_before_any_launch():
    """trivance_copy_device checks size, alignment and overlap on the host; a zero-byte copy is a
    no-op. None of these cases reaches the GPU."""
    lib = T.binding._lib()
    P = ctypes.c_void_p
    EINVAL = -1
    assert lib.trivance_copy_device(P(4096), P(8192), 0, None) == 0
    assert lib.trivance_copy_device(None, None, 0, None) == 0
    assert lib.trivance_copy_device(P(4096), P(8192), -16, None) == EINVAL
    assert lib.trivance_copy_device(P(4096), P(8192), 24, None) == EINVAL    # not a multiple of 16
    assert lib.trivance_copy_device(P(4104), P(8192), 16, None) == EINVAL    # dst misaligned
    assert lib.trivance_copy_device(P(4096), P(8200), 16, None) == EINVAL    # src misaligned
    assert lib.trivance_copy_device(None, P(8192), 16, None) == EINVAL
    assert lib.trivance_copy_device(P(4096), P(4096 + 32), 64, None) == EINVAL  # overlap
    assert lib.trivance_copy_device(P(4096 + 32), P(4096), 64, None) == EINVAL  # overlap


# ---- latency-optimal plans on sides that are not powers of three (slot programs) ----

LATENCY_TREES = [(2,), (4,), (5,), (7,), (8,), (10,), (20,), (32,), (64,), (100,), (728,),
                 (4, 4), (2, 3), (3, 8), (8, 3), (5, 7), (1, 8), (2, 3, 4), (4, 4, 4), (2, 2, 2, 2),
                 (32, 32), (8, 64), (16, 16, 16), (10, 3, 3)]


@pytest.mark.parametrize("dims", LATENCY_TREES, ids=lambda d: "x".join(map(str, d)))
def test_latency_slot_plan_matches_oracle_program(dims):
    """The plan's passes (dimension and distance per collective, step index) equal the oracle's
    rotation; per pass and collective, the byte accounting (every partial held before the pass
    read once, every one after it written once) equals the oracle's partial counts; the
    workspace holds the most partials of any state between passes."""
    from oracle import latency_nonpow3, nonpow3, partition

    dims = tuple(dims)
    D = len(dims)
    n = int(np.prod(dims))
    p = T.trivance_plan(dims, "L")
    S = sum(nonpow3.dim_steps(s) for s in dims)
    assert p.num_steps == S and p.num_passes == S
    E = 64 * D * 3 + 37  # unequal segments and a ragged tail
    seg = [e - b for b, e in partition.segment_bounds(E, D)]
    progs = [latency_nonpow3.program(dims, c) for c in range(D)]
    rot = [nonpow3.torus_rotation(dims, c) for c in range(D)]
    most = 1
    for t in range(S):
        assert T.trivance_plan_step_index(p, t) == t
        want = 0
        for c in range(D):
            phase, dim, d = T.trivance_plan_step(p, t, c)
            assert (phase, dim, d) == (0, rot[c][t][0], nonpow3.distances(dims[rot[c][t][0]])[rot[c][t][1]])
            needed = progs[c][0]
            want += (len(needed[t]) + len(needed[t + 1])) * n * seg[c] * 4
            most = max(most, len(needed[t]))
        assert T.trivance_pass_bytes(p, E, t) == want
    halves = 2 if S >= 3 else 1
    assert T.trivance_workspace_bytes(p, E) == halves * most * n * E * 4
    assert T.trivance_workspace_bytes(p, E, T.I32) == halves * most * n * E * 4


def test_latency_slot_plan_needs_its_workspace():
    """The in-place entry points refuse a plan that keeps partials between passes (ESIZE), before
    any launch; so does the workspace form with a workspace below the required size."""
    import ctypes

    lib = T.binding._lib()
    p = T.trivance_plan((8,), "L")
    need = T.trivance_workspace_bytes(p, 1000)
    assert need > 0
    fake = ctypes.c_void_p(1 << 40)  # never dereferenced: the size check comes first
    assert lib.trivance_allreduce_emulated(fake, 8, 1000, 0, p.handle, None) == -5
    assert lib.trivance_allreduce_emulated_steps(fake, 8, 1000, 0, p.handle, None, 0, 1) == -5
    assert lib.trivance_allreduce_emulated_ws(fake, 8, 1000, 0, p.handle, fake, need - 1, None) == -5
    assert lib.trivance_allreduce_emulated_ws(fake, 8, 1000, 0, p.handle, None, need, None) == -5
    # elems == 0 is a no-op, and plans that run in place need no workspace
    assert lib.trivance_allreduce_emulated(fake, 8, 0, 0, p.handle, None) == 0
    for dims, v in [((9,), "L"), ((8,), "B"), ((27, 27), "B"), ((9, 3), "L")]:
        assert T.trivance_workspace_bytes(T.trivance_plan(dims, v), 12345) == 0
    assert lib.trivance_workspace_bytes(None, 10, 0) == -1
    assert lib.trivance_workspace_bytes(p.handle, -1, 0) == -1
    assert lib.trivance_workspace_bytes(p.handle, 10, 7) == -1


def test_missing_library_fails_loudly():
    """Every call of the binding reaches the native library through one loader, and every use
    starts with a plan: without the library, the loader and plan construction raise RuntimeError
    (there is no fallback path). Checked in a child process whose binding points at a library
    that does not exist."""
    import subprocess
    import sys

    code = (
        "import paper_2602_17254_amd as T\n"
        "T.binding.LIB_PATH = '/nonexistent/libtrivance.so'\n"
        "T.binding._LIB = None\n"
        "for call in (lambda: T.trivance_plan((9,), 'L'), lambda: T.trivance_plan((3, 3), 'B'),\n"
        "             T.binding._lib):\n"
        "    try:\n"
        "        call()\n"
        "    except RuntimeError as e:\n"
        "        assert 'not built' in str(e)\n"
        "    else:\n"
        "        raise SystemExit('no error')\n"
        "print('raised')\n")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, cwd=root,
                         timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.strip().endswith("raised")
