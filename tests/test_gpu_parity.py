"""GPU parity: the HIP path (through the C ABI) against the CPU oracle, element by element.

Run on an MI355X: python -u -m pytest tests -m gpu -x -v --timeout 120 --timeout-method thread
Bars: int32 and congestion bit-exact; fp32 within 1e-6 relative of the schedule-ordered oracle
(expected and asserted: identical bits) and within 4 S 2^-23 sum|v| of an fp64 sum.
"""

import sys

import numpy as np
import pytest

from gpu_util import assert_matches_oracle, run_hip
from oracle import allreduce, congestion, partition, schedule

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu_present():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2602_17254_amd as T

    T.binding._lib()  # fails loudly when the native library is missing
    yield


# (dims, elements) spanning several work tiles, ragged tails, the 16-byte path (E % 4 == 0) and
# the scalar path (odd E), empty blocks (E < 64 n) and E = 0.
SHAPES = [
    ((1,), 5), ((3,), 1), ((3,), 4), ((3,), 64 * 3 * 5 + 4), ((3,), 1001),
    ((9,), 0), ((9,), 7), ((9,), 64), ((9,), 1024), ((9,), 64 * 9 * 3 + 20), ((9,), 12345),
    ((27,), 64 * 27 * 4 + 4), ((27,), 5003),
    ((81,), 64 * 81 * 2 + 8), ((81,), 20001),
    ((243,), 64 * 243 * 2 + 4), ((729,), 64 * 729 + 8),
    ((3, 3), 5), ((3, 3), 64 * 9 * 4 + 12), ((3, 3), 3333),
    ((9, 9), 64 * 81 * 3 + 4), ((9, 9), 7777),
    ((3, 3, 3), 64 * 27 * 3 + 16), ((3, 3, 3), 999),
    ((27, 27), 64 * 729 + 36),
    ((9, 9, 9), 64 * 729 * 2 + 100),
    # rectangular tori (unequal sides; rotation reading in include/trivance.h)
    ((3, 9), 64 * 27 * 3 + 4), ((9, 3), 777), ((3, 27), 64 * 81 * 2 + 12),
    ((27, 3), 64 * 81 + 8), ((3, 3, 9), 64 * 81 * 2 + 4), ((9, 27), 64 * 243 + 4),
    ((3, 9, 9), 64 * 243 + 4),
]


def _ids(p):
    dims, E = p
    return "x".join(map(str, dims)) + f"-E{E}"


@pytest.mark.parametrize("variant", ["L", "B"])
@pytest.mark.parametrize("dtype", ["f32", "i32"])
@pytest.mark.parametrize("shape", SHAPES, ids=_ids)
def test_parity_small(shape, dtype, variant):
    dims, E = shape
    n = schedule.Torus(dims).n
    seed = 1000 * len(dims) + n + E + (0 if variant == "L" else 7)
    rng = np.random.default_rng(seed)
    _say(f"[parity] dims={dims} E={E} dtype={dtype} variant={variant} seed={seed}")
    if dtype == "f32":
        V = rng.standard_normal((n, E), dtype=np.float32)
    else:
        V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    got = run_hip(V, dims, variant)
    assert_matches_oracle(got, V, dims, variant, what=f"{dims} E={E} {dtype} {variant}")
    if dtype == "i32":
        np.testing.assert_array_equal(got, np.broadcast_to(allreduce.exact_int_sum(V), got.shape))


# Latency-optimal only (the bandwidth-optimal oracle takes minutes at this many ranks): 9-row
# cycles in each of four dimensions, one wave per cycle.
@pytest.mark.parametrize("dtype", ["f32", "i32"])
def test_parity_latency_4d_torus(dtype):
    dims, E = (9, 9, 9, 9), 64 * 4 + 45
    n = 6561
    rng = np.random.default_rng(94 + E)
    _say(f"[parity] dims={dims} E={E} dtype={dtype} variant=L")
    if dtype == "f32":
        V = rng.standard_normal((n, E), dtype=np.float32)
    else:
        V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    got = run_hip(V, dims, "L")
    assert_matches_oracle(got, V, dims, "L", what=f"{dims} E={E} {dtype} L")
    if dtype == "i32":
        np.testing.assert_array_equal(got, np.broadcast_to(allreduce.exact_int_sum(V), got.shape))


@pytest.mark.parametrize("dims,variants", [((9,), "LB"), ((8,), "B"), ((4, 4), "B"), ((81,), "L"),
                                           ((243,), "L"), ((3, 9, 9), "LB")])
def test_misaligned_rows_use_scalar_path(dims, variants):
    """A [n, E] view whose start is not 16-byte aligned still gives the oracle's result (block,
    latency and tree steps; latency tiles of 3-, 9-, 81- and 243-row cycles, with one and with
    several waves per cycle)."""
    import paper_2602_17254_amd as T

    n = int(np.prod(dims))
    E = 64 * n * len(dims) * 2 + 8
    rng = np.random.default_rng(3)
    V = rng.standard_normal((n, E), dtype=np.float32)
    for variant in variants:
        _say(f"[misaligned] dims={dims} variant={variant}")
        flat = torch.zeros(n * E + 1, dtype=torch.float32, device="cuda")
        view = flat[1:].view(n, E)
        view.copy_(torch.from_numpy(V))
        assert view.data_ptr() % 16 != 0
        T.trivance_allreduce_emulated(view, T.trivance_plan(dims, variant))
        torch.cuda.synchronize()
        assert_matches_oracle(view.cpu().numpy(), V, dims, variant, what="misaligned")


@pytest.mark.parametrize("dims", [(27,), (9, 9), (3, 3, 3), (3, 9)])
def test_step_hook_coverage(dims):
    """Lemma 2 on the GPU: with one-hot int32 inputs, after each latency-optimal pass every rank
    holds each source of its covered window exactly once; passes run one call at a time equal the
    oracle after the same number of steps."""
    import paper_2602_17254_amd as T

    t = schedule.Torus(dims)
    n, D = t.n, t.D
    E = n * D * 64
    V = np.zeros((n, E), dtype=np.int32)
    for c in range(D):
        V[np.arange(n), c * n * 64 + np.arange(n)] = 1
    plan = T.trivance_plan(dims, "L")
    buf = torch.from_numpy(V).cuda()
    for p in range(plan.num_passes):
        _say(f"[step-hook] dims={dims} pass={p}")
        T.trivance_allreduce_emulated_steps(buf, plan, p, p + 1)
        torch.cuda.synchronize()
        want = allreduce.latency_optimal(V, dims, passes=p + 1)
        np.testing.assert_array_equal(buf.cpu().numpy(), want)
    assert (buf.cpu().numpy()[:, [c * n * 64 + u for c in range(D) for u in range(n)]] == 1).all()


@pytest.mark.parametrize("dims", [(27,), (9, 9), (8,), (64,), (4, 4), (3, 8), (2, 3, 4)])
def test_step_hook_reduce_scatter_then_resume(dims):
    """After the reduce-scatter passes alone, rank r's block r is final (int32 exact sum);
    resuming with the all-gather passes completes the AllReduce."""
    import paper_2602_17254_amd as T

    n, D = int(np.prod(dims)), len(dims)
    E = 64 * n * 2 + 4
    rng = np.random.default_rng(41)
    V = rng.integers(-1000, 1000, size=(n, E), dtype=np.int32)
    plan = T.trivance_plan(dims, "B")
    S = plan.num_steps
    buf = torch.from_numpy(V).cuda()
    _say(f"[rs-resume] dims={dims}")
    T.trivance_allreduce_emulated_steps(buf, plan, 0, S)
    torch.cuda.synchronize()
    mid = buf.cpu().numpy()
    total = allreduce.exact_int_sum(V)
    bb = partition.block_bounds(E, D, n)
    for c in range(D):
        for r in range(n):
            b, e = bb[c][r]
            np.testing.assert_array_equal(mid[r, b:e], total[b:e])
    T.trivance_allreduce_emulated_steps(buf, plan, S, 2 * S)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(buf.cpu().numpy(), np.broadcast_to(total, (n, E)))


@pytest.mark.parametrize("dims", [(7,), (8,), (10,), (32,), (4, 4), (3, 8), (5, 2), (2, 3, 4)])
def test_step_hook_tree_partials(dims):
    """Sides that are not powers of three, one pass at a time: after reduce-scatter step t every
    rank that still holds a partial of block j holds exactly the int32 sum of the contributions
    whose paths (oracle) have reached it; the all-gather then leaves the exact sum everywhere."""
    import paper_2602_17254_amd as T
    from oracle import nonpow3

    n, D = int(np.prod(dims)), len(dims)
    E = 64 * n * D + 20
    rng = np.random.default_rng(43 + n)
    V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    plan = T.trivance_plan(dims, "B")
    S = plan.num_steps
    bb = partition.block_bounds(E, D, n)
    paths = {(c, j): nonpow3.torus_paths(dims, j, c) for c in range(D) for j in range(n)}
    buf = torch.from_numpy(V).cuda()
    for t in range(S):
        _say(f"[tree-partials] dims={dims} step={t}")
        T.trivance_allreduce_emulated_steps(buf, plan, t, t + 1)
        torch.cuda.synchronize()
        mid = buf.cpu().numpy()
        for c in range(D):
            for j in range(n):
                b, e = bb[c][j]
                pos = paths[(c, j)][t + 1]
                for x in set(pos):
                    want = np.zeros(e - b, dtype=np.int64)
                    for u in range(n):
                        if pos[u] == x:
                            want += V[u, b:e]
                    np.testing.assert_array_equal(mid[x, b:e], want.astype(np.int32))
    T.trivance_allreduce_emulated_steps(buf, plan, S, 2 * S)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(buf.cpu().numpy(),
                                  np.broadcast_to(allreduce.exact_int_sum(V), (n, E)))


@pytest.mark.parametrize("dims,variant,routing", [
    ((9,), "L", "scheduled"), ((81,), "L", "scheduled"), ((243,), "B", "scheduled"),
    ((27, 27), "B", "scheduled"), ((9, 9, 9), "B", "scheduled"), ((27, 27), "L", "shortest"),
    ((9,), "BRUCK", "scheduled"), ((81,), "BRUCK", "scheduled"), ((9,), "BRUCK", "shortest"),
    ((243,), "BRUCK", "shortest"), ((3, 3), "B", "shortest"), ((1,), "L", "scheduled"),
    ((9, 27), "B", "scheduled"), ((3, 9), "L", "shortest"), ((3, 3, 9), "B", "scheduled"),
])
def test_congestion_bit_exact(dims, variant, routing):
    import paper_2602_17254_amd as T

    _say(f"[congestion] dims={dims} variant={variant} routing={routing}")
    plan = T.trivance_plan(dims, variant)
    got = T.trivance_congestion(plan, routing)
    want = congestion.link_loads(dims, variant, routing)
    assert got.shape == want.shape
    np.testing.assert_array_equal(got, want)
    out = torch.full((got.size,), -7, dtype=torch.int64, device="cuda")
    T.trivance_congestion_device(plan, out, routing)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy().reshape(got.shape), want)


def test_errors_surface():
    import paper_2602_17254_amd as T

    plan = T.trivance_plan((9,), "BRUCK")
    buf = torch.zeros((9, 16), dtype=torch.float32, device="cuda")
    with pytest.raises(T.TrivanceError):
        T.trivance_allreduce_emulated(buf, plan)
    with pytest.raises(ValueError):
        T.trivance_allreduce_emulated(buf, T.trivance_plan((27,), "L"))


def test_fill_hash_uniform_matches_host_generator():
    import paper_2602_17254_amd as T
    from paper_2602_17254_amd import inputs

    n, E = 7, 10007
    buf = torch.empty((n, E), dtype=torch.float32, device="cuda")
    T.trivance_fill_hash_uniform(buf, 4)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(buf.cpu().numpy(), inputs.hash_uniform(4, E, np.arange(n), np.arange(E)))


NONPOW3 = [(2, 100), (4, 64 * 4 * 3 + 4), (5, 999), (7, 64 * 7 * 5 + 12), (8, 64 * 8 * 4),
           (10, 3001), (16, 64 * 16 * 2 + 8), (20, 64 * 20 * 3 + 4), (32, 64 * 32 + 20),
           (50, 7777), (64, 64 * 64 + 4), (100, 64 * 100 + 36), (250, 64 * 250 + 4),
           (728, 64 * 728 + 8),
           # blocks filling whole 256-element chunks: one unit per wave (the others above take two
           # in the reduce-scatter and eight in the all-gather)
           (8, 8 * 256 * 3 + 4), (20, 20 * 256 * 2)]


@pytest.mark.parametrize("dtype", ["f32", "i32"])
@pytest.mark.parametrize("n,E", NONPOW3, ids=[f"n{n}-E{E}" for n, E in NONPOW3])
def test_parity_nonpower3_ring(n, E, dtype):
    """Sec. 4.4 rings (bandwidth-optimal): the tree-driven kernels against the oracle."""
    rng = np.random.default_rng(n * 7 + E)
    _say(f"[nonpow3] n={n} E={E} dtype={dtype}")
    if dtype == "f32":
        V = rng.standard_normal((n, E), dtype=np.float32)
    else:
        V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    got = run_hip(V, (n,), "B")
    assert_matches_oracle(got, V, (n,), "B", what=f"ring {n} E={E} {dtype}")
    if dtype == "i32":
        np.testing.assert_array_equal(got, np.broadcast_to(allreduce.exact_int_sum(V), got.shape))


@pytest.mark.parametrize("n", [4, 7, 8, 10, 32, 100])
def test_congestion_nonpower3_ring(n):
    import paper_2602_17254_amd as T

    _say(f"[nonpow3 congestion] n={n}")
    got = T.trivance_congestion(T.trivance_plan((n,), "B"))
    np.testing.assert_array_equal(got, congestion.link_loads((n,), "B"))


# tori with a side that is not a power of three (one tree per dimension), including mixed sides,
# a side of 1, four dimensions, empty blocks (E < 64 n D), ragged tails and the scalar path
NONPOW3_TORI = [((4, 4), 64 * 16 * 2 * 3 + 4), ((2, 3), 101), ((8, 8), 64 * 64 * 2 + 12),
                ((5, 7), 7777), ((3, 8), 64 * 24 * 2 * 2 + 8), ((8, 3), 3001),
                ((1, 8), 64 * 8 * 2 + 4), ((9, 2), 64 * 18 * 2 * 3 + 4),
                ((4, 4, 4), 64 * 64 * 3 + 20), ((2, 3, 4), 999), ((2, 2, 2, 2), 64 * 16 * 4 + 4),
                ((10, 3, 3), 64 * 90 * 3 + 4), ((16, 16), 64 * 256 * 2 + 36), ((4, 4), 5),
                ((8, 8), 0),
                # blocks filling whole 256-element chunks: one unit per wave in both phases (the
                # partly filled ones above take two units per wave (2D) or one (3D, 4D) in the
                # reduce-scatter, and eight (2D) or two (3D, 4D) in the all-gather)
                ((4, 4), 2 * 16 * 256 * 2), ((2, 3, 4), 3 * 24 * 256 + 12),
                ((2, 2, 2), 3 * 8 * 4096 + 192), ((2, 2, 2, 2), 4 * 16 * 256 * 2),
                # more than 64 offset-table entries per pass on 2D and 4D tori (the long table)
                ((20, 20), 64 * 400 * 2 // 3 + 4), ((5, 5, 5, 5), 4001)]


@pytest.mark.parametrize("dtype", ["f32", "i32"])
@pytest.mark.parametrize("dims,E", NONPOW3_TORI, ids=[_ids(p) for p in NONPOW3_TORI])
def test_parity_nonpower3_torus(dims, E, dtype):
    """Tori with a side that is not a power of three (bandwidth-optimal): against the oracle."""
    n = int(np.prod(dims))
    rng = np.random.default_rng(n * 11 + E)
    _say(f"[nonpow3 torus] dims={dims} E={E} dtype={dtype}")
    if dtype == "f32":
        V = rng.standard_normal((n, E), dtype=np.float32)
    else:
        V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    got = run_hip(V, dims, "B")
    assert_matches_oracle(got, V, dims, "B", what=f"torus {dims} E={E} {dtype}")
    if dtype == "i32":
        np.testing.assert_array_equal(got, np.broadcast_to(allreduce.exact_int_sum(V), got.shape))


@pytest.mark.parametrize("dims", [(4, 4), (5, 7), (8, 3), (1, 8), (4, 4, 4), (2, 3, 4), (16, 16),
                                  (8, 64), (2,), (2, 2)])
def test_congestion_nonpower3_torus(dims):
    """Both routings: every tree distance is at most half its side (a tie at exactly half keeps
    the offset's sign), so shortest-path routing counts what scheduled routing counts."""
    import paper_2602_17254_amd as T

    _say(f"[nonpow3 torus congestion] dims={dims}")
    plan = T.trivance_plan(dims, "B")
    want = congestion.link_loads(dims, "B")
    np.testing.assert_array_equal(T.trivance_congestion(plan), want)
    np.testing.assert_array_equal(T.trivance_congestion(plan, "shortest"), want)


def _seeded_shapes(seed, count, max_n):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        D = int(rng.integers(1, 4))
        dims = tuple(int(x) for x in rng.integers(1, 12 if D > 1 else 250, size=D))
        n = int(np.prod(dims))
        E = int(rng.integers(1, 64 * D * n * 3))
        if 2 <= n <= max_n and dims not in [d for d, _ in out]:
            out.append((dims, E))
    return out


SEEDED = _seeded_shapes(2026, 24, 200)


@pytest.mark.parametrize("dtype", ["f32", "i32"])
@pytest.mark.parametrize("dims,E", SEEDED, ids=[_ids(p) for p in SEEDED])
def test_parity_seeded_random_shapes(dims, E, dtype):
    """Seeded random rings and tori (sides that are and are not powers of three, 1-3 dimensions,
    random E: vector and scalar paths, empty blocks, ragged tails), bandwidth-optimal, and the
    latency-optimal variant where every side is a power of three."""
    from oracle import nonpow3

    n = int(np.prod(dims))
    rng = np.random.default_rng(n + E)
    if dtype == "f32":
        V = rng.standard_normal((n, E), dtype=np.float32)
    else:
        V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    variants = "B" if nonpow3.is_tree(dims) else "LB"
    for variant in variants:
        _say(f"[seeded] dims={dims} E={E} {dtype} {variant}")
        got = run_hip(V, dims, variant)
        assert_matches_oracle(got, V, dims, variant, what=f"{dims} E={E} {dtype} {variant}")


@pytest.mark.parametrize("n", [1000, 2200])
def test_parity_largest_rings_sampled(n):
    """Rings up to the 2200-rank limit (receiver tables of several hundred entries per step):
    int32 and fp32 on a column sample (first, last and two random elements of every block)
    against the oracle's gather form, which equals the mailbox form bit for bit."""
    import paper_2602_17254_amd as T
    from gpu_util import sample_columns

    E = 64 * n * 2 + 12
    plan = T.trivance_plan((n,), "B")
    cols, seg, blk = sample_columns(E, 1, n, "B", seed=n)
    for dtype in ("i32", "f32"):
        _say(f"[large ring] n={n} E={E} {dtype}")
        rng = np.random.default_rng(n + 7)
        if dtype == "f32":
            V = rng.standard_normal((n, E), dtype=np.float32)
        else:
            V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
        buf = torch.from_numpy(V).cuda()
        T.trivance_allreduce_emulated(buf, plan)
        torch.cuda.synchronize()
        got = buf.index_select(1, torch.from_numpy(cols).cuda()).cpu().numpy()
        assert_matches_oracle(got, np.ascontiguousarray(V[:, cols]), (n,), "B", col_seg=seg,
                              col_blk=blk, what=f"ring {n} {dtype}")
        del buf


def test_two_streams_concurrently():
    """Independent AllReduces enqueued on two streams (default priority) both match the oracle."""
    import paper_2602_17254_amd as T

    jobs = [((27,), "B", 64 * 27 * 3 + 4), ((3, 8), "B", 64 * 24 * 2 * 2 + 8), ((9,), "L", 4096)]
    streams = [torch.cuda.Stream() for _ in jobs]
    data = []
    for (dims, variant, E), s in zip(jobs, streams):
        n = int(np.prod(dims))
        V = np.random.default_rng(E).standard_normal((n, E), dtype=np.float32)
        buf = torch.from_numpy(V).cuda()
        data.append((dims, variant, V, buf))
    torch.cuda.synchronize()
    for (dims, variant, V, buf), s in zip(data, streams):
        _say(f"[streams] {dims} {variant}")
        T.trivance_allreduce_emulated(buf, T.trivance_plan(dims, variant), stream=s)
    for s in streams:
        s.synchronize()
    for dims, variant, V, buf in data:
        assert_matches_oracle(buf.cpu().numpy(), V, dims, variant, what=f"stream {dims}")


@pytest.mark.parametrize("dims,variant", [((27,), "B"), ((9,), "L"), ((3, 8), "B"), ((9, 9), "B")])
def test_graph_capture_replays(dims, variant):
    """The enqueued passes can be captured in a HIP graph: every replay (with eager refills and
    synchronisation between replays) reproduces the eager result bit for bit."""
    import paper_2602_17254_amd as T

    n = int(np.prod(dims))
    E = 64 * n * len(dims) * 2 + 4
    plan = T.trivance_plan(dims, variant)
    V = np.random.default_rng(n + E).standard_normal((n, E), dtype=np.float32)
    src = torch.from_numpy(V).cuda()
    buf = src.clone()
    T.trivance_allreduce_emulated(buf, plan)
    torch.cuda.synchronize()
    eager = buf.clone()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    buf.copy_(src)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        T.trivance_allreduce_emulated(buf, plan)
    for k in range(3):
        _say(f"[graph] {dims} {variant} replay {k}")
        buf.copy_(src)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(buf, eager), f"replay {k} differs from the eager result"


# Message-contiguous block placement (TRIVANCE_PLACE_BY_SCHEDULE): bandwidth-optimal,
# power-of-three sides; against the oracle with the placed block labels
PLACED = [((3,), 64 * 3 * 5 + 4), ((9,), 7), ((9,), 64 * 9 * 3 + 20), ((27,), 5003),
          ((81,), 64 * 81 * 2 + 8), ((243,), 64 * 243 * 2 + 4), ((729,), 64 * 729 + 8),
          ((3, 3), 3333), ((9, 9), 64 * 81 * 3 + 4), ((27, 27), 64 * 729 + 36),
          ((3, 3, 3), 64 * 27 * 3 + 16), ((9, 9, 9), 64 * 729 * 2 + 100),
          ((3, 3, 3, 3), 64 * 81 * 4 + 12), ((1,), 5), ((9,), 0),
          # unequal sides (the step order of the rotation reading)
          ((3, 9), 64 * 27 * 3 + 4), ((9, 3), 777), ((3, 27), 64 * 81 * 2 + 12),
          ((3, 3, 9), 64 * 81 * 2 + 4), ((9, 27), 64 * 243 + 4), ((1, 9), 64 * 9 * 2 + 4)]


@pytest.mark.parametrize("dtype", ["f32", "i32"])
@pytest.mark.parametrize("dims,E", PLACED, ids=[_ids(p) for p in PLACED])
def test_parity_placed(dims, E, dtype):
    from gpu_util import placement_labels

    n = int(np.prod(dims))
    rng = np.random.default_rng(31 * n + E)
    _say(f"[placed] dims={dims} E={E} dtype={dtype}")
    if dtype == "f32":
        V = rng.standard_normal((n, E), dtype=np.float32)
    else:
        V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    got = run_hip(V, dims, "B", placement="schedule")
    seg, blk = placement_labels(E, dims)
    assert_matches_oracle(got, V, dims, "B", col_seg=seg, col_blk=blk,
                          what=f"placed {dims} E={E} {dtype}")
    if dtype == "i32":
        np.testing.assert_array_equal(got, np.broadcast_to(allreduce.exact_int_sum(V), got.shape))


@pytest.mark.parametrize("dims", [(9,), (3, 3)])
def test_placed_misaligned_rows_use_scalar_path(dims):
    """Placed plans on a [n, E] view whose start is not 16-byte aligned (4-byte accesses)."""
    import paper_2602_17254_amd as T
    from gpu_util import placement_labels

    n = int(np.prod(dims))
    E = 64 * n * len(dims) * 2 + 8
    V = np.random.default_rng(5).standard_normal((n, E), dtype=np.float32)
    _say(f"[placed misaligned] dims={dims}")
    flat = torch.zeros(n * E + 1, dtype=torch.float32, device="cuda")
    view = flat[1:].view(n, E)
    view.copy_(torch.from_numpy(V))
    assert view.data_ptr() % 16 != 0
    T.trivance_allreduce_emulated(view, T.trivance_plan(dims, "B", placement="schedule"))
    torch.cuda.synchronize()
    seg, blk = placement_labels(E, dims)
    assert_matches_oracle(view.cpu().numpy(), V, dims, "B", col_seg=seg, col_blk=blk,
                          what="placed misaligned")


@pytest.mark.parametrize("dims", [(27,), (9, 9), (3, 3, 3)])
def test_placed_step_hook_reduce_scatter_then_resume(dims):
    """Placed plans: the state after the reduce-scatter passes equals the oracle's, and resuming
    with the all-gather passes completes the AllReduce."""
    import paper_2602_17254_amd as T
    from gpu_util import placement_labels

    n = int(np.prod(dims))
    E = 64 * n * len(dims) + 28
    V = np.random.default_rng(n).standard_normal((n, E), dtype=np.float32)
    seg, blk = placement_labels(E, dims)
    plan = T.trivance_plan(dims, "B", placement="schedule")
    S = plan.num_steps
    _say(f"[placed step hook] dims={dims} E={E}")
    buf = torch.from_numpy(V).cuda()
    T.trivance_allreduce_emulated_steps(buf, plan, 0, S)
    torch.cuda.synchronize()
    want_rs = allreduce.bandwidth_optimal(V, dims, col_seg=seg, col_blk=blk, ag_passes=0)
    np.testing.assert_array_equal(buf.cpu().numpy(), want_rs)
    T.trivance_allreduce_emulated_steps(buf, plan, S, 2 * S)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(buf.cpu().numpy(),
                                  allreduce.bandwidth_optimal(V, dims, col_seg=seg, col_blk=blk))
