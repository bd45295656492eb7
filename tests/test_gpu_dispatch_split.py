"""GPU: launches issued as several dispatches.

A dispatch carries its grid size as a 32-bit count of work-items; every launch of the library
goes through a split into dispatches of at most the plan's limit (2^31 work-items, lowered on a
derived plan by trivance_plan_with_dispatch_limit). Here a limit of 1024 work-items (one to sixteen workgroups per dispatch) forces the split on small
inputs for every kernel family, against the oracle; and a bandwidth-optimal call whose first
pass holds 3^18 waves (2.5e10 work-items) runs at the default limit, against exact column sums.
"""

import sys

import numpy as np
import pytest

from gpu_util import assert_matches_oracle, run_hip
from oracle import allreduce, congestion

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


# every launch path: latency steps with 3-, 9- (three waves per cycle on rings, one on tori of
# three or more dimensions), 27-, 81-, 243- and 729-rank cycles and the generic cycle kernel
# (2187); block steps; tree steps on rings and tori, with the short and the long offset table. The 10 x 10 x 10 torus takes 65,536 work-items per dispatch
# (about 500 dispatches per pass), the others 1024.
CASES = [
    ((3,), "L", 64 * 3 * 40 + 4), ((9,), "L", 64 * 9 * 6 + 8), ((9, 9, 9), "L", 64 * 27 + 12),
    ((27,), "L", 64 * 27 * 3 + 4), ((81,), "L", 64 * 81 * 2 + 8), ((243,), "L", 64 * 243 + 4),
    ((729,), "L", 2003), ((2187,), "L", 333), ((27,), "B", 64 * 27 * 6 + 4), ((9, 9), "B", 64 * 81 * 2 * 3 + 12),
    ((8,), "B", 8 * 256 * 3 + 4), ((50,), "B", 7777), ((4, 8), "B", 64 * 32 * 2 * 3 + 12),
    ((4, 4, 4), "B", 64 * 64 * 3 + 20), ((10, 10, 10), "B", 3001),
]


def _id(c):
    dims, variant, E = c
    return "x".join(map(str, dims)) + f"-{variant}-E{E}"


@pytest.mark.parametrize("dtype", ["f32", "i32"])
@pytest.mark.parametrize("dims,variant,E", CASES, ids=[_id(c) for c in CASES])
def test_split_dispatches_match_oracle(dims, variant, E, dtype):
    n = int(np.prod(dims))
    seed = 17 * n + E + (0 if variant == "L" else 5)
    limit = 65536 if n >= 1000 and len(dims) > 1 else 1024
    rng = np.random.default_rng(seed)
    _say(f"[split] dims={dims} variant={variant} E={E} dtype={dtype} seed={seed} limit={limit}")
    if dtype == "f32":
        V = rng.standard_normal((n, E), dtype=np.float32)
    else:
        V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    got = run_hip(V, dims, variant, dispatch_items=limit)
    assert_matches_oracle(got, V, dims, variant, what=f"split {dims} {variant} E={E} {dtype}")
    if dtype == "i32":
        np.testing.assert_array_equal(got, np.broadcast_to(allreduce.exact_int_sum(V), got.shape))


@pytest.mark.parametrize("dims,E", [((243,), 64 * 243 + 4), ((9, 9, 9), 64 * 729 + 100)])
def test_split_dispatches_placed(dims, E):
    """Message-contiguous placement with one to sixteen workgroups per dispatch."""
    from gpu_util import placement_labels

    n = int(np.prod(dims))
    V = np.random.default_rng(n + E).integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    _say(f"[split placed] dims={dims} E={E} limit=1024")
    got = run_hip(V, dims, "B", placement="schedule", dispatch_items=1024)
    seg, blk = placement_labels(E, dims)
    assert_matches_oracle(got, V, dims, "B", col_seg=seg, col_blk=blk, what=f"split placed {dims}")


@pytest.mark.parametrize("dims,variant", [((27, 27), "B"), ((81,), "L"), ((8,), "B"),
                                          ((4, 4, 4), "B"), ((9,), "BRUCK")])
def test_split_congestion_matches_oracle(dims, variant):
    import paper_2602_17254_amd as T

    _say(f"[split congestion] dims={dims} variant={variant} limit=1024")
    plan = T.trivance_plan_with_dispatch_limit(T.trivance_plan(dims, variant), 1024)
    got = T.trivance_congestion(plan)
    np.testing.assert_array_equal(got, congestion.link_loads(dims, variant))


def test_grid_above_32_bit_work_items_is_whole():
    """27 x 27 x 27 ranks, bandwidth-optimal, 472,512 int32 per rank (37 GB): the first
    reduce-scatter pass launches 3^18 one-wave units (2.5e10 work-items); in one dispatch only a
    part of its workgroups would run. Sampled columns against the exact sums of the inputs,
    which are read back before the call."""
    import paper_2602_17254_amd as T

    dims, E = (27, 27, 27), 472_512
    plan = T.trivance_plan(dims, "B")
    n = plan.n
    _say(f"[split] dims={dims} variant=B E={E} int32 default limit")
    torch.cuda.empty_cache()
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    buf = torch.randint(-1000, 1000, (n, E), dtype=torch.int32, device="cuda", generator=g)
    try:
        cols = torch.linspace(0, E - 1, 1024, device="cuda").round().long().unique()
        want = buf[:, cols].cpu().numpy().astype(np.int64).sum(axis=0).astype(np.int32)
        T.trivance_allreduce_emulated(buf, plan)
        torch.cuda.synchronize()
        got = buf[:, cols].cpu().numpy()
        bad = np.argwhere(got != want[None, :])
        assert bad.size == 0, f"{bad.shape[0]} of {got.size} sampled cells differ, e.g. {bad[:3].tolist()}"
        # every rank holds the same vector: first, middle and last rank in full
        rows = buf[[0, n // 2, n - 1]].cpu().numpy()
        assert (rows == rows[0][None]).all()
    finally:
        del buf
        torch.cuda.empty_cache()
