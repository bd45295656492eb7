"""GPU parity of the latency-optimal variant on rings and tori whose sides are not all powers of
three (Sec. 4.2 with Sec. 4.4): the slot-step kernels through the C ABI against the oracle
(oracle/latency_nonpow3.py), element by element; int32 bit-exact, fp32 identical bits (and within
the summation bound). The workspace is filled with NaN before every call, so a read of stale
partials would show.
"""

import sys

import numpy as np
import pytest

from gpu_util import assert_matches_oracle, run_hip
from oracle import allreduce, congestion, latency_nonpow3

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


# rings and tori: one to four steps, one to 64 partials per rank, the 16-byte path (E % 4 == 0)
# and the scalar one (odd E), ragged tails, empty segments (E < 64 D) and E = 0
CASES = [((2,), 1001), ((2,), 64 * 2 * 3 + 4), ((4,), 64 * 4 + 12), ((5,), 777), ((7,), 64 * 7 * 2 + 4),
         ((8,), 64 * 8 * 3 + 8), ((8,), 5), ((10,), 1234), ((20,), 64 * 20 + 4), ((32,), 64 * 32 + 4),
         ((32,), 3001), ((64,), 64 * 64 + 8), ((100,), 2001), ((728,), 64 * 4 + 4), ((2200,), 260),
         ((4, 4), 64 * 16 * 2 + 12), ((2, 3), 101), ((3, 8), 64 * 24 + 4), ((8, 3), 999),
         ((5, 7), 64 * 35 + 20), ((1, 8), 300), ((2, 3, 4), 64 * 24 * 3 + 8),
         ((4, 4, 4), 64 * 3 + 4), ((2, 2, 2, 2), 64 * 4 + 4), ((32, 32), 64 * 2 * 3 + 8),
         ((8, 64), 64 * 2 * 2 + 4), ((16, 16, 16), 64 * 3 + 12), ((4, 4), 0), ((8,), 0),
         ((9, 8), 64 * 2 + 4), ((3, 3, 2), 64 * 3 + 4)]


def _id(c):
    dims, E = c
    return "x".join(map(str, dims)) + f"-E{E}"


@pytest.mark.parametrize("dtype", ["f32", "i32"])
@pytest.mark.parametrize("dims,E", CASES, ids=[_id(c) for c in CASES])
def test_latency_nonpow3_matches_oracle(dims, E, dtype):
    n = int(np.prod(dims))
    seed = 5 * n + E + (1 if dtype == "i32" else 0)
    rng = np.random.default_rng(seed)
    _say(f"[latency nonpow3] dims={dims} E={E} dtype={dtype} seed={seed}")
    if dtype == "f32":
        V = (rng.standard_normal((n, E)) * np.logspace(-3, 3, max(E, 1))[:E]).astype(np.float32)
    else:
        V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    got = run_hip(V, dims, "L")
    assert_matches_oracle(got, V, dims, "L", what=f"L {dims} E={E} {dtype}")
    if dtype == "i32":
        np.testing.assert_array_equal(got, np.broadcast_to(allreduce.exact_int_sum(V), got.shape))


@pytest.mark.parametrize("dims", [(8,), (32,), (5, 7)], ids=lambda d: "x".join(map(str, d)))
def test_latency_nonpow3_pass_ranges_and_split_dispatches(dims):
    """Pass ranges run one after another with one workspace equal one full call; a plan whose
    launches are split into dispatches of 1024 work-items gives the same bits."""
    import paper_2602_17254_amd as T

    n = int(np.prod(dims))
    E = 64 * len(dims) * 3 + 4
    V = np.random.default_rng(n).standard_normal((n, E)).astype(np.float32)
    _say(f"[latency nonpow3 steps] dims={dims} E={E}")
    plan = T.trivance_plan(dims, "L")
    ws = torch.full(((T.trivance_workspace_bytes(plan, E) + 3) // 4,), float("nan"),
                    dtype=torch.float32, device="cuda")
    buf = torch.from_numpy(V).cuda()
    for p in range(plan.num_passes):
        T.trivance_allreduce_emulated_steps_ws(buf, plan, ws, p, p + 1)
    torch.cuda.synchronize()
    want = latency_nonpow3.latency_optimal(V, dims)
    got = buf.cpu().numpy()
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    split = run_hip(V, dims, "L", dispatch_items=1024)
    assert np.array_equal(split.view(np.uint32), want.view(np.uint32))


def test_latency_nonpow3_misaligned_rows_and_workspace():
    """A [n, E] view that is not 16-byte aligned, and a workspace that is not either: the scalar
    path gives the same bits."""
    import paper_2602_17254_amd as T

    dims, E = (7,), 64 * 7 * 2 + 8
    n = 7
    V = np.random.default_rng(77).standard_normal((n, E)).astype(np.float32)
    plan = T.trivance_plan(dims, "L")
    flat = torch.zeros(n * E + 1, dtype=torch.float32, device="cuda")
    view = flat[1:].view(n, E)
    view.copy_(torch.from_numpy(V))
    nws = (T.trivance_workspace_bytes(plan, E) + 3) // 4
    wflat = torch.full((nws + 1,), float("nan"), dtype=torch.float32, device="cuda")
    ws = wflat[1:]
    assert view.data_ptr() % 16 != 0 and ws.data_ptr() % 16 != 0
    T.trivance_allreduce_emulated_ws(view, plan, ws)
    torch.cuda.synchronize()
    assert_matches_oracle(view.cpu().numpy(), V, dims, "L", what="misaligned L 7")


@pytest.mark.parametrize("dims", [(8,), (7,), (32,), (64,), (4, 4), (5, 7), (32, 32), (8, 64)],
                         ids=lambda d: "x".join(map(str, d)))
def test_latency_nonpow3_congestion(dims):
    """Per-link message counts: a rank sends towards a side when its peer there takes a partial
    from it; the GPU counter against the oracle's link walk."""
    import paper_2602_17254_amd as T

    _say(f"[latency nonpow3 congestion] dims={dims}")
    got = T.trivance_congestion(T.trivance_plan(dims, "L"))
    np.testing.assert_array_equal(got, congestion.link_loads(dims, "L"))
