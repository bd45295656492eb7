"""The AllReduce call under HIP stream capture: every kernel family's passes recorded into one graph.

A call enqueues kernel launches only (no allocation, copy or memset through the runtime), so a
caller can capture it once and replay it. Each case captures trivance_allreduce_emulated (with
the workspace form for the partial-sum programs of sides that are not powers of three), then
replays the graph three times; before every replay the inputs are restored eagerly, outside the
graph, and after it the result must equal the eager call's bit for bit. The first case also runs
an eager call between two replays.
"""

import sys

import numpy as np
import pytest

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


# (dims, variant, elems): latency steps (split tiles and the generic kernel), block steps, tree
# steps on rings and tori, partial-sum programs with one pass (result copied back), two passes
# and four, the scalar path (odd elems)
CASES = [((9,), "L", 1024), ((81,), "L", 64 * 81 + 4), ((2187,), "L", 260), ((27, 27), "B", 4100),
         ((3, 3, 3), "B", 3001), ((8,), "B", 5000), ((5, 7), "B", 64 * 35 + 4), ((2,), "L", 1000),
         ((2,), "L", 999), ((7,), "L", 64 * 7 + 4), ((4, 4), "L", 64 * 32 + 4), ((32,), "L", 3001)]


def _id(c):
    dims, v, E = c
    return "x".join(map(str, dims)) + f"-{v}-E{E}"


@pytest.mark.parametrize("dims,variant,E", CASES, ids=[_id(c) for c in CASES])
def test_captured_allreduce_replays_equal_the_eager_call(dims, variant, E):
    import paper_2602_17254_amd as T

    n = int(np.prod(dims))
    _say(f"[graph] dims={dims} variant={variant} E={E}")
    plan = T.trivance_plan(dims, variant)
    V = torch.from_numpy(np.random.default_rng(11 * n + E).standard_normal((n, E))
                         .astype(np.float32)).cuda()
    wsb = T.trivance_workspace_bytes(plan, E)
    ws = torch.empty(((wsb + 3) // 4,), dtype=torch.float32, device="cuda") if wsb else None

    def call(buf):
        if ws is None:
            T.trivance_allreduce_emulated(buf, plan)
        else:
            T.trivance_allreduce_emulated_ws(buf, plan, ws)

    want = V.clone()
    call(want)
    torch.cuda.synchronize()

    buf = torch.empty_like(V)
    buf.copy_(V)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(buf)  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(buf)
    torch.cuda.synchronize()
    for k in range(3):
        buf.copy_(V)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(buf.view(torch.int32), want.view(torch.int32)), f"replay {k}"
        if k == 0 and dims == (9,):
            other = V.clone()
            call(other)  # eager work between replays
            torch.cuda.synchronize()
            assert torch.equal(other.view(torch.int32), want.view(torch.int32))
    del g
