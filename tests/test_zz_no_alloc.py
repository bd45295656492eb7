"""GPU: trivance_congestion_noalloc, the allocation-free form of trivance_congestion, called
through the C ABI, against trivance_congestion and the oracle's link walk, on two calls in a row
(the second with a smaller plan, so the scratch still holds the first call's larger contents),
with routing variants and the size limit."""

import ctypes
import sys

import numpy as np
import pytest

from oracle import congestion

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _noalloc(plan, routing="scheduled"):
    """Direct C-ABI call: length query, then the call into a host array."""
    import paper_2602_17254_amd as T

    lib = T.binding._lib()
    topo = T.binding._topology(plan, routing)
    need = lib.trivance_congestion_noalloc(plan.handle, ctypes.byref(topo), None, 0)
    assert need == plan.num_passes * plan.n * 2 * plan.D
    out = np.full(need, -7, dtype=np.int64)
    rc = lib.trivance_congestion_noalloc(plan.handle, ctypes.byref(topo),
                                         out.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), need)
    assert rc == 0, T.binding._lib().trivance_strerror(rc)
    return out.reshape(plan.num_passes, plan.n, 2 * plan.D)


def test_noalloc_congestion_matches_allocating_form_twice():
    import paper_2602_17254_amd as T

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    T.binding._lib()
    cases = [((27, 27), "B", "scheduled"), ((9,), "L", "scheduled"), ((16, 16, 16), "B", "scheduled"),
             ((8,), "B", "scheduled"), ((27,), "BRUCK", "shortest"), ((3,), "L", "scheduled")]
    for dims, variant, routing in cases:
        _say(f"[noalloc] dims={dims} variant={variant} routing={routing}")
        plan = T.trivance_plan(dims, variant)
        got = _noalloc(plan, routing)
        want = T.trivance_congestion(plan, routing)
        np.testing.assert_array_equal(got, want)
        np.testing.assert_array_equal(got, congestion.link_loads(dims, variant, routing))


def test_noalloc_congestion_rejects_plans_beyond_the_scratch():
    import paper_2602_17254_amd as T

    lib = T.binding._lib()
    plan = T.trivance_plan((27, 27, 27), "B")  # 18 passes x 19683 ranks x 6 ports > 2^20
    topo = T.binding._topology(plan, "scheduled")
    need = lib.trivance_congestion_noalloc(plan.handle, ctypes.byref(topo), None, 0)
    assert need == 18 * 19683 * 6 > 2 ** 20
    out = np.zeros(need, dtype=np.int64)
    rc = lib.trivance_congestion_noalloc(plan.handle, ctypes.byref(topo),
                                         out.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), need)
    assert rc == -6 and lib.trivance_strerror(rc) == b"request exceeds the fixed device scratch"
    assert not out.any()
    small = np.zeros(3, dtype=np.int64)
    p9 = T.trivance_plan((9,), "L")
    t9 = T.binding._topology(p9, "scheduled")
    assert lib.trivance_congestion_noalloc(p9.handle, ctypes.byref(t9),
                                           small.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                           3) == -5
    # after a rejected call the scratch still serves a valid one
    np.testing.assert_array_equal(_noalloc(p9), congestion.link_loads((9,), "L"))
