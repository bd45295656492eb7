"""Large rank counts on the GPU, checked by properties that hold at any size (CPU-side numpy).

* int32: every rank ends with the exact column sums (Sec. 2.2), wrapping modulo 2^32, checked
  on every column of every rank.
* fp32: every element within 4 ceil(log3 n) 2^-23 sum|v| of the fp64 column sum.

Cases: 59,049 ranks (3^10) on a ring and on a 243 x 243 torus, latency-optimal, with 1,028
elements per rank (the first four ring passes run the generic cycle kernel on cycles of up to
59,049 rows); 531,441 ranks (3^12) on a ring with one 16-byte vector per rank; 6,561 ranks
bandwidth-optimal on a ring and on a 27 x 27 x 9 torus with 820 and 823 granules per rank, so that
most of the 6,561 blocks of a segment are empty and the rest hold one granule (millions of work
units per pass, most of them exiting at once).
"""

import sys

import numpy as np
import pytest

from gpu_util import run_hip

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


def _exact_sums(V):
    out = np.empty(V.shape[1], dtype=np.int32)
    for e0 in range(0, V.shape[1], 4096):
        s = V[:, e0:e0 + 4096].astype(np.int64).sum(axis=0)
        out[e0:e0 + 4096] = ((s + 2 ** 31) % 2 ** 32 - 2 ** 31).astype(np.int32)
    return out


def _ceil_log3(n):
    s, p = 0, 1
    while p < n:
        p *= 3
        s += 1
    return s


CASES = [((59049,), "L", 1028), ((243, 243), "L", 1028), ((531441,), "L", 4),
         ((6561,), "B", 820 * 64), ((27, 27, 9), "B", 823 * 64)]


@pytest.mark.parametrize("dims,variant,E", CASES,
                         ids=["x".join(map(str, c[0])) + f"-{c[1]}-E{c[2]}" for c in CASES])
def test_int32_exact_sums_at_large_rank_counts(dims, variant, E):
    n = int(np.prod(dims))
    _say(f"[max sizes] dims={dims} variant={variant} E={E} int32")
    V = np.random.default_rng(n + E).integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    want = _exact_sums(V)
    got = run_hip(V, dims, variant)
    for r0 in range(0, n, 4096):
        bad = np.nonzero((got[r0:r0 + 4096] != want[None, :]).any(axis=1))[0]
        assert bad.size == 0, f"rank {r0 + bad[0]} differs from the exact column sums"


def test_fp32_bound_at_59049_ranks():
    dims, E = (59049,), 1028
    n = dims[0]
    _say(f"[max sizes] dims={dims} variant=L E={E} fp32")
    V = np.random.default_rng(7).standard_normal((n, E), dtype=np.float32)
    got = run_hip(V, dims, "L")
    exact = V.astype(np.float64).sum(axis=0)
    bound = 4.0 * _ceil_log3(n) * 2.0 ** -23 * np.abs(V).astype(np.float64).sum(axis=0)
    for r0 in range(0, n, 4096):
        err = np.abs(got[r0:r0 + 4096].astype(np.float64) - exact[None, :])
        assert (err <= bound[None, :]).all(), f"ranks {r0}.. exceed the fp64 bound"
