"""Parity on a seeded random sample of shapes: rings and tori of one to three dimensions with sides
of 1 to 30 (powers of three or not, equal or not), both variants, fp32 and int32, against the
oracle element by element (fp32 identical bits, int32 exact).

The sample (128 shapes) is drawn once from a fixed seed, so every case has a stable name; it
complements the hand-picked shapes of the other parity tests with combinations nobody chose:
unequal sides mixing trees and powers of three, sides of 1 inside tori, element counts with ragged
tails, the scalar path (E % 4 != 0) and empty segments (E < 64 D). Shapes a plan rejects by design (more partial
sums than a latency-optimal plan keeps) are skipped with the reason.
"""

import sys

import numpy as np
import pytest

from gpu_util import assert_matches_oracle, run_hip

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


def _sample(count=128, seed=20260217, max_ranks=240):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        D = int(rng.integers(1, 4))
        dims = tuple(int(rng.integers(1, 31)) for _ in range(D))
        n = int(np.prod(dims))
        if n < 2 or n > max_ranks:
            continue
        kind = int(rng.integers(0, 4))
        if kind == 0:
            E = int(rng.integers(1, 64 * D))                      # empty segments
        elif kind == 1:
            E = 64 * D * n * int(rng.integers(1, 3)) + 4 * int(rng.integers(0, 16))
        elif kind == 2:
            E = int(rng.integers(64 * D, 64 * D * n * 2)) | 1     # odd: the scalar path
        else:
            E = int(rng.integers(64 * D, 64 * D * n * 3)) & ~3    # the 16-byte path, ragged
        out.append((dims, E))
    return out


CASES = _sample()


@pytest.mark.parametrize("variant", ["L", "B"])
@pytest.mark.parametrize("dims,E", CASES, ids=["x".join(map(str, d)) + f"-E{E}" for d, E in CASES])
def test_random_shape_matches_oracle(dims, E, variant):
    import paper_2602_17254_amd as T

    try:
        T.trivance_plan(dims, variant)
    except RuntimeError as e:
        assert "unsupported" in str(e)
        pytest.skip(f"plan rejects {dims} {variant}: {e}")
    n = int(np.prod(dims))
    seed = 7 * n + 3 * E + (variant == "B")
    _say(f"[random] dims={dims} E={E} variant={variant} seed={seed}")
    rng = np.random.default_rng(seed)
    V = (rng.standard_normal((n, E)) * np.logspace(-4, 4, E)[None, :]).astype(np.float32)
    assert_matches_oracle(run_hip(V, dims, variant), V, dims, variant,
                          what=f"{dims} {variant} E={E} f32")
    Vi = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    assert_matches_oracle(run_hip(Vi, dims, variant), Vi, dims, variant,
                          what=f"{dims} {variant} E={E} i32")
