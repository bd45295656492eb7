"""GPU parity on paths and values the other tests leave out.

* The generic latency-optimal kernel (cycles of 2187 ranks and more) on the 16-byte path: rings
  of 2187 and a 2187 x 3 torus with E % 4 == 0, fp32 and int32, in full.
* IEEE fp32 specials through every kernel family (latency-optimal steps, block steps, tree steps):
  subnormal inputs (from 2^-149 up to about 1e-38), signed zeros, sums that overflow to +/-inf,
  inf - inf and NaN inputs. The oracle adds in numpy float32 (IEEE round-to-nearest-even, no
  flush to zero); the results must agree bit for bit, a NaN matching any NaN (the GPU and the
  host write different NaN payloads for an invalid operation).
* The 243-ring bandwidth-optimal workload's int32 companion (8,388,608 int32 per rank) compared
  in every column against the exact column sums, and every rank against rank 0.
"""

import sys

import numpy as np
import pytest

from gpu_util import assert_matches_oracle, assert_same_bits, run_hip
from oracle import allreduce, nonpow3, partition
from paper_2602_17254_amd import inputs

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


# ---- the generic latency kernel with 16-byte vectors ----

@pytest.mark.parametrize("dtype", ["f32", "i32"])
@pytest.mark.parametrize("dims,E", [((2187,), 1028), ((2187,), 64 * 4 * 3 + 4), ((2187, 3), 1028)],
                         ids=["2187-E1028", "2187-E772", "2187x3-E1028"])
def test_generic_latency_kernel_16_byte_path(dims, E, dtype):
    n = int(np.prod(dims))
    assert E % 4 == 0
    seed = 2187 + E + len(dims)
    rng = np.random.default_rng(seed)
    _say(f"[edge] generic latency kernel dims={dims} E={E} dtype={dtype} seed={seed}")
    if dtype == "f32":
        V = rng.standard_normal((n, E), dtype=np.float32)
    else:
        V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, E), dtype=np.int32)
    got = run_hip(V, dims, "L")
    assert_matches_oracle(got, V, dims, "L", what=f"{dims} E={E} {dtype} L")
    if dtype == "i32":
        np.testing.assert_array_equal(got, np.broadcast_to(allreduce.exact_int_sum(V), got.shape))


# ---- IEEE fp32 specials ----

def _special_inputs(n: int, E: int, seed: int) -> np.ndarray:
    """Columns cycle through six kinds of values:
    0 subnormals k 2^-149 with |k| < 2^20 (their sums stay subnormal or reach small normals);
    1 random signs of zero (a column of -0 alone sums to -0, any +0 makes +0);
    2 huge values of one sign per column (sums overflow to +inf or -inf);
    3 huge values of random signs (overflow to inf in one order, inf - inf = NaN in another);
    4 N(0,1) with every fourth value replaced by a subnormal or a signed zero;
    5 N(0,1) with one NaN or inf input per column."""
    rng = np.random.default_rng(seed)
    V = rng.standard_normal((n, E)).astype(np.float32)
    kind = np.arange(E) % 6
    tiny = np.float32(2.0 ** -149)
    for c in np.nonzero(kind == 0)[0]:
        V[:, c] = rng.integers(-(2 ** 20), 2 ** 20, n).astype(np.float32) * tiny
    for c in np.nonzero(kind == 1)[0]:
        V[:, c] = np.where(rng.random(n) < (0.5 if c % 12 == 1 else 0.0), 0.0, -0.0)
    for c in np.nonzero(kind == 2)[0]:
        V[:, c] = np.float32(3.0e38) * (1 if c % 4 < 2 else -1) * rng.uniform(0.2, 1.0, n)
    for c in np.nonzero(kind == 3)[0]:
        V[:, c] = np.float32(3.0e38) * np.where(rng.random(n) < 0.5, 1, -1) * rng.uniform(0.5, 1.0, n)
    for c in np.nonzero(kind == 4)[0]:
        rows = rng.random(n) < 0.25
        V[rows, c] = np.where(rng.random(rows.sum()) < 0.5,
                              rng.integers(-1000, 1000, rows.sum()).astype(np.float32) * tiny,
                              -0.0)
    for c in np.nonzero(kind == 5)[0]:
        V[rng.integers(n), c] = [np.nan, np.inf, -np.inf][c % 3]
    return V.astype(np.float32)


def _oracle(V, dims, variant):
    with np.errstate(over="ignore", invalid="ignore"):
        if variant == "L":
            return allreduce.latency_optimal(V, dims)
        if nonpow3.is_tree(dims):
            if len(dims) == 1:
                return nonpow3.bandwidth_optimal_ring(V)
            seg, blk = partition.column_labels(V.shape[1], len(dims), V.shape[0])
            return nonpow3.bandwidth_optimal_torus_columns(V, dims, seg, blk)
        return allreduce.bandwidth_optimal(V, dims)


SPECIAL_CASES = [((9,), "L", 64 * 9 + 36), ((27,), "L", 64 * 27 * 2 + 12), ((9, 9), "L", 64 * 81 + 4),
                 ((27,), "B", 64 * 27 * 3 + 8), ((243,), "B", 64 * 243 + 4), ((9, 9), "B", 64 * 81 * 2),
                 ((3, 3, 3), "B", 64 * 27 * 3 + 20), ((8,), "B", 64 * 8 * 4 + 4),
                 ((64,), "B", 64 * 64 * 2 + 8), ((4, 8), "B", 64 * 32 * 2 * 2 + 12),
                 ((9,), "L", 1001), ((8,), "B", 999)]


@pytest.mark.parametrize("dims,variant,E", SPECIAL_CASES,
                         ids=["x".join(map(str, d)) + f"-{v}-E{e}" for d, v, e in SPECIAL_CASES])
def test_fp32_specials_bit_exact(dims, variant, E):
    n = int(np.prod(dims))
    seed = 31 * n + E
    _say(f"[edge] fp32 specials dims={dims} variant={variant} E={E} seed={seed}")
    V = _special_inputs(n, E, seed)
    got = run_hip(V, dims, variant)
    want = _oracle(V, dims, variant)
    assert_same_bits(got, want, f"specials {dims} {variant} E={E}")
    # the inputs do reach every kind of result
    assert np.isnan(want).any() and np.isposinf(want).any() and np.isneginf(want).any()
    z = (want == 0) & np.signbit(want)
    assert z.any() and ((want == 0) & ~np.signbit(want)).any()
    sub = (want != 0) & (np.abs(want) < np.finfo(np.float32).tiny)
    assert sub.any()


# ---- the 243-ring int32 companion in every column ----

def test_ring243_int32_companion_every_column():
    import paper_2602_17254_amd as T

    w = inputs.WORKLOADS["ring243_B_32MiB"]
    _say(f"[edge] {w.name} int32, all {w.elems} columns against the exact sums")
    Vi = inputs.uniform_i32(w.int_seed, w.n, w.elems, *w.int_range)
    buf = torch.from_numpy(Vi).cuda()
    T.trivance_allreduce_emulated(buf, T.trivance_plan(w.dims, w.variant))
    torch.cuda.synchronize()
    try:
        # every rank holds rank 0's vector
        assert bool((buf[1:] == buf[0:1]).all().item())
        row0 = buf[0].cpu().numpy()
        step = 1 << 20
        for e0 in range(0, w.elems, step):
            want = allreduce.exact_int_sum(Vi[:, e0:e0 + step])
            bad = np.nonzero(row0[e0:e0 + step] != want)[0]
            assert bad.size == 0, f"columns {(e0 + bad[:5]).tolist()} differ from the exact sums"
    finally:
        del buf
        torch.cuda.empty_cache()
