"""Dead-partial poisoning on the GPU: a pass must read only partials that are still live.

The passes run one at a time through the C ABI (trivance_allreduce_emulated_steps[_ws]). After
each pass every location that no later pass may read before writing it is overwritten with NaN:

* bandwidth-optimal variant: after reduce-scatter step t a block j of collective c is live on
  rank r only while, in every dimension q, the offset (r_q - j_q) mod side_q is one the tree of
  that side has not forwarded yet after the steps collective c took along q (multiples of 3^k on
  sides that are powers of three, Sec. 4.3; the plan's own tables otherwise, Sec. 4.4). The
  all-gather pass of step t restores the live set from before that step.
* latency-optimal variant on sides that are not powers of three: between passes the rank buffers
  and the workspace half that does not hold the current partial sums are dead.

A read of a dead partial would carry a NaN into the result; the final buffers must instead equal
the unpoisoned run, and the oracle, bit for bit. The host checker of the same sets is
tests/test_race_free.py.
"""

import os
import shutil
import sys

import numpy as np
import pytest

from gpu_util import assert_matches_oracle, run_hip

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu_present():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2602_17254_amd as T

    T.binding._lib()  # fails loudly when the native library is missing
    yield


def _is_pow3(s):
    while s % 3 == 0:
        s //= 3
    return s == 1


def _levels(s):
    k, p = 0, 1
    while p < s:
        p *= 3
        k += 1
    return k


@pytest.fixture(scope="module")
def tree_alive(tmp_path_factory):
    """alive[side][m]: offsets of the plan's tree of that side not forwarded before step m."""
    if shutil.which("g++") is None:
        pytest.skip("g++ not found")
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import test_nonpow3_trees as tt

    sides = [7, 8, 20, 32, 4, 5, 2, 100]
    trees = tt.plan_trees(sides, str(tmp_path_factory.mktemp("poison")))
    return {s: trees[s]["alive"] for s in sides}


def _alive(side, m, tree_alive):
    if _is_pow3(side):
        return np.arange(side) % 3 ** m == 0
    out = np.zeros(side, dtype=bool)
    out[tree_alive[side][m]] = True
    return out


def _live_mask(plan, E, taken, tree_alive):
    """[n, E] boolean: columns whose partial is live on each rank when collective c has taken
    taken[c][q] reduce-scatter steps along dimension q."""
    import paper_2602_17254_amd as T

    dims, n, D = plan.dims, plan.n, plan.D
    coords = np.array(np.unravel_index(np.arange(n), dims, order="F")).T  # [n, D], dim 0 fastest
    live = np.ones((D, n, n), dtype=bool)
    for c in range(D):
        for q, s in enumerate(dims):
            ok = _alive(s, taken[c][q], tree_alive)
            off = (coords[:, None, q] - coords[None, :, q]) % s
            live[c] &= ok[off]
    col_seg = np.full(E, -1, dtype=np.int64)
    col_blk = np.full(E, -1, dtype=np.int64)
    for c in range(D):
        for j in range(n):
            b, e = T.trivance_block_range(plan, E, c, j)
            col_seg[b:e], col_blk[b:e] = c, j
    assert (col_seg >= 0).all(), "blocks of all segments tile the buffer"
    return live[col_seg[None, :], np.arange(n)[:, None], col_blk[None, :]]


B_CASES = [(9,), (27,), (3, 3), (9, 9), (3, 3, 3), (3, 9), (7,), (8,), (20,), (32,), (100,),
           (4, 4), (5, 7), (9, 8), (2, 3, 4)]


@pytest.mark.parametrize("dims", B_CASES, ids=lambda d: "x".join(map(str, d)))
def test_bandwidth_optimal_reads_only_live_partials(dims, tree_alive):
    import paper_2602_17254_amd as T

    n, D = int(np.prod(dims)), len(dims)
    E = 64 * D * n * 2 + 12
    V = (np.random.default_rng(31 * n + D).standard_normal((n, E)) *
         np.logspace(-3, 3, E)).astype(np.float32)
    _say(f"[poison B] dims={dims} E={E}")
    plan = T.trivance_plan(dims, "B")
    S, P = plan.num_steps, plan.num_passes
    assert P == 2 * S
    # steps taken along each dimension after the first m reduce-scatter passes, per collective
    taken = [[[0] * D for _ in range(D)]]
    for t in range(S):
        nxt = [list(x) for x in taken[-1]]
        for c in range(D):
            _, dim, _ = T.trivance_plan_step(plan, t, c)
            nxt[c][dim] += 1
        taken.append(nxt)
    for c in range(D):
        assert taken[S][c] == [_levels(s) for s in dims]
    buf = torch.from_numpy(V).cuda()
    nan = torch.tensor(float("nan"), device="cuda")
    poisoned = 0
    for p in range(P):
        T.trivance_allreduce_emulated_steps(buf, plan, p, p + 1)
        m = p + 1 if p < S else 2 * S - 1 - p
        dead = ~torch.from_numpy(_live_mask(plan, E, taken[m], tree_alive)).cuda()
        poisoned += int(dead.sum())
        buf = torch.where(dead, nan, buf)
    torch.cuda.synchronize()
    assert poisoned > 0
    got = buf.cpu().numpy()
    assert not np.isnan(got).any()
    clean = run_hip(V, dims, "B")
    assert np.array_equal(got.view(np.uint32), clean.view(np.uint32))
    assert_matches_oracle(got, V, dims, "B", what=f"poisoned B {dims}")


L_CASES = [(2,), (4,), (8,), (7,), (32,), (100,), (4, 4), (5, 7), (2, 3, 4), (9, 8)]


@pytest.mark.parametrize("dims", L_CASES, ids=lambda d: "x".join(map(str, d)))
def test_latency_slots_read_only_the_current_state(dims):
    import paper_2602_17254_amd as T

    n, D = int(np.prod(dims)), len(dims)
    E = 64 * D * 3 + 4
    V = (np.random.default_rng(17 * n + D).standard_normal((n, E)) *
         np.logspace(-3, 3, E)).astype(np.float32)
    _say(f"[poison L] dims={dims} E={E}")
    plan = T.trivance_plan(dims, "L")
    S = plan.num_passes
    nws = T.trivance_workspace_bytes(plan, E) // 4
    halves = 2 if S >= 3 else 1
    half = nws // halves
    assert nws > 0 and half * halves == nws
    ws = torch.full((nws,), float("nan"), dtype=torch.float32, device="cuda")
    buf = torch.from_numpy(V).cuda()
    for p in range(S):
        T.trivance_allreduce_emulated_steps_ws(buf, plan, ws, p, p + 1)
        if p < S - 1:
            # state p + 1 sits in half p % 2: the rank buffers and the other half are dead
            buf.fill_(float("nan"))
            if halves == 2:
                o = (p + 1) % 2
                ws[o * half:(o + 1) * half].fill_(float("nan"))
    torch.cuda.synchronize()
    got = buf.cpu().numpy()
    assert not np.isnan(got).any()
    clean = run_hip(V, dims, "L")
    assert np.array_equal(got.view(np.uint32), clean.view(np.uint32))
    assert_matches_oracle(got, V, dims, "L", what=f"poisoned L {dims}")
