"""Helpers of the GPU parity tests: run the HIP path, run the oracle, compare."""

from __future__ import annotations

import numpy as np

from oracle import allreduce, nonpow3, partition, schedule

VARIANT_NAMES = {"L": "latency-optimal", "B": "bandwidth-optimal"}


def run_hip(V: np.ndarray, dims, variant: str, placement: str = "natural",
            dispatch_items: int | None = None) -> np.ndarray:
    """Run the HIP path on a copy of V; with dispatch_items, on a plan whose launches are split
    into dispatches of at most that many work-items."""
    import torch

    import paper_2602_17254_amd as T

    plan = T.trivance_plan(dims, variant, placement)
    if dispatch_items is not None:
        plan = T.trivance_plan_with_dispatch_limit(plan, dispatch_items)
    buf = torch.from_numpy(np.ascontiguousarray(V)).cuda()
    ws_bytes = T.trivance_workspace_bytes(plan, V.shape[1])
    if ws_bytes:
        # the partial sums of the latency-optimal variant on sides that are not powers of three;
        # filled with NaN so that a read of stale contents would show
        ws = torch.full(((ws_bytes + 3) // 4,), float("nan"), dtype=torch.float32, device="cuda")
        T.trivance_allreduce_emulated_ws(buf, plan, ws)
    else:
        T.trivance_allreduce_emulated(buf, plan)
    torch.cuda.synchronize()
    return buf.cpu().numpy()


def assert_matches_oracle(got: np.ndarray, V: np.ndarray, dims, variant: str, col_seg=None,
                          col_blk=None, what: str = "") -> dict:
    """Element-by-element comparison against the schedule-ordered oracle.

    int32: bit-exact. fp32: |g - o| <= 1e-6 |o| elementwise (the oracle's order is the kernel's,
    so the difference is expected to be exactly zero, which is asserted as well), and every
    element within 4 S 2^-23 sum|v| of the fp64 sum."""
    if variant == "L" and nonpow3.is_tree(dims):
        from oracle import latency_nonpow3

        want = latency_nonpow3.latency_optimal(V, dims, col_seg=col_seg)
    elif variant == "L":
        want = allreduce.latency_optimal(V, dims, col_seg=col_seg)
    elif nonpow3.is_tree(dims) and len(dims) == 1 and dims[0] <= 300:
        want = nonpow3.bandwidth_optimal_ring(V, col_blk=col_blk)
    elif nonpow3.is_tree(dims):
        # the gather form, equal bit for bit to the mailbox form (pinned in the oracle tests)
        if col_seg is None or col_blk is None:
            col_seg, col_blk = partition.column_labels(V.shape[1], len(dims), V.shape[0])
        want = nonpow3.bandwidth_optimal_torus_columns(V, dims, col_seg, col_blk)
    else:
        want = allreduce.bandwidth_optimal(V, dims, col_seg=col_seg, col_blk=col_blk)
    info = {}
    if V.dtype == np.int32:
        bad = np.argwhere(got != want)
        assert bad.size == 0, f"{what}: int32 mismatch at {bad[:5].tolist()}"
        info["int_exact"] = True
        return info
    g = got.astype(np.float64)
    o = want.astype(np.float64)
    diff = np.abs(g - o)
    rel_ok = diff <= 1e-6 * np.abs(o)
    assert rel_ok.all(), f"{what}: fp32 beyond 1e-6 relative at {np.argwhere(~rel_ok)[:5].tolist()}"
    assert_same_bits(got, want, what)
    err = np.abs(g - allreduce.fp64_sum(V)[None, :])
    bound = allreduce.fp32_error_bound(V)[None, :]
    assert (err <= bound).all(), f"{what}: fp32 outside the fp64 summation bound"
    info["max_rel_vs_oracle"] = float((diff / np.maximum(np.abs(o), 1e-300)).max()) if o.size else 0.0
    info["fp64_bound_margin"] = float((err / np.maximum(bound, 1e-300)).max()) if o.size else 0.0
    return info


def assert_same_bits(got: np.ndarray, want: np.ndarray, what: str = "") -> None:
    """fp32 results identical bit for bit (so +0 and -0 differ); a NaN matches any NaN, since the
    GPU and the host write different NaN payloads for an invalid operation such as inf - inf."""
    assert got.shape == want.shape, f"{what}: shape {got.shape} != {want.shape}"
    g = np.ascontiguousarray(got).view(np.uint32)
    w = np.ascontiguousarray(want).view(np.uint32)
    both_nan = np.isnan(got) & np.isnan(want)
    bad = np.argwhere((g != w) & ~both_nan)
    assert bad.size == 0, (f"{what}: fp32 differs in bits from the schedule-ordered oracle at "
                           f"{bad[:5].tolist()}")


def sample_columns(E: int, D: int, n: int, variant: str, seed: int, per_block: int = 2,
                   max_blocks: int | None = None, dims=None, placement: str = "natural"):
    """Deterministic column sample of a large run: for every (segment, block) its first and last
    element and `per_block` seeded random ones (variant B), or segment ends plus random columns
    (variant L). With max_blocks, only that many seeded blocks per segment (always including the
    first and last) are sampled. Returns sorted unique columns with their labels."""
    rng = np.random.default_rng(seed)
    cols = []
    if variant == "B":
        for row in partition.block_bounds(E, D, n):
            pick = range(len(row))
            if max_blocks is not None and max_blocks < len(row):
                pick = sorted({0, len(row) - 1} |
                              set(rng.choice(len(row), max_blocks - 2, replace=False).tolist()))
            for i in pick:
                b, e = row[i]
                if e > b:
                    cols += [b, e - 1] + rng.integers(b, e, per_block).tolist()
    else:
        for (b, e) in partition.segment_bounds(E, D):
            if e > b:
                cols += [b, e - 1] + rng.integers(b, e, 2000).tolist()
    cols = np.unique(np.array(cols, dtype=np.int64))
    if placement == "schedule":
        # the same granule ranges, now labelled with the block placed there
        seg, blk = placement_labels(E, dims, cols)
    else:
        seg, blk = partition.column_labels(E, D, n, cols)
    return cols, seg, blk


def placement_labels(E: int, dims, cols=None):
    from oracle import placement

    return placement.column_labels(E, dims, cols)
