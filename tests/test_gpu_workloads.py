"""GPU parity at the five named workload sizes, through the same entry point the benchmark times.

Small workloads are compared in full; large ones on a deterministic column sample (for the
bandwidth-optimal variant: first, last and two random elements of every block of every segment;
every step acts column-wise inside a block, so the oracle on those columns with their original
block labels is exact). Congestion counts are compared in full.
"""

import sys

import numpy as np
import pytest

from gpu_util import assert_matches_oracle, sample_columns
from oracle import congestion
from paper_2602_17254_amd import inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _run_full(w, V):
    import paper_2602_17254_amd as T

    plan = T.trivance_plan(w.dims, w.variant, w.placement)
    buf = torch.from_numpy(V).cuda()
    T.trivance_allreduce_emulated(buf, plan)
    torch.cuda.synchronize()
    return buf


def _check_sampled(w, V, buf, seed):
    D = len(w.dims)
    cols, seg, blk = sample_columns(w.elems, D, w.n, w.variant, seed, dims=w.dims,
                                    placement=w.placement)
    idx = torch.from_numpy(cols).cuda()
    got = buf.index_select(1, idx).cpu().numpy()
    return assert_matches_oracle(got, np.ascontiguousarray(V[:, cols]), w.dims, w.variant,
                                 col_seg=seg, col_blk=blk, what=w.name)


def _congestion(w):
    import paper_2602_17254_amd as T

    plan = T.trivance_plan(w.dims, w.variant)
    got = T.trivance_congestion(plan)
    np.testing.assert_array_equal(got, congestion.link_loads(w.dims, w.variant))


def test_ring9_latency_4KiB():
    w = inputs.WORKLOADS["ring9_L_4KiB"]
    _say(f"[workload] {w.name} f32")
    V = inputs.normal_f32(w.seed, w.n, w.elems)
    assert_matches_oracle(_run_full(w, V).cpu().numpy(), V, w.dims, w.variant, what=w.name)
    _say(f"[workload] {w.name} i32")
    Vi = inputs.uniform_i32(w.int_seed, w.n, w.elems, *w.int_range)
    assert_matches_oracle(_run_full(w, Vi).cpu().numpy(), Vi, w.dims, w.variant, what=w.name)
    _congestion(w)


def test_ring81_latency_8MiB():
    w = inputs.WORKLOADS["ring81_L_8MiB"]
    _say(f"[workload] {w.name} f32 (full comparison)")
    V = inputs.normal_f32(w.seed, w.n, w.elems)
    buf = _run_full(w, V)
    assert_matches_oracle(buf.cpu().numpy(), V, w.dims, w.variant, what=w.name)
    _congestion(w)


def test_ring243_bandwidth_32MiB():
    w = inputs.WORKLOADS["ring243_B_32MiB"]
    _say(f"[workload] {w.name} f32 (column sample)")
    V = inputs.normal_f32(w.seed, w.n, w.elems)
    buf = _run_full(w, V)
    _check_sampled(w, V, buf, seed=w.seed)
    del buf
    _say(f"[workload] {w.name} i32 (column sample)")
    Vi = inputs.uniform_i32(w.int_seed, w.n, w.elems, *w.int_range)
    buf = _run_full(w, Vi)
    _check_sampled(w, Vi, buf, seed=w.int_seed)
    # every rank must hold identical bits after the all-gather
    assert bool((buf[1:] == buf[0:1]).all().item())
    del buf
    torch.cuda.empty_cache()


def test_torus27x27_bandwidth_4MiB():
    w = inputs.WORKLOADS["torus27x27_B_4MiB"]
    _say(f"[workload] {w.name} f32 (column sample)")
    V = inputs.normal_f32(w.seed, w.n, w.elems)
    buf = _run_full(w, V)
    _check_sampled(w, V, buf, seed=w.seed)
    assert bool((buf[1:] == buf[0:1]).all().item())
    del buf
    torch.cuda.empty_cache()
    _congestion(w)


def test_torus9x9x9_bandwidth_128MiB():
    import paper_2602_17254_amd as T

    w = inputs.WORKLOADS["torus9x9x9_B_128MiB"]
    _say(f"[workload] {w.name} f32, device-generated inputs (column sample)")
    buf = torch.empty((w.n, w.elems), dtype=torch.float32, device="cuda")
    T.trivance_fill_hash_uniform(buf, w.seed)
    plan = T.trivance_plan(w.dims, w.variant)
    T.trivance_allreduce_emulated(buf, plan)
    torch.cuda.synchronize()
    cols, seg, blk = sample_columns(w.elems, 3, w.n, w.variant, w.seed)
    got = buf.index_select(1, torch.from_numpy(cols).cuda()).cpu().numpy()
    Vs = inputs.hash_uniform(w.seed, w.elems, np.arange(w.n), cols)
    assert_matches_oracle(got, Vs, w.dims, w.variant, col_seg=seg, col_blk=blk, what=w.name)
    del buf
    torch.cuda.empty_cache()


def test_ring8_bandwidth_32MiB_nonpower3():
    """Sec. 4.4 ring of 8 (not a power of three), compared in full, fp32 and int32."""
    w = inputs.WORKLOADS["ring8_B_32MiB"]
    _say(f"[workload] {w.name} f32 (full comparison)")
    V = inputs.normal_f32(w.seed, w.n, w.elems)
    buf = _run_full(w, V)
    assert_matches_oracle(buf.cpu().numpy(), V, w.dims, w.variant, what=w.name)
    _say(f"[workload] {w.name} i32 (full comparison)")
    Vi = inputs.uniform_i32(w.int_seed, w.n, w.elems, *w.int_range)
    assert_matches_oracle(_run_full(w, Vi).cpu().numpy(), Vi, w.dims, w.variant, what=w.name)
    _congestion(w)


def test_ring64_bandwidth_8MiB_nonpower3():
    w = inputs.WORKLOADS["ring64_B_8MiB"]
    _say(f"[workload] {w.name} f32 (column sample)")
    V = inputs.normal_f32(w.seed, w.n, w.elems)
    buf = _run_full(w, V)
    _check_sampled(w, V, buf, seed=w.seed)
    assert bool((buf[1:] == buf[0:1]).all().item())
    _congestion(w)


def _device_hash_workload(w, max_blocks=None):
    """Device-generated U(-1, 1) inputs, one run, then a column sample against the oracle (the
    gather form on the sampled columns with their block labels) and identical bits on all ranks."""
    import paper_2602_17254_amd as T

    D = len(w.dims)
    buf = torch.empty((w.n, w.elems), dtype=torch.float32, device="cuda")
    T.trivance_fill_hash_uniform(buf, w.seed)
    plan = T.trivance_plan(w.dims, w.variant, w.placement)
    T.trivance_allreduce_emulated(buf, plan)
    torch.cuda.synchronize()
    cols, seg, blk = sample_columns(w.elems, D, w.n, w.variant, w.seed, max_blocks=max_blocks,
                                    dims=w.dims, placement=w.placement)
    got = buf.index_select(1, torch.from_numpy(cols).cuda()).cpu().numpy()
    Vs = inputs.hash_uniform(w.seed, w.elems, np.arange(w.n), cols)
    assert_matches_oracle(got, Vs, w.dims, w.variant, col_seg=seg, col_blk=blk, what=w.name)
    assert bool((buf[1:] == buf[0:1]).all().item())
    del buf
    torch.cuda.empty_cache()


def test_torus32x32_bandwidth_8MiB_nonpower3():
    w = inputs.WORKLOADS["torus32x32_B_8MiB"]
    _say(f"[workload] {w.name} f32, device-generated inputs (column sample)")
    _device_hash_workload(w)
    _congestion(w)


def test_torus8x64_bandwidth_8MiB_nonpower3():
    w = inputs.WORKLOADS["torus8x64_B_8MiB"]
    _say(f"[workload] {w.name} f32, device-generated inputs (column sample)")
    _device_hash_workload(w)
    _congestion(w)


def test_torus16x16x16_bandwidth_8MiB_nonpower3():
    w = inputs.WORKLOADS["torus16x16x16_B_8MiB"]
    _say(f"[workload] {w.name} f32, device-generated inputs (column sample of 64 blocks per "
         "segment)")
    _device_hash_workload(w, max_blocks=64)


# The latency-optimal variant on sides that are not powers of three (partials in a workspace).
def _run_full_ws(w, buf):
    import paper_2602_17254_amd as T

    plan = T.trivance_plan(w.dims, w.variant, w.placement)
    ws = torch.empty(T.trivance_workspace_bytes(plan, w.elems), dtype=torch.uint8, device="cuda")
    T.trivance_allreduce_emulated_ws(buf, plan, ws)
    torch.cuda.synchronize()
    del ws
    torch.cuda.empty_cache()
    return buf


def test_ring8_latency_8MiB_nonpower3():
    w = inputs.WORKLOADS["ring8_L_8MiB"]
    _say(f"[workload] {w.name} f32 (full comparison)")
    V = inputs.normal_f32(w.seed, w.n, w.elems)
    buf = _run_full_ws(w, torch.from_numpy(V).cuda())
    assert_matches_oracle(buf.cpu().numpy(), V, w.dims, w.variant, what=w.name)
    _say(f"[workload] {w.name} i32 (full comparison)")
    Vi = inputs.uniform_i32(w.int_seed, w.n, w.elems, *w.int_range)
    buf = _run_full_ws(w, torch.from_numpy(Vi).cuda())
    assert_matches_oracle(buf.cpu().numpy(), Vi, w.dims, w.variant, what=w.name)
    _congestion(w)


def _device_hash_latency(w):
    import paper_2602_17254_amd as T

    D = len(w.dims)
    buf = torch.empty((w.n, w.elems), dtype=torch.float32, device="cuda")
    T.trivance_fill_hash_uniform(buf, w.seed)
    _run_full_ws(w, buf)
    cols, seg, _ = sample_columns(w.elems, D, w.n, "L", w.seed)
    got = buf.index_select(1, torch.from_numpy(cols).cuda()).cpu().numpy()
    del buf
    torch.cuda.empty_cache()
    Vs = inputs.hash_uniform(w.seed, w.elems, np.arange(w.n), cols)
    assert_matches_oracle(got, Vs, w.dims, w.variant, col_seg=seg, what=w.name)


def test_ring64_latency_8MiB_nonpower3():
    w = inputs.WORKLOADS["ring64_L_8MiB"]
    _say(f"[workload] {w.name} f32, device-generated inputs (column sample)")
    _device_hash_latency(w)
    _congestion(w)


def test_torus32x32_latency_8MiB_nonpower3():
    """1024 ranks of 8 MiB with up to nine partials per rank: 8.6 GB of rank data and a 155 GB
    workspace."""
    w = inputs.WORKLOADS["torus32x32_L_8MiB"]
    _say(f"[workload] {w.name} f32, device-generated inputs (column sample)")
    _device_hash_latency(w)
    _congestion(w)


# The power-of-three bandwidth-optimal workloads with message-contiguous block placement: the
# same column sample, labelled with the block placed at each column's granule range.
def test_ring243_bandwidth_32MiB_placed():
    w = inputs.WORKLOADS["ring243_Bp_32MiB"]
    _say(f"[workload] {w.name} f32 (column sample)")
    V = inputs.normal_f32(w.seed, w.n, w.elems)
    buf = _run_full(w, V)
    _check_sampled(w, V, buf, seed=w.seed)
    del buf
    _say(f"[workload] {w.name} i32 (column sample)")
    Vi = inputs.uniform_i32(w.int_seed, w.n, w.elems, *w.int_range)
    buf = _run_full(w, Vi)
    _check_sampled(w, Vi, buf, seed=w.int_seed)
    assert bool((buf[1:] == buf[0:1]).all().item())
    del buf
    torch.cuda.empty_cache()


def test_torus27x27_bandwidth_4MiB_placed():
    w = inputs.WORKLOADS["torus27x27_Bp_4MiB"]
    _say(f"[workload] {w.name} f32 (column sample)")
    V = inputs.normal_f32(w.seed, w.n, w.elems)
    buf = _run_full(w, V)
    _check_sampled(w, V, buf, seed=w.seed)
    assert bool((buf[1:] == buf[0:1]).all().item())
    del buf
    torch.cuda.empty_cache()


def test_torus9x9x9_bandwidth_128MiB_placed():
    w = inputs.WORKLOADS["torus9x9x9_Bp_128MiB"]
    _say(f"[workload] {w.name} f32, device-generated inputs (column sample)")
    _device_hash_workload(w)
