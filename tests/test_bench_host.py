"""Host-side logic of bench.py (no GPU): phase grouping of the timed region, the power-of-three
test that picks the kernel family, the CPU-baseline column sample and its repetition, and the
--gpus refusal."""

import subprocess
import sys

import numpy as np
import pytest

import bench
from paper_2602_17254_amd import inputs

T = pytest.importorskip("paper_2602_17254_amd")


@pytest.mark.parametrize("dims,variant", [((81,), "L"), ((243,), "B"), ((27, 27), "B"), ((8,), "B"),
                                          ((4, 4, 4), "B"), ((3, 9), "L")])
def test_phase_groups_cover_the_plan(dims, variant):
    plan = T.trivance_plan(dims, variant)
    phases = [T.trivance_plan_step(plan, p)[0] for p in range(plan.num_passes)]
    groups = bench.phase_groups(phases)
    if variant == "L":
        assert groups == [[0, plan.num_passes, 0]]
    else:
        S = plan.num_steps
        assert groups == [[0, S, 1], [S, 2 * S, 2]]
    assert bench.phase_groups([]) == []
    assert bench.phase_groups([1, 1, 2, 1]) == [[0, 2, 1], [2, 3, 2], [3, 4, 1]]


def test_is_pow3():
    assert [v for v in range(1, 100) if bench._is_pow3(v)] == [1, 3, 9, 27, 81]


@pytest.mark.parametrize("name", sorted(inputs.WORKLOADS))
def test_baseline_sample_is_in_range(name):
    w = inputs.WORKLOADS[name]
    budget = min(60_000, (1 << 24) // w.n)
    cols = bench._sample_for_baseline(w, min(budget, w.elems))
    assert cols.dtype == np.int64 and cols.min() >= 0 and cols.max() < w.elems
    assert len(cols) == min(budget, w.elems)
    assert (np.diff(cols) == 1).all()


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr


@pytest.mark.parametrize("name", ["ring9_L_4KiB", "ring243_B_32MiB", "ring243_Bp_32MiB"])
def test_cpu_baseline_repeats_short_samples(name):
    """The baseline reruns a short sample up to the time target (capped), reports the number of
    runs and compares the first result: here the oracle's own, so it must match."""
    from oracle import allreduce, partition, placement

    w = inputs.WORKLOADS[name]
    cols = bench._sample_for_baseline(w, min(300, w.elems))
    V_cols = np.random.default_rng(w.seed).standard_normal((w.n, cols.size), dtype=np.float32)
    if w.placement == "schedule":
        seg, blk = placement.column_labels(w.elems, w.dims, cols)
    else:
        seg, blk = partition.column_labels(w.elems, len(w.dims), w.n, cols)
    first = (allreduce.latency_optimal(V_cols, w.dims, col_seg=seg) if w.variant == "L" else
             allreduce.allreduce(V_cols, w.dims, "B", col_seg=seg, col_blk=blk))
    out = bench.cpu_baseline(w, first, cols, V_cols, seconds_target=0.05, max_runs=3)
    assert 1 <= out["runs"] <= 3 and out["matches_gpu_on_sample"] is True
    assert out["value"] > 0 and out["cores"] == 1 and f"{out['runs']} run(s)" in out["sample"]
    assert out["gpu_fp64_bound_ratio_on_sample"] <= 1.0


@pytest.mark.parametrize("key", sorted(bench.MEASURED_TRAFFIC), ids=lambda k: f"{k[0]}-{k[1]}")
def test_measured_traffic_matches_the_workload(key):
    """Each stored counter figure belongs to its workload and kernel family: within 5% of that
    family's algorithmic bytes per launch computed from the plan (the profiles show 0.9999 to
    1.022), so an entry keyed to the wrong workload or family fails."""
    name, kernel = key
    w = inputs.WORKLOADS[name]
    plan = T.trivance_plan(w.dims, w.variant, w.placement)
    phases = [T.trivance_plan_step(plan, p)[0] for p in range(plan.num_passes)]
    want = 0 if kernel in ("latency_split_kernel", "slot_step_kernel") else (
        1 if kernel.endswith("<reduce>") else 2)
    passes = [p for p in range(plan.num_passes) if phases[p] == want]
    assert passes, f"{name} has no pass of the {kernel} family"
    alg = sum(T.trivance_pass_bytes(plan, w.elems, p) for p in passes) / len(passes)
    ratio = bench.MEASURED_TRAFFIC[key]["bytes_per_launch"] / alg
    assert 0.99 <= ratio <= 1.05, f"{name} {kernel}: traffic / algorithmic = {ratio:.4f}"
