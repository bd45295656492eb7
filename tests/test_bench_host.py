"""Host-side logic of bench.py (no GPU): phase grouping of the timed region, the power-of-three
test that picks the kernel family, the CPU-baseline column sample and the --gpus refusal."""

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
