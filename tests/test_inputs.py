"""The seeded input generators (CPU only)."""

import json
import os

import numpy as np

from paper_2602_17254_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_published_outputs():
    with open(os.path.join(GOLDEN, "splitmix64_state0.json")) as f:
        want = [int(h, 16) for h in json.load(f)["outputs_hex"]]
    k = np.arange(1, 4, dtype=np.uint64)
    with np.errstate(over="ignore"):
        got = inputs._splitmix64_mix(k * inputs.GOLDEN_GAMMA)
    assert [int(x) for x in got] == want


def test_hash_uniform_grid_and_range():
    E = 1000
    full = inputs.hash_uniform(4, E, np.arange(5), np.arange(E))
    assert full.dtype == np.float32 and full.shape == (5, E)
    assert (full >= -1).all() and (full < 1).all()
    # every value is on the 2^-23 grid, and a sub-grid regenerates the same values
    assert np.all((full.astype(np.float64) + 1) * 2 ** 23 == np.round((full.astype(np.float64) + 1) * 2 ** 23))
    sub = inputs.hash_uniform(4, E, [3, 1], [999, 0, 17])
    np.testing.assert_array_equal(sub, full[[3, 1]][:, [999, 0, 17]])
    # first value of seed 0 is the top 24 bits of the first SplitMix64 output
    v = inputs.hash_uniform(0, 10, [0], [0])[0, 0]
    assert v == np.float32((0xE220A8397B1DCDAF >> 40) * 2.0 ** -23 - 1)
    # mean and spread of U(-1, 1)
    assert abs(full.mean()) < 0.02 and abs(full.var() - 1 / 3) < 0.02


def test_workload_table():
    w = inputs.WORKLOADS
    assert inputs.HEADLINE in w
    assert [x.n for x in w.values()] == [9, 81, 243, 729, 729, 8, 64, 1024, 512, 4096,
                                         8, 64, 1024, 243, 729, 729]
    placed = [x for x in w.values() if x.placement == "schedule"]
    assert [x.name for x in placed] == ["ring243_Bp_32MiB", "torus27x27_Bp_4MiB",
                                        "torus9x9x9_Bp_128MiB"]
    for x in placed:  # same inputs as the default-partition workload of the same shape and size
        twin = w[x.name.replace("_Bp_", "_B_")]
        assert (twin.dims, twin.elems, twin.dist, twin.seed, twin.int_range) == \
            (x.dims, x.elems, x.dist, x.seed, x.int_range) and twin.placement == "natural"
    assert w["torus9x9x9_B_128MiB"].rank_bytes == 128 * 2 ** 20
    assert w["ring81_L_8MiB"].rank_bytes == 8 * 2 ** 20
    a = inputs.normal_f32(1, 3, 10)
    np.testing.assert_array_equal(a, inputs.normal_f32(1, 3, 10))
    b = inputs.uniform_i32(5, 4, 100, -3, 3)
    assert b.dtype == np.int32 and b.min() >= -3 and b.max() <= 3
