"""Seeded synthetic inputs and the named workloads (shared by tests and the benchmark).

This module holds no arithmetic of the AllReduce method: it only produces the per-rank input
vectors and describes the workload shapes. Both the HIP path and the CPU oracle are fed from it.

Generators
----------
normal_f32     numpy's default_rng(seed).standard_normal((n, E), float32), row r = rank r.
uniform_i32    numpy's default_rng(seed).integers(lo, hi, endpoint=True) as int32.
hash_uniform   counter-based U(-1, 1) fp32 from SplitMix64 (Steele, Lea, Flood, "Fast splittable
               pseudorandom number generators", OOPSLA 2014). Value (rank, e) of seed s is the
               k-th SplitMix64 output of a generator started at state 0, k = s * 2^40 + rank * E +
               e + 1, i.e. mix(k * 0x9E3779B97F4A7C15 mod 2^64); the top 24 bits h >> 40 give
               u = h * 2^-23 - 1, an exact fp32 value in [-1, 1). The device library implements
               the same definition (trivance_fill_hash_uniform) so that a 93 GB input never has
               to cross PCIe and any column can be regenerated on the host.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

GOLDEN_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def normal_f32(seed: int, n: int, E: int) -> np.ndarray:
    return np.random.default_rng(seed).standard_normal((n, E), dtype=np.float32)


def uniform_i32(seed: int, n: int, E: int, lo: int, hi: int) -> np.ndarray:
    return np.random.default_rng(seed).integers(lo, hi, size=(n, E), endpoint=True,
                                                dtype=np.int32)


def _splitmix64_mix(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def hash_uniform(seed: int, E: int, ranks, cols) -> np.ndarray:
    """U(-1, 1) values for the grid ranks x cols of an (n, E) input (see module docstring)."""
    ranks = np.asarray(ranks, dtype=np.uint64).reshape(-1, 1)
    cols = np.asarray(cols, dtype=np.uint64).reshape(1, -1)
    with np.errstate(over="ignore"):
        k = np.uint64(seed) * np.uint64(1 << 40) + ranks * np.uint64(E) + cols + np.uint64(1)
        h = _splitmix64_mix(k * GOLDEN_GAMMA)
    u = (h >> np.uint64(40)).astype(np.float64) * 2.0 ** -23 - 1.0
    return u.astype(np.float32)


@dataclass(frozen=True)
class Workload:
    """One named emulated-AllReduce workload.

    dims      ring (one entry) or torus sides
    variant   'L' latency-optimal or 'B' bandwidth-optimal (reduce-scatter + all-gather)
    elems     elements per rank vector
    dist      'normal' (N(0,1) fp32 from numpy) or 'hash_uniform' (U(-1,1), generated on device)
    seed      seed of the fp32 input
    int_range inclusive int32 range of the bit-exact integer companion run, or None
    congestion whether the bench line also reports the plan's per-link message counts checked
              against the oracle's link walk (congestion_exact)
    placement 'natural' (block j at the j-th granule range) or 'schedule' (blocks placed by the
              digits the schedule fixes, TRIVANCE_PLACE_BY_SCHEDULE)
    """

    name: str
    dims: tuple
    variant: str
    elems: int
    dist: str
    seed: int
    int_range: tuple | None = None
    congestion: bool = False
    tags: tuple = field(default_factory=tuple)
    placement: str = "natural"

    @property
    def n(self) -> int:
        out = 1
        for d in self.dims:
            out *= d
        return out

    @property
    def int_seed(self) -> int:
        return self.seed + 1000

    @property
    def rank_bytes(self) -> int:
        return 4 * self.elems


WORKLOADS = {
    w.name: w
    for w in [
        Workload("ring9_L_4KiB", (9,), "L", 1024, "normal", 0, (-1000, 1000), True),
        Workload("ring81_L_8MiB", (81,), "L", 2_097_152, "normal", 1, None, True),
        Workload("ring243_B_32MiB", (243,), "B", 8_388_608, "normal", 2, (-(2 ** 20), 2 ** 20),
                 True),
        Workload("torus27x27_B_4MiB", (27, 27), "B", 1_048_576, "normal", 3, None, True),
        Workload("torus9x9x9_B_128MiB", (9, 9, 9), "B", 33_554_432, "hash_uniform", 4, None,
                 True),
        # rings whose size is not a power of three (the paper's 8- and 64-node rings)
        Workload("ring8_B_32MiB", (8,), "B", 8_388_608, "normal", 5, (-(2 ** 20), 2 ** 20), True,
                 ("nonpower3",)),
        Workload("ring64_B_8MiB", (64,), "B", 2_097_152, "normal", 6, None, True, ("nonpower3",)),
        # the paper's tori whose sides are not powers of three
        Workload("torus32x32_B_8MiB", (32, 32), "B", 2_097_152, "hash_uniform", 7, None, True,
                 ("nonpower3",)),
        Workload("torus8x64_B_8MiB", (8, 64), "B", 2_097_152, "hash_uniform", 8, None, True,
                 ("nonpower3",)),
        Workload("torus16x16x16_B_8MiB", (16, 16, 16), "B", 2_097_152, "hash_uniform", 9, None,
                 False, ("nonpower3",)),
        # the latency-optimal variant on the paper's sides that are not powers of three (partial
        # sums in a caller-owned workspace: 0.5, 4 and 144 GiB)
        Workload("ring8_L_8MiB", (8,), "L", 2_097_152, "normal", 10, (-(2 ** 20), 2 ** 20), True,
                 ("nonpower3",)),
        Workload("ring64_L_8MiB", (64,), "L", 2_097_152, "hash_uniform", 11, None, True,
                 ("nonpower3",)),
        Workload("torus32x32_L_8MiB", (32, 32), "L", 2_097_152, "hash_uniform", 12, None, True,
                 ("nonpower3",)),
        # the power-of-three bandwidth-optimal workloads with message-contiguous block placement
        # (same inputs as their default-partition counterparts)
        Workload("ring243_Bp_32MiB", (243,), "B", 8_388_608, "normal", 2, (-(2 ** 20), 2 ** 20),
                 False, ("placed",), "schedule"),
        Workload("torus27x27_Bp_4MiB", (27, 27), "B", 1_048_576, "normal", 3, None, False,
                 ("placed",), "schedule"),
        Workload("torus9x9x9_Bp_128MiB", (9, 9, 9), "B", 33_554_432, "hash_uniform", 4, None,
                 False, ("placed",), "schedule"),
    ]
}

# The headline single-GPU workload: the largest configuration of the metric's 8-128 MiB range, a
# 9 x 9 x 9 torus of 729 virtual ranks, bandwidth-optimal, 128 MiB per rank (97.8 GB resident).
HEADLINE = "torus9x9x9_B_128MiB"
