"""Planted mistakes in the oracle of sides that are not powers of three must be caught (CPU only).

Each mutation patches one piece of `oracle.nonpow3` with a plausible bug and re-runs a compact
set of the pins of `test_oracle_nonpow3.py`; at least one must fail (or the oracle must abort).
"""

import json
import os

import numpy as np
import pytest

from oracle import allreduce, congestion, nonpow3, partition

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "n7_nonpower3.json")))


def _clear():
    for f in (nonpow3._digits_to, nonpow3.families, nonpow3.path_digits):
        f.cache_clear()


def _pins_hold() -> bool:
    try:
        rng = np.random.default_rng(303)
        # exact integer sums and one forward per block and phase, rings and tori (mailbox form)
        for n in (7, 8, 10, 32):
            V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, 64 * n + 5), dtype=np.int32)
            stats = {}
            out = nonpow3.bandwidth_optimal_ring(V, stats=stats)
            if not (out == allreduce.exact_int_sum(V)[None]).all():
                return False
            if not (stats["blocks_sent"].sum(axis=(0, 2)) == n - 1).all():
                return False
        for dims in ((3, 8), (4, 4), (2, 3, 4)):
            n = int(np.prod(dims))
            V = rng.integers(-(2 ** 31), 2 ** 31 - 1, size=(n, 64 * len(dims) * n + 5),
                             dtype=np.int32)
            stats = {}
            out = nonpow3.bandwidth_optimal_torus(V, dims, stats=stats)
            if not (out == allreduce.exact_int_sum(V)[None]).all():
                return False
            if not (stats["sent"].sum(axis=(0, 3)) == n - 1).all():
                return False
        # the 7-node figure: 2 steps, final distance 2, 2 blocks per direction then 1
        if len(nonpow3.distances(7)) != GOLDEN["n7_steps"]["value"]:
            return False
        if nonpow3.distances(7)[-1] != GOLDEN["n7_final_distance"]["value"]:
            return False
        stats = {}
        nonpow3.bandwidth_optimal_ring(np.zeros((7, 7 * 64), np.int32), stats=stats)
        if stats["blocks_sent"].max(axis=(1, 2)).tolist() != GOLDEN["n7_blocks_per_direction"]["value"]:
            return False
        # final step uniform with congestion d
        for n in (8, 32):
            loads = congestion.link_loads((n,), "B")
            S = len(nonpow3.distances(n))
            if not (loads[S - 1] == nonpow3.levels(n)[1]).all():
                return False
        # the ordinary schedule whenever every side is a power of three, bits and link loads
        for dims in ((9,), (27,), (3, 9)):
            n = int(np.prod(dims))
            V = rng.standard_normal((n, 64 * len(dims) * n + 3), dtype=np.float32)
            want = allreduce.bandwidth_optimal(V, dims)
            got = nonpow3.bandwidth_optimal_ring(V) if len(dims) == 1 else \
                nonpow3.bandwidth_optimal_torus(V, dims)
            if not np.array_equal(got, want):
                return False
            if len(dims) > 1 and not np.array_equal(nonpow3.link_loads_torus(dims),
                                                    congestion.link_loads(dims, "B")):
                return False
        # a 1 x 8 torus is the ring of 8 on each segment
        V = rng.standard_normal((8, 128 * 8 + 9), dtype=np.float32)
        seg, blk = partition.column_labels(V.shape[1], 2, 8)
        if not np.array_equal(nonpow3.bandwidth_optimal_torus(V, (1, 8)),
                              nonpow3.bandwidth_optimal_ring(V, col_blk=blk)):
            return False
        # the gather form equals the mailbox form, bits and link loads
        for dims in ((4, 4), (3, 8)):
            n = int(np.prod(dims))
            V = rng.standard_normal((n, 64 * 2 * n + 37), dtype=np.float32)
            seg, blk = partition.column_labels(V.shape[1], 2, n)
            if not np.array_equal(nonpow3.bandwidth_optimal_torus_columns(V, dims, seg, blk),
                                  nonpow3.bandwidth_optimal_torus(V, dims)):
                return False
            if not np.array_equal(nonpow3.link_loads_torus(dims, "columns"),
                                  nonpow3.link_loads_torus(dims, "mailbox")):
                return False
        return True
    except (AssertionError, ValueError, KeyError, IndexError, StopIteration, TypeError):
        return False


def test_unmutated_nonpow3_oracle_passes():
    _clear()
    assert _pins_hold()


_levels = nonpow3.levels
_torus_rotation = nonpow3.torus_rotation
_digits_to = nonpow3._digits_to.__wrapped__
_families = nonpow3.families.__wrapped__
_tree_tables = nonpow3._tree_tables
_joint = nonpow3._joint
_gather_joint = nonpow3._gather_joint


def _final_distance_floor(n):
    f, d = _levels(n)
    return (f, (n - 3 ** f) // 2) if d else (f, 0)


def _rotation_without_skip(dims, c):
    D = len(dims)
    S = sum(nonpow3.dim_steps(s) for s in dims)
    return [((c + t) % D, t // D) for t in range(S)]


def _digits_reversed(f, value):
    e = _digits_to(f, value)
    return None if e is None else tuple(reversed(e))


def _no_closure(n):
    f, d = _levels(n)
    R = (3 ** f - 1) // 2
    return {o: (0 if abs(o) <= R else (1 if o > R else -1)) for o in nonpow3.offsets(n)}


def _send_step_late(side):
    send, digit = _tree_tables(side)
    return np.minimum(send + 1, max(nonpow3.dim_steps(side), 1)), digit


def _joint_right_first(parts):
    acc = None
    for side in ("own", "right", "left"):
        if side in parts:
            acc = parts[side].copy() if acc is None else np.add(acc, parts[side],
                                                                 dtype=parts[side].dtype)
    return acc


def _joint_children_first(parts):
    kids = [parts[s] for s in ("left", "right") if s in parts]
    if not kids:
        return parts["own"].copy()
    k = kids[0] if len(kids) == 1 else np.add(kids[0], kids[1], dtype=kids[0].dtype)
    return np.add(parts["own"], k, dtype=k.dtype) if "own" in parts else k


def _gather_sides_swapped(own, left, right, from_left, from_right):
    return _gather_joint(own, right, left, from_right, from_left)


def _gather_drops_right(own, left, right, from_left, from_right):
    return np.where(from_left, np.add(own, left, dtype=own.dtype), own)


MUTATIONS = {
    "final distance rounded down": ("levels", _final_distance_floor),
    "rotation keeps exhausted dimensions": ("torus_rotation", _rotation_without_skip),
    "path digits taken highest first": ("_digits_to", _digits_reversed),
    "tree closure skipped": ("families", _no_closure),
    "send step one late (gather form)": ("_tree_tables", _send_step_late),
    "joint reduction takes the right child first": ("_joint", _joint_right_first),
    "joint reduction adds the children first": ("_joint", _joint_children_first),
    "gather form swaps the children's sides": ("_gather_joint", _gather_sides_swapped),
    "gather form drops the right child": ("_gather_joint", _gather_drops_right),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_nonpow3_mutation_is_caught(name, monkeypatch):
    attr, repl = MUTATIONS[name]
    _clear()
    monkeypatch.setattr(nonpow3, attr, repl)
    try:
        assert not _pins_hold(), f"pins did not catch: {name}"
    finally:
        monkeypatch.undo()
        _clear()
