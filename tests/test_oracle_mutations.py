"""Planted mistakes in the oracle must be caught by the pins (CPU only).

Each mutation patches one piece of the oracle with a plausible bug (a wrong sign, a swapped
operand, a dropped term, a wrong index) and re-runs a compact set of pin checks taken from the
other oracle tests; at least one must fail. This shows the pins constrain every part they cover.
"""

import numpy as np
import pytest

from oracle import allreduce, congestion, partition, schedule


def _pins_hold() -> bool:
    """A compact selection of the pins; False as soon as one fails (or the oracle aborts)."""
    try:
        rng = np.random.default_rng(101)
        # brute-force integer sums, ring and torus, both variants
        for dims in [(9,), (27,), (3, 3), (9, 9), (3, 3, 3)]:
            n = schedule.Torus(dims).n
            V = rng.integers(-1000, 1000, size=(n, 64 * n + 7), dtype=np.int32)
            want = allreduce.exact_int_sum(V)
            for v in "LB":
                if not (allreduce.allreduce(V, dims, v) == want[None]).all():
                    return False
        # n = 9 explicit tree (worked example of Sec. 4.3)
        V = (rng.standard_normal((9, 64)) * np.logspace(-6, 6, 64)).astype(np.float32)
        v = V
        want = (((v[0] + v[8]) + v[1]) + ((v[6] + v[5]) + v[7])) + ((v[3] + v[2]) + v[4])
        if not (allreduce.allreduce(V, (9,), "L")[0] == want).all():
            return False
        # association witness
        e = np.float32(2.0 ** -24)
        if allreduce.allreduce(np.array([[1.0], [e], [e]], np.float32), (3,), "L")[0, 0] != 1.0:
            return False
        # Lemma 2 windows on 27 nodes
        Vh = np.eye(27, dtype=np.int32)
        for k in range(3):
            out = allreduce.latency_optimal(Vh, (27,), passes=k + 1)
            Rk = (3 ** (k + 1) - 1) // 2
            for r in range(27):
                want = [1 if schedule.ring_distance(u, r, 27) <= Rk else 0 for u in range(27)]
                if out[r].tolist() != want:
                    return False
        # closed form of Sec. 4.3
        t9 = schedule.Torus((27,))
        for k in range(3):
            for p in range(27):
                if schedule.message_blocks(t9, 0, p, k) != schedule.pi_closed_form_ring(27, p, k):
                    return False
        # congestion: uniform 3^k, Fig. 1 values, Appendix B factors
        for dims, var in [((9,), "L"), ((27, 27), "B")]:
            t = schedule.Torus(dims)
            loads = congestion.link_loads(dims, var)
            for pi, (_, step) in enumerate(schedule.pass_list(t, var)):
                if not (loads[pi] == 3 ** (step // t.D)).all():
                    return False
        if congestion.link_loads((9,), "BRUCK").max(axis=(1, 2)).tolist() != [3, 9]:
            return False
        from fractions import Fraction
        if congestion.transmission_delay_factor((9, 9, 9), "B") != Fraction(260, 243):
            return False
        # B block j equals L at owner j (bitwise)
        Vf = rng.standard_normal((27, 2 * 64 * 27 + 5), dtype=np.float32)
        L = allreduce.allreduce(Vf, (27,), "L")
        B = allreduce.allreduce(Vf, (27,), "B")
        _, blk = partition.column_labels(Vf.shape[1], 1, 27)
        for j in range(27):
            if not (B[0, blk == j] == L[j, blk == j]).all():
                return False
        return True
    except (AssertionError, ValueError, KeyError, IndexError):
        return False


def test_unmutated_oracle_passes():
    assert _pins_hold()


def _swap_assoc(own, a, b):
    return np.add(own, np.add(a, b, dtype=own.dtype), dtype=own.dtype)


def _left_right_swapped(own, a, b):
    return np.add(np.add(own, b, dtype=own.dtype), a, dtype=own.dtype)


def _wrong_rotation(torus, c, t):
    return c % torus.D, 3 ** (t // torus.D)  # forgets to switch dimensions


def _wrong_distance(torus, c, t):
    return (c + t) % torus.D, 2 ** (t // torus.D)  # doubling instead of tripling


def _message_reach_same_step(torus, c, receiver, t):
    return sorted({receiver} | set(schedule.reach(torus, c, receiver, t)))  # t instead of t + 1


def _message_without_receiver(torus, c, receiver, t):
    return sorted(set(schedule.reach(torus, c, receiver, t + 1)))


def _route_short_by_one(offset, size, routing):
    fwd = offset % size
    if fwd == 0:
        return +1, 0
    return (1, max(offset - 1, 0)) if offset > 0 else (-1, max(-offset - 1, 0))


def _bruck_same_as_trivance(torus, variant, c, r, t):
    dim, dist = schedule.step_dim_and_distance(torus, c, t)
    return [(dim, -dist), (dim, +dist)]


def _partition_floor_swapped(E, D, n):
    # rounds every block start up instead of down
    out = []
    G = -(-E // 64)
    for c in range(D):
        g0, g1 = (c * G) // D, ((c + 1) * G) // D
        row = []
        for j in range(n):
            b = g0 + -(-(j * (g1 - g0)) // n)
            e = g0 + -(-((j + 1) * (g1 - g0)) // n)
            row.append((min(b * 64, E), min(e * 64, E)))
        out.append(row)
    return out


MUTATIONS = {
    "association own+(left+right)": (allreduce, "_reduce3", _swap_assoc),
    "left and right swapped": (allreduce, "_reduce3", _left_right_swapped),
    "no dimension rotation": (schedule, "step_dim_and_distance", _wrong_rotation),
    "distance 2^k": (schedule, "step_dim_and_distance", _wrong_distance),
    "reachability from the current step": (schedule, "message_blocks", _message_reach_same_step),
    "message drops the receiver's block": (schedule, "message_blocks", _message_without_receiver),
    "route one hop short": (congestion, "_route", _route_short_by_one),
    "Bruck pattern symmetric": (congestion, "_messages", _bruck_same_as_trivance),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    mod, attr, repl = MUTATIONS[name]
    schedule._reach_cached.cache_clear()
    monkeypatch.setattr(mod, attr, repl)
    try:
        assert not _pins_hold(), f"pins did not catch: {name}"
    finally:
        schedule._reach_cached.cache_clear()


def test_partition_mutation_changes_float_trees(monkeypatch):
    """The partition decides each element's owner, hence its fp32 tree: a different rounding rule
    must change some fp32 bits of the B result on a ragged shape, while integer results (which
    do not depend on it) stay correct."""
    rng = np.random.default_rng(5)
    V = (rng.standard_normal((27, 64 * 40 + 3)) * np.logspace(-5, 5, 64 * 40 + 3)).astype(np.float32)
    ref = allreduce.allreduce(V, (27,), "B")
    monkeypatch.setattr(partition, "block_bounds", _partition_floor_swapped)
    mutated = allreduce.allreduce(V, (27,), "B")
    assert not np.array_equal(ref, mutated)
