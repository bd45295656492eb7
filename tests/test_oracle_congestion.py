"""Pins of the oracle's link-load walk and transmission-delay factors (CPU only)."""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import congestion, schedule

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_n9_figure1_congestion():
    """Fig. 1 (fig:trivancevsrecursivedoublingbruck) on nine nodes: Trivance max congestion 1, 3;
    Bruck routed in one direction 3, 9."""
    with open(os.path.join(GOLDEN, "n9_example.json")) as f:
        g = json.load(f)
    tri = congestion.link_loads((9,), "L").max(axis=(1, 2)).tolist()
    bru = congestion.link_loads((9,), "BRUCK").max(axis=(1, 2)).tolist()
    assert tri == g["trivance_max_link_congestion"]["value"]
    assert bru == g["bruck_max_link_congestion"]["value"]


@pytest.mark.parametrize("dims,variant", [((9,), "L"), ((81,), "L"), ((243,), "B"),
                                          ((27, 27), "B"), ((9, 9, 9), "B"), ((27, 27), "L"),
                                          ((3, 3), "B")])
def test_trivance_congestion_is_uniform_3k(dims, variant):
    """Sec. 4.1/4.2: every directed link carries exactly 3^k messages at step k; on a torus each
    collective uses a distinct dimension per step (Sec. 5), so that holds per link as well."""
    t = schedule.Torus(dims)
    loads = congestion.link_loads(dims, variant)
    for pi, (_, step) in enumerate(schedule.pass_list(t, variant)):
        assert (loads[pi] == 3 ** (step // t.D)).all()
    # shortest-path routing is the same schedule for Trivance (Appendix E: distances < n_d / 2)
    np.testing.assert_array_equal(loads, congestion.link_loads(dims, variant, "shortest"))


@pytest.mark.parametrize("n", [3, 9, 27, 81, 243])
def test_bruck_is_three_times_trivance(n):
    """Appendix B: Bruck's per-step congestion 3 * 3^k is exactly three times Trivance's."""
    tri = congestion.link_loads((n,), "L").max(axis=(1, 2))
    bru = congestion.link_loads((n,), "BRUCK").max(axis=(1, 2))
    np.testing.assert_array_equal(bru, 3 * tri)
    assert congestion.transmission_delay_factor((n,), "BRUCK") == \
        3 * congestion.transmission_delay_factor((n,), "L")


def test_bruck_shortest_path_n9():
    """Appendix C reroutes Bruck along shortest paths; on nine nodes the 2*3^k offset then goes
    backwards at step 1 (6 > 9/2): both steps peak at 3."""
    assert congestion.link_loads((9,), "BRUCK", "shortest").max(axis=(1, 2)).tolist() == [3, 3]


@pytest.mark.parametrize("n", [9, 27, 81, 243])
def test_table1_ring_factors(n):
    """Table 1 / Appendix B (rings): Trivance(L) = sum_k 3^k = (n - 1)/2 -> n/2;
    Trivance(B) = 1/3 per step over 2 log3 n steps = (2/3) log3 n."""
    s = schedule.log3_exact(n)
    assert congestion.transmission_delay_factor((n,), "L") == Fraction(n - 1, 2)
    assert congestion.transmission_delay_factor((n,), "B") == Fraction(2 * s, 3)


@pytest.mark.parametrize("dims", [(9, 9), (27, 27), (3, 3, 3), (9, 9, 9)])
def test_table2_torus_factors(dims):
    """Appendix B (tori), relative to m*beta/D as Table 2:
    Trivance(B) = 2 sum_d sum_k 3^k / 3^(1 + d + D k), which tends to (3^D - 1)/(3^D - 3);
    Trivance(L) = D sum_k 3^k, which tends to (D/2) n^(1/D)."""
    D = len(dims)
    K = schedule.log3_exact(dims[0])
    want_b = 2 * sum(Fraction(3 ** k, 3 ** (1 + d + D * k)) for d in range(D) for k in range(K))
    want_l = D * sum(3 ** k for k in range(K))
    assert congestion.transmission_delay_factor(dims, "B") == want_b
    assert congestion.transmission_delay_factor(dims, "L") == want_l


def test_table2_limits():
    """The finite-n torus factors approach Table 2's closed forms as the sides grow."""
    for D in (2, 3, 4):
        lim = Fraction(3 ** D - 1, 3 ** D - 3)
        K = 12
        val = 2 * sum(Fraction(3 ** k, 3 ** (1 + d + D * k)) for d in range(D) for k in range(K))
        assert abs(float(val - lim)) < 1e-4
    assert congestion.transmission_delay_factor((27, 27), "B") == Fraction(104, 81)
    assert congestion.transmission_delay_factor((9, 9, 9), "B") == Fraction(260, 243)


def test_loads_shape_and_ports():
    loads = congestion.link_loads((27, 27), "B")
    assert loads.shape == (12, 729, 4)
    assert loads.dtype == np.int64


@pytest.mark.parametrize("dims,variant", [((3, 9), "B"), ((9, 27), "L"), ((3, 3, 9), "B")])
def test_rectangular_link_loads(dims, variant):
    """With unequal sides two collectives can share a dimension in a step; every directed link of
    dimension d then carries sum over the collectives using d of 3^(their per-dimension step)."""
    t = schedule.Torus(dims)
    loads = congestion.link_loads(dims, variant)
    for pi, (_, step) in enumerate(schedule.pass_list(t, variant)):
        want = [0] * t.D
        for c in range(t.D):
            d, dist = schedule.step_dim_and_distance(t, c, step)
            want[d] += dist
        for d in range(t.D):
            assert (loads[pi][:, 2 * d] == want[d]).all()
            assert (loads[pi][:, 2 * d + 1] == want[d]).all()
