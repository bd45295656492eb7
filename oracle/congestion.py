"""Per-link congestion of a schedule, by walking every message hop by hop (oracle side).

Test infrastructure only (see the package docstring).

Sec. 2.1 defines the congestion c_k of a step as the number of chunks (messages) that share a link.
The network model (Sec. 2, Appendix E) is a ring or torus with one port per direction and
dimension, deterministic routing, and transmissions that stay inside one dimension.

Output layout: loads[pass][rank][port] (int64), port 2d = link leaving `rank` towards +d,
port 2d+1 = link leaving `rank` towards -d. A message from r over offset o along dimension d
crosses the links leaving r, r+1, ..., r+o-1 (for o > 0) in the + direction.

Schedules
---------
'L', 'B'  Trivance (Sec. 4.1/4.2): every rank sends to r - 3^k and r + 3^k along the collective's
          dimension; 'B' has S reduce-scatter passes followed by S all-gather passes (same peers).
'BRUCK'   ring-only comparison pattern (Sec. 2.4 and Fig. 1): at step k every rank sends to the
          offsets +3^k and +2*3^k, both in the + direction as the original algorithm does.
Routing
-------
'scheduled'  a message travels in the direction of the sign of its offset.
'shortest'   a message takes the shorter way round its ring (Appendix C's modified Bruck); a tie at
             exactly half the ring keeps the sign of the offset. For Trivance every distance is
             below half the ring, so both routings agree (Appendix E).
"""

from __future__ import annotations

from fractions import Fraction

import numpy as np

from . import nonpow3, schedule


def _messages(torus: schedule.Torus, variant: str, c: int, r: int, t: int):
    """(dimension, signed offset) of every message rank r sends at global step t."""
    dim, dist = schedule.step_dim_and_distance(torus, c, t)
    if variant in ("L", "B"):
        return [(dim, -dist), (dim, +dist)]
    if variant == "BRUCK":
        return [(dim, +dist), (dim, +2 * dist)]
    raise ValueError(f"unknown schedule {variant!r}")


def _route(offset: int, size: int, routing: str) -> tuple:
    """(direction +1/-1, hop count) for a message over `offset` on a ring of `size` nodes."""
    fwd = offset % size
    if fwd == 0:
        return +1, 0
    if routing == "scheduled":
        return (1, offset) if offset > 0 else (-1, -offset)
    if routing == "shortest":
        back = size - fwd
        if fwd < back:
            return +1, fwd
        if back < fwd:
            return -1, back
        return (1, fwd) if offset > 0 else (-1, back)
    raise ValueError(f"unknown routing {routing!r}")


def passes_of(torus: schedule.Torus, variant: str) -> list:
    if variant == "BRUCK":
        if torus.D != 1:
            raise ValueError("the Bruck comparison pattern is defined on rings only")
        return [("L", t) for t in range(torus.steps)]
    return schedule.pass_list(torus, variant)


def _link_loads_latency_tree(dims, routing):
    """Latency-optimal schedule on sides that are not all powers of three: a rank sends towards a
    side in a pass when its peer there takes some partial from it (latency_nonpow3)."""
    from . import latency_nonpow3

    dims = tuple(int(x) for x in dims)
    D = len(dims)
    n = int(np.prod(dims))
    S = sum(nonpow3.dim_steps(s) for s in dims)
    loads = np.zeros((S, n, 2 * D), dtype=np.int64)
    strides = np.cumprod((1,) + dims[:-1])
    for c in range(D):
        rot = nonpow3.torus_rotation(dims, c)
        for t, ((dim, k), (plus, minus)) in enumerate(zip(rot, latency_nonpow3.message_slots(dims, c))):
            dist = nonpow3.distances(dims[dim])[k]
            for r in range(n):
                for off, count in ((+dist, plus), (-dist, minus)):
                    if not count:
                        continue
                    direction, hops = _route(off, dims[dim], routing)
                    port = 2 * dim + (0 if direction > 0 else 1)
                    node = r
                    for _ in range(hops):
                        loads[t, node, port] += 1
                        x = (node // strides[dim]) % dims[dim]
                        node += (((x + direction) % dims[dim]) - x) * strides[dim]
    return loads


def link_loads(dims, variant: str, routing: str = "scheduled") -> np.ndarray:
    if variant == "L" and nonpow3.is_tree(dims):
        return _link_loads_latency_tree(dims, routing)
    if variant == "B" and nonpow3.is_tree(dims):
        # Sec. 4.4 trees; every distance is below half its side, so both routings agree
        if len(dims) == 1:
            return nonpow3.link_loads_ring(dims[0])
        return nonpow3.link_loads_torus(dims)
    torus = schedule.Torus(tuple(dims))
    plist = passes_of(torus, variant)
    n, D = torus.n, torus.D
    loads = np.zeros((len(plist), n, 2 * D), dtype=np.int64)
    for pi, (_, t) in enumerate(plist):
        for c in range(D):
            for r in range(n):
                for dim, off in _messages(torus, variant, c, r, t):
                    direction, hops = _route(off, torus.dims[dim], routing)
                    port = 2 * dim + (0 if direction > 0 else 1)
                    node = r
                    for _ in range(hops):
                        loads[pi, node, port] += 1
                        node = torus.shift(node, dim, direction)
    return loads


def message_fraction(torus: schedule.Torus, variant: str, phase: str, t: int) -> Fraction:
    """Size of one message as a fraction of the whole vector m.

    L / Bruck: a whole segment (1/D). B: the blocks of Algorithm 1, each 1/(n D) of m; in the
    all-gather a rank forwards everything it holds, which at step t is the same count as the
    reduce-scatter message of that step (Sec. 4.1: sizes triple as the distance shrinks)."""
    if variant in ("L", "BRUCK"):
        return Fraction(1, torus.D)
    nblk = len(schedule.message_blocks(torus, 0, 0, t))
    return Fraction(nblk, torus.n * torus.D)


def transmission_delay_factor(dims, variant: str, routing: str = "scheduled") -> Fraction:
    """Theta of Tables 1 and 2: sum over steps of (message fraction x max link load), expressed
    relative to the ideal m*beta/D (for a ring, D = 1, that is m*beta)."""
    torus = schedule.Torus(tuple(dims))
    loads = link_loads(dims, variant, routing)
    total = Fraction(0)
    for pi, (phase, t) in enumerate(passes_of(torus, variant)):
        total += message_fraction(torus, variant, phase, t) * int(loads[pi].max())
    return total * torus.D
