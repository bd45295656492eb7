"""Trivance communication schedule, written from the paper (oracle side).

Test infrastructure only (see the package docstring).

Sources in the paper:
  * Sec. 4.1: peer function pi(r, k, n) = (r - 3^k, r + 3^k) mod n, distance tripling per step.
  * Sec. 4.2 / Theorem 1: a ring of n = 3^s nodes needs s steps.
  * Sec. 4.3, Algorithm 1 (BlockPropagation): recursive forward-reachability from a node, used
    to decide which blocks a node forwards to a peer; and the closed form Pi(n, r, p, k).
  * Sec. 5: on a D-dimensional torus one collective per dimension runs on 1/D of the vector, and
    the collectives switch dimensions every step. Appendix B indexes the data fraction of global
    step t by t = d + D*k (d = dimension offset, k = per-dimension step), which fixes the reading
    used here: collective c works at global step t on dimension (c + t) mod D at distance
    3^(t div D).

Rank numbering on a torus (a reading; the paper does not fix one): rank = sum_d x_d * stride_d,
dimension 0 fastest. Block j of a collective's segment is owned by rank j (Sec. 4.1 generalised).

Unequal sides (rectangular tori) are outside Sec. 5. Reading used for them: collective c at global
step t takes the first dimension, in cyclic order starting at (c + t) mod D, in which it still has
steps left; its distance there is 3^(steps it already took in that dimension). With equal sides
this is the rule above.
"""

from __future__ import annotations

from dataclasses import dataclass
from functools import lru_cache
from itertools import product


def log3_exact(n: int) -> int:
    """Return s with 3**s == n; raise ValueError if n is not a power of three (n >= 1)."""
    if n < 1:
        raise ValueError(f"size must be positive, got {n}")
    s, m = 0, 1
    while m < n:
        m *= 3
        s += 1
    if m != n:
        raise ValueError(f"{n} is not a power of three")
    return s


@dataclass(frozen=True)
class Torus:
    """A ring (one dimension) or a D-dimensional torus with power-of-three sides."""

    dims: tuple

    def __post_init__(self):
        if len(self.dims) < 1:
            raise ValueError("need at least one dimension")
        for d in self.dims:
            log3_exact(d)

    @property
    def D(self) -> int:
        return len(self.dims)

    @property
    def n(self) -> int:
        out = 1
        for d in self.dims:
            out *= d
        return out

    @property
    def steps(self) -> int:
        """Total number of steps S = sum_d log3(n_d) = log3(n) (Theorem 1, Sec. 5)."""
        return sum(log3_exact(d) for d in self.dims)

    def coords(self, r: int) -> tuple:
        out = []
        for d in self.dims:
            out.append(r % d)
            r //= d
        return tuple(out)

    def rank(self, xs) -> int:
        r, stride = 0, 1
        for x, d in zip(xs, self.dims):
            r += (x % d) * stride
            stride *= d
        return r

    def shift(self, r: int, dim: int, off: int) -> int:
        xs = list(self.coords(r))
        xs[dim] = (xs[dim] + off) % self.dims[dim]
        return self.rank(xs)


def step_dim_and_distance(torus: Torus, c: int, t: int) -> tuple:
    """(dimension, distance) used by collective c at global step t.

    Ring: distance 3^t (Sec. 4.1). Torus: the collectives rotate through the dimensions
    (Sec. 5), with per-dimension step k = t div D (Appendix B, t = d + D k). Unequal sides: see
    the module docstring."""
    return _rotation(torus, c)[t]


@lru_cache(maxsize=None)
def _rotation(torus: Torus, c: int) -> tuple:
    D = torus.D
    left = [log3_exact(d) for d in torus.dims]
    taken = [0] * D
    out = []
    for t in range(torus.steps):
        order = [(c + t + i) % D for i in range(D)]
        dim = next(d for d in order if taken[d] < left[d])
        out.append((dim, 3 ** taken[dim]))
        taken[dim] += 1
    return tuple(out)


def peers(torus: Torus, c: int, r: int, t: int) -> tuple:
    """(left, right) peers of rank r for collective c at global step t (Sec. 4.1 pi)."""
    dim, dist = step_dim_and_distance(torus, c, t)
    return torus.shift(r, dim, -dist), torus.shift(r, dim, +dist)


def peers_ring(r: int, k: int, n: int) -> tuple:
    """pi(r, k, n) of Sec. 4.1 on a ring: (r - 3^k mod n, r + 3^k mod n)."""
    return (r - 3 ** k) % n, (r + 3 ** k) % n


def remaining_reach(torus: Torus, c: int, p: int, t: int) -> frozenset:
    """Ranks (p included) that data held by p can still travel to in global steps t .. S-1.

    Each remaining step may move a partial by -d, 0 or +d along that step's dimension and distance
    (Sec. 4.1: every rank exchanges with both peers and every partial moves at most once per step),
    so the set grows step by step: everything reached so far, shifted by each of the three moves.
    This is the reachability that Algorithm 1 (BlockPropagation) computes recursively; `reach` below
    transcribes that algorithm, and the tests check that both agree."""
    cur = {p}
    for t2 in range(t, torus.steps):
        dim, dist = step_dim_and_distance(torus, c, t2)
        cur = {torus.shift(x, dim, e * dist) for x in cur for e in (-1, 0, +1)}
    return frozenset(cur)


def reach(torus: Torus, c: int, p: int, t: int) -> frozenset:
    """Algorithm 1 (BlockPropagation) as printed, generalised to the torus step list: from p, every
    later step contacts both peers, and every contacted rank continues from the following step. p
    itself is never marked (the algorithm only marks peers). A cross-check of remaining_reach."""
    return _reach_cached(torus, c, p, t)


@lru_cache(maxsize=None)
def _reach_cached(torus: Torus, c: int, p: int, t: int) -> frozenset:
    marked = set()
    for t2 in range(t, torus.steps):
        for q in peers(torus, c, p, t2):
            marked.add(q)
            marked |= _reach_cached(torus, c, q, t2 + 1)
    return frozenset(marked)


@lru_cache(maxsize=None)
def _message_cached(torus: Torus, c: int, receiver: int, t: int) -> tuple:
    return tuple(sorted(remaining_reach(torus, c, receiver, t + 1)))


def message_blocks(torus: Torus, c: int, receiver: int, t: int) -> list:
    """Blocks a rank sends to `receiver` at reduce-scatter step t (Sec. 4.1, 4.3).

    The sender forwards the block destined for the receiver plus the blocks of every node the
    receiver will reach in the remaining steps t+1 .. S-1 (remaining_reach, which includes the
    receiver itself). The set does not depend on which side sends. Returned sorted, which also
    fixes the order of the values inside a message."""
    return list(_message_cached(torus, c, receiver, t))


def pi_closed_form_ring(n: int, p: int, k: int) -> list:
    """Closed form Pi(n, r, p, k) of Sec. 4.3: {p + sum_{i=k+1}^{s-1} e_i 3^i mod n}, e_i in
    {-1, 0, 1}. Independent of r. Used only to pin `message_blocks`."""
    s = log3_exact(n)
    out = set()
    for eps in product((-1, 0, 1), repeat=max(s - 1 - k, 0)):
        off = sum(e * 3 ** (k + 1 + i) for i, e in enumerate(eps))
        out.add((p + off) % n)
    return sorted(out)


def ring_distance(a: int, b: int, n: int) -> int:
    d = (a - b) % n
    return min(d, n - d)


def pass_list(torus: Torus, variant: str) -> list:
    """Ordered passes of one AllReduce as (phase, t).

    'L' (latency-optimal, Sec. 4.2): one phase of S steps, whole segments every step.
    'B' (bandwidth-optimal, Sec. 4.1): reduce-scatter steps t = 0..S-1, then all-gather steps in
    reverse order t = S-1..0 (distance divided and data multiplied by three each step)."""
    S = torus.steps
    if variant == "L":
        return [("L", t) for t in range(S)]
    if variant == "B":
        return [("RS", t) for t in range(S)] + [("AG", t) for t in reversed(range(S))]
    raise ValueError(f"unknown variant {variant!r}")
