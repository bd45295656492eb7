"""The congestion-aware cost model of Sec. 2.1 evaluated on the oracle's own schedules (oracle side).

Test infrastructure only (see the package docstring).

Sec. 2.1 prices an AllReduce A of m bytes as C(m, A) = steps(A) alpha + sum_k beta m_k c_k: every
step pays the start-up latency alpha, and its transmission takes beta times the bytes of its chunks
weighted by how many chunks share a link. Written per directed link, the transmission of a step
lasts as long as its busiest link needs: beta times the bytes of every message that crosses that
link (for chunks of one size m_k that is m_k c_k). That is what this module computes, from nothing
but messages walked hop by hop:

  * latency-optimal variant: every rank sends its whole segment (m / D) to both peers;
  * bandwidth-optimal variant, sides that are powers of three: the message to peer p at step t
    holds the blocks of Algorithm 1 (schedule.message_blocks), each m / (n D); the all-gather
    message of step t retraces it from the receiver back to the sender (Sec. 4.1);
  * sides that are not powers of three (Sec. 4.4): the number of blocks every rank forwards per
    step and direction, counted by the tree emulations of nonpow3 (the ring's mailbox form, the
    torus's gather form with one column per block), each m / (n D) again;
  * latency-optimal variant on sides that are not powers of three: every message carries the
    partials its receiver takes from the sender (latency_nonpow3), each m / D;
  * the Bruck comparison pattern on a ring (Sec. 2.4, Table 1): whole segments to the offsets
    +3^k and +2 3^k, or Algorithm 1's blocks for its bandwidth-optimal form (Sec. 2.4 says its
    data follows Trivance's pattern), for the threefold-congestion pin only.

Each message of b bytes over a signed offset crosses its hops in the direction the routing picks
(congestion._route), adding b to each link it leaves. Sizes are exact fractions of m.

Theta, the transmission-delay factor of Tables 1 and 2, is the transmission term relative to
m beta / D (relative to m beta on a ring).
"""

from __future__ import annotations

from fractions import Fraction

import numpy as np

from . import congestion, nonpow3, schedule


def _walk(add, torus_dims, r, dim, offset, size, routing):
    """Add `size` to every directed link a message from rank r over `offset` along `dim` crosses."""
    dims = tuple(torus_dims)
    direction, hops = congestion._route(offset, dims[dim], routing)
    port = 2 * dim + (0 if direction > 0 else 1)
    stride = 1
    for d in range(dim):
        stride *= dims[d]
    node = r
    for _ in range(hops):
        add(node, port, size)
        x = (node // stride) % dims[dim]
        node += (((x + direction) % dims[dim]) - x) * stride


def _messages_pow3(dims, variant):
    """[(pass, rank, dim, signed offset, size as a fraction of m)] of a power-of-three schedule."""
    torus = schedule.Torus(tuple(dims))
    n, D = torus.n, torus.D
    out = []
    plist = congestion.passes_of(torus, "L" if variant == "BRUCK_B" else variant)
    if variant == "BRUCK_B":
        plist = [("RS", t) for t in range(torus.steps)] + \
                [("AG", t) for t in reversed(range(torus.steps))]
    for pi, (phase, t) in enumerate(plist):
        for c in range(D):
            dim, dist = schedule.step_dim_and_distance(torus, c, t)
            for r in range(n):
                if variant == "L":
                    for off in (-dist, +dist):
                        out.append((pi, r, dim, off, Fraction(1, D)))
                elif variant == "BRUCK":
                    for off in (+dist, +2 * dist):
                        out.append((pi, r, dim, off, Fraction(1, D)))
                else:
                    offs = (+dist, +2 * dist) if variant == "BRUCK_B" else (-dist, +dist)
                    for off in offs:
                        to = torus.shift(r, dim, off)
                        # Bruck's blocks follow the same reachability (Sec. 2.4, Appendix C)
                        nblk = len(schedule.message_blocks(torus, c, to, t)) \
                            if variant != "BRUCK_B" else torus.n // 3 ** (t + 1)
                        size = Fraction(nblk, n * D)
                        if phase == "RS":
                            out.append((pi, r, dim, off, size))
                        else:  # the all-gather message of step t goes from `to` back to r
                            out.append((pi, to, dim, -off, size))
    return len(plist), out


def _messages_latency_tree(dims):
    """Latency-optimal schedule on sides that are not all powers of three: every message carries
    the distinct partials its receiver takes from the sender (latency_nonpow3), each m / D."""
    from . import latency_nonpow3

    dims = tuple(int(x) for x in dims)
    D = len(dims)
    n = int(np.prod(dims))
    out = []
    S = 0
    for c in range(D):
        rot = nonpow3.torus_rotation(dims, c)
        S = len(rot)
        for t, ((dim, k), (plus, minus)) in enumerate(zip(rot, latency_nonpow3.message_slots(dims, c))):
            dist = nonpow3.distances(dims[dim])[k]
            for r in range(n):
                if plus:
                    out.append((t, r, dim, +dist, Fraction(plus, D)))
                if minus:
                    out.append((t, r, dim, -dist, Fraction(minus, D)))
    return S, out


def _messages_tree(dims):
    """The same list for the Sec. 4.4 trees, from the emulations' per-message block counts."""
    dims = tuple(int(x) for x in dims)
    D = len(dims)
    n = int(np.prod(dims))
    stats = {}
    if D == 1:
        nonpow3.bandwidth_optimal_ring(np.zeros((n, 0), np.int32), stats=stats)
        sent = stats["blocks_sent"][:, None, :, :]  # [S][collective][rank][port]
        rot = [[(0, k) for k in range(sent.shape[0])]]
    else:
        seg = np.repeat(np.arange(D), n)
        blk = np.tile(np.arange(n), D)
        nonpow3.bandwidth_optimal_torus_columns(np.zeros((n, D * n), np.int32), dims, seg, blk,
                                                stats=stats)
        sent = stats["sent"]
        rot = [nonpow3.torus_rotation(dims, c) for c in range(D)]
    S = sent.shape[0]
    out = []
    for c in range(D):
        for t, (dim, k) in enumerate(rot[c]):
            dist = nonpow3.distances(dims[dim])[k]
            for r in range(n):
                for port, sign in ((0, +1), (1, -1)):
                    nblk = int(sent[t, c, r, port])
                    if nblk == 0:
                        continue
                    size = Fraction(nblk, n * D)
                    out.append((t, r, dim, sign * dist, size))
                    # all-gather pass 2S - 1 - t: the receiver sends the blocks back
                    xs = nonpow3._coords(dims, r)
                    xs[dim] += sign * dist
                    out.append((2 * S - 1 - t, nonpow3._rank(dims, xs), dim, -sign * dist, size))
    return 2 * S, out


def link_bytes(dims, variant: str, routing: str = "scheduled") -> np.ndarray:
    """Bytes (as fractions of m) crossing every directed link in every pass: an object array
    [pass][rank][port] of Fractions, port 2d towards +d and 2d+1 towards -d.

    variant 'L' or 'B' (Trivance), 'BRUCK' (latency-optimal comparison pattern) or 'BRUCK_B'
    (its bandwidth-optimal form)."""
    dims = tuple(int(x) for x in dims)
    n = int(np.prod(dims))
    D = len(dims)
    if variant == "B" and nonpow3.is_tree(dims):
        P, msgs = _messages_tree(dims)
    elif variant == "L" and nonpow3.is_tree(dims):
        P, msgs = _messages_latency_tree(dims)
    else:
        P, msgs = _messages_pow3(dims, variant)
    acc = np.empty((P, n, 2 * D), dtype=object)
    acc.fill(Fraction(0))

    for pi, r, dim, off, size in msgs:
        def add(node, port, b, pi=pi):
            acc[pi, node, port] += b
        _walk(add, dims, r, dim, off, size, routing)
    return acc


def pass_link_peaks(dims, variant: str, routing: str = "scheduled") -> list:
    """Per pass, the bytes (fraction of m) of the busiest directed link."""
    lb = link_bytes(dims, variant, routing)
    return [max(lb[p].ravel().tolist()) for p in range(lb.shape[0])]


def theta(dims, variant: str, routing: str = "scheduled") -> Fraction:
    """Transmission-delay factor: sum over passes of the busiest link's bytes, relative to
    m / D (Tables 1 and 2)."""
    return sum(pass_link_peaks(dims, variant, routing), Fraction(0)) * len(tuple(dims))


def cost(dims, variant: str, m: float, alpha: float, beta: float,
         routing: str = "scheduled") -> dict:
    """C(m, A) = passes alpha + beta sum_pass (busiest link's bytes) for an AllReduce of m bytes
    per rank; seconds when alpha is in seconds and beta in seconds per byte."""
    peaks = pass_link_peaks(dims, variant, routing)
    trans = beta * m * float(sum(peaks, Fraction(0)))
    lat = alpha * len(peaks)
    return {"total": lat + trans, "latency": lat, "transmission": trans, "passes": len(peaks),
            "pass_peaks": peaks}
