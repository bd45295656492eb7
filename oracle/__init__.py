"""CPU oracle for the Trivance AllReduce (Juerss, Addanki, Schmid, arXiv 2602.17254).

TEST INFRASTRUCTURE ONLY. This package is a plain, slow, obviously-correct CPU model of what the
emulated AllReduce computes. Only the test suite, the smoke check and the CPU-baseline leg of the
benchmark may import it. The product path (the HIP library and its Python binding) never imports,
calls or falls back to anything in here, and nothing in here imports the product path: the two
share no code. The seeded input generators live in a module of their own that holds none of the
method's arithmetic.

Modules
-------
schedule    peers, per-step distances, torus dimension rotation, reachability (Algorithm 1) and
            the closed-form block sets of Sec. 4.3.
partition   the rule that splits a rank's vector into per-collective segments and blocks
            (the paper assumes m/n-sized blocks; the rounding rule is a reading, see the module).
allreduce   message-passing emulation of both variants, step by step, with an explicit
            barrier between posting and reducing (Sec. 4.1, 4.2, 4.3, 5), plus reference sums.
congestion  hop-by-hop link-load walk (cost model of Sec. 2.1) and the transmission-delay
            factors of Tables 1 and 2 / Appendix B.
nonpow3     rings and tori whose sides are not all powers of three (Sec. 4.4): the final-step
            distance, the reduction tree of every side, a mailbox emulation of the bandwidth-
            optimal variant and a column-by-column gather form of it, and their link loads.
latency_nonpow3
            the latency-optimal variant on sides that are not all powers of three: the partial
            sums every rank keeps (windows, and the sub-window partials the final step of a side
            needs), worked out backwards from the result, and the schedule run on them.
cost        the congestion-aware cost model of Sec. 2.1 on the oracle's own messages, walked hop
            by hop.
placement   an optional block placement (not the default partition): block j at the position
            spelled by its base-3 digits in the order the schedule fixes them, which makes every
            kept set and message contiguous.

Parity status: every function here is pinned by a `-m "not gpu"` test against values the paper
prints, closed forms or brute force, except the floating-point summation order of the joint
reduction, which the paper leaves open; that order is a stated reading (own + left) + right,
pinned only through the invariants listed in tests/test_oracle_allreduce.py. The reduction trees
of sides that are not powers of three are a reading too (nonpow3): integer sums, forwarding
counts, the 7-node figure, the final-step congestion and agreement with the ordinary schedule on
powers of three pin them; the fp32 association they produce beyond that is parity unpinned.
The optional placement is pinned by the digit reversal it reduces to on a ring, by the contiguity
of the kept sets Algorithm 1 yields, and by the per-block equality with the latency-optimal
result at the block's owner.
"""

from . import schedule, partition, allreduce, congestion, placement  # noqa: F401
