"""The step kernels write with one of two cache policies, chosen per pass from the pass's
algorithmic bytes (`kKeepPassBytes` in csrc/device.h): SC1 alone up to the threshold, NT|SC1 above
it. The policy changes no value, so only the parity tests can show that each compiled form
computes the same results. This host-side check keeps them covering both: for every kernel family
the full-size workloads that tests/test_gpu_workloads.py compares with the oracle include a pass on
each side of the threshold (no GPU needed: plan and byte counts are host calls)."""

import os
import re

import pytest

from paper_2602_17254_amd import inputs

T = pytest.importorskip("paper_2602_17254_amd")

HERE = os.path.dirname(os.path.abspath(__file__))
DEVICE_H = os.path.join(HERE, "..", "paper_2602_17254_amd", "csrc", "device.h")


def _threshold():
    m = re.search(r"kKeepPassBytes\s*=\s*\(int64_t\)1\s*<<\s*(\d+)", open(DEVICE_H).read())
    assert m, "kKeepPassBytes not found in csrc/device.h"
    return 1 << int(m.group(1))


def _is_pow3(v):
    while v > 1 and v % 3 == 0:
        v //= 3
    return v == 1


def _family(w):
    pow3 = all(_is_pow3(s) for s in w.dims)
    if w.variant == "L":
        return "latency tiles" if pow3 else "slot steps"
    return "block steps" if pow3 else "tree steps"


def test_every_family_meets_both_policies():
    limit = _threshold()
    seen = {}
    for w in inputs.WORKLOADS.values():
        plan = T.trivance_plan(w.dims, w.variant, getattr(w, "placement", "natural"))
        sides = seen.setdefault(_family(w), set())
        for p in range(plan.num_passes):
            sides.add(T.trivance_pass_bytes(plan, w.elems, p) <= limit)
    assert set(seen) == {"latency tiles", "slot steps", "block steps", "tree steps"}
    for family, sides in seen.items():
        assert sides == {True, False}, f"{family}: the workloads reach only one store policy"
